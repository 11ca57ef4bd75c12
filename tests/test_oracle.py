"""The CPU oracle against what the paper and the mathematics fix."""
import types

import pytest

import oracle
from tests import oracle_pins


def _ns():
    return types.SimpleNamespace(**{k: getattr(oracle, k) for k in dir(oracle) if not k.startswith("_")})


@pytest.mark.parametrize("pin", oracle_pins.ALL_PINS, ids=lambda p: p.__name__)
def test_pin(pin):
    pin(_ns())
