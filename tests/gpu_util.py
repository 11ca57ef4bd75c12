"""Helpers for the GPU tests: move seeded inputs to the device with padded
rows whose padding holds NaN (so any use of padding shows up), and bring
outputs back as float64."""
import numpy as np
import pytest
import torch

NAN_BF16 = 0x7FC0


def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    return torch.device("cuda:0")


def dev_mat(storage, dtype, device, pad_value=float("nan"), align=None):
    """Device tensor [R][C] with a leading dimension rounded up to the
    library's alignment and NaN in the padding columns."""
    storage = np.ascontiguousarray(storage)
    R, C = storage.shape
    if align is None:
        align = 8 if dtype == "bf16" else 4
    ld = max((C + align - 1) // align * align, align)
    if dtype == "bf16":
        full = np.full((R, ld), NAN_BF16, dtype=np.uint16)
        full[:, :C] = storage
        t = torch.from_numpy(full.view(np.int16)).view(torch.bfloat16)
    else:
        full = np.full((R, ld), pad_value, dtype=np.float32)
        full[:, :C] = storage
        t = torch.from_numpy(full)
    return t.to(device)[:, :C]


def out_mat(R, C, dtype, device, fill=float("nan")):
    """Output tensor [R][C] (padded leading dimension) prefilled with `fill`,
    so unwritten entries and writes into padding are visible."""
    align = 8 if dtype == "bf16" else 4
    ld = max((C + align - 1) // align * align, align)
    tdt = torch.bfloat16 if dtype == "bf16" else torch.float32
    return torch.full((R, ld), fill, dtype=tdt, device=device)[:, :C]


def host64(t):
    return t.float().cpu().numpy().astype(np.float64)


def padding(t):
    """The padding columns [C, ld) of a padded 2-D view, as a host array."""
    R, C = t.shape
    ld = t.stride(0)
    base = t.as_strided((R, ld), (ld, 1))
    return base[:, C:].float().cpu().numpy()
