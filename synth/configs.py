"""The five layer workloads of the projected linear layer, and smaller variants.

Shapes follow the paper's tensor-parallel-folded layer table (Appendix B.2,
Table 2) for Llama2-7B and GPT3-22B; the token counts follow the paper's
prefill setting (batch 1, sequence length 4096 for Llama2, Section 4.1) and add
decode-sized token counts.  Storage convention: W[M][K] (output features by
input features), Pt[L][K] (the K×L projection stored column-major), X[N][K]
(token-major), Y[N][M].
"""
from dataclasses import dataclass, replace

SEED = 241005437


@dataclass(frozen=True)
class Workload:
    cfg: int            # which of the five workloads (0..4)
    name: str
    K: int              # input features (reduction depth of the dense layer)
    M: int              # output features
    L: int              # retained principal components
    N: int              # tokens
    dtype: str          # "f32" or "bf16"
    recipe: str         # "gaussian": X = Q·diag(sqrt(lam))·G ; "silu_gated": SiLU(a)*b
    lam_floor: float    # spectrum lam_i = 1/i + lam_floor
    proj: str           # "leading": P = Q[:, :L] ; "calibrated": top-L eigvecs of sample X·Xᵀ
    cov_key: int        # seed key of Q (workloads sharing a covariance share it)
    w_key: int          # seed key of W
    n_cal: int = 0      # calibration tokens for proj == "calibrated"
    layer: str = ""

    @property
    def compression(self):
        """Per-layer inference compression 1 - L(K+M)/(KM) (Section 2.2)."""
        return 1.0 - self.L * (self.K + self.M) / (self.K * self.M)

    @property
    def flops(self):
        """Algorithmic flops of Y = (W·P)·(Pᵀ·X): 2·L·N·(K+M)."""
        return 2 * self.L * self.N * (self.K + self.M)

    @property
    def dense_flops(self):
        return 2 * self.M * self.K * self.N

    def scaled(self, **kw):
        """Same recipe and seeds, other sizes (for fast tests)."""
        return replace(self, **kw)

    def key(self):
        return (self.cfg, self.name, self.K, self.M, self.L, self.N, self.dtype,
                self.recipe, self.lam_floor, self.proj, self.cov_key, self.w_key,
                self.n_cal, self.layer)


def _base():
    return {
        0: Workload(0, "tiny-fp32", K=256, M=256, L=64, N=128, dtype="f32",
                    recipe="gaussian", lam_floor=0.0, proj="leading",
                    cov_key=0, w_key=0),
        1: Workload(1, "llama2-7b-qkv", K=4096, M=12288, L=1536, N=4096,
                    dtype="bf16", recipe="gaussian", lam_floor=1e-4,
                    proj="leading", cov_key=1, w_key=1),
        2: Workload(2, "llama2-7b-ffn-upgate", K=4096, M=22016, L=1536, N=4096,
                    dtype="bf16", recipe="gaussian", lam_floor=1e-4,
                    proj="leading", cov_key=1, w_key=2),
        3: Workload(3, "llama2-7b-ffn-down", K=11008, M=4096, L=1536, N=4096,
                    dtype="bf16", recipe="silu_gated", lam_floor=0.0,
                    proj="calibrated", cov_key=3, w_key=3, n_cal=16384),
        4: Workload(4, "gpt3-22b-ffn-up", K=6144, M=24576, L=2458, N=8192,
                    dtype="bf16", recipe="gaussian", lam_floor=0.0,
                    proj="leading", cov_key=4, w_key=4, layer="up"),
    }


CONFIGS = _base()


def workloads(cfg):
    """Every (layer, L, N) case of one workload."""
    b = CONFIGS[cfg]
    if cfg == 2:
        return [b.scaled(N=n) for n in (4096, 1, 8, 16)]
    if cfg == 4:
        out = []
        for layer, K, M, key in (("up", 6144, 24576, 4), ("down", 24576, 6144, 5)):
            for L in (3686, 2458, 1966):
                for N in (8192, 1, 16):
                    out.append(b.scaled(name=f"gpt3-22b-ffn-{layer}", K=K, M=M,
                                        L=L, N=N, cov_key=key, w_key=key,
                                        layer=layer))
        return out
    return [b]


def workload(cfg, **kw):
    """One case of a workload; keyword arguments select among its cases."""
    for w in workloads(cfg):
        if all(getattr(w, k) == v for k, v in kw.items()):
            return w
    raise KeyError((cfg, kw))
