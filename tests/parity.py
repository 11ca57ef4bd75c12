"""Element-wise parity criteria for the GPU path against the float64 oracle.

Three criteria, all asserted on whole outputs:

1. every output entry is finite (outputs are NaN-prefilled, so an entry the
   kernels never write shows up);
2. every entry lies within a rounding bound derived from the arithmetic the
   GPU performs (below), computed entry by entry from float64 quantities of
   the oracle;
3. the relative Frobenius error of the whole output is at most `tol` (1e-2 for
   bfloat16, 1e-5 for float32), and so is that of every 64 x 64 block of it
   (relative to the block's norm, or to its share of the whole output's norm
   when that is larger), so that an error confined to one kernel tile cannot
   hide in the global norm.

The bound.  The GPU computes each product with bfloat16 (or float32) operands,
exact products, fp32 accumulation, and one round-to-nearest-even to the
storage type (unit roundoff u = 2^-8 for bfloat16, 2^-24 for float32).  For
one product C = A·Bᵀ of depth D with exact inputs, accumulation over D terms
in fp32 errs by at most γ_D·Σ_k |a_k||b_k| with γ_n = n·v/(1 - n·v); v = 2^-23
(twice fp32's unit roundoff, so that an accumulation that does not round to
nearest is covered too).  By Cauchy-Schwarz Σ_k |a_k||b_k| <= ||a||·||b||, so

    |C_gpu - C| <= u·|C| + (1 + u)·γ_D·||a_r||·||b_c||          (fold, project, dense)

For the layer Y = W'·Z with W' = fold(W, P) and Z = project(P, X) both rounded
on the GPU, eZ = γ_K·||x_n||·||p_l|| and eW = γ_K·||w_m||·||p_l|| bound the
accumulation errors of the two inputs, so |Z_gpu - Z| <= dZ = u·|Z| + (1+u)·eZ
and |Z_gpu| <= mZ = |Z| + dZ (the same for W').  The expansion adds the
accumulation of depth L and the final rounding:

    |Y_gpu - Y| <= u·|Y| + (1 + u)·E,
    E = γ_L·Σ_l mZ·mW + Σ_l dZ·mW + Σ_l |Z|·dW,

which expands into |Z|·|W'|ᵀ (one product of the layer's size) and rank-one
products of the norms, each with its own coefficient (layer_bound).

The bound is a worst case (every rounding error aligned): it catches gross
errors (a wrong index, an unwritten or doubly written entry, a lost product),
while the per-block Frobenius criterion catches a small error confined to a
region (one depth half of one tile lost).  The typical error is about
sqrt(3)·1.6e-3 ≈ 3e-3 relative: three roundings of relative RMS
u/sqrt(3)·E[1/m] ≈ 1.6e-3 each.
"""
import numpy as np

U_BF16 = 2.0 ** -8
U_F32 = 2.0 ** -24
V_ACC = 2.0 ** -23
TOL = {"bf16": 1e-2, "f32": 1e-5}
UNIT = {"bf16": U_BF16, "f32": U_F32}
BLOCK = 64


def gamma(n):
    return n * V_ACC / (1.0 - n * V_ACC)


def row_norms(A):
    A = np.asarray(A, dtype=np.float64)
    return np.sqrt(np.einsum("ij,ij->i", A, A))


def product_bound(C, a_norms, b_norms, depth, u):
    """Entry bound of one product C = A·Bᵀ (exact float64 C) rounded to the
    storage type: rows of A have norms a_norms, rows of B b_norms."""
    return u * np.abs(C) + (1.0 + u) * gamma(depth) * np.outer(a_norms, b_norms)


def layer_bound(Y, Z, Wf, x_norms, p_norms, w_norms, K, L, u):
    """Entry bound of Y = Wf·Z computed from the GPU's rounded Z (from X and P,
    depth K) and its rounded fold Wf (from W and P, depth K).  Pass w_norms=None
    when Wf is an exact input rather than the GPU's fold."""
    gK, gL, v = gamma(K), gamma(L), 1.0 + u
    az = np.abs(Z)
    bw = np.abs(Wf)
    s_zw = az @ bw.T                                          # Σ |Z||W'|
    s_ezw = gK * np.outer(x_norms, bw @ p_norms)              # Σ eZ |W'|
    if w_norms is None:
        s_zew = np.zeros_like(s_zw)
        s_ee = s_zew
    else:
        s_zew = gK * np.outer(az @ p_norms, w_norms)          # Σ |Z| eW
        s_ee = gK * gK * float(p_norms @ p_norms) * np.outer(x_norms, w_norms)
    E = ((gL * v * v + u * v + u) * s_zw + (gL * v * v + v * v) * s_ezw
         + (gL * v * v + u * v + v) * s_zew + (gL * v * v + v * v) * s_ee)
    return u * np.abs(Y) + v * E


def block_rel_errors(got, ref, block=BLOCK):
    """Relative Frobenius error of every block x block tile: ||E_t|| divided by
    max(||ref_t||, ||ref||·sqrt(n_t / n)), the tile's norm or its share of
    the whole output's norm."""
    R, C = ref.shape
    d2 = (got - ref) ** 2
    r2 = ref ** 2
    nr = -(-R // block)
    nc = -(-C // block)
    pr = nr * block - R
    pc = nc * block - C
    d2 = np.pad(d2, ((0, pr), (0, pc))).reshape(nr, block, nc, block).sum(axis=(1, 3))
    r2 = np.pad(r2, ((0, pr), (0, pc))).reshape(nr, block, nc, block).sum(axis=(1, 3))
    rows = np.minimum(block, R - block * np.arange(nr))
    cols = np.minimum(block, C - block * np.arange(nc))
    share = r2.sum() * np.outer(rows, cols) / (R * C)
    return np.sqrt(d2 / np.maximum(np.maximum(r2, share), 1e-300))


def check(got, ref, bound, tol, what=""):
    """Assert the three criteria; returns (rel_fro, worst block error, worst
    ratio of error to bound) for reporting."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert got.shape == ref.shape, (what, got.shape, ref.shape)
    if got.size == 0:
        return 0.0, 0.0, 0.0
    finite = np.isfinite(got)
    if not finite.all():
        bad = np.argwhere(~finite)
        raise AssertionError(f"{what}: {len(bad)} non-finite (unwritten?) entries, first at {bad[:4].tolist()}")
    err = np.abs(got - ref)
    over = err > bound
    if over.any():
        bad = np.argwhere(over)
        i, j = bad[0]
        raise AssertionError(f"{what}: {len(bad)} entries outside the rounding bound, first at ({i}, {j}): "
                             f"got {got[i, j]!r}, oracle {ref[i, j]!r}, bound {bound[i, j]!r}")
    den = np.linalg.norm(ref)
    rel = float(np.linalg.norm(got - ref) / den) if den > 0 else float(np.linalg.norm(got - ref))
    assert rel <= tol, f"{what}: relative Frobenius error {rel:.3e} > {tol}"
    blk = block_rel_errors(got, ref)
    worst = float(blk.max())
    if worst > tol:
        bi, bj = np.unravel_index(int(np.argmax(blk)), blk.shape)
        raise AssertionError(f"{what}: block ({bi * BLOCK}, {bj * BLOCK}) relative error {worst:.3e} > {tol}")
    ratio = float(np.max(err / np.maximum(bound, 1e-300)))
    return rel, worst, ratio
