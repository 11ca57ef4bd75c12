/*
 * espace.h - C ABI of the ESPACE projected linear layer on MI355X (gfx950).
 *
 * The layer (Sakr & Khailany, "ESPACE: Dimensionality Reduction of Activations
 * for Model Compression", Section 2.2, Eq. 3) replaces a dense linear layer
 * Y = W·X (Section 2.1, Eq. 1) at inference by
 *
 *        Y = (W·P)·(Pᵀ·X)
 *
 * where P (K×L, orthonormal columns) is a static projection calibrated before
 * deployment and the folded weight W' = W·P (M×L) is computed once, before
 * deployment.  Each call computes the projection Z = Pᵀ·X and then Y = W'·Z.
 *
 * Letters: K input features, M output features, L retained components, N tokens.
 *
 * Storage (all matrices row-major with an explicit leading dimension "ld",
 * counted in elements):
 *     W  [M][K]   weight, output features by input features
 *     Pt [L][K]   the projection P stored column-major (row l = column p_l)
 *     Wf [M][L]   folded weight W' = W·P
 *     X  [N][K]   activations, token-major (row n = token x_n)
 *     Z  [N][L]   projected activations (row n = Pᵀ·x_n)
 *     Y  [N][M]   output, token-major
 * With this storage every product reduces over the contiguous dimension of
 * both operands.
 *
 * Conventions shared by every entry point:
 *  - Pointers are DEVICE pointers owned by the caller; the library never
 *    allocates, frees or keeps caller memory.
 *  - A matrix with R rows and leading dimension ld occupies R·ld elements:
 *    the library may read the padding columns [cols, round_up(cols, 8)) of a
 *    row but never uses their values, and never writes outside [0, cols).
 *  - ld >= cols, ld a multiple of 8 elements (bf16) or 4 elements (f32);
 *    every base pointer 16-byte aligned (workspace: 256-byte aligned).
 *  - Shapes: M, N >= 0 (0 = empty, nothing is launched); K >= 1; 1 <= L <= K
 *    (P has L orthonormal columns of length K).  Orthonormality of P is the
 *    caller's contract and is not checked: the library computes the products
 *    for any P.
 *  - The output must not overlap any input or the workspace.
 *  - dtype: ESPACE_BF16 (bfloat16 storage, fp32 accumulation, outputs and the
 *    intermediate Z rounded to bfloat16 with round-to-nearest-even) or
 *    ESPACE_F32 (float32 throughout).
 *  - workspace: device scratch of at least espace_workspace_bytes(...) bytes
 *    for the same op, shapes and dtype; NULL only when that size is 0.  Its
 *    contents need no initialisation and are undefined after the call.  Calls
 *    that run concurrently must not share a workspace.
 *  - Every call is asynchronous and stream-ordered on `stream` (NULL = the
 *    default stream).  ESPACE_OK means "validated and enqueued"; faults during
 *    execution surface at the caller's next synchronisation.  Any other status
 *    means nothing was enqueued and no memory was written; espace_last_error()
 *    then gives a description (thread-local).
 */
#ifndef ESPACE_H
#define ESPACE_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ESPACE_ABI_VERSION 7

typedef enum {
    ESPACE_F32 = 0,
    ESPACE_BF16 = 1
} espace_dtype;

typedef enum {
    ESPACE_OK = 0,
    ESPACE_ERR_NULL = 1,       /* a required pointer is NULL */
    ESPACE_ERR_SHAPE = 2,      /* a size or leading dimension is invalid */
    ESPACE_ERR_ALIGN = 3,      /* a pointer or leading dimension is misaligned */
    ESPACE_ERR_DTYPE = 4,      /* unknown dtype */
    ESPACE_ERR_ALIAS = 5,      /* the output overlaps an input or the workspace */
    ESPACE_ERR_WORKSPACE = 6,  /* workspace missing or too small */
    ESPACE_ERR_HIP = 7,        /* the HIP runtime reported an error */
    ESPACE_ERR_DEVICE = 8      /* the current device is not gfx950 */
} espace_status;

typedef enum {
    ESPACE_OP_FOLD = 0,
    ESPACE_OP_PROJECT = 1,
    ESPACE_OP_EXPAND = 2,
    ESPACE_OP_PROJECTED_LINEAR = 3,
    ESPACE_OP_DENSE = 4,
    ESPACE_OP_AUTOCORR = 5,    /* espace_autocorrelation_update: uses K, N */
    ESPACE_OP_PCA = 6,         /* espace_principal_components: uses K, L */
    ESPACE_OP_SYMPRODUCT = 7,  /* espace_symmetrized_product: uses K */
    ESPACE_OP_BACKWARD = 8,    /* espace_projected_linear_backward: uses M, K, L, N */
    ESPACE_OP_DENSE_BACKWARD = 9,  /* espace_dense_linear_backward: uses M, K, N */
    ESPACE_OP_PROJECTED_LINEAR_MXFP8 = 10  /* espace_projected_linear_mxfp8: uses L, N */
} espace_op;

/* Folded weight Wf = W·P (Section 2.2: the paper's PᵀW, "pre-computed before
 * deployment", stored transposed).  Wf[m][l] = sum_k W[m][k]·Pt[l][k].
 * In: W [M][K] (ldw), Pt [L][K] (ldp).  Out: Wf [M][L] (ldwf). */
espace_status espace_fold_weights(const void* W, int64_t ldw,
                                  const void* Pt, int64_t ldp,
                                  void* Wf, int64_t ldwf,
                                  int64_t M, int64_t K, int64_t L,
                                  espace_dtype dt,
                                  void* workspace, size_t workspace_bytes,
                                  hipStream_t stream);

/* Projection Z = Pᵀ·X (Section 2.2, Eq. 3, right factor; Eq. 6 gives its
 * entries as the inner products <p_l, x_n>).  Z[n][l] = sum_k X[n][k]·Pt[l][k].
 * In: Pt [L][K] (ldp), X [N][K] (ldx).  Out: Z [N][L] (ldz). */
espace_status espace_project(const void* Pt, int64_t ldp,
                             const void* X, int64_t ldx,
                             void* Z, int64_t ldz,
                             int64_t K, int64_t L, int64_t N,
                             espace_dtype dt,
                             void* workspace, size_t workspace_bytes,
                             hipStream_t stream);

/* Expansion Y = Wf·Z (Section 2.2, Eq. 3: the folded weight times the
 * projected activations).  Y[n][m] = sum_l Z[n][l]·Wf[m][l].
 * In: Z [N][L] (ldz), Wf [M][L] (ldwf).  Out: Y [N][M] (ldy). */
espace_status espace_expand(const void* Z, int64_t ldz,
                            const void* Wf, int64_t ldwf,
                            void* Y, int64_t ldy,
                            int64_t M, int64_t L, int64_t N,
                            espace_dtype dt,
                            void* workspace, size_t workspace_bytes,
                            hipStream_t stream);

/* The projected linear layer Y = Wf·(Pᵀ·X) (Section 2.2, Eq. 3, inference
 * view), i.e. espace_project followed by espace_expand with Z kept in the
 * workspace (bf16: Z is rounded to bfloat16 between the two products).
 * In: X [N][K] (ldx), Pt [L][K] (ldp), Wf [M][L] (ldwf).  Out: Y [N][M] (ldy).
 * Needs espace_workspace_bytes(ESPACE_OP_PROJECTED_LINEAR, M, K, L, N, dt). */
espace_status espace_projected_linear(const void* X, int64_t ldx,
                                      const void* Pt, int64_t ldp,
                                      const void* Wf, int64_t ldwf,
                                      void* Y, int64_t ldy,
                                      int64_t M, int64_t K, int64_t L, int64_t N,
                                      espace_dtype dt,
                                      void* workspace, size_t workspace_bytes,
                                      hipStream_t stream);

/* The dense layer Y = W·X it replaces (Section 2.1, Eq. 1): the baseline.
 * Y[n][m] = sum_k X[n][k]·W[m][k].
 * In: X [N][K] (ldx), W [M][K] (ldw).  Out: Y [N][M] (ldy). */
espace_status espace_dense_linear(const void* X, int64_t ldx,
                                  const void* W, int64_t ldw,
                                  void* Y, int64_t ldy,
                                  int64_t M, int64_t K, int64_t N,
                                  espace_dtype dt,
                                  void* workspace, size_t workspace_bytes,
                                  hipStream_t stream);

/* ---- Training view (Section 2.2, "during training/finetuning") -----------
 *
 * While training, the layer is Y = W·(P·Pᵀ·X): P stays fixed, W is learnt.
 * The forward pass is espace_fold_weights (Wf = W·P, every step) followed by
 * espace_project (Z, kept for the backward pass) and espace_expand.
 * Gradients for an upstream gradient dY = ∂ℓ/∂Y [N][M]:
 *     dX = (dY·Wf)·Pt         dX[n][k] = Σ_l (Σ_m dY[n][m]·Wf[m][l])·Pt[l][k]
 *     dW = (dYᵀ·Z)·Pt         dW[m][k] = Σ_l (Σ_n dY[n][m]·Z[n][l])·Pt[l][k]
 * i.e. ∂ℓ/∂X = P·Pᵀ·(Wᵀ-side gradient) and ∂ℓ/∂W = dYᵀ·X̃ with X̃ = P·Pᵀ·X.
 * bf16: the intermediate products dY·Wf and dYᵀ·Z are rounded to bf16 (as Z
 * in the forward pass).  In: dY [N][M], Z [N][L] (for dW), Pt [L][K], Wf
 * [M][L] (for dX).  Out: dX [N][K] and/or dW [M][K] (either may be NULL).
 * Needs espace_workspace_bytes(ESPACE_OP_BACKWARD, M, K, L, N, dt). */
espace_status espace_projected_linear_backward(const void* dY, int64_t lddy,
                                               const void* Z, int64_t ldz,
                                               const void* Pt, int64_t ldp,
                                               const void* Wf, int64_t ldwf,
                                               void* dX, int64_t lddx,
                                               void* dW, int64_t lddw,
                                               int64_t M, int64_t K, int64_t L, int64_t N,
                                               espace_dtype dt,
                                               void* workspace, size_t workspace_bytes,
                                               hipStream_t stream);

/* Gradients of the dense layer Y = W·X it replaces (the baseline):
 * dX = dY·W, dW = dYᵀ·X.  In: dY [N][M], X [N][K] (for dW), W [M][K] (for
 * dX).  Out: dX [N][K] and/or dW [M][K] (either may be NULL).
 * Needs espace_workspace_bytes(ESPACE_OP_DENSE_BACKWARD, M, K, 0, N, dt). */
espace_status espace_dense_linear_backward(const void* dY, int64_t lddy,
                                           const void* X, int64_t ldx,
                                           const void* W, int64_t ldw,
                                           void* dX, int64_t lddx,
                                           void* dW, int64_t lddw,
                                           int64_t M, int64_t K, int64_t N,
                                           espace_dtype dt,
                                           void* workspace, size_t workspace_bytes,
                                           hipStream_t stream);

/* ---- Calibration of P (before deployment) --------------------------------
 *
 * Activation autocorrelation update (Section 3.1, Eq. 5; Corollary 1):
 *
 *        C += alpha · Σ_n x̂_n x̂_nᵀ      over the N tokens x_n (rows) of X,
 *
 * with x̂_n = x_n, or x̂_n = x_n / ||x_n||₂ when normalize != 0 (a zero token
 * then contributes nothing).  With alpha = 1/(N_i·B) for each of B batches
 * the calls accumulate Eq. 5's batch-averaged estimate C_X; with normalize,
 * Corollary 1's input-normalised Ĉ_X.  C[r][c] += alpha·Σ_n x̂_n[r]·x̂_n[c].
 * In: X [N][K] (ldx, dt).  In/out: C [K][K] (ldc, always float32; initialise
 * it, e.g. to zero, before the first batch).  bf16: products of bfloat16
 * values are exact in fp32 and summed in fp32; with normalize the scaled
 * tokens are rounded to bfloat16 first (1/||x_n|| from an fp64 sum of
 * squares).  f32: float32 throughout.  Limits: K·round_up(N, 8) and
 * K·round_up(K, 8) below 2^31 (split larger batches into several calls).
 * Needs espace_workspace_bytes(ESPACE_OP_AUTOCORR, 0, K, 0, N, dt). */
espace_status espace_autocorrelation_update(const void* X, int64_t ldx,
                                            float* C, int64_t ldc,
                                            int64_t K, int64_t N,
                                            int normalize, float alpha,
                                            espace_dtype dt,
                                            void* workspace, size_t workspace_bytes,
                                            hipStream_t stream);

/* GO-MSE and NL-MSE candidate matrices (Section 3.3, Theorem 2):
 *
 *        C = beta·C + alpha·(A·Bᵀ + B·Aᵀ)
 *
 * C[r][c] = beta·C[r][c] + alpha·(Σ_k A[r][k]·B[c][k] + Σ_k B[r][k]·A[c][k]),
 * float32 throughout (one fp32 product added to its transpose: exactly
 * symmetric when beta·C is); C is not read when beta == 0.  For the
 * symmetric autocorrelations A = C_X and B = C_W (espace_autocorrelation_update
 * over the rows of W) with alpha = 1, beta = 0 this is Theorem 2's GO-MSE
 * matrix C_X·C_W + C_W·C_X; with both normalised, its Ĉ.  The NL-MSE matrix
 * is accumulated per calibration sequence i (the proof of Theorem 2): A and B
 * the autocorrelations of the sequence's activations and of their loss
 * gradients (alpha = 1/M_i in each update), then alpha = 1/B, beta = 1.
 * In: A, B [K][K] (lda, ldb, float32).  In/out: C [K][K] (ldc, float32).
 * Needs espace_workspace_bytes(ESPACE_OP_SYMPRODUCT, 0, K, 0, 0, ESPACE_F32). */
espace_status espace_symmetrized_product(const float* A, int64_t lda,
                                         const float* B, int64_t ldb,
                                         float* C, int64_t ldc, int64_t K,
                                         float alpha, float beta,
                                         void* workspace, size_t workspace_bytes,
                                         hipStream_t stream);

/* Principal activation components (Theorem 1; Corollary 1 with Ĉ_X;
 * Theorem 2 with by_magnitude): row l of Pt is the eigenvector of the l-th
 * largest eigenvalue of the symmetric C — with by_magnitude != 0, of the
 * l-th largest in absolute value (the rule Theorem 2's proof gives when C is
 * not positive semi-definite; equal magnitudes: the larger value first) —
 * for l < L, signed so that its entry of largest magnitude (the first such on
 * ties) is positive.  Only the upper triangle of C (c >= r) is read.
 * The decomposition runs in float64 (rocSOLVER's divide-and-conquer dsyevd,
 * loaded at the first call; ESPACE_ERR_HIP if it cannot be loaded).
 * In: C [K][K] (ldc, float32).  Out: Pt [L][K] (ldp, dt); eigenvalues: all K
 * in the selection order (float32, device, may be NULL); info: one device int
 * (may be NULL), 0 on success, > 0 when the solver did not converge.
 * Exception to the conventions above: the first call on a device creates a
 * rocBLAS handle, and the solver may allocate device scratch of its own
 * (kept by that handle), so the call is not for graph capture.
 * Limits: K <= 32768.  Needs espace_workspace_bytes(ESPACE_OP_PCA, 0, K, L,
 * 0, dt). */
espace_status espace_principal_components(const float* C, int64_t ldc,
                                          void* Pt, int64_t ldp,
                                          float* eigenvalues, int* info,
                                          int64_t K, int64_t L, int by_magnitude,
                                          espace_dtype dt,
                                          void* workspace, size_t workspace_bytes,
                                          hipStream_t stream);

/* ---- MX-FP8 layer -------------------------------------------------------------
 * The paper notes that the activation projection can be carried out in low
 * precision (Section 1.1) and leaves combining ESPACE with quantisation to
 * future work (Section 5), without fixing a number format.  This path uses
 * the OCP Microscaling format MX-FP8, which gfx950's block-scaled MFMA
 * consumes directly:
 *  - elements: FP8 E4M3 (exponent bias 7, 3 mantissa bits, subnormals below
 *    2^-6, largest magnitude 448, no infinities), one byte each;
 *  - blocks: 32 consecutive elements of a row (the reduction dimension of both
 *    products) share the scale 2^S, stored as the byte S + 127 (E8M0), with
 *    S = floor(log2(max |v|)) - 8, the byte clamped to [0, 254] and 0 for a
 *    block of zeros; an element is v / 2^S rounded to the nearest E4M3 value
 *    (ties to even), magnitudes above 448 clamped to 448.
 * An MX-FP8 matrix of R rows and C columns is stored as
 *     codes  Q [R][ldq]  uint8, ldq >= round_up(C, 128) and a multiple of 16,
 *                        16-byte aligned; the columns [C, round_up(C, 128))
 *                        must hold zeros (espace_quantize_mxfp8 and
 *                        espace_project_mxfp8 write them);
 *     scales S [R][lds]  uint8, lds >= round_up(C, 128) / 32 and a multiple of
 *                        4, 4-byte aligned; byte b scales columns [32b, 32b + 32)
 *                        (the bytes up to round_up(C, 128) / 32 are written).
 *                        Where lds is a multiple of 16 and S is 16-byte
 *                        aligned for both operands, the projection loads four
 *                        steps' scales at a time (faster; same results).
 * Both products accumulate in fp32 through the MFMA.
 * Shapes as for the bf16 layer (1 <= L <= K; M, N >= 0); every code matrix
 * must span less than 2^31 bytes.  Other conventions (device pointers,
 * stream order, statuses, no overlap of outputs and inputs) as above. */

/* Quantise a bfloat16 matrix A [R][C] (lda, a multiple of 8) to MX-FP8 along
 * its rows: the activations X (per token, along K) at run time, the
 * projection Pt (along K) and the folded weight Wf (along L) once, like the
 * fold.  Out: Q [R][ldq], S [R][lds]. */
espace_status espace_quantize_mxfp8(const void* A, int64_t lda, int64_t R, int64_t C,
                                    void* Q, int64_t ldq, void* S, int64_t lds,
                                    hipStream_t stream);

/* Projection Z = Pᵀ·X from MX-FP8 operands (Section 2.2, Eq. 3, right
 * factor), accumulated in fp32 and written in MX-FP8 along L (per token).
 * In: Pt codes/scales [L][K] (ldpq, ldps), X codes/scales [N][K] (ldxq,
 * ldxs).  Out: Z codes/scales [N][L] (ldzq, ldzs). */
espace_status espace_project_mxfp8(const void* Ptq, int64_t ldpq, const void* Pts, int64_t ldps,
                                   const void* Xq, int64_t ldxq, const void* Xs, int64_t ldxs,
                                   void* Zq, int64_t ldzq, void* Zs, int64_t ldzs,
                                   int64_t K, int64_t L, int64_t N, hipStream_t stream);

/* Expansion Y = Wf·Z from MX-FP8 operands (Section 2.2, Eq. 3), fp32
 * accumulation, Y bfloat16 (round to nearest even).
 * In: Z codes/scales [N][L] (ldzq, ldzs), Wf codes/scales [M][L] (ldwq,
 * ldws).  Out: Y [N][M] (ldy, a multiple of 8). */
espace_status espace_expand_mxfp8(const void* Zq, int64_t ldzq, const void* Zs, int64_t ldzs,
                                  const void* Wfq, int64_t ldwq, const void* Wfs, int64_t ldws,
                                  void* Y, int64_t ldy,
                                  int64_t M, int64_t L, int64_t N, hipStream_t stream);

/* The MX-FP8 layer: espace_project_mxfp8 then espace_expand_mxfp8 with Z in
 * the workspace (espace_workspace_bytes(ESPACE_OP_PROJECTED_LINEAR_MXFP8, M,
 * K, L, N, ESPACE_BF16) bytes, 256-byte aligned); computes exactly what the
 * two calls compute.
 * In: X, Pt, Wf codes/scales.  Out: Y [N][M] bfloat16 (ldy). */
espace_status espace_projected_linear_mxfp8(const void* Xq, int64_t ldxq, const void* Xs, int64_t ldxs,
                                            const void* Ptq, int64_t ldpq, const void* Pts, int64_t ldps,
                                            const void* Wfq, int64_t ldwq, const void* Wfs, int64_t ldws,
                                            void* Y, int64_t ldy,
                                            int64_t M, int64_t K, int64_t L, int64_t N,
                                            void* workspace, size_t workspace_bytes,
                                            hipStream_t stream);

/* Workspace bytes needed by `op` for these sizes (0 when none is needed).
 * Arguments an op does not use are ignored (e.g. L for ESPACE_OP_DENSE).
 * Returns SIZE_MAX for invalid sizes. */
size_t espace_workspace_bytes(espace_op op, int64_t M, int64_t K, int64_t L,
                              int64_t N, espace_dtype dt);

const char* espace_status_string(espace_status s);
const char* espace_last_error(void);
int espace_abi_version(void);

/* Allocation-free variant of espace_projected_linear, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, computation and results
 * as espace_projected_linear without the workspace: Z and the partial sums
 * live in a static device array of ESPACE_NOALLOC_SCRATCH_BYTES that the
 * library holds on every device it runs on until the process ends.  Calls
 * neither hipMalloc, hipFree nor any allocating library routine (the first
 * call on a device looks up that device's copy of the array).
 *  - Sizes whose workspace (espace_workspace_bytes(ESPACE_OP_PROJECTED_LINEAR,
 *    ...)) exceeds ESPACE_NOALLOC_SCRATCH_BYTES return ESPACE_ERR_WORKSPACE
 *    and enqueue nothing.
 *  - All calls on one device share the array: calls that can overlap on one
 *    device (other streams, other threads, other processes are not affected)
 *    race and must be serialised by the caller.  Nothing in it needs to start
 *    at zero (its state words carry a per-call tag). */
#define ESPACE_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

espace_status espace_projected_linear_noalloc(const void* X, int64_t ldx,
                                              const void* Pt, int64_t ldp,
                                              const void* Wf, int64_t ldwf,
                                              void* Y, int64_t ldy,
                                              int64_t M, int64_t K, int64_t L, int64_t N,
                                              espace_dtype dt, hipStream_t stream);

/* Bounded waits.  Some kernels wait for other workgroups of the same launch
 * (the combine of two depth halves of a tile).  Every such wait gives up after a
 * limit of polls; the waiting workgroup then writes NaN to the outputs it
 * could not complete (the call's result shows the failure) and adds one to a
 * per-device count.  These waits end within microseconds when the launch runs
 * alone on the device; the limit (about seconds) only matters if workgroups
 * of a launch are kept from running.
 *
 * espace_wait_timeouts: the current device's count of waits that gave up
 * since the process loaded the library, written to *count.  It reads device
 * memory synchronously: call it after the streams that ran the kernels have
 * been synchronised.  ESPACE_ERR_NULL for a NULL count.
 *
 * espace_set_wait_limit: the number of polls after which later launches give
 * up (process-wide; 0 restores the default).  Meant for tests of the failure
 * path: a limit of 1 makes a workgroup that finds its partner's results not
 * yet there give up at once. */
espace_status espace_wait_timeouts(unsigned long long* count);
espace_status espace_set_wait_limit(unsigned spins);

#ifdef __cplusplus
}
#endif

#endif /* ESPACE_H */
