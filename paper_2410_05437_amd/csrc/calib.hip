// Calibration of the projection (paper Section 3.1-3.2): the activation
// autocorrelation C_X = E[x xᵀ] estimated from calibration batches (Eq. 5),
// its input-normalised variant Ĉ_X (Corollary 1), and the projection made of
// its L principal eigenvectors (Theorem 1).
//
//  * Autocorrelation update C += alpha · Σ_n x̂_n x̂_nᵀ over the M tokens of a
//    batch X[M][K] (x̂_n = x_n, or x_n / ||x_n|| when normalising): the tokens
//    are transposed (and scaled) into Xt[K][M] so that the sum over tokens is
//    the contiguous dimension of a "TN" product Xt·Xtᵀ, which runs on the
//    MFMA GEMM kernels with fp32 results per depth range; the product is
//    symmetric, so (bf16) only the 256 x 256 tiles on and above the diagonal
//    are computed, and a last pass adds alpha times the sum of the ranges to
//    C in fixed order, reading the mirrored entry below the diagonal tiles.
//  * GO-MSE / NL-MSE candidates (Theorem 2): C = beta·C + alpha·(A·Bᵀ + B·Aᵀ),
//    for the symmetric autocorrelations A = C_X and B = C_W (or, per
//    calibration sequence, C_G of the activation gradients) the matrix
//    C_X·C_W + C_W·C_X: one fp32 "TN" product A·Bᵀ, then C[r][c] =
//    beta·C[r][c] + alpha·(P[r][c] + P[c][r]) (64 x 64 tiles of P and of its
//    transpose through LDS), exactly symmetric.
//  * Principal components: C (fp32, upper triangle read) is widened to fp64
//    and handed to rocSOLVER's symmetric divide-and-conquer eigensolver
//    (dsyevd, loaded at the first call: the library is large and only
//    calibration needs it); the eigenvectors of the L largest eigenvalues (or
//    largest in magnitude, Theorem 2's rule for an indefinite C) become the
//    rows of Pt, each with the sign that makes its entry of largest magnitude
//    positive.
#include <dlfcn.h>
#include <math.h>
#include <mutex>

#include <rocblas/rocblas.h>
#include <rocsolver/rocsolver-extra-types.h>

#include "common.hpp"
#include "kernels.hpp"

namespace espace {

namespace {

__device__ __forceinline__ float load_f(const uint16_t* p) { return bf16_to_f32(*p); }
__device__ __forceinline__ float load_f(const float* p) { return *p; }
__device__ __forceinline__ void store_f(uint16_t* p, float v) { *p = (uint16_t)bf16_rne(v); }
__device__ __forceinline__ void store_f(float* p, float v) { *p = v; }

// 1 / ||x_n|| for each token of a bfloat16 X (0 for a zero token), the sum of
// squares in fp64.  One wave per token, 16-byte loads: lane l adds the
// squares of chunks l, l + 64, ... in order, then a fixed butterfly.
__global__ __launch_bounds__(256) void token_inv_norm_bf16_kernel(const uint16_t* __restrict__ X, int64_t ldx,
                                                                  int M, int K, float* __restrict__ inv) {
    const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (n >= M) return;
    const uint16_t* row = X + (int64_t)n * ldx;
    double s = 0.0;
    for (int k = lane * 8; k < K; k += 512) {
        const u32x4_t v = mask_chunk(*reinterpret_cast<const u32x4_t*>(row + k), K - k);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const double lo = (double)bf16_to_f32(v[e] & 0xffffu), hi = (double)bf16_to_f32(v[e] >> 16);
            s += lo * lo;
            s += hi * hi;
        }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0) inv[n] = s > 0.0 ? (float)(1.0 / sqrt(s)) : 0.f;
}

// 1 / ||x_n|| for each token (0 for a zero token), the sum of squares in fp64.
// One wave per token.
template <typename T>
__global__ __launch_bounds__(256) void token_inv_norm_kernel(const T* __restrict__ X, int64_t ldx, int M,
                                                             int K, float* __restrict__ inv) {
    const int n = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (n >= M) return;
    const T* row = X + (int64_t)n * ldx;
    double s = 0.0;
    for (int k = lane; k < K; k += 64) {
        const double v = (double)load_f(row + k);
        s += v * v;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane == 0) inv[n] = s > 0.0 ? (float)(1.0 / sqrt(s)) : 0.f;
}

// Xt[k][n] = X[n][k] (times inv[n] when inv is given), rounded to T.  64 x 64
// tiles through LDS so that both the reads and the writes are row-contiguous.
template <typename T>
__global__ __launch_bounds__(256) void transpose_scale_kernel(const T* __restrict__ X, int64_t ldx,
                                                              const float* __restrict__ inv,
                                                              T* __restrict__ Xt, int64_t ldt, int M, int K) {
    __shared__ float tile[64][65];
    const int n0 = blockIdx.x * 64, k0 = blockIdx.y * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
#pragma unroll 4
    for (int i = 0; i < 16; ++i) {
        const int n = n0 + ty * 16 + i, k = k0 + tx;
        float v = 0.f;
        if (n < M && k < K) {
            v = load_f(X + (int64_t)n * ldx + k);
            if (inv) v *= inv[n];
        }
        tile[ty * 16 + i][tx] = v;
    }
    __syncthreads();
#pragma unroll 4
    for (int i = 0; i < 16; ++i) {
        const int k = k0 + ty * 16 + i, n = n0 + tx;
        if (k < K && n < M) store_f(Xt + (int64_t)k * ldt + n, tile[tx][ty * 16 + i]);
    }
}

// dst[c][r] = src[r][c] for bfloat16: 64 x 64 tiles, 16-byte loads and
// stores.  A thread loads 8 consecutive elements of a source row into the
// LDS tile and stores 8 consecutive source rows of one column as a 16-byte
// piece of a destination row.  Rows of both matrices are padded to a
// multiple of 8 elements (16 bytes), so a piece that starts inside a row
// stays inside it; the destination's padding may be written (the caller's
// own scratch), its rows beyond `cols` are not.
__global__ __launch_bounds__(256) void transpose_bf16_kernel(const uint16_t* __restrict__ src, int64_t lds,
                                                             uint16_t* __restrict__ dst, int64_t ldd, int rows,
                                                             int cols) {
    __shared__ uint16_t t[64][66];
    const int r0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
    const int part = threadIdx.x & 7, line = threadIdx.x >> 3;    // 8 pieces of 8 elements, 32 lines
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int r = line + 32 * h;
        u32x4_t v = {0u, 0u, 0u, 0u};
        if (r0 + r < rows && c0 + part * 8 < cols)
            v = *reinterpret_cast<const u32x4_t*>(src + (int64_t)(r0 + r) * lds + c0 + part * 8);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            t[r][part * 8 + 2 * e] = (uint16_t)(v[e] & 0xffffu);
            t[r][part * 8 + 2 * e + 1] = (uint16_t)(v[e] >> 16);
        }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int c = line + 32 * h;
        if (c0 + c >= cols || r0 + part * 8 >= rows) continue;
        u32x4_t v;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            v[e] = (uint32_t)t[part * 8 + 2 * e][c] | ((uint32_t)t[part * 8 + 2 * e + 1][c] << 16);
        *reinterpret_cast<u32x4_t*>(dst + (int64_t)(c0 + c) * ldd + r0 + part * 8) = v;
    }
}

// Xt[k][n] = bf16(X[n][k] · inv[n]) for bfloat16 X: the 16-byte transpose
// below with each token's scale applied as its row is loaded (the product in
// fp32, rounded to nearest even, as the element-wise kernel above does).
__global__ __launch_bounds__(256) void transpose_scale_bf16_kernel(const uint16_t* __restrict__ src, int64_t lds,
                                                                   const float* __restrict__ inv,
                                                                   uint16_t* __restrict__ dst, int64_t ldd,
                                                                   int rows, int cols) {
    __shared__ uint16_t t[64][66];
    const int r0 = blockIdx.x * 64, c0 = blockIdx.y * 64;
    const int part = threadIdx.x & 7, line = threadIdx.x >> 3;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int r = line + 32 * h;
        u32x4_t v = {0u, 0u, 0u, 0u};
        if (r0 + r < rows && c0 + part * 8 < cols) {
            v = *reinterpret_cast<const u32x4_t*>(src + (int64_t)(r0 + r) * lds + c0 + part * 8);
            const float sc = inv[r0 + r];
#pragma unroll
            for (int e = 0; e < 4; ++e)
                v[e] = pack_bf16x2(bf16_to_f32(v[e] & 0xffffu) * sc, bf16_to_f32(v[e] >> 16) * sc);
        }
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            t[r][part * 8 + 2 * e] = (uint16_t)(v[e] & 0xffffu);
            t[r][part * 8 + 2 * e + 1] = (uint16_t)(v[e] >> 16);
        }
    }
    __syncthreads();
#pragma unroll
    for (int h = 0; h < 2; ++h) {
        const int c = line + 32 * h;
        if (c0 + c >= cols || r0 + part * 8 >= rows) continue;
        u32x4_t v;
#pragma unroll
        for (int e = 0; e < 4; ++e)
            v[e] = (uint32_t)t[part * 8 + 2 * e][c] | ((uint32_t)t[part * 8 + 2 * e + 1][c] << 16);
        *reinterpret_cast<u32x4_t*>(dst + (int64_t)(c0 + c) * ldd + r0 + part * 8) = v;
    }
}

// C[r][c] += alpha · Σ_s P_s[r][c], the depth ranges added in order.  With
// tile > 0 only the tiles on and above the diagonal of P (tile x tile, a
// multiple of 64) hold sums: a 64 x 64 block below them reads its mirror
// block of P row by row and transposes the sums through LDS.
__global__ __launch_bounds__(256) void accumulate_kernel(const float* __restrict__ P, int S, int64_t stride,
                                                         int64_t ldp, float* __restrict__ C, int64_t ldc,
                                                         int R, int Cc, float alpha, int tile) {
    __shared__ float t[64][65];
    const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    const bool mirror = tile > 0 && r0 / tile > c0 / tile;    // uniform over the block
    if (!mirror) {
        for (int i = ty; i < 64; i += 4) {
            const int r = r0 + i, c = c0 + tx;
            if (r >= R || c >= Cc) continue;
            const int64_t at = (int64_t)r * ldp + c;
            float s = 0.f;
            for (int q = 0; q < S; ++q) s += P[q * stride + at];
            float* o = C + (int64_t)r * ldc + c;
            *o = fmaf(alpha, s, *o);
        }
        return;
    }
    for (int i = ty; i < 64; i += 4) {
        const int pr = c0 + i, pc = r0 + tx;    // P[pr][pc] is the mirror of C[pc][pr]
        float s = 0.f;
        if (pr < Cc && pc < R) {
            const int64_t at = (int64_t)pr * ldp + pc;
            for (int q = 0; q < S; ++q) s += P[q * stride + at];
        }
        t[i][tx] = s;
    }
    __syncthreads();
    for (int i = ty; i < 64; i += 4) {
        const int r = r0 + i, c = c0 + tx;
        if (r >= R || c >= Cc) continue;
        float* o = C + (int64_t)r * ldc + c;
        *o = fmaf(alpha, t[tx][i], *o);
    }
}

// A[r][c] = C[r][c] in fp64 (K x K, leading dimension K).
__global__ __launch_bounds__(256) void widen_kernel(const float* __restrict__ C, int64_t ldc,
                                                    double* __restrict__ A, int K) {
    const int64_t total = (int64_t)K * K;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int r = (int)(i / K), c = (int)(i % K);
        A[i] = (double)C[(int64_t)r * ldc + c];
    }
}

// C[r][c] = beta·C[r][c] + alpha·(P[r][c] + P[c][r]) for r, c < K (C is not
// read when beta == 0): a 64 x 64 tile of P and the mirrored tile, the latter
// read row-contiguously and transposed in LDS.
__global__ __launch_bounds__(256) void symmetrize_kernel(const float* __restrict__ P, int64_t ldp,
                                                         float* __restrict__ C, int64_t ldc, int K, float alpha,
                                                         float beta) {
    __shared__ float t[64][65];
    const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
#pragma unroll 4
    for (int i = 0; i < 16; ++i) {
        const int rr = c0 + ty * 16 + i, cc = r0 + tx;      // P[c0 + i'][r0 + j']
        t[ty * 16 + i][tx] = (rr < K && cc < K) ? P[(int64_t)rr * ldp + cc] : 0.f;
    }
    __syncthreads();
#pragma unroll 4
    for (int i = 0; i < 16; ++i) {
        const int r = r0 + ty * 16 + i, c = c0 + tx;
        if (r < K && c < K) {
            const float v = alpha * (P[(int64_t)r * ldp + c] + t[tx][ty * 16 + i]);
            float* o = C + (int64_t)r * ldc + c;
            *o = beta != 0.f ? fmaf(beta, *o, v) : v;
        }
    }
}

// The order in which eigenvalues D (ascending, from the solver) are taken:
// decreasing value, or decreasing magnitude (by_magnitude; from both ends of
// D, the larger magnitude first, the upper end on ties).  One thread.
__global__ void order_kernel(const double* __restrict__ D, int K, int by_magnitude, int* __restrict__ idx) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    int lo = 0, hi = K - 1;
    for (int l = 0; l < K; ++l) {
        if (!by_magnitude || fabs(D[hi]) >= fabs(D[lo])) idx[l] = hi--;
        else idx[l] = lo++;
    }
}

// Row l of Pt: the eigenvector of eigenvalue idx[l] (column idx[l] of the
// solver's column-major V, contiguous), signed so that its entry of largest
// magnitude (the first such) is positive.  One workgroup per row; workgroup
// 0 also writes the eigenvalues in the order of idx.
template <typename T>
__global__ __launch_bounds__(256) void select_kernel(const double* __restrict__ V, const double* __restrict__ D,
                                                     const int* __restrict__ idx, int K, int L,
                                                     T* __restrict__ Pt, int64_t ldp, float* __restrict__ evals) {
    __shared__ double best_v[256];
    __shared__ int best_i[256];
    const int l = blockIdx.x;
    const double* v = V + (int64_t)idx[l] * K;
    double bv = -1.0;
    int bi = K;
    for (int k = threadIdx.x; k < K; k += 256) {
        const double a = fabs(v[k]);
        if (a > bv) { bv = a; bi = k; }       // first index of the largest within the thread
    }
    best_v[threadIdx.x] = bv;
    best_i[threadIdx.x] = bi;
    __syncthreads();
    for (int off = 128; off > 0; off >>= 1) {
        if (threadIdx.x < off) {
            const double ov = best_v[threadIdx.x + off];
            const int oi = best_i[threadIdx.x + off];
            if (ov > best_v[threadIdx.x] || (ov == best_v[threadIdx.x] && oi < best_i[threadIdx.x])) {
                best_v[threadIdx.x] = ov;
                best_i[threadIdx.x] = oi;
            }
        }
        __syncthreads();
    }
    const double sign = v[best_i[0]] < 0.0 ? -1.0 : 1.0;
    for (int k = threadIdx.x; k < K; k += 256) store_f(Pt + (int64_t)l * ldp + k, (float)(sign * v[k]));
    if (l == 0 && evals)
        for (int i = threadIdx.x; i < K; i += 256) evals[i] = (float)D[idx[i]];
}

inline int ceil_div_i(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

// ---- rocSOLVER, loaded on first use ----------------------------------------

typedef rocblas_status (*create_handle_fn)(rocblas_handle*);
typedef rocblas_status (*set_stream_fn)(rocblas_handle, hipStream_t);
typedef rocblas_status (*dsyevd_fn)(rocblas_handle, const rocblas_evect, const rocblas_fill, const rocblas_int,
                                    double*, const rocblas_int, double*, double*, rocblas_int*);

struct Solver {
    bool ok = false;
    create_handle_fn create = nullptr;
    set_stream_fn set_stream = nullptr;
    dsyevd_fn dsyevd = nullptr;
    rocblas_handle handles[64] = {};   // one per device, created on first use
    std::mutex mu;
};

Solver& solver() {
    static Solver s;
    static std::once_flag once;
    std::call_once(once, [] {
        void* blas = dlopen("librocblas.so.5", RTLD_NOW | RTLD_GLOBAL);
        void* sol = dlopen("librocsolver.so.0", RTLD_NOW | RTLD_GLOBAL);
        if (!blas || !sol) return;
        s.create = (create_handle_fn)dlsym(blas, "rocblas_create_handle");
        s.set_stream = (set_stream_fn)dlsym(blas, "rocblas_set_stream");
        s.dsyevd = (dsyevd_fn)dlsym(sol, "rocsolver_dsyevd");
        s.ok = s.create && s.set_stream && s.dsyevd;
    });
    return s;
}

}  // namespace

size_t autocorr_workspace_bytes(int64_t M, int64_t K, bool f32) {
    const int64_t ldt = (M + 7) / 8 * 8;
    size_t b = (size_t)K * ldt * (f32 ? 4 : 2);               // Xt
    b = (b + 255) / 256 * 256;
    b += (size_t)((M + 63) / 64 * 64) * 4;                    // inverse norms
    b = (b + 255) / 256 * 256;
    b += (size_t)autocorr_ranges(M, K, f32) * K * splitk_ld((int)K) * 4;   // fp32 sums per depth range
    return b;
}

int autocorr_ranges(int64_t M, int64_t K, bool f32) {
    if (f32) return 1;
    // enough depth ranges to give the chip up to 256 workgroups in one
    // round, each range at least 16 steps of 64 tokens deep
    const int64_t n = (K + 255) / 256;
    const int64_t tiles = n * (n + 1) / 2;
    const int64_t steps = (M + 63) / 64;
    int64_t S = 256 / tiles;
    if (S > steps / 16) S = steps / 16;
    if (S < 1) S = 1;
    // the GEMM uses ceil(steps / ceil(steps / S)) non-empty ranges
    const int64_t per = (steps + S - 1) / S;
    return (int)((steps + per - 1) / per);
}

hipError_t launch_autocorr_update(const void* X, int64_t ldx, int M, int K, bool f32, bool normalize,
                                  float alpha, float* C, int64_t ldc, void* workspace, hipStream_t stream) {
    const int64_t ldt = (M + 7) / 8 * 8;
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    size_t off = (size_t)K * ldt * (f32 ? 4 : 2);
    off = (off + 255) / 256 * 256;
    float* inv = reinterpret_cast<float*>(ws + off);
    off += (size_t)((M + 63) / 64 * 64) * 4;
    off = (off + 255) / 256 * 256;
    float* part = reinterpret_cast<float*>(ws + off);
    const int S = autocorr_ranges(M, K, f32);
    const int64_t ldp = splitk_ld(K);

    if (normalize) {
        if (f32)
            hipLaunchKernelGGL(token_inv_norm_kernel<float>, dim3(ceil_div_i(M, 4)), dim3(256), 0, stream,
                               static_cast<const float*>(X), ldx, M, K, inv);
        else
            hipLaunchKernelGGL(token_inv_norm_bf16_kernel, dim3(ceil_div_i(M, 4)), dim3(256), 0, stream,
                               static_cast<const uint16_t*>(X), ldx, M, K, inv);
    }
    const dim3 tgrid(ceil_div_i(M, 64), ceil_div_i(K, 64));
    if (f32)
        hipLaunchKernelGGL(transpose_scale_kernel<float>, tgrid, dim3(256), 0, stream, static_cast<const float*>(X),
                           ldx, normalize ? inv : nullptr, reinterpret_cast<float*>(ws), ldt, M, K);
    else if (normalize)
        hipLaunchKernelGGL(transpose_scale_bf16_kernel, tgrid, dim3(256), 0, stream,
                           static_cast<const uint16_t*>(X), ldx, inv, reinterpret_cast<uint16_t*>(ws), ldt, M, K);
    else
        hipLaunchKernelGGL(transpose_bf16_kernel, tgrid, dim3(256), 0, stream, static_cast<const uint16_t*>(X),
                           ldx, reinterpret_cast<uint16_t*>(ws), ldt, M, K);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;

    if (f32) {
        const float* Xt = reinterpret_cast<const float*>(ws);
        e = launch_gemm_tn_f32(Xt, ldt, Xt, ldt, part, ldp, K, K, M, stream);
    } else {
        GemmArgs g{};
        g.A = reinterpret_cast<const uint16_t*>(ws);
        g.lda = ldt;
        g.B = g.A;
        g.ldb = ldt;
        g.R = K;
        g.Cc = K;
        g.D = M;
        g.tile = TILE_256x256;
        g.splits = S;
        g.partial = part;
        int used = 0;
        e = launch_gemm_tn_bf16_v3_ranges(g, true, &used, stream);
        if (e == hipSuccess && used != S) return hipErrorInvalidValue;
    }
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(accumulate_kernel, dim3(ceil_div_i(K, 64), ceil_div_i(K, 64)), dim3(256), 0, stream, part,
                       S, (int64_t)K * ldp, ldp, C, ldc, K, K, alpha, f32 ? 0 : 256);
    return hipGetLastError();
}

hipError_t launch_transpose(const void* src, int64_t lds, int rows, int cols, void* dst, int64_t ldd, bool f32,
                            hipStream_t stream) {
    const dim3 grid(ceil_div_i(rows, 64), ceil_div_i(cols, 64));
    if (f32)
        hipLaunchKernelGGL(transpose_scale_kernel<float>, grid, dim3(256), 0, stream, static_cast<const float*>(src),
                           lds, nullptr, static_cast<float*>(dst), ldd, rows, cols);
    else
        hipLaunchKernelGGL(transpose_bf16_kernel, grid, dim3(256), 0, stream, static_cast<const uint16_t*>(src), lds,
                           static_cast<uint16_t*>(dst), ldd, rows, cols);
    return hipGetLastError();
}

size_t pca_workspace_bytes(int64_t K) {
    size_t b = (size_t)K * K * 8;          // the matrix, then its eigenvectors
    b += (size_t)K * 8 * 2;                // eigenvalues, off-diagonal scratch
    b += 256;                              // solver status
    b += (size_t)K * 4;                    // selection order
    return (b + 255) / 256 * 256;
}

size_t symprod_workspace_bytes(int64_t K) { return (size_t)K * splitk_ld((int)K) * 4; }

hipError_t launch_symmetrized_product(const float* A, int64_t lda, const float* B, int64_t ldb, float* C,
                                      int64_t ldc, int K, float alpha, float beta, void* workspace,
                                      hipStream_t stream) {
    float* P = static_cast<float*>(workspace);
    const int64_t ldp = splitk_ld(K);
    hipError_t e = launch_gemm_tn_f32(A, lda, B, ldb, P, ldp, K, K, K, stream);
    if (e != hipSuccess) return e;
    hipLaunchKernelGGL(symmetrize_kernel, dim3(ceil_div_i(K, 64), ceil_div_i(K, 64)), dim3(256), 0, stream, P,
                       ldp, C, ldc, K, alpha, beta);
    return hipGetLastError();
}

bool pca_available() { return solver().ok; }

hipError_t launch_principal_components(const float* C, int64_t ldc, int K, int L, bool by_magnitude, void* Pt,
                                       int64_t ldp, bool f32, float* evals, int* info, void* workspace,
                                       hipStream_t stream) {
    Solver& s = solver();
    if (!s.ok) return hipErrorSharedObjectInitFailed;
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= 64) return hipErrorInvalidDevice;
    unsigned char* ws = static_cast<unsigned char*>(workspace);
    double* A = reinterpret_cast<double*>(ws);
    double* D = A + (int64_t)K * K;
    double* E = D + K;
    rocblas_int* st = reinterpret_cast<rocblas_int*>(E + K);
    int* idx = reinterpret_cast<int*>(reinterpret_cast<unsigned char*>(st) + 256);
    const int64_t total = (int64_t)K * K;
    const int blocks = (int)(total / 256 < 4096 ? (total + 255) / 256 : 4096);
    hipLaunchKernelGGL(widen_kernel, dim3(blocks), dim3(256), 0, stream, C, ldc, A, K);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    {
        // one handle per device, shared by the calls on it: the stream is set
        // and the solver enqueued under the lock
        std::lock_guard<std::mutex> lk(s.mu);
        if (!s.handles[dev] && s.create(&s.handles[dev]) != rocblas_status_success) {
            s.handles[dev] = nullptr;
            return hipErrorSharedObjectInitFailed;
        }
        rocblas_handle h = s.handles[dev];
        if (s.set_stream(h, stream) != rocblas_status_success) return hipErrorInvalidHandle;
        // A row-major is Aᵀ column-major; the lower triangle of that is the
        // upper triangle (c >= r) of C
        const rocblas_status rs = s.dsyevd(h, rocblas_evect_original, rocblas_fill_lower, K, A, K, D, E, st);
        if (rs != rocblas_status_success) return hipErrorLaunchFailure;
    }
    hipLaunchKernelGGL(order_kernel, dim3(1), dim3(64), 0, stream, D, K, by_magnitude ? 1 : 0, idx);
    if (f32)
        hipLaunchKernelGGL(select_kernel<float>, dim3(L), dim3(256), 0, stream, A, D, idx, K, L,
                           static_cast<float*>(Pt), ldp, evals);
    else
        hipLaunchKernelGGL(select_kernel<uint16_t>, dim3(L), dim3(256), 0, stream, A, D, idx, K, L,
                           static_cast<uint16_t*>(Pt), ldp, evals);
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    if (info) e = hipMemcpyAsync(info, st, sizeof(int), hipMemcpyDeviceToDevice, stream);
    return e;
}

}  // namespace espace
