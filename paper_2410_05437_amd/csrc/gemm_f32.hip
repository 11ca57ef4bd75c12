// float32 "TN" product C[r][c] = sum_k A[r][k] * B[c][k] with fp32 FMA.
//
// The fp32 layer variant is small (it serves the float32 workloads and the
// exactness checks); a 64x64 tile per 256-thread workgroup, 16-deep LDS
// steps, 4x4 outputs per thread.  Tiles are stored k-major in LDS so each
// thread reads its four rows / four columns as one 16-byte vector.
#include "common.hpp"
#include "kernels.hpp"

namespace espace {

namespace {

constexpr int FT = 64;    // tile edge
constexpr int FK = 16;    // depth step
constexpr int FPAD = 4;

__device__ __forceinline__ f32x4_t load4_masked(const float* row, int k, int depth) {
    f32x4_t v = {0.f, 0.f, 0.f, 0.f};
    const int nvalid = depth - k;
    if (nvalid >= 4) {
        v = *reinterpret_cast<const f32x4_t*>(row + k);
    } else if (nvalid > 0) {
        const f32x4_t t = *reinterpret_cast<const f32x4_t*>(row + k);
#pragma unroll
        for (int e = 0; e < 4; ++e) v[e] = e < nvalid ? t[e] : 0.f;
    }
    return v;
}

__global__ __launch_bounds__(256)
void gemm_tn_f32_kernel(const float* __restrict__ A, int64_t lda,
                        const float* __restrict__ B, int64_t ldb,
                        float* __restrict__ C, int64_t ldc, int R, int Cc, int D) {
    __shared__ float As[FK][FT + FPAD];
    __shared__ float Bs[FK][FT + FPAD];
    const int tid = threadIdx.x;
    const int tx = tid & 15;
    const int ty = tid >> 4;
    const int row0 = blockIdx.y * FT;
    const int col0 = blockIdx.x * FT;
    // loader: row tid/4, 4 consecutive k at (tid%4)*4
    const int lr = tid >> 2;
    const int lk = (tid & 3) * 4;
    int ar = row0 + lr;
    ar = ar < R ? ar : R - 1;
    int bc = col0 + lr;
    bc = bc < Cc ? bc : Cc - 1;
    const float* arow = A + (int64_t)ar * lda;
    const float* brow = B + (int64_t)bc * ldb;

    float acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = 0.f;

    for (int k0 = 0; k0 < D; k0 += FK) {
        const f32x4_t va = load4_masked(arow, k0 + lk, D);
        const f32x4_t vb = load4_masked(brow, k0 + lk, D);
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            As[lk + e][lr] = va[e];
            Bs[lk + e][lr] = vb[e];
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < FK; ++kk) {
            const f32x4_t a = *reinterpret_cast<const f32x4_t*>(&As[kk][ty * 4]);
            const f32x4_t b = *reinterpret_cast<const f32x4_t*>(&Bs[kk][tx * 4]);
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = __builtin_fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int r = row0 + ty * 4 + i;
        if (r >= R) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int c = col0 + tx * 4 + j;
            if (c < Cc) C[(int64_t)r * ldc + c] = acc[i][j];
        }
    }
}

}  // namespace

hipError_t launch_gemm_tn_f32(const float* A, int64_t lda, const float* B, int64_t ldb,
                              float* C, int64_t ldc, int R, int Cc, int D, hipStream_t stream) {
    dim3 grid((Cc + FT - 1) / FT, (R + FT - 1) / FT);
    hipLaunchKernelGGL(gemm_tn_f32_kernel, grid, dim3(256), 0, stream, A, lda, B, ldb, C, ldc,
                       R, Cc, D);
    return hipGetLastError();
}

}  // namespace espace
