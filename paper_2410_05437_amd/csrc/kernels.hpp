// Host-side launchers of the gfx950 kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace espace {

enum TileKind {
    TILE_256x256 = 0,
    TILE_256x128 = 1,
    TILE_128x256 = 2,
    TILE_128x128 = 3,
    TILE_256x256_W8 = 4,     // 8 waves as 2 x 4 (128 x 64 each)
    TILE_256x256_W8T = 5,    // 8 waves as 4 x 2 (64 x 128 each)
    SKINNY_RG1_W4 = 10,
    SKINNY_RG2_W4 = 11,
    SKINNY_RG1_W8 = 12,
    SKINNY_RG2_W8 = 13,
};

// One "TN" product C[r][c] = sum_k A[r][k] * B[c][k]  (bf16 in, fp32 accumulate).
struct GemmArgs {
    const uint16_t* A;
    int64_t lda;
    const uint16_t* B;
    int64_t ldb;
    void* C;            // bf16 output (or fp32 when c_f32)
    int64_t ldc;
    int R;              // rows of A and C
    int Cc;             // rows of B = columns of C
    int D;              // reduced dimension
    int c_f32;          // 1: write fp32 output
    int tile;           // TileKind
    int splits;         // depth ranges; > 1 needs `partial`
    float* partial;     // splits * R * splitk_ld(Cc) fp32 (workspace)
    int variant = 0;    // kernel variant (tuning)
};

// leading dimension of split-K partial sums
inline int64_t splitk_ld(int Cc) { return (Cc + 7) / 8 * 8; }

hipError_t launch_gemm_tn_bf16(const GemmArgs& g, hipStream_t stream);
hipError_t launch_gemm_tn_bf16_v2(const GemmArgs& g, hipStream_t stream);
hipError_t launch_gemm_tn_bf16_pp(const GemmArgs& g, hipStream_t stream);
hipError_t launch_skinny_tn_bf16(const GemmArgs& g, hipStream_t stream);
hipError_t launch_splitk_reduce(const float* P, int S, int64_t split_stride, int64_t ldp,
                                void* C, int64_t ldc, int R, int Cc, int out_bf16,
                                hipStream_t stream);
hipError_t launch_gemm_tn_f32(const float* A, int64_t lda, const float* B, int64_t ldb,
                              float* C, int64_t ldc, int R, int Cc, int D, hipStream_t stream);

}  // namespace espace
