// Host-side launchers of the gfx950 kernels (internal to the library).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace espace {

enum TileKind {
    TILE_256x256 = 0,
    TILE_256x128 = 1,
    TILE_128x256 = 2,
    TILE_128x128 = 3,
    TILE_256x256_W8 = 4,     // 8 waves as 2 x 4 (128 x 64 each)
    TILE_256x256_W8T = 5,    // 8 waves as 4 x 2 (64 x 128 each)
    TILE_128x192 = 6,        // 8 waves as 4 x 2 (32 x 96 each)
    TILE_256x192_W8 = 7,     // 8 waves as 4 x 2 (64 x 96 each)
    SKINNY_RG1_W4 = 10,
    SKINNY_RG2_W4 = 11,
    SKINNY_RG1_W8 = 12,
    SKINNY_RG2_W8 = 13,
    SKINNY_RG1_W4_U8 = 14,   // as above with 8 steps of loads in flight per wave
    SKINNY_RG2_W4_U8 = 15,
    SKINNY_RG1_W8_U8 = 16,
    SKINNY_RG2_W8_U8 = 17,
    SKINNY_RG1_W8_U6 = 18,   // 6 steps in flight (48-step depths split evenly over 8 waves)
    SKINNY_RG2_W4_U6 = 19,
    SKINNY_RG1_W16_U8 = 20,  // 16 waves: one workgroup keeps 128 steps in flight
    SKINNY_RG1_W16_U4 = 21,
    SKINNY_SEG2_W8_U8 = 22,  // 8 rows x 2 depth segments per MFMA operand, N <= 8
    SKINNY_SEG2_W16_U4 = 23,
    SKINNY_SEG2_TG2_W8_U8 = 24,   // the same with two groups of 8 tokens, N <= 16
    SKINNY_SEG2_TG2_W16_U4 = 25,
};

// Limit of the bounded cross-workgroup waits and the device counter of the
// waits that gave up (see note_timeout).
struct WaitCfg {
    unsigned spins = 1u << 22;
    unsigned long long* timeouts = nullptr;
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
    float* partial;     // splits * R * splitk_ld(Cc) fp32 (workspace); with `pair`:
                        // tiles * tile area fp32, then one 8-byte state word per tile
    int cus = 256;      // compute units of the device (persistent grids)
    WaitCfg wait;       // bounded waits of the pair combine
    int pair = 0;       // splits == 2 combined inside the kernel (no reduce pass)
    unsigned long long epoch = 0;   // per-call tag of the pair state words
    // Row-pair layout (a matrix the library keeps to itself: Z in the layer's
    // workspace).  Element (r, k) sits at (r / 2) * ld + (k / 32) * 64 +
    // (r % 2) * 32 + k % 32: every 128-byte block holds 32 consecutive
    // elements of two neighbouring rows, so a 32-deep load of a row pair is
    // one whole cache line.  ld (elements per row pair) is a multiple of 64.
    int a_pairs = 0;    // A is in the row-pair layout (lda its pair pitch)
    int c_pairs = 0;    // write C (bf16) in the row-pair layout (ldc its pair pitch)
};

// offset (elements) of element (r, k) of a row-pair matrix with pair pitch ld
__host__ __device__ inline int64_t pair_offset(int64_t r, int64_t k, int64_t ld) {
    return (r >> 1) * ld + (k >> 5) * 64 + (r & 1) * 32 + (k & 31);
}

// Tile size of a TileKind in the pair-combine kernel (rows, columns).
void tile_dims(int tile, int* bm, int* bn);

// leading dimension of split-K partial sums
inline int64_t splitk_ld(int Cc) { return (Cc + 7) / 8 * 8; }

hipError_t launch_gemm_tn_bf16(const GemmArgs& g, hipStream_t stream);
hipError_t launch_gemm_tn_bf16_v2(const GemmArgs& g, hipStream_t stream);
// Four-wave 256 x 256 and 256 x 192 kernel with a hand-ordered main loop;
// hipErrorInvalidValue for products it does not take (other tiles, fp32
// output, >= 2^31 elements).
hipError_t launch_gemm_tn_bf16_v3(const GemmArgs& g, hipStream_t stream);
hipError_t launch_skinny_tn_bf16(const GemmArgs& g, hipStream_t stream);
// Vector-ALU product for 1 <= R <= 2 tokens with whole-row streaming (tile,
// splits, partial unused); gemv_supported says whether the tokens fit its LDS.
bool gemv_supported(int R, int D);
hipError_t launch_gemv_tn_bf16(const GemmArgs& g, hipStream_t stream);
// Persistent streaming product for up to 16 tokens with the many-row operand
// streamed through an LDS ring (tile, splits, partial unused); stream_supported
// says whether the tokens and depth fit (depth up to 6144).
bool stream_supported(int R, int D);
hipError_t launch_stream_tn_bf16(const GemmArgs& g, hipStream_t stream);
// out_bf16: 0 fp32 output, 1 bf16, 2 bf16 in the row-pair layout
hipError_t launch_splitk_reduce(const float* P, int S, int64_t split_stride, int64_t ldp,
                                void* C, int64_t ldc, int R, int Cc, int out_bf16,
                                hipStream_t stream);
hipError_t launch_gemm_tn_f32(const float* A, int64_t lda, const float* B, int64_t ldb,
                              float* C, int64_t ldc, int R, int Cc, int D, hipStream_t stream);

// fp32 sums of the depth ranges of a 256 x 256 or 256 x 192 tiled product
// (g.splits ranges requested; *ranges receives the number of non-empty ones),
// range s at g.partial + s * R * splitk_ld(Cc); not combined.  upper (square
// 256 x 256 tiling only): just the tiles on and above the diagonal.
hipError_t launch_gemm_tn_bf16_v3_ranges(const GemmArgs& g, bool upper, int* ranges, hipStream_t stream);

// Calibration (autocorrelation of calibration tokens, principal components).
int autocorr_ranges(int64_t M, int64_t K, bool f32);
size_t autocorr_workspace_bytes(int64_t M, int64_t K, bool f32);
hipError_t launch_autocorr_update(const void* X, int64_t ldx, int M, int K, bool f32, bool normalize,
                                  float alpha, float* C, int64_t ldc, void* workspace, hipStream_t stream);
size_t pca_workspace_bytes(int64_t K);
bool pca_available();
hipError_t launch_principal_components(const float* C, int64_t ldc, int K, int L, bool by_magnitude, void* Pt,
                                       int64_t ldp, bool f32, float* evals, int* info, void* workspace,
                                       hipStream_t stream);
size_t symprod_workspace_bytes(int64_t K);
// dst[c][r] = src[r][c] for r < rows, c < cols (bf16 or fp32; values copied
// exactly).  Both leading dimensions are multiples of 8 elements; the bf16
// kernel may write the padding columns of dst's rows (scratch only).
hipError_t launch_transpose(const void* src, int64_t lds, int rows, int cols, void* dst, int64_t ldd, bool f32,
                            hipStream_t stream);
hipError_t launch_symmetrized_product(const float* A, int64_t lda, const float* B, int64_t ldb, float* C,
                                      int64_t ldc, int K, float alpha, float beta, void* workspace,
                                      hipStream_t stream);

// ---- MX-FP8 products (gemm_mxfp8.hip) ----------------------------------------
// out[r][c] = sum_d T[r][d]·W[c][d] over MX-FP8 operands (codes with zero
// padding up to round_up(D, 128), one E8M0 scale byte per 32 along d).
struct MxGemmArgs {
    const uint8_t* T;  int64_t ldt;     // token-side codes [R][ldt]
    const uint8_t* Ts; int64_t ldts;    // its scale bytes [R][ldts]
    const uint8_t* W;  int64_t ldw;     // weight-side codes [C][ldw]
    const uint8_t* Ws; int64_t ldws;    // its scale bytes [C][ldws]
    void* out;         int64_t ldo;     // bf16 Y [R][ldo], or MX-FP8 codes [R][ldo]
    uint8_t* outs;     int64_t ldos;    // MX-FP8 output: scale bytes [R][ldos]
    int R, C, D;
    int cpad;                           // MX-FP8 output: columns written, round_up(C, 128)
    // Row pairs (the MX-FP8 layer's Z in its workspace): code (r, c) at
    // (r / 2) * ld + (c / 64) * 128 + (r % 2) * 64 + c % 64, ld (bytes per
    // row pair) a multiple of 128; the scale bytes stay one row per token.
    int t_pairs = 0;                    // the token codes T (bf16 output only)
    int out_pairs = 0;                  // the MX-FP8 output codes
};
// Tile of the MX GEMM for R x C outputs (0: 256 x 256, 1: 256 x 128, 2: 128 x 128;
// 2 only for MX-FP8 output).
int mx_gemm_tile(int R, int C, int cus, int out_mx);
// out_mx: write MX-FP8 (codes and scales along the columns) instead of bf16.
// hipErrorInvalidValue when an operand spans 2^31 bytes or more.
hipError_t launch_gemm_mx(const MxGemmArgs& a, int out_mx, int cus, hipStream_t stream);
hipError_t launch_mx_quantize(const uint16_t* A, int64_t lda, int R, int C, uint8_t* Q, int64_t ldq, uint8_t* S,
                              int64_t lds, hipStream_t stream);

}  // namespace espace
