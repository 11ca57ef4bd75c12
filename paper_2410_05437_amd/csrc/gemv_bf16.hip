// Bandwidth-oriented bfloat16 product for one or two tokens (decode):
//
//     C[n][j] = sum_k A[n][k] * B[j][k],   n < R <= 2 (tokens), j < Cc
//
// One wave streams whole rows of B: lane l reads the 8-element chunks l,
// l + 64, l + 128, ... of a row, so every load instruction of a wave covers
// 1 KB of contiguous memory (the MFMA kernel's loads cover 16 rows x 64 B,
// which the memory system serves at a lower rate).  The arithmetic is on the
// vector ALU with bf16 pair dot products accumulating in fp32 (with so few
// tokens the 16 columns of an MFMA operand would be mostly empty): each lane
// adds its chunks in order, then a butterfly over the 64 lanes gives the sum,
// and the lane of a token writes it.  The order is fixed, so results do not
// depend on scheduling.
//
// Rows of at most 2048 elements (four 512-element passes) take the first
// kernel: every lane keeps its chunks of the tokens in registers, loaded
// once, so nothing waits for a workgroup-wide staging step, and a wave loads
// two rows per iteration.  Longer rows take the second kernel, which stages
// the tokens in LDS once per workgroup and walks each row in blocks of up to
// eight passes (kept there from five passes on: at eight passes the register
// form needs twice the registers and was slower, e.g. 34.7 against 33.6 µs
// on a 22016 x 4096 weight at one token).
#include "common.hpp"
#include "kernels.hpp"

namespace espace {

namespace {

constexpr int GV_WAVES = 4;
constexpr int GV_MAX_UB = 8;                   // 1 KB loads in flight per wave
constexpr int GV_LDS_MAX = 64 * 1024;          // token staging per workgroup
// Rows are spread over about this many waves (one or two rows per wave on
// the decode layers).  Measured at one token against 4096 waves: the
// Llama2-7B up+gate expansion 13.8 -> 13.0 µs, the QKV one 9.4 -> 8.4 µs;
// long rows (the LDS form) at one token gain again from one row per wave
// (32768: the up+gate dense weight 32.7 -> 30.3 µs, GPT3-22B's 53.7 ->
// 51.1 µs), short rows and two tokens do not.
constexpr int GV_TARGET_WAVES = 16384;
constexpr int GV_TARGET_WAVES_LONG1 = 32768;

int gv_tokens(int R) { return R <= 1 ? 1 : 2; }
int gv_passes(int D) { return ((D + 7) / 8 + 63) / 64; }

// acc + sum of the products of two chunks of 8 bfloat16 values, in element
// order, two products per instruction (v_dot2c_f32_bf16: the product of two
// bfloat16 values is exact in fp32).  The four words are named one by one:
// a bit cast of a subscripted vector element inside a loop compiled to the
// first element every time with this compiler.
__device__ __forceinline__ float dot2(uint32_t a, uint32_t b, float acc) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2_t, a), __builtin_bit_cast(bf16x2_t, b),
                                           acc, false);
}

__device__ __forceinline__ float dot_chunk(u32x4_t a, u32x4_t b, float acc) {
    acc = dot2(a.x, b.x, acc);
    acc = dot2(a.y, b.y, acc);
    acc = dot2(a.z, b.z, acc);
    return dot2(a.w, b.w, acc);
}

// Sum over the wave of each token's partial sums (fixed butterfly), written
// by the lane of the token.
template <int NT>
__device__ __forceinline__ void finish_row(const float (&acc)[NT], int lane, int R, int j,
                                           void* __restrict__ Cout, int64_t ldc, int out_f32) {
    float out = 0.f;
#pragma unroll
    for (int n = 0; n < NT; ++n) {
        float v = acc[n];
#pragma unroll
        for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m);
        out = lane == n ? v : out;
    }
    if (lane < NT && lane < R) {
        if (out_f32) reinterpret_cast<float*>(Cout)[(int64_t)lane * ldc + j] = out;
        else reinterpret_cast<uint16_t*>(Cout)[(int64_t)lane * ldc + j] = (uint16_t)bf16_rne(out);
    }
}

// Rows of at most UB passes; RB rows per iteration.
template <int NT, int UB, int RB>
__global__ __launch_bounds__(GV_WAVES * 64)
void gemv_rows_bf16_kernel(const uint16_t* __restrict__ A, int64_t lda,
                           const uint16_t* __restrict__ B, int64_t ldb,
                           void* __restrict__ Cout, int64_t ldc,
                           int R, int Cc, int D, int rows_per_wave, int out_f32) {
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nfull = D >> 9;           // passes entirely inside the row

    // chunk u of this lane: elements 8 * (64 * u + lane) ...; keep[u] masks
    // the elements at or beyond D (passes past the row: all of them, and
    // their loads read the row's first chunk)
    int off[UB];
    u32x4_t keep[UB];
#pragma unroll
    for (int u = 0; u < UB; ++u) {
        const int c = u * 64 + lane;
        const int valid = D - 8 * c;
        off[u] = valid > 0 ? 8 * c : 0;
        keep[u] = mask_chunk(u32x4_t{0xffffffffu, 0xffffffffu, 0xffffffffu, 0xffffffffu}, valid);
    }
    // Token chunks as loaded (masked where used, in the partial pass): these
    // loads stay in flight with the first rows'.  Token rows >= R load row
    // R - 1; their sums are never written.
    u32x4_t t[NT][UB];
#pragma unroll
    for (int n = 0; n < NT; ++n) {
        const uint16_t* arow = A + (int64_t)min(n, R - 1) * lda;
#pragma unroll
        for (int u = 0; u < UB; ++u) t[n][u] = *reinterpret_cast<const u32x4_t*>(arow + off[u]);
    }

    const int j_begin = (blockIdx.x * GV_WAVES + wave) * rows_per_wave;
    const int j_end = j_begin + rows_per_wave < Cc ? j_begin + rows_per_wave : Cc;
    for (int j = j_begin; j < j_end; j += RB) {
        u32x4_t w[RB][UB];
#pragma unroll
        for (int r = 0; r < RB; ++r) {
            // rows past the wave's range load its last row (not used)
            const int jr = j + r < j_end ? j + r : j_end - 1;
            const uint16_t* brow = B + (int64_t)jr * ldb;
#pragma unroll
            for (int u = 0; u < UB; ++u) w[r][u] = *reinterpret_cast<const u32x4_t*>(brow + off[u]);
        }
        __builtin_amdgcn_sched_barrier(0);   // all loads of the iteration issue before the first use
#pragma unroll
        for (int r = 0; r < RB; ++r) {
            float acc[NT];
#pragma unroll
            for (int n = 0; n < NT; ++n) acc[n] = 0.f;
#pragma unroll
            for (int u = 0; u < UB; ++u) {
                if (u < nfull) {
#pragma unroll
                    for (int n = 0; n < NT; ++n) acc[n] = dot_chunk(w[r][u], t[n][u], acc[n]);
                } else {
                    // both operands masked: the padding after D may hold
                    // anything.  The empty asm keeps the masked tokens from
                    // being hoisted out of the loop, which would make the
                    // prologue wait for the token loads.
                    u32x4_t k = keep[u];
                    asm volatile("" : "+v"(k));
#pragma unroll
                    for (int n = 0; n < NT; ++n) acc[n] = dot_chunk(w[r][u] & k, t[n][u] & k, acc[n]);
                }
            }
            if (j + r < j_end) finish_row<NT>(acc, lane, R, j + r, Cout, ldc, out_f32);
        }
    }
}

// Rows longer than UB passes: tokens staged in LDS, blocks of UB passes.
template <int NT, int UB>
__global__ __launch_bounds__(GV_WAVES * 64)
void gemv_tn_bf16_kernel(const uint16_t* __restrict__ A, int64_t lda,
                         const uint16_t* __restrict__ B, int64_t ldb,
                         void* __restrict__ Cout, int64_t ldc,
                         int R, int Cc, int D, int rows_per_wave, int out_f32) {
    extern __shared__ u32x4_t tok[];    // [NT][ldt] chunks of 8 bf16

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nch = (D + 7) >> 3;       // chunks per row
    const int npass = (nch + 63) >> 6;  // 64-chunk passes per row
    const int ldt = npass << 6;

    // staging: four chunks per thread in flight; chunks outside the tokens
    // load the first chunk of A and are zeroed
    constexpr int SU = 4;
    for (int i0 = threadIdx.x; i0 < NT * ldt; i0 += SU * GV_WAVES * 64) {
        u32x4_t v[SU];
        int valid[SU];
#pragma unroll
        for (int s = 0; s < SU; ++s) {
            const int i = i0 + s * GV_WAVES * 64;
            const int n = i / ldt;
            const int c = i - n * ldt;
            valid[s] = (i < NT * ldt && n < R && c < nch) ? D - 8 * c : 0;
            v[s] = *reinterpret_cast<const u32x4_t*>(A + (valid[s] > 0 ? (int64_t)n * lda + 8 * c : 0));
        }
#pragma unroll
        for (int s = 0; s < SU; ++s) {
            const int i = i0 + s * GV_WAVES * 64;
            if (i < NT * ldt) tok[i] = mask_chunk(v[s], valid[s]);
        }
    }
    __syncthreads();

    const int j_begin = (blockIdx.x * GV_WAVES + wave) * rows_per_wave;
    const int j_end = j_begin + rows_per_wave < Cc ? j_begin + rows_per_wave : Cc;
    for (int j = j_begin; j < j_end; ++j) {
        const uint16_t* brow = B + (int64_t)j * ldb;
        float acc[NT];
#pragma unroll
        for (int n = 0; n < NT; ++n) acc[n] = 0.f;
        for (int p0 = 0; p0 < npass; p0 += UB) {
            // UB passes of loads in flight; passes past the row load its
            // first chunk and are masked
            u32x4_t w[UB];
            int valid[UB];
#pragma unroll
            for (int u = 0; u < UB; ++u) {
                const int c = (p0 + u) * 64 + lane;
                valid[u] = p0 + u < npass ? D - 8 * c : 0;
                w[u] = *reinterpret_cast<const u32x4_t*>(brow + (valid[u] > 0 ? 8 * c : 0));
            }
            if ((p0 + UB) * 512 <= D) {
                // every chunk of these passes lies inside the row
#pragma unroll
                for (int u = 0; u < UB; ++u)
#pragma unroll
                    for (int n = 0; n < NT; ++n)
                        acc[n] = dot_chunk(w[u], tok[n * ldt + (p0 + u) * 64 + lane], acc[n]);
            } else {
#pragma unroll
                for (int u = 0; u < UB; ++u) {
                    const u32x4_t wv = mask_chunk(w[u], valid[u]);
                    const uint32_t keep = valid[u] > 0 ? 0xffffffffu : 0u;
                    const int c = valid[u] > 0 ? (p0 + u) * 64 + lane : 0;
#pragma unroll
                    for (int n = 0; n < NT; ++n) acc[n] = dot_chunk(wv, tok[n * ldt + c] & keep, acc[n]);
                }
            }
        }
        finish_row<NT>(acc, lane, R, j, Cout, ldc, out_f32);
    }
}

template <int NT, int UB>
hipError_t launch_ub(const GemmArgs& g, int rows_per_wave, hipStream_t stream) {
    const size_t lds = (size_t)NT * gv_passes(g.D) * 64 * 16;
    const int waves = (g.Cc + rows_per_wave - 1) / rows_per_wave;
    dim3 grid((waves + GV_WAVES - 1) / GV_WAVES), block(GV_WAVES * 64);
    hipLaunchKernelGGL((gemv_tn_bf16_kernel<NT, UB>), grid, block, lds, stream, g.A, g.lda, g.B, g.ldb,
                       g.C, g.ldc, g.R, g.Cc, g.D, rows_per_wave, g.c_f32);
    return hipGetLastError();
}

template <int NT, int UB, int RB>
hipError_t launch_rows(const GemmArgs& g, int rows_per_wave, hipStream_t stream) {
    rows_per_wave = (rows_per_wave + RB - 1) / RB * RB;
    const int waves = (g.Cc + rows_per_wave - 1) / rows_per_wave;
    dim3 grid((waves + GV_WAVES - 1) / GV_WAVES), block(GV_WAVES * 64);
    hipLaunchKernelGGL((gemv_rows_bf16_kernel<NT, UB, RB>), grid, block, 0, stream, g.A, g.lda, g.B, g.ldb,
                       g.C, g.ldc, g.R, g.Cc, g.D, rows_per_wave, g.c_f32);
    return hipGetLastError();
}

template <int NT>
hipError_t launch_nt(const GemmArgs& g, int rows_per_wave, hipStream_t stream) {
    switch (gv_passes(g.D)) {
        case 1: return launch_rows<NT, 1, 2>(g, rows_per_wave, stream);
        case 2: return launch_rows<NT, 2, 2>(g, rows_per_wave, stream);
        case 3: return launch_rows<NT, 3, 2>(g, rows_per_wave, stream);
        case 4: return launch_rows<NT, 4, 2>(g, rows_per_wave, stream);
        case 5: return launch_ub<NT, 5>(g, rows_per_wave, stream);
        case 6: return launch_ub<NT, 6>(g, rows_per_wave, stream);
        case 7: return launch_ub<NT, 7>(g, rows_per_wave, stream);
        case 8: return launch_ub<NT, 8>(g, rows_per_wave, stream);
        default: return launch_ub<NT, GV_MAX_UB>(g, rows_per_wave, stream);
    }
}

}  // namespace

bool gemv_supported(int R, int D) {
    return R >= 1 && R <= 2 && D >= 1 && (int64_t)gv_tokens(R) * gv_passes(D) * 64 * 16 <= GV_LDS_MAX;
}

hipError_t launch_gemv_tn_bf16(const GemmArgs& g, hipStream_t stream) {
    if (!gemv_supported(g.R, g.D) || g.Cc < 1) return hipErrorInvalidValue;
    const int target = (gv_passes(g.D) > 4 && g.R == 1) ? GV_TARGET_WAVES_LONG1 : GV_TARGET_WAVES;
    int rows_per_wave = (g.Cc + target - 1) / target;
    if (rows_per_wave < 1) rows_per_wave = 1;
    return gv_tokens(g.R) == 1 ? launch_nt<1>(g, rows_per_wave, stream) : launch_nt<2>(g, rows_per_wave, stream);
}

}  // namespace espace
