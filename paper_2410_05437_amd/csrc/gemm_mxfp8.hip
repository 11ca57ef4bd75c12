// The low-precision projected linear layer on gfx950's block-scaled MFMA:
// operands in MX-FP8 (E4M3 elements, one power-of-two E8M0 scale per 32
// elements along the reduction dimension), the two products of Section 2.2,
// Eq. 3 with fp32 accumulation.  The projection's epilogue writes Z back in
// MX-FP8 along L, so the expansion consumes it as it consumes the folded
// weight.
//
// v_mfma_scale_f32_16x16x128_f8f6f4 (operands "A" then "B", scale bytes in
// byte 0 of a VGPR per lane):
//   - lane l of an operand holds row l % 16 of its 16 x 128 slice: bytes
//     0..15 are depth 16 (l / 16) .. +15 and bytes 16..31 are depth
//     64 + 16 (l / 16) .. +15;
//   - the scale byte of lane l applies to row l % 16 over depth block
//     32 (l / 16) .. +31;
//   - lane l of the result holds rows 4 (l / 16) + {0..3} (from A) of column
//     l % 16 (from B).
// The weight-side slice is passed as A and the token-side slice as B, so a
// lane's four results are four consecutive output features of one token.
//
// The scaled MFMA adds the running sum C with limited precision (on gfx950
// the result differs from the exact C + sum of products by up to about
// 2^-12 (|C| + sum |a·b|)); the accumulators stay in the MFMA chain, and the
// parity tests bound the error accordingly.
#include "common.hpp"
#include "kernels.hpp"

namespace espace {

namespace {

typedef int i32x8_t __attribute__((ext_vector_type(8)));
typedef int i32x4_t __attribute__((ext_vector_type(4)));

constexpr int MX_BK = 128;   // depth of one step: one block-scaled MFMA

// 16-byte chunk c of LDS row r sits at chunk c ^ mx_swz(r): the 16 rows one
// fragment read touches then fall on distinct bank groups
__device__ __forceinline__ int mx_swz(int r) { return (r >> 1) & 7; }

// Tile BT tokens x BW output columns, 4 waves as 2 x 2, each BT/2 x BW/2.
// A stage holds the tile's BT + BW rows of 128 code bytes (token rows first),
// then one scale dword (the 4 blocks of the step) per row.
template <int BT, int BW>
struct MxCfg {
    static constexpr int ROWS = BT + BW;
    static constexpr int DATA = ROWS * MX_BK;
    static constexpr int STAGE = DATA + ROWS * 4;
    static constexpr int SMEM = 2 * STAGE;
    static constexpr int WT = BT / 2, WW = BW / 2;
    static constexpr int NI = WT / 16, NJ = WW / 16;
    static constexpr int NDL = ROWS / 8;    // 1 KB code loads per stage (8 rows each)
    static constexpr int NSL = ROWS / 64;   // 256-byte scale loads per stage (64 rows each)
    static_assert(BT % 64 == 0 && BW % 64 == 0 && NDL % 4 == 0, "tile");
};

// Issue the direct-to-LDS loads of depth step t into `stage`: codes (16
// bytes per lane) and scale dwords (4 bytes per lane).  Rows past the matrix
// read its last row (their results are never stored).
template <int BT, int BW>
__device__ __forceinline__ void mx_issue(unsigned char* stage, const MxGemmArgs& a, int row0, int col0, int t,
                                         int wave, int lane) {
    using C = MxCfg<BT, BW>;
    const auto tr = __builtin_amdgcn_make_buffer_rsrc((void*)a.T, (short)0, (int)(a.R * a.ldt), 0x00020000);
    const auto wr = __builtin_amdgcn_make_buffer_rsrc((void*)a.W, (short)0, (int)(a.C * a.ldw), 0x00020000);
    const auto ts = __builtin_amdgcn_make_buffer_rsrc((void*)a.Ts, (short)0, (int)(a.R * a.ldts), 0x00020000);
    const auto ws = __builtin_amdgcn_make_buffer_rsrc((void*)a.Ws, (short)0, (int)(a.C * a.ldws), 0x00020000);
#pragma unroll
    for (int j = 0; j < C::NDL / 4; ++j) {
        const int q = wave + 4 * j;
        const int rr = 8 * q + (lane >> 3);
        const int c = (lane & 7) ^ mx_swz(rr);
        if (8 * q < BT) {
            const int g = min(row0 + rr, a.R - 1);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(tr, (__attribute__((address_space(3))) void*)(stage + q * 1024), 16,
                                                     (int)(g * a.ldt + 16 * c), t * MX_BK, 0, 0);
        } else {
            const int g = min(col0 + rr - BT, a.C - 1);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(wr, (__attribute__((address_space(3))) void*)(stage + q * 1024), 16,
                                                     (int)(g * a.ldw + 16 * c), t * MX_BK, 0, 0);
        }
    }
    for (int s = wave; s < C::NSL; s += 4) {
        const int rr = 64 * s + lane;
        if (64 * s < BT) {
            const int g = min(row0 + rr, a.R - 1);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ts, (__attribute__((address_space(3))) void*)(stage + C::DATA + s * 256),
                                                     4, (int)(g * a.ldts), 4 * t, 0, 0);
        } else {
            const int g = min(col0 + rr - BT, a.C - 1);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ws, (__attribute__((address_space(3))) void*)(stage + C::DATA + s * 256),
                                                     4, (int)(g * a.ldws), 4 * t, 0, 0);
        }
    }
}

// The lane's 32 code bytes of LDS row rr of a stage, in MFMA operand order.
__device__ __forceinline__ i32x8_t mx_frag(const unsigned char* stage, int rr, int lane) {
    const unsigned char* row = stage + rr * MX_BK;
    const int s = mx_swz(rr);
    const i32x4_t lo = *reinterpret_cast<const i32x4_t*>(row + (((lane >> 4) ^ s) << 4));
    const i32x4_t hi = *reinterpret_cast<const i32x4_t*>(row + (((4 + (lane >> 4)) ^ s) << 4));
    return i32x8_t{lo[0], lo[1], lo[2], lo[3], hi[0], hi[1], hi[2], hi[3]};
}

__device__ __forceinline__ void mx_wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0F70); }

// MX-FP8 code byte of x (already divided by its block scale): clamp to the
// largest E4M3 magnitude, then the hardware's round-to-nearest-even
// conversion (which turns magnitudes past 464 into NaN, hence the clamp).
__device__ __forceinline__ uint32_t mx_pack4(float x0, float x1, float x2, float x3) {
    x0 = fminf(fmaxf(x0, -448.f), 448.f);
    x1 = fminf(fmaxf(x1, -448.f), 448.f);
    x2 = fminf(fmaxf(x2, -448.f), 448.f);
    x3 = fminf(fmaxf(x3, -448.f), 448.f);
    uint32_t r = (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(x0, x1, 0, false);
    return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(x2, x3, (int)r, true);
}

// Scale exponent S of a block with largest magnitude amax: floor(log2 amax)
// - 8 with the byte S + 127 clamped to [0, 254]; byte 0 for a zero block.
__device__ __forceinline__ int mx_scale_byte(float amax) {
    if (!(amax > 0.f)) return 0;
    const int e = __builtin_amdgcn_frexp_expf(amax) - 1;   // floor(log2 amax)
    const int b = e - 8 + 127;
    return b < 0 ? 0 : (b > 254 ? 254 : b);
}

template <int BT, int BW, int OUT>
__global__ __launch_bounds__(256, (BT + BW) <= 256 ? 2 : 1)
void gemm_mx_kernel(MxGemmArgs a) {
    using C = MxCfg<BT, BW>;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[C::SMEM];

    const int tiles_c = (a.C + BW - 1) / BW;
    const int tiles = tiles_c * ((a.R + BT - 1) / BT);
    int tile_r, tile_c;
    tile_coords<8>(blockIdx.x, tiles, tiles_c, 0, tile_r, tile_c);
    const int row0 = tile_r * BT, col0 = tile_c * BW;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wt0 = (wave >> 1) * C::WT;          // the wave's token rows in the tile
    const int ww0 = (wave & 1) * C::WW;           // its output columns
    const int lr = lane & 15, q = lane >> 4;

    f32x4_t acc[C::NI][C::NJ];
#pragma unroll
    for (int i = 0; i < C::NI; ++i)
#pragma unroll
        for (int j = 0; j < C::NJ; ++j) acc[i][j] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    const int steps = (a.D + MX_BK - 1) / MX_BK;
    mx_issue<BT, BW>(smem, a, row0, col0, 0, wave, lane);
    mx_wait_vm0();
    __syncthreads();
    for (int t = 0; t < steps; ++t) {
        const unsigned char* cur = smem + (t & 1) * C::STAGE;
        // the other stage was last read in step t - 1, before the barrier
        // that ended it
        if (t + 1 < steps) mx_issue<BT, BW>(smem + ((t + 1) & 1) * C::STAGE, a, row0, col0, t + 1, wave, lane);
        i32x8_t tf[C::NI];
        int tsc[C::NI];
#pragma unroll
        for (int i = 0; i < C::NI; ++i) {
            const int rr = wt0 + 16 * i + lr;
            tf[i] = mx_frag(cur, rr, lane);
            tsc[i] = cur[C::DATA + 4 * rr + q];
        }
#pragma unroll
        for (int j = 0; j < C::NJ; ++j) {
            const int rr = BT + ww0 + 16 * j + lr;
            const i32x8_t wf = mx_frag(cur, rr, lane);
            const int wsc = cur[C::DATA + 4 * rr + q];
#pragma unroll
            for (int i = 0; i < C::NI; ++i)
                acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(wf, tf[i], acc[i][j], 0, 0, 0, wsc, 0,
                                                                            tsc[i]);
        }
        // step t + 1 has landed in the other stage, and every wave is done
        // with this one before the next step's loads overwrite it
        mx_wait_vm0();
        __syncthreads();
    }

    // ---- epilogue: lane holds token row wt0 + 16 i + lr, output columns
    // ww0 + 16 j + 4 q + {0..3}
    if constexpr (OUT == 0) {
        uint16_t* Y = static_cast<uint16_t*>(a.out);
#pragma unroll
        for (int i = 0; i < C::NI; ++i) {
            const int n = row0 + wt0 + 16 * i + lr;
            if (n >= a.R) continue;
#pragma unroll
            for (int j = 0; j < C::NJ; ++j) {
                const int m = col0 + ww0 + 16 * j + 4 * q;
                const f32x4_t v = acc[i][j];
                uint16_t* p = Y + (int64_t)n * a.ldo + m;
                if (m + 4 <= a.C) {
                    *reinterpret_cast<u32x2_t*>(p) = u32x2_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (m + e < a.C) p[e] = (uint16_t)bf16_rne(v[e]);
                }
            }
        }
    } else {
        // MX-FP8 along the columns: block pair (j, j + 1) is one 32-column
        // block; its largest magnitude over the 4 lanes of the token row
        uint8_t* Zq = static_cast<uint8_t*>(a.out);
#pragma unroll
        for (int i = 0; i < C::NI; ++i) {
            const int n = row0 + wt0 + 16 * i + lr;
#pragma unroll
            for (int j = 0; j < C::NJ; j += 2) {
                const int cb = col0 + ww0 + 16 * j;          // first column of the block
                float v[8];
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    v[e] = (cb + 4 * q + e < a.C) ? acc[i][j][e] : 0.f;
                    v[4 + e] = (cb + 16 + 4 * q + e < a.C) ? acc[i][j + 1][e] : 0.f;
                }
                float amax = 0.f;
#pragma unroll
                for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf(v[e]));
                amax = fmaxf(amax, __shfl_xor(amax, 16));
                amax = fmaxf(amax, __shfl_xor(amax, 32));
                const int sb = mx_scale_byte(amax);
                const int nsh = 127 - sb;                    // multiply by 2^-S
                if (n < a.R && cb < a.cpad) {
                    uint8_t* p = Zq + (int64_t)n * a.ldo + cb + 4 * q;
                    *reinterpret_cast<uint32_t*>(p) =
                        mx_pack4(__builtin_amdgcn_ldexpf(v[0], nsh), __builtin_amdgcn_ldexpf(v[1], nsh),
                                 __builtin_amdgcn_ldexpf(v[2], nsh), __builtin_amdgcn_ldexpf(v[3], nsh));
                    *reinterpret_cast<uint32_t*>(p + 16) =
                        mx_pack4(__builtin_amdgcn_ldexpf(v[4], nsh), __builtin_amdgcn_ldexpf(v[5], nsh),
                                 __builtin_amdgcn_ldexpf(v[6], nsh), __builtin_amdgcn_ldexpf(v[7], nsh));
                    if (q == 0) a.outs[(int64_t)n * a.ldos + cb / 32] = (uint8_t)sb;
                }
            }
        }
    }
}

// bfloat16 A [R][C] -> MX-FP8: one thread per 32-element block of a row
// (blocks up to round_up(C, 128) / 32; blocks past C are written as zeros
// with scale byte 0).
__global__ __launch_bounds__(256)
void mx_quantize_kernel(const uint16_t* A, int64_t lda, int R, int C, uint8_t* Q, int64_t ldq, uint8_t* S,
                        int64_t lds, int nbp) {
    const int64_t id = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (id >= (int64_t)R * nbp) return;
    const int r = (int)(id / nbp), b = (int)(id - (int64_t)r * nbp);
    const int c0 = 32 * b;
    const uint16_t* row = A + (int64_t)r * lda;
    float v[32];
    if (c0 + 32 <= C) {
#pragma unroll
        for (int h = 0; h < 4; ++h) {
            const u32x4_t w = *reinterpret_cast<const u32x4_t*>(row + c0 + 8 * h);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                v[8 * h + 2 * e] = bf16_to_f32(w[e] & 0xffffu);
                v[8 * h + 2 * e + 1] = bf16_to_f32(w[e] >> 16);
            }
        }
    } else {
#pragma unroll
        for (int e = 0; e < 32; ++e) v[e] = (c0 + e < C) ? bf16_to_f32(row[c0 + e]) : 0.f;
    }
    float amax = 0.f;
#pragma unroll
    for (int e = 0; e < 32; ++e) amax = fmaxf(amax, fabsf(v[e]));
    const int sb = mx_scale_byte(amax);
    const int nsh = 127 - sb;
    u32x4_t lo, hi;
#pragma unroll
    for (int w = 0; w < 4; ++w) {
        lo[w] = mx_pack4(__builtin_amdgcn_ldexpf(v[4 * w], nsh), __builtin_amdgcn_ldexpf(v[4 * w + 1], nsh),
                         __builtin_amdgcn_ldexpf(v[4 * w + 2], nsh), __builtin_amdgcn_ldexpf(v[4 * w + 3], nsh));
        hi[w] = mx_pack4(__builtin_amdgcn_ldexpf(v[16 + 4 * w], nsh), __builtin_amdgcn_ldexpf(v[17 + 4 * w], nsh),
                         __builtin_amdgcn_ldexpf(v[18 + 4 * w], nsh), __builtin_amdgcn_ldexpf(v[19 + 4 * w], nsh));
    }
    uint8_t* qp = Q + (int64_t)r * ldq + c0;
    *reinterpret_cast<u32x4_t*>(qp) = lo;
    *reinterpret_cast<u32x4_t*>(qp + 16) = hi;
    S[(int64_t)r * lds + b] = (uint8_t)sb;
}

template <int BT, int BW, int OUT>
hipError_t launch_tile(const MxGemmArgs& a, hipStream_t stream) {
    const int tiles = ((a.R + BT - 1) / BT) * ((a.C + BW - 1) / BW);
    hipLaunchKernelGGL((gemm_mx_kernel<BT, BW, OUT>), dim3(tiles), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

int mx_gemm_tile(int R, int C, int cus) {
    // the largest tile that still gives every CU a tile, else the smallest
    const long long t256 = (long long)((R + 255) / 256) * ((C + 255) / 256);
    const long long t128 = (long long)((R + 255) / 256) * ((C + 127) / 128);
    if (t256 >= cus) return 0;
    if (t128 >= cus) return 1;
    return 2;
}

hipError_t launch_gemm_mx(const MxGemmArgs& a, int out_mx, int cus, hipStream_t stream) {
    const int64_t lim = (int64_t)1 << 31;
    if (a.R < 1 || a.C < 1 || a.D < 1 || a.R * a.ldt >= lim || a.C * a.ldw >= lim || a.R * a.ldts >= lim ||
        a.C * a.ldws >= lim)
        return hipErrorInvalidValue;
    switch (mx_gemm_tile(a.R, a.C, cus) * 2 + (out_mx ? 1 : 0)) {
        case 0: return launch_tile<256, 256, 0>(a, stream);
        case 1: return launch_tile<256, 256, 1>(a, stream);
        case 2: return launch_tile<256, 128, 0>(a, stream);
        case 3: return launch_tile<256, 128, 1>(a, stream);
        case 4: return launch_tile<128, 128, 0>(a, stream);
        default: return launch_tile<128, 128, 1>(a, stream);
    }
}

hipError_t launch_mx_quantize(const uint16_t* A, int64_t lda, int R, int C, uint8_t* Q, int64_t ldq, uint8_t* S,
                              int64_t lds, hipStream_t stream) {
    const int nbp = ((C + 127) / 128) * 4;
    const int64_t n = (int64_t)R * nbp;
    if (n <= 0) return hipSuccess;
    hipLaunchKernelGGL(mx_quantize_kernel, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, A, lda, R, C, Q,
                       ldq, S, lds, nbp);
    return hipGetLastError();
}

}  // namespace espace
