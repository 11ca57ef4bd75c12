// The low-precision projected linear layer on gfx950's block-scaled MFMA:
// operands in MX-FP8 (E4M3 elements, one power-of-two E8M0 scale per 32
// elements along the reduction dimension), the two products of Section 2.2,
// Eq. 3 with fp32 accumulation.  The projection's epilogue writes Z back in
// MX-FP8 along L, so the expansion consumes it as it consumes the folded
// weight.  Two GEMM kernels:
//
// * The expansion (bf16 output) runs the four-wave bfloat16 kernel's
//   pipeline (gemm_bf16_v3.hip) on fp8 operands: a depth step of 128 codes is
//   two sub-steps of 64, each with its own LDS half-stage of 64-byte rows laid
//   out as the bf16 kernel's (same loads; the chunk swizzle suits reads of
//   32 rows), plus
//   one scale dword per row (the four 32-blocks of the step), loaded with
//   the first half-stage only.  Per sub-step a
//   wave issues NI x NJ v_mfma_scale_f32_32x32x64_f8f6f4 (16 for the
//   256 x 256 tile, as long on the matrix pipe as the bf16 kernel's 64
//   16x16x32 MFMAs) with the fragment reads of the next sub-step and the
//   loads of step + 2 between them; persistent tiles, the next tile's first
//   two steps loaded during the last two of the current one.
// * The projection (MX-FP8 output, a few hundred tiles at most) runs a
//   simpler kernel on v_mfma_scale_f32_16x16x128_f8f6f4 with tiles small
//   enough to give every CU work: for the 4096 x 1536 projections 128 x 192
//   tiles (256 of them) with three LDS stages, the loads of a step issued two
//   steps ahead (measured on operands rotated through HBM: 38 against 41 us
//   with 128 x 128 tiles on two stages and two workgroups per CU at depth
//   4096, 110 against 131 us at depth 11008; the pipelined kernel's 256 x 128
//   or 256 x 256 tiles on 192 or 96 CUs took 54-60 us at depth 4096).
//
// v_mfma_scale_f32_32x32x64_f8f6f4 (operands "A" then "B"), as measured on
// the device:
//   - lane l of an operand holds row l % 32 of its 32 x 64 slice: bytes
//     0..15 are depth 16 (l / 32) .. +15 and bytes 16..31 are depth
//     32 + 16 (l / 32) .. +15, i.e. 16-byte chunks l / 32 and 2 + l / 32 of
//     the 64-byte row;
//   - the scale byte of lane l applies to row l % 32 over depth block
//     32 (l / 32) .. +31; the instruction's op_sel picks the byte of the
//     scale register (byte 0 for the first sub-step of a step, byte 2 for
//     the second, each lane's dword shifted right by 8 (l / 32) beforehand);
//   - register i of lane l of the result holds row 8 (i / 4) + 4 (l / 32) +
//     i % 4 (from A) of column l % 32 (from B).
// v_mfma_scale_f32_16x16x128_f8f6f4:
//   - lane l of an operand holds row l % 16 of its 16 x 128 slice: bytes
//     0..15 are depth 16 (l / 16) .. +15 and bytes 16..31 are depth
//     64 + 16 (l / 16) .. +15;
//   - the scale byte of lane l applies to row l % 16 over depth block
//     32 (l / 16) .. +31;
//   - lane l of the result holds rows 4 (l / 16) + {0..3} (from A) of column
//     l % 16 (from B).
// In both the weight-side slice is passed as A and the token-side slice as
// B, so a lane's results are runs of consecutive output features of one
// token.
//
// The scaled MFMAs add the running sum C with limited precision (on gfx950
// the result differs from the exact C + sum of products by up to about
// 2^-11.5 (|C| + sum |a·b|), either form); the accumulators stay in the MFMA
// chain, and the parity tests bound the error accordingly.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"
#include "v3_core.hpp"

namespace espace {

namespace {

typedef int i32x8_t __attribute__((ext_vector_type(8)));
typedef int i32x4_t __attribute__((ext_vector_type(4)));

// Tile 256 tokens x BW output columns (BW = 256 or 128), four waves as 2 x 2,
// each owning 128 tokens x BW/2 columns as NI x NJ blocks of 32 x 32.  The
// code half-stages are the bf16 kernel's (V3Cfg<BW>: token rows first, 64
// bytes each); after the four of them, two scale areas of one dword per row,
// one per stage (the scale loads of a step go with its first half-stage: a
// scale load gathers 64 rows, one memory line each; loaded with both halves
// they took 88 against 82 us on the 4096 x 12288 x 1536 expansion).
template <int BW, int SS>
struct MxCfg {
    using V = V3Cfg<BW>;
    static constexpr int NI = 4, NJ = BW / 64;
    static constexpr int ROWS = V::ROWS;
    static constexpr int SROW = 4 * SS;               // scale bytes per row in an area
    static constexpr int SCB = ROWS * SROW;           // bytes of a scale area
    static constexpr int NSC = ROWS / 64;             // scale loads (64 rows each) per area
    static constexpr int LSC = (NSC + 3) / 4;         // per wave (uniform: extra ones repeat a load)
    // loads per wave of a step's first half-stage when it carries scales
    // (codes, and SS steps' scale dwords, which only that half loads) and of
    // a half-stage of codes alone
    static constexpr int LPH0 = V::LPH + LSC, LPH1 = V::LPH;
    static constexpr int LPS = LPH0 + LPH1;           // per step with scales
    static constexpr int NMF = NI * NJ;               // MFMAs per sub-step
    static constexpr int NRD = 2 * (NI + NJ);         // code fragment reads per sub-step
    static constexpr int NSR = NI + NJ;               // scale dword reads per step
    static constexpr int NST = 2 * NI * NJ;           // 16-byte stores per wave (bf16 output)
    static constexpr int SMEM = 4 * V::HS + 2 * SCB;
    static_assert(BW == 256 || BW == 128, "tile");
    static_assert(SS == 1 || SS == 4, "scale steps");
    static_assert(LPS + NST < 64, "vmcnt");
    // whether step kt's first half carries scales, and its loads per wave
    static __device__ __forceinline__ constexpr bool scales_with(int kt) { return SS == 1 || (kt & 3) == 0; }
    static __device__ __forceinline__ constexpr int n0(int kt) { return scales_with(kt) ? LPH0 : LPH1; }
    // MFMA after which load y of a sub-step's n is issued
    static constexpr int load_slot(int y, int n) { return y * NMF / n + NMF / (2 * n); }
    // MFMA after which read x of a sub-step is issued (n reads in all)
    static constexpr int read_slot(int x, int n) { return x * NMF / n; }
};

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

// ---- the projection's kernel ------------------------------------------------

constexpr int MX_BK = 128;   // depth of one step: one block-scaled MFMA

// 16-byte chunk c of LDS row r sits at chunk c ^ mx_swz(r): the 16 rows one
// fragment read touches then fall on distinct bank groups
__device__ __forceinline__ int mx_swz(int r) { return (r >> 1) & 7; }

// Tile BT tokens x BW output columns, 4 waves as 2 x 2, each BT/2 x BW/2,
// NS LDS stages (the loads of step t + NS - 1 are issued at the start of
// step t).  A stage holds the tile's BT + BW rows of 128 code bytes (token
// rows first).  The scale dwords (the 4 blocks of a step) of SS steps are
// loaded together: SS = 1, one dword per row after the codes of each stage;
// SS = 4 (scale rows 16-byte aligned), 16 bytes per row into one of two
// areas after the stages, with the codes of every fourth step.  A scale load
// gathers 64 rows, one memory line each, so a quarter of them as 16-byte
// loads saves most of their cost (4096 x 1536 projections: 37.6 -> 36.7 us
// at depth 4096, 107.7 -> 89.6 us at depth 11008).
template <int BT, int BW, int NS, int SS>
struct MxZCfg {
    static constexpr int ROWS = BT + BW;
    static constexpr int DATA = ROWS * MX_BK;
    static constexpr int STAGE = SS == 1 ? DATA + ROWS * 4 : DATA;
    static constexpr int SAREA = ROWS * 16;           // four steps' scale dwords (SS = 4)
    static constexpr int SMEM = NS * STAGE + (SS == 1 ? 0 : 2 * SAREA);
    static constexpr int WT = BT / 2, WW = BW / 2;
    static constexpr int NI = WT / 16, NJ = WW / 16;
    static constexpr int NDL = ROWS / 8;    // 1 KB code loads per stage (8 rows each)
    static constexpr int NSL = ROWS / 64;   // 256-byte scale loads per stage (64 rows each)
    static constexpr int LPD = NDL / 4;     // code loads per wave and stage
    static constexpr int LPS = (NSL + 3) / 4;   // scale loads per wave (uniform: extra ones repeat a load)
    static constexpr int LPW = LPD + LPS;
    static_assert(BT % 64 == 0 && BW % 64 == 0 && NDL % 4 == 0, "tile");
    static_assert((NS == 2 || NS == 3) && (NS - 2) * LPW < 64 && SMEM <= 160 * 1024, "stages");
    static_assert(SS == 1 || SS == 4, "scale steps");
    // whether step t's loads include scales, and where step t's scale bytes are
    static __device__ __forceinline__ bool scales_with(int t) { return SS == 1 || (t & 3) == 0; }
    static __device__ __forceinline__ int scale_area(int t) {
        return SS == 1 ? (t % NS) * STAGE + DATA : NS * STAGE + ((t >> 2) & 1) * SAREA;
    }
};

// s_barrier that the compiler moves no memory access across (the loads of
// other waves into LDS are invisible to it), after this wave's LDS reads
// have completed; unlike __syncthreads() it does not wait for this wave's
// loads still in flight
__device__ __forceinline__ void mx_barrier() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// Issue the direct-to-LDS loads of depth step t into its stage: codes (16
// bytes per lane) and, with the steps that carry them, scale dwords (4 or 16
// bytes per lane).  Rows past the matrix read its last row (their results
// are never stored); the 16-byte scale loads of a last group may read past
// the matrix's steps (bytes never used; past the buffer they read zeros).
template <int BT, int BW, int NS, int SS>
__device__ __forceinline__ void mx_issue(unsigned char* smem, const MxGemmArgs& a, int row0, int col0, int t,
                                         int wave, int lane) {
    using C = MxZCfg<BT, BW, NS, SS>;
    unsigned char* stage = smem + (t % NS) * C::STAGE;
    const auto tr = __builtin_amdgcn_make_buffer_rsrc((void*)a.T, (short)0, (int)(a.R * a.ldt), 0x00020000);
    const auto wr = __builtin_amdgcn_make_buffer_rsrc((void*)a.W, (short)0, (int)(a.C * a.ldw), 0x00020000);
    const auto ts = __builtin_amdgcn_make_buffer_rsrc((void*)a.Ts, (short)0, (int)(a.R * a.ldts), 0x00020000);
    const auto ws = __builtin_amdgcn_make_buffer_rsrc((void*)a.Ws, (short)0, (int)(a.C * a.ldws), 0x00020000);
#pragma unroll
    for (int j = 0; j < C::LPD; ++j) {
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
    if (!C::scales_with(t)) return;
    unsigned char* area = smem + C::scale_area(t);
#pragma unroll
    for (int j = 0; j < C::LPS; ++j) {
        const int s = (wave + 4 * j) % C::NSL;
        const int rr = 64 * s + lane;
        const bool tok = 64 * s < BT;
        const int g = tok ? min(row0 + rr, a.R - 1) : min(col0 + rr - BT, a.C - 1);
        const int off = g * (int)(tok ? a.ldts : a.ldws);
        if constexpr (SS == 1)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(tok ? ts : ws, (__attribute__((address_space(3))) void*)(area + s * 256),
                                                     4, off, 4 * t, 0, 0);
        else
            __builtin_amdgcn_raw_ptr_buffer_load_lds(tok ? ts : ws, (__attribute__((address_space(3))) void*)(area + s * 1024),
                                                     16, off, 4 * t, 0, 0);
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

// Tile BT tokens x BW columns, MX-FP8 output along the columns (codes and
// one scale byte per 32 columns, up to cpad columns); one workgroup per tile.
template <int BT, int BW, int NS, int SS>
__global__ __launch_bounds__(256, (BT + BW) <= 256 ? 2 : 1)
void gemm_mx_z_kernel(MxGemmArgs a) {
    using C = MxZCfg<BT, BW, NS, SS>;
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
    for (int t = 0; t < NS - 1 && t < steps; ++t) mx_issue<BT, BW, NS, SS>(smem, a, row0, col0, t, wave, lane);
    for (int t = 0; t < steps; ++t) {
        // this wave's loads of step t have landed (those of the newer steps
        // may stay in flight); after the barrier every wave's have, and
        // every wave is done with step t - 1, whose stage receives step
        // t + NS - 1 (and whose scale area, with four-step groups, is not
        // rewritten before step t + 4)
        if (NS == 3 && t + 1 < steps) {
            if (C::scales_with(t + 1)) v3_wait_vm<C::LPW>();
            else v3_wait_vm<C::LPD>();
        } else {
            v3_wait_vm<0>();
        }
        mx_barrier();
        if (t + NS - 1 < steps) mx_issue<BT, BW, NS, SS>(smem, a, row0, col0, t + NS - 1, wave, lane);
        const unsigned char* cur = smem + (t % NS) * C::STAGE;
        const unsigned char* sc = smem + C::scale_area(t) + (SS == 1 ? 0 : 4 * (t & 3));
        i32x8_t tf[C::NI];
        int tsc[C::NI];
#pragma unroll
        for (int i = 0; i < C::NI; ++i) {
            const int rr = wt0 + 16 * i + lr;
            tf[i] = mx_frag(cur, rr, lane);
            tsc[i] = sc[4 * SS * rr + q];
        }
#pragma unroll
        for (int j = 0; j < C::NJ; ++j) {
            const int rr = BT + ww0 + 16 * j + lr;
            const i32x8_t wf = mx_frag(cur, rr, lane);
            const int wsc = sc[4 * SS * rr + q];
#pragma unroll
            for (int i = 0; i < C::NI; ++i)
                acc[i][j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(wf, tf[i], acc[i][j], 0, 0, 0, wsc, 0,
                                                                            tsc[i]);
        }
    }

    // ---- epilogue: lane holds token row wt0 + 16 i + lr, output columns
    // ww0 + 16 j + 4 q + {0..3}
    {
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
                    // row pairs: columns cb .. cb + 31 lie in one 64-code block
                    const int c = cb + 4 * q;
                    uint8_t* p = Zq + (a.out_pairs ? (int64_t)(n >> 1) * a.ldo + (c >> 6) * 128 + (n & 1) * 64 + (c & 63)
                                                   : (int64_t)n * a.ldo + c);
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

// ---- the expansion's kernel -------------------------------------------------

// v_mfma_scale_f32_32x32x64_f8f6f4 by inline assembly, so that the
// accumulators stay in the AGPRs and the order is the one written; SEL is
// the op_sel_hi bit of both scale operands (0: byte 0, 1: byte 2).
#define MX_MFMA(acc, w, t, ws, ts, SEL)                                                                \
    asm volatile("v_mfma_scale_f32_32x32x64_f8f6f4 %0, %1, %2, %0, %3, %4 op_sel_hi:[" SEL "," SEL ",0]" \
                 : "+a"(acc) : "v"(w), "v"(t), "v"(ws), "v"(ts))
#define MX_MFMA0(acc, w, t, ws, ts, SEL)                                                              \
    asm volatile("v_mfma_scale_f32_32x32x64_f8f6f4 %0, %1, %2, 0, %3, %4 op_sel_hi:[" SEL "," SEL ",0]" \
                 : "=a"(acc) : "v"(w), "v"(t), "v"(ws), "v"(ts))
#define MX_READ(dst, addr, off) \
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(dst) : "v"(addr), "i"(off))
#define MX_READ32(dst, addr, off) \
    asm volatile("ds_read_b32 %0, %1 offset:%2" : "=v"(dst) : "v"(addr), "i"(off))

// Code fragments of one sub-step: 32 bytes per lane and block, read as the
// two 16-byte chunks of the 64-byte row.
template <int NJ>
struct MxFrag {
    i32x4_t tl[4], th[4], wl[NJ], wh[NJ];
};

// LDS addresses of one half-stage for this lane: its token and weight rows'
// two chunks, and its token and weight scale dwords.
struct MxAddr {
    unsigned tl, th, wl, wh, ts, ws;
};

// Code read x of a sub-step, in the order the MFMAs use them: token block 0,
// weight blocks 0 .. NJ-1, token blocks 1 .. 3 (two reads per block; blocks
// are 32 rows, 2048 bytes, apart).
template <int NJ>
__device__ __forceinline__ void mx_read(int x, MxFrag<NJ>& f, const MxAddr& a) {
#define MX_R(n)                                                                                     \
    if constexpr (n < 2 * (4 + NJ)) {                                                               \
        if (x == n) {                                                                               \
            constexpr int b = n / 2;                                                                \
            if constexpr (b == 0) {                                                                 \
                if constexpr (n % 2) MX_READ(f.th[0], a.th, 0); else MX_READ(f.tl[0], a.tl, 0);     \
            } else if constexpr (b <= NJ) {                                                         \
                if constexpr (n % 2) MX_READ(f.wh[b - 1], a.wh, (b - 1) * 2048);                    \
                else MX_READ(f.wl[b - 1], a.wl, (b - 1) * 2048);                                    \
            } else {                                                                                \
                if constexpr (n % 2) MX_READ(f.th[b - NJ], a.th, (b - NJ) * 2048);                  \
                else MX_READ(f.tl[b - NJ], a.tl, (b - NJ) * 2048);                                  \
            }                                                                                       \
        }                                                                                           \
    }
    MX_R(0) MX_R(1) MX_R(2) MX_R(3) MX_R(4) MX_R(5) MX_R(6) MX_R(7)
    MX_R(8) MX_R(9) MX_R(10) MX_R(11) MX_R(12) MX_R(13) MX_R(14) MX_R(15)
#undef MX_R
}

// Scale read x of a step (token blocks 0 .. 3, then weight blocks; 32 rows,
// 32 SROW bytes, apart) into the raw dwords.
template <int NJ, int SROW>
__device__ __forceinline__ void mx_read_scale(int x, int* tsr, int* wsr, const MxAddr& a) {
#define MX_S(n)                                                                           \
    if constexpr (n < 4 + NJ) {                                                           \
        if (x == n) {                                                                     \
            if constexpr (n < 4) MX_READ32(tsr[n], a.ts, n * 32 * SROW);                  \
            else MX_READ32(wsr[n - 4], a.ws, (n - 4) * 32 * SROW);                        \
        }                                                                                 \
    }
    MX_S(0) MX_S(1) MX_S(2) MX_S(3) MX_S(4) MX_S(5) MX_S(6) MX_S(7)
#undef MX_S
}

// What a sub-step's loads need: the code operands as 16-bit arrays (the
// bf16 kernel's load helpers; one step of 128 codes is 64 of their
// elements), the scale arrays, and this lane's per-load row offsets.
// APAIR: the token codes in row pairs (each 128-byte block holds 64
// consecutive codes of two neighbouring tokens).
template <int BW, int SS, bool APAIR = false>
struct MxLoad {
    using C = MxCfg<BW, SS>;
    const uint16_t* T;
    const uint16_t* W;
    unsigned tbytes, wbytes;
    const uint8_t* Ts;
    const uint8_t* Ws;
    unsigned tsbytes, wsbytes;
    int voff[C::V::LPH];
    int soff[C::LSC];
    int wave;

    // scale load j covers rows 64 s .. 64 s + 63 of the tile, s = (wave + 4 j) % NSC
    __device__ __forceinline__ void scale_offsets(const MxGemmArgs& a, int row0, int col0, int lane) {
#pragma unroll
        for (int j = 0; j < C::LSC; ++j) {
            const int s = (wave + 4 * j) % C::NSC;
            const int rr = 64 * s + lane;
            soff[j] = rr < 256 ? min(row0 + rr, a.R - 1) * (int)a.ldts
                               : min(col0 + rr - 256, a.C - 1) * (int)a.ldws;
        }
    }

    // load y of half h of step kt into half-stage u; a scale load (SS
    // steps' dwords per row, only with a step that carries them) goes to
    // scale area `area` (SS = 1: the stage's own, u / 2).  The 16-byte loads
    // of a last group may read past the matrix's steps: bytes never used,
    // zeros past the buffer.
    __device__ __forceinline__ void load(unsigned char* smem, int kt, int h, int u, int y, int area) const {
        if (y < C::V::LPH) {
            v3_load<typename C::V, APAIR>(smem, T, W, tbytes, wbytes, voff, wave, kt, h, u, y);
        } else if (C::scales_with(kt)) {
            const int j = y - C::V::LPH;
            const int s = (wave + 4 * j) % C::NSC;
            const bool tok = s < 4;
            const auto rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)(tok ? Ts : Ws), (short)0,
                                                                (int)(tok ? tsbytes : wsbytes), 0x00020000);
            const int ar = SS == 1 ? (u >> 1) : area;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rsrc,
                (__attribute__((address_space(3))) void*)(smem + 4 * C::V::HS + ar * C::SCB + 64 * C::SROW * s),
                C::SROW, soff[j], 4 * kt, 0, 0);
        }
    }
};

// One sub-step: NMF MFMAs on (cur, the shifted scales tsc / wsc) with
// op_sel_hi SEL; between them the NRD code reads of the next sub-step into
// nxt from rd, with SREADS also the NSR scale dwords of the next step from
// sd into tsr / wsr, and with do_load the loads of half h of step lkt into
// half-stage u (h = SEL1: LPH0 loads in sub-step 0, LPH1 in sub-step 1).
// FIRST: the accumulators start from zero.
template <int BW, int SS, bool FIRST, bool SEL1, bool SREADS, class LD>
__device__ __forceinline__ void mx_substep(f32x16_t (&acc)[4][BW / 64], const MxFrag<BW / 64>& cur,
                                           const int* tsc, const int* wsc, MxFrag<BW / 64>& nxt,
                                           const MxAddr& rd, const MxAddr& sd, int* tsr, int* wsr,
                                           unsigned char* smem, const LD& ld, int lkt, int h, int u,
                                           int area, bool do_load) {
    using C = MxCfg<BW, SS>;
    constexpr int NJ = C::NJ;
    constexpr int NR = C::NRD + (SREADS ? C::NSR : 0);
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < NJ; ++j) {
            const i32x8_t w = __builtin_shufflevector(cur.wl[j], cur.wh[j], 0, 1, 2, 3, 4, 5, 6, 7);
            const i32x8_t t = __builtin_shufflevector(cur.tl[i], cur.th[i], 0, 1, 2, 3, 4, 5, 6, 7);
            if constexpr (FIRST) {
                if constexpr (SEL1) MX_MFMA0(acc[i][j], w, t, wsc[j], tsc[i], "1");
                else MX_MFMA0(acc[i][j], w, t, wsc[j], tsc[i], "0");
            } else {
                if constexpr (SEL1) MX_MFMA(acc[i][j], w, t, wsc[j], tsc[i], "1");
                else MX_MFMA(acc[i][j], w, t, wsc[j], tsc[i], "0");
            }
            const int m = i * NJ + j;
#pragma unroll
            for (int x = 0; x < NR; ++x)
                if (C::read_slot(x, NR) == m) {
                    if (x < C::NRD) mx_read<NJ>(x, nxt, rd);
                    else mx_read_scale<NJ, C::SROW>(x - C::NRD, tsr, wsr, sd);
                }
            constexpr int NL = SEL1 ? C::LPH1 : C::LPH0;
#pragma unroll
            for (int y = 0; y < NL; ++y)
                if (C::load_slot(y, NL) == m && do_load) ld.load(smem, lkt, h, u, y, area);
        }
}

// vmcnt(n) for the counts the steps need (half-steps of LPH0 or LPH1 and
// LPH1 loads, plus the previous tile's NST stores); any other n waits for
// everything
template <class C>
__device__ __forceinline__ void mx_wait_vm_n(int n) {
    constexpr int L0 = C::LPH0, L1 = C::LPH1, S = C::NST;
    if (n == 0) v3_wait_vm<0>();
    else if (n == L1) v3_wait_vm<L1>();
    else if (n == 2 * L1) v3_wait_vm<2 * L1>();
    else if (n == L0 + L1) v3_wait_vm<L0 + L1>();
    else if (n == S) v3_wait_vm<S>();
    else if (n == S + L1) v3_wait_vm<S + L1>();
    else if (n == S + 2 * L1) v3_wait_vm<S + 2 * L1>();
    else if (n == S + L0 + L1) v3_wait_vm<S + L0 + L1>();
    else v3_wait_vm<0>();
}

// Copy of an accumulator block in VGPRs (the accumulators are named only by
// inline assembly with AGPR operands).
__device__ __forceinline__ f32x16_t mx_acc_read(const f32x16_t& a) {
    f32x16_t v;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        float x;
        asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(x) : "a"(a[r]));
        v[r] = x;
    }
    return v;
}

// The MX GEMM: out[n][c] = sum_k T[n][k] W[c][k] over MX-FP8 codes and
// scales, n < R tokens, c < C columns, depth D (the codes are zero-padded to
// whole steps of 128).  Persistent: min(tiles, CUs) workgroups,
// each taking tiles blockIdx.x, blockIdx.x + gridDim.x, ...  As in the bf16
// kernel, when the output is bf16 with C a multiple of 8, the last two steps
// of a tile load the next tile's first two, and the tile's results leave with
// exactly NST stores per wave.  Output: bf16 Y [R][ldo].  SS = 4 (scale
// rows 16-byte aligned): the scale dwords of four steps per 16-byte load,
// with every fourth step, into two areas taken in turn by the workgroup's
// successive groups of four steps (tile after tile), so that a group's area
// is rewritten only after its last step's scales were read.
template <int BW, int SS, int APAIR = 0>
__global__ __launch_bounds__(256, 1)
void gemm_mx_kernel(MxGemmArgs a, int tiles_c, int ntiles) {
    using C = MxCfg<BW, SS>;
    using V = typename C::V;
    constexpr int NJ = C::NJ;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[C::SMEM];

    const int ktiles = (a.D + 127) / 128;           // the codes are zero-padded to whole steps
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wrow0 = (wave >> 1) * 128;              // the wave's tokens in the tile
    const int wcol0 = (wave & 1) * (BW / 2);          // its output columns
    const bool ahead_ok = (a.C & 7) == 0 && ktiles >= 2;

    MxLoad<BW, SS, APAIR != 0> ld;
    ld.T = reinterpret_cast<const uint16_t*>(a.T);
    ld.W = reinterpret_cast<const uint16_t*>(a.W);
    ld.tbytes = (unsigned)((uint64_t)(APAIR ? (a.R + 1) / 2 : a.R) * a.ldt);
    ld.wbytes = (unsigned)((uint64_t)a.C * a.ldw);
    ld.Ts = a.Ts;
    ld.Ws = a.Ws;
    ld.tsbytes = (unsigned)((uint64_t)a.R * a.ldts);
    ld.wsbytes = (unsigned)((uint64_t)a.C * a.ldws);
    ld.wave = wave;

    // fragment addresses: a lane reads row lane % 32 of each 32-row block,
    // chunks lh and 2 + lh; the swizzle depends on the row only through
    // lane % 32 (blocks start at multiples of 32 rows).  Chunk c of a row
    // sits at c ^ ((row >> 2) & 3): with the bf16 kernel's (row >> 1) & 3
    // these reads of 32 rows took two passes of the LDS banks each (measured
    // with the bank-conflict counter, on the kernel and on a probe of the
    // read pattern alone; the kernel's time did not change measurably)
    const int lr = lane & 31;
    const int lh = lane >> 5;
    const int sw = (lr >> 2) & 3;
    const unsigned sbase = (unsigned)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)smem;
    const unsigned c_lo = (unsigned)((lh ^ sw) * 16), c_hi = (unsigned)(((2 + lh) ^ sw) * 16);
    const unsigned trow = sbase + (unsigned)((wrow0 + lr) * V3_ROWB);
    const unsigned wrow = sbase + (unsigned)((V3_BM + wcol0 + lr) * V3_ROWB);
    const unsigned tsca = sbase + (unsigned)(4 * V::HS + C::SROW * (wrow0 + lr));
    const unsigned wsca = sbase + (unsigned)(4 * V::HS + C::SROW * (V3_BM + wcol0 + lr));
    auto addr = [&](int u) {
        MxAddr m;
        m.tl = trow + c_lo + (unsigned)(u * V::HS);
        m.th = trow + c_hi + (unsigned)(u * V::HS);
        m.wl = wrow + c_lo + (unsigned)(u * V::HS);
        m.wh = wrow + c_hi + (unsigned)(u * V::HS);
        m.ts = tsca + (unsigned)((u >> 1) * C::SCB);   // a stage's scale area (first half-stages only)
        m.ws = wsca + (unsigned)((u >> 1) * C::SCB);
        return m;
    };
    const int shift = 8 * lh;                         // block lh of a sub-step at byte 0 (or 2)
    int gb = 0;             // SS = 4: the workgroup's group count at this tile's first step
    // scale addresses of step k of this tile (SS = 1: its stage's area, as
    // in the stage's addresses st)
    auto sca = [&](const MxAddr& st, int k) {
        MxAddr m = st;
        if constexpr (SS == 4) {
            const unsigned off = (unsigned)(((gb + (k >> 2)) & 1) * C::SCB + 4 * (k & 3));
            m.ts = tsca + off;
            m.ws = wsca + off;
        }
        return m;
    };
    // vmcnt with the loads of half 0 of step k (and a half 1) in flight
    auto wait_step = [&](int k) {
        if (C::scales_with(k)) v3_wait_vm<C::LPS>();
        else v3_wait_vm<2 * C::LPH1>();
    };

    f32x16_t acc[4][NJ];
    MxFrag<NJ> f0, f1;
    int tsr[4], wsr[NJ], tsc[4], wsc[NJ];

    int item = blockIdx.x;
    int tile_r, tile_c;
    tile_coords<4>(item, ntiles, tiles_c, 0, tile_r, tile_c);
    bool ahead = false;     // this tile's first two steps were loaded by the previous one
    int s0 = 0;             // stage of this tile's first step (half-stages 2 s0, 2 s0 + 1)
    while (true) {
        const int row0 = tile_r * V3_BM;
        const int col0 = tile_c * BW;
        const int next = item + (int)gridDim.x;
        const bool ahead_next = ahead_ok && next < ntiles;
        const int gb_next = gb + (ktiles + 3) / 4;
        int ntr = 0, ntc = 0;
        if (next < ntiles) tile_coords<4>(next, ntiles, tiles_c, 0, ntr, ntc);

        // half-stage of (stage relative to s0, half)
        auto hs = [&](int rel, int h) { return ((rel ^ s0) << 1) | h; };
        const MxAddr A0 = addr(hs(0, 0)), A1 = addr(hs(0, 1)), A2 = addr(hs(1, 0)), A3 = addr(hs(1, 1));

        if (ahead) {
            // the first step's loads, then the second's and the previous
            // tile's stores were issued
            v3_wait_vm<C::n0(1) + C::LPH1 + C::NST>();
        } else {
            // the half-stages may still be read by a wave finishing the previous tile
            if (item != (int)blockIdx.x) __syncthreads();
            v3_offsets<V, 2, APAIR != 0>(ld.voff, row0, col0, a.R, a.C, a.ldt / 2, a.ldw / 2, wave, lane);
            ld.scale_offsets(a, row0, col0, lane);
#pragma unroll
            for (int y = 0; y < C::LPH0; ++y) ld.load(smem, 0, 0, hs(0, 0), y, gb & 1);
#pragma unroll
            for (int y = 0; y < C::LPH1; ++y) ld.load(smem, 0, 1, hs(0, 1), y, gb & 1);
            if (ktiles > 1) {
#pragma unroll
                for (int y = 0; y < C::LPH0; ++y) ld.load(smem, 1, 0, hs(1, 0), y, gb & 1);
#pragma unroll
                for (int y = 0; y < C::LPH1; ++y) ld.load(smem, 1, 1, hs(1, 1), y, gb & 1);
                v3_wait_vm<C::n0(1) + C::LPH1>();
            } else {
                v3_wait_vm<0>();
            }
        }
        __builtin_amdgcn_s_barrier();
#pragma unroll
        for (int x = 0; x < C::NRD; ++x) mx_read<NJ>(x, f0, A0);
#pragma unroll
        for (int x = 0; x < C::NSR; ++x) mx_read_scale<NJ, C::SROW>(x, tsr, wsr, sca(A0, 0));
        v3_wait_lgkm0();
        // the first sub-step loads step 2 into the half-stage just read:
        // every wave's reads of it must be complete before any wave issues them
        __builtin_amdgcn_s_barrier();

        int kt = 0;
        int rel = 0;          // stage of step kt relative to s0
        // the loads of sub-step h of step kt: half h of step kt + 2 of this
        // tile, or of the next tile's first steps once this one has none left
        // (step lkt of that tile, scale area larea); false: none
        auto load_kind = [&](int h, int& lkt, int& larea) -> bool {
            if (kt + 2 < ktiles) {
                lkt = kt + 2;
                larea = (gb + (lkt >> 2)) & 1;
                return true;
            }
            lkt = kt + 2 - ktiles;
            larea = (gb_next + (lkt >> 2)) & 1;
            if (!ahead_next) return false;
            if (kt + 2 == ktiles && h == 0) {
                v3_offsets<V, 2, APAIR != 0>(ld.voff, ntr * V3_BM, ntc * BW, a.R, a.C, a.ldt / 2, a.ldw / 2, wave, lane);
                ld.scale_offsets(a, ntr * V3_BM, ntc * BW, lane);
            }
            return true;
        };
        // the step's scale dwords, each lane's shifted right by 8 lh: inline
        // assembly, so that the shifts stay after the lgkmcnt wait that
        // completes the reads (the compiler does not know them as LDS reads)
        auto shift_scales = [&]() {
#pragma unroll
            for (int i = 0; i < 4; ++i) asm volatile("v_lshrrev_b32 %0, %1, %2" : "=v"(tsc[i]) : "v"(shift), "v"(tsr[i]));
#pragma unroll
            for (int j = 0; j < NJ; ++j) asm volatile("v_lshrrev_b32 %0, %1, %2" : "=v"(wsc[j]) : "v"(shift), "v"(wsr[j]));
        };
        // one step with the stage chosen at run time (the first one and the
        // last ones); FIRST: the accumulators start at zero
        auto generic_step = [&](auto first) {
            constexpr bool F = decltype(first)::value;
            // after a tile loaded ahead, its first step has the previous
            // tile's stores in flight behind the loads of its second step
            const int stores = (F && ahead) ? C::NST : 0;
            shift_scales();
            int lkt, larea;
            const bool k0 = load_kind(0, lkt, larea);
            mx_substep<BW, SS, F, false, false>(acc, f0, tsc, wsc, f1, rel ? A3 : A1, A0, tsr, wsr, smem, ld, lkt,
                                                0, hs(rel, 0), larea, k0);
            const int n0 = k0 ? C::n0(lkt) : 0;
            v3_wait_lgkm0();
            if (kt + 1 < ktiles || ahead_next) {
                // the next step's first half has landed (the loads just issued may stay in flight)
                if (kt + 1 < ktiles) mx_wait_vm_n<C>(C::LPH1 + stores + n0);
                __builtin_amdgcn_s_barrier();
            }
            // sub-step 1: fragments and scales of the next step's sub-step 0
            // (after the last step the reads are of no use but harmless)
            const bool k1 = load_kind(1, lkt, larea);
            mx_substep<BW, SS, false, true, true>(acc, f1, tsc, wsc, f0, rel ? A0 : A2, sca(rel ? A0 : A2, kt + 1),
                                                  tsr, wsr, smem, ld, lkt, 1, hs(rel, 1), larea, k1);
            const int n1 = k1 ? C::LPH1 : 0;
            v3_wait_lgkm0();
            if (kt + 1 < ktiles) {
                // the next step's second half has landed
                mx_wait_vm_n<C>(stores + n0 + n1);
                __builtin_amdgcn_s_barrier();
            }
            rel ^= 1;
            ++kt;
        };
        generic_step(std::true_type{});
        // steady state, two steps per iteration (relative stages 1 and 0):
        // the loads issued in them are this tile's; each barrier waits for the
        // half-stage the next sub-step reads, with the two newer half-steps of
        // loads in flight
        while (kt + 3 < ktiles) {
            const int a2 = (gb + ((kt + 2) >> 2)) & 1, a3 = (gb + ((kt + 3) >> 2)) & 1;
            shift_scales();
            mx_substep<BW, SS, false, false, false>(acc, f0, tsc, wsc, f1, A3, A3, tsr, wsr, smem, ld, kt + 2, 0,
                                                    hs(1, 0), a2, true);
            v3_wait_lgkm0();
            wait_step(kt + 2);
            __builtin_amdgcn_s_barrier();
            mx_substep<BW, SS, false, true, true>(acc, f1, tsc, wsc, f0, A0, sca(A0, kt + 1), tsr, wsr, smem, ld,
                                                  kt + 2, 1, hs(1, 1), a2, true);
            v3_wait_lgkm0();
            wait_step(kt + 2);
            __builtin_amdgcn_s_barrier();
            shift_scales();
            mx_substep<BW, SS, false, false, false>(acc, f0, tsc, wsc, f1, A1, A1, tsr, wsr, smem, ld, kt + 3, 0,
                                                    hs(0, 0), a3, true);
            v3_wait_lgkm0();
            wait_step(kt + 3);
            __builtin_amdgcn_s_barrier();
            mx_substep<BW, SS, false, true, true>(acc, f1, tsc, wsc, f0, A2, sca(A2, kt + 2), tsr, wsr, smem, ld,
                                                  kt + 3, 1, hs(0, 1), a3, true);
            v3_wait_lgkm0();
            wait_step(kt + 3);
            __builtin_amdgcn_s_barrier();
            kt += 2;
        }
        while (kt < ktiles) generic_step(std::false_type{});

        // the accumulators are written by inline assembly the compiler does
        // not know as MFMAs: wait out the MFMA-to-VALU read hazard
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);

        // ---- epilogue: register r of block (i, j) holds token row
        // wrow0 + 32 i + lr and output column wcol0 + 32 j + 8 (r / 4) + 4 lh + r % 4
        uint16_t* Y = static_cast<uint16_t*>(a.out);
        if (ahead_ok) {
            // two 16-byte stores per block: after the swap with the lane
            // 32 away, lane lh holds columns 16 g + 8 lh .. + 7 (g = 0, 1)
            // of its row; lanes outside the matrix get an offset past
            // the buffer, which its range check drops
            const unsigned ybytes = (unsigned)((uint64_t)a.R * a.ldo * 2u);
            const auto yr = __builtin_amdgcn_make_buffer_rsrc((void*)Y, (short)0, (int)ybytes, 0x00020000);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int n = row0 + wrow0 + 32 * i + lr;
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    const f32x16_t v = mx_acc_read(acc[i][j]);
#pragma unroll
                    for (int g = 0; g < 2; ++g) {
                        const auto s0v = __builtin_amdgcn_permlane32_swap(
                            pack_bf16x2(v[8 * g], v[8 * g + 1]), pack_bf16x2(v[8 * g + 4], v[8 * g + 5]), false,
                            false);
                        const auto s1v = __builtin_amdgcn_permlane32_swap(
                            pack_bf16x2(v[8 * g + 2], v[8 * g + 3]), pack_bf16x2(v[8 * g + 6], v[8 * g + 7]),
                            false, false);
                        const u32x4_t out = u32x4_t{s0v[0], s1v[0], s0v[1], s1v[1]};
                        const int c = col0 + wcol0 + 32 * j + 16 * g + 8 * lh;
                        const unsigned off =
                            (n < a.R && c < a.C) ? ((unsigned)n * (unsigned)a.ldo + (unsigned)c) * 2u : 0xFFFFFFF0u;
                        __builtin_amdgcn_raw_buffer_store_b128(out, yr, (int)off, 0, 0);
                    }
                }
            }
        } else {
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int n = row0 + wrow0 + 32 * i + lr;
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    const f32x16_t v = mx_acc_read(acc[i][j]);
                    if (n >= a.R) continue;
#pragma unroll
                    for (int g = 0; g < 4; ++g) {
                        const int c = col0 + wcol0 + 32 * j + 8 * g + 4 * lh;
                        uint16_t* p = Y + (int64_t)n * a.ldo + c;
                        if (c + 4 <= a.C) {
                            *reinterpret_cast<u32x2_t*>(p) =
                                u32x2_t{pack_bf16x2(v[4 * g], v[4 * g + 1]), pack_bf16x2(v[4 * g + 2], v[4 * g + 3])};
                        } else {
#pragma unroll
                            for (int e = 0; e < 4; ++e)
                                if (c + e < a.C) p[e] = (uint16_t)bf16_rne(v[4 * g + e]);
                        }
                    }
                }
            }
        }
        if (next >= ntiles) break;
        item = next;
        tile_r = ntr;
        tile_c = ntc;
        s0 = (s0 + ktiles) & 1;
        gb = gb_next;
        ahead = ahead_next;
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

bool scale_rows_16(const MxGemmArgs& a) {
    return a.ldts % 16 == 0 && a.ldws % 16 == 0 && (uintptr_t)a.Ts % 16 == 0 && (uintptr_t)a.Ws % 16 == 0;
}

template <int BW>
hipError_t launch_pipelined(const MxGemmArgs& a, int cus, hipStream_t stream) {
    const int tiles_c = (a.C + BW - 1) / BW;
    const int ntiles = tiles_c * ((a.R + 255) / 256);
    const int grid = ntiles < cus ? ntiles : cus;
    // four steps' scales per 16-byte load where every scale row starts on 16 bytes
    if (scale_rows_16(a)) {
        if (a.t_pairs)
            hipLaunchKernelGGL((gemm_mx_kernel<BW, 4, 1>), dim3(grid), dim3(256), 0, stream, a, tiles_c, ntiles);
        else
            hipLaunchKernelGGL((gemm_mx_kernel<BW, 4>), dim3(grid), dim3(256), 0, stream, a, tiles_c, ntiles);
    } else {
        if (a.t_pairs)
            hipLaunchKernelGGL((gemm_mx_kernel<BW, 1, 1>), dim3(grid), dim3(256), 0, stream, a, tiles_c, ntiles);
        else
            hipLaunchKernelGGL((gemm_mx_kernel<BW, 1>), dim3(grid), dim3(256), 0, stream, a, tiles_c, ntiles);
    }
    return hipGetLastError();
}

template <int BT, int BW, int NS>
hipError_t launch_z(const MxGemmArgs& a, hipStream_t stream) {
    const int tiles = ((a.R + BT - 1) / BT) * ((a.C + BW - 1) / BW);
    // four steps' scales per 16-byte load where every scale row starts on 16 bytes
    if (scale_rows_16(a)) hipLaunchKernelGGL((gemm_mx_z_kernel<BT, BW, NS, 4>), dim3(tiles), dim3(256), 0, stream, a);
    else hipLaunchKernelGGL((gemm_mx_z_kernel<BT, BW, NS, 1>), dim3(tiles), dim3(256), 0, stream, a);
    return hipGetLastError();
}

}  // namespace

int mx_gemm_tile(int R, int C, int cus, int out_mx) {
    const long long t256 = (long long)((R + 255) / 256) * ((C + 255) / 256);
    const long long t128 = (long long)((R + 255) / 256) * ((C + 127) / 128);
    if (out_mx) {
        // the largest tile that still gives every CU a tile; else 128 x 192
        // tiles with three stages when they make one round on more than half
        // of the CUs; else the smallest
        const long long t192 = (long long)((R + 127) / 128) * ((C + 191) / 192);
        if (t256 >= cus) return 0;
        if (t128 >= cus) return 1;
        if (2 * t192 > cus && t192 <= cus) return 3;
        return 2;
    }
    // 256 x 256 tiles when they give every CU a tile or when 256 x 128 tiles
    // (half the work each) need twice the rounds or more
    const long long r256 = (t256 + cus - 1) / cus, r128 = (t128 + cus - 1) / cus;
    return (t256 >= cus || 2 * r256 <= r128) ? 0 : 1;
}

hipError_t launch_gemm_mx(const MxGemmArgs& a, int out_mx, int cus, hipStream_t stream) {
    const int64_t lim = (int64_t)1 << 31;
    if (a.R < 1 || a.C < 1 || a.D < 1 || a.R * a.ldt >= lim || a.C * a.ldw >= lim || a.R * a.ldts >= lim ||
        a.C * a.ldws >= lim || a.ldt % 16 || a.ldw % 16 || a.ldts % 4 || a.ldws % 4 ||
        (!out_mx && (int64_t)a.R * a.ldo * 2 >= lim))
        return hipErrorInvalidValue;
    // row pairs: token codes read by the expansion, codes written by the
    // projection; pair pitches of whole 128-byte blocks
    if ((a.t_pairs && (out_mx || a.ldt % 128)) || (a.out_pairs && (!out_mx || a.ldo % 128)))
        return hipErrorNotSupported;
    const int tile = mx_gemm_tile(a.R, a.C, cus, out_mx);
    if (out_mx) {
        switch (tile) {
            case 0: return launch_z<256, 256, 2>(a, stream);
            case 1: return launch_z<256, 128, 2>(a, stream);
            case 3: return launch_z<128, 192, 3>(a, stream);
            default: return launch_z<128, 128, 2>(a, stream);
        }
    }
    return tile == 0 ? launch_pipelined<256>(a, cus, stream) : launch_pipelined<128>(a, cus, stream);
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
