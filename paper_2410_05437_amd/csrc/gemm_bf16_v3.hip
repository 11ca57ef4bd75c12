// Four-wave 256 x 256 bfloat16 "TN" GEMM for gfx950 with a hand-ordered
// main loop:
//
//     C[r][c] = sum_k A[r][k] * B[c][k]        (fp32 accumulation)
//
// A [R][D] and B [Cc][D] row-major with the reduced dimension contiguous.
//
// One wave per SIMD; wave (wr, wc) owns the 128 x 128 sub-tile at
// (128 wr, 128 wc) as 8 x 8 blocks of v_mfma_f32_16x16x32_bf16.  The MFMAs
// and the LDS fragment reads are written as inline assembly so that their
// order is exactly the one below (the compiler's scheduler otherwise groups
// the loads of a step together and leaves the matrix pipe idle while they
// issue, and splits the accumulators between AGPRs and VGPRs with copies in
// the loop); the accumulators are pinned to the AGPRs.
//
// Depth step 64 in two LDS stages of 64 KB (A rows then B rows, 128 bytes
// per row, 16-byte chunk c of row r stored at slot c ^ ((r >> 1) & 7), which
// makes the fragment reads conflict free).  Per step and wave:
//   sub-step 0: 64 MFMAs on fragment buffer 0; the 16 fragment reads of
//               sub-step 1 (same stage) go between the first 16 of them.
//   wait for the own reads and the own loads of the next stage, barrier.
//   sub-step 1: 64 MFMAs on buffer 1; between the first 32 of them the 16
//               fragment reads of the next step's sub-step 0 (next stage)
//               and the 16 buffer_load ... lds of step + 2 into the stage
//               just released.
// The loads of a step thus have one step of time to land.
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace espace {

namespace {

constexpr int V3_BM = 256, V3_BN = 256, V3_BK = 64;
constexpr int V3_NW = 4;                          // waves, 2 x 2
constexpr int V3_WT = 128;                        // wave tile edge
constexpr int V3_NB = 8;                          // 16 x 16 blocks per wave-tile edge
constexpr int V3_ROWB = 128;                      // bytes per LDS tile row
constexpr int V3_STAGE = (V3_BM + V3_BN) * V3_ROWB;   // 64 KB
constexpr int V3_LPW = (V3_BM + V3_BN) / 8 / V3_NW;   // 1 KB wave-loads per wave and stage (16)
constexpr int V3_EPI_LD = V3_WT * 2 + 16;         // epilogue staging row stride (bytes)
constexpr int V3_EPI = V3_NW * V3_WT * V3_EPI_LD;
constexpr int V3_SMEM = (2 * V3_STAGE > V3_EPI) ? 2 * V3_STAGE : V3_EPI;

__device__ __forceinline__ int v3_swz(int r) { return (r >> 1) & 7; }

// s_waitcnt with one counter and the others left free (gfx9 encoding)
__device__ __forceinline__ void v3_wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }
__device__ __forceinline__ void v3_wait_vm0() { __builtin_amdgcn_s_waitcnt(0x0F70); }

#define V3_MFMA(acc, a, b) \
    asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, %0" : "+a"(acc) : "v"(a), "v"(b))
#define V3_READ(dst, addr, off) \
    asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(dst) : "v"(addr), "i"(off))

// Copy of an accumulator block in VGPRs.  The accumulators are only ever
// named by inline assembly with AGPR operands, so the register allocator has
// no reason to give them a VGPR home (with copies in the loop).
__device__ __forceinline__ f32x4_t v3_acc_read(const f32x4_t& a) {
    f32x4_t v;
    float x0, x1, x2, x3;
    asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(x0) : "a"(a[0]));
    asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(x1) : "a"(a[1]));
    asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(x2) : "a"(a[2]));
    asm volatile("v_accvgpr_read_b32 %0, %1" : "=v"(x3) : "a"(a[3]));
    v[0] = x0; v[1] = x1; v[2] = x2; v[3] = x3;
    return v;
}

// Fragment reads of one sub-step into fa/fb (block i of A at +2048 i, of B at
// +2048 j from the lane's row address), in the order the MFMAs use them.
// Read x is issued after MFMA x of the enclosing sub-step when x < 16.
template <int X>
__device__ __forceinline__ void v3_read(bf16x8_t* fa, bf16x8_t* fb, unsigned aa, unsigned ab) {
    // order: fa0, fb0..fb7, fa1..fa7
    if constexpr (X == 0) V3_READ(fa[0], aa, 0);
    else if constexpr (X <= 8) V3_READ(fb[X - 1], ab, (X - 1) * 2048);
    else V3_READ(fa[X - 8], aa, (X - 8) * 2048);
}

// The loads of depth step kt (full depth) into stage st: wave-load j covers
// rows 8q .. 8q+7 of the combined A|B tile, q = wave + 4j; j < 8 are A rows.
__device__ __forceinline__ void v3_load(unsigned char* smem, const uint16_t* A, const uint16_t* B,
                                        unsigned a_bytes, unsigned b_bytes, const int* voff,
                                        int wave, int kt, int st, int j) {
    const int q = wave + 4 * j;
    const auto rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)(j < 8 ? A : B), (short)0,
                                                        (int)(j < 8 ? a_bytes : b_bytes), 0x00020000);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rsrc, (__attribute__((address_space(3))) void*)(smem + st * V3_STAGE + q * 1024), 16,
        voff[j], kt * V3_BK * 2, 0, 0);
}

// Sub-step 0 of a step: MFMAs on (fa0, fb0), the reads of sub-step 1 into
// (fa1, fb1) between the first 16.
__device__ __forceinline__ void v3_sub0(f32x4_t (&acc)[V3_NB][V3_NB], const bf16x8_t* fa0,
                                        const bf16x8_t* fb0, bf16x8_t* fa1, bf16x8_t* fb1,
                                        unsigned aa, unsigned ab) {
#pragma unroll
    for (int i = 0; i < V3_NB; ++i)
#pragma unroll
        for (int j = 0; j < V3_NB; ++j) {
            V3_MFMA(acc[i][j], fb0[j], fa0[i]);
            const int x = i * V3_NB + j;
            if (x < 16) {
                // template dispatch over the constant x after unrolling
#define V3_R(n) if (x == n) v3_read<n>(fa1, fb1, aa, ab);
                V3_R(0) V3_R(1) V3_R(2) V3_R(3) V3_R(4) V3_R(5) V3_R(6) V3_R(7)
                V3_R(8) V3_R(9) V3_R(10) V3_R(11) V3_R(12) V3_R(13) V3_R(14) V3_R(15)
#undef V3_R
            }
        }
}


// The loads of depth step kt into stage st for any step: full-depth steps by
// buffer_load ... lds, the depth tail through registers with the elements at
// or beyond D zeroed.
__device__ __forceinline__ void v3_load_any(unsigned char* smem, const uint16_t* A, const uint16_t* B,
                                            unsigned a_bytes, unsigned b_bytes, const int* voff,
                                            int wave, int lane, int kt, int st, int D) {
    if ((kt + 1) * V3_BK <= D) {
#pragma unroll
        for (int j = 0; j < V3_LPW; ++j) v3_load(smem, A, B, a_bytes, b_bytes, voff, wave, kt, st, j);
        return;
    }
    const int k0 = kt * V3_BK;
#pragma unroll
    for (int j = 0; j < V3_LPW; ++j) {
        const int q = wave + 4 * j;
        const int rr = q * 8 + (lane >> 3) - (j < 8 ? 0 : V3_BM);
        const int lc = (lane & 7) ^ v3_swz(rr);
        const uint16_t* rowp = (j < 8 ? A : B) + ((unsigned)voff[j] >> 1) - lc * 8;
        const u32x4_t v = load_chunk_masked(rowp, k0 + lc * 8, D);
        *reinterpret_cast<u32x4_t*>(smem + st * V3_STAGE + q * 1024 + lane * 16) = v;
    }
}

// The 16 fragment reads of one sub-step, back to back.
__device__ __forceinline__ void v3_read_all(bf16x8_t* fa, bf16x8_t* fb, unsigned aa, unsigned ab) {
    v3_read<0>(fa, fb, aa, ab);  v3_read<1>(fa, fb, aa, ab);  v3_read<2>(fa, fb, aa, ab);
    v3_read<3>(fa, fb, aa, ab);  v3_read<4>(fa, fb, aa, ab);  v3_read<5>(fa, fb, aa, ab);
    v3_read<6>(fa, fb, aa, ab);  v3_read<7>(fa, fb, aa, ab);  v3_read<8>(fa, fb, aa, ab);
    v3_read<9>(fa, fb, aa, ab);  v3_read<10>(fa, fb, aa, ab); v3_read<11>(fa, fb, aa, ab);
    v3_read<12>(fa, fb, aa, ab); v3_read<13>(fa, fb, aa, ab); v3_read<14>(fa, fb, aa, ab);
    v3_read<15>(fa, fb, aa, ab);
}

// 64 MFMAs of a sub-step with nothing between them.
__device__ __forceinline__ void v3_mfmas(f32x4_t (&acc)[V3_NB][V3_NB], const bf16x8_t* fa,
                                         const bf16x8_t* fb) {
#pragma unroll
    for (int i = 0; i < V3_NB; ++i)
#pragma unroll
        for (int j = 0; j < V3_NB; ++j) V3_MFMA(acc[i][j], fb[j], fa[i]);
}

// Sub-step 0 of a tile's first step: the accumulators start from zero (the
// inline constant 0 as the addend); reads of sub-step 1 between the first 16.
__device__ __forceinline__ void v3_sub0_first(f32x4_t (&acc)[V3_NB][V3_NB], const bf16x8_t* fa0,
                                              const bf16x8_t* fb0, bf16x8_t* fa1, bf16x8_t* fb1,
                                              unsigned aa, unsigned ab) {
#pragma unroll
    for (int i = 0; i < V3_NB; ++i)
#pragma unroll
        for (int j = 0; j < V3_NB; ++j) {
            asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0"
                         : "=a"(acc[i][j]) : "v"(fb0[j]), "v"(fa0[i]));
            const int x = i * V3_NB + j;
#define V3_R(n) if (x == n) v3_read<n>(fa1, fb1, aa, ab);
            V3_R(0) V3_R(1) V3_R(2) V3_R(3) V3_R(4) V3_R(5) V3_R(6) V3_R(7)
            V3_R(8) V3_R(9) V3_R(10) V3_R(11) V3_R(12) V3_R(13) V3_R(14) V3_R(15)
#undef V3_R
        }
}

// Sub-step 1 of a steady-state step: MFMAs on (fa1, fb1); between the first
// 32, alternately a read of the next step's sub-step 0 into (fa0, fb0) and
// one of this wave's 16 loads of step kt into stage ST.
template <int ST>
__device__ __forceinline__ void v3_sub1_steady(f32x4_t (&acc)[V3_NB][V3_NB], const bf16x8_t* fa1,
                                               const bf16x8_t* fb1, bf16x8_t* fa0, bf16x8_t* fb0,
                                               unsigned aa, unsigned ab, unsigned char* smem,
                                               const uint16_t* A, const uint16_t* B, unsigned a_bytes,
                                               unsigned b_bytes, const int* voff, int wave, int kt) {
#pragma unroll
    for (int i = 0; i < V3_NB; ++i)
#pragma unroll
        for (int j = 0; j < V3_NB; ++j) {
            V3_MFMA(acc[i][j], fb1[j], fa1[i]);
            const int x = i * V3_NB + j;
            if (x < 32) {
                if (x & 1) {
                    v3_load(smem, A, B, a_bytes, b_bytes, voff, wave, kt, ST, x >> 1);
                } else {
#define V3_R(n) if ((x >> 1) == n) v3_read<n>(fa0, fb0, aa, ab);
                    V3_R(0) V3_R(1) V3_R(2) V3_R(3) V3_R(4) V3_R(5) V3_R(6) V3_R(7)
                    V3_R(8) V3_R(9) V3_R(10) V3_R(11) V3_R(12) V3_R(13) V3_R(14) V3_R(15)
#undef V3_R
                }
            }
        }
}

enum { V3_BF16 = 0, V3_F32 = 1 };

// Matrices handed to this kernel hold fewer than 2^31 elements (the launcher
// checks), so byte offsets fit in 32 bits.  Every depth range is non-empty.
template <int MODE>
__global__ __launch_bounds__(256, 1)
void gemm_tn_bf16_v3_kernel(const uint16_t* __restrict__ A, int64_t lda,
                            const uint16_t* __restrict__ B, int64_t ldb,
                            void* __restrict__ Cout, int64_t ldc,
                            int R, int Cc, int D, int tiles_c, int ktiles_per_split,
                            int64_t split_stride, int map) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[V3_SMEM];

    int tile_r, tile_c;
    tile_coords<4>(blockIdx.x, gridDim.x, tiles_c, map, tile_r, tile_c);
    const int row0 = tile_r * V3_BM;
    const int col0 = tile_c * V3_BN;

    const int ktiles = (D + V3_BK - 1) / V3_BK;
    const int kt0 = blockIdx.y * ktiles_per_split;
    const int kt_end = kt0 + ktiles_per_split < ktiles ? kt0 + ktiles_per_split : ktiles;
    const int nfull = D / V3_BK < kt_end ? D / V3_BK : kt_end;   // end of the full-depth steps

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wrow0 = (wave >> 1) * V3_WT;
    const int wcol0 = (wave & 1) * V3_WT;

    // byte offset of this lane's 16-byte chunk of wave-load j, depth offset
    // excluded: row 8q + lane/8 of the A|B tile, logical chunk
    // (lane % 8) ^ swz(row); rows past the matrix are clamped to its last row
    int voff[V3_LPW];
#pragma unroll
    for (int j = 0; j < V3_LPW; ++j) {
        const int q = wave + 4 * j;
        const bool isA = j < 8;
        const int rr = q * 8 + (lane >> 3) - (isA ? 0 : V3_BM);
        const int lc = (lane & 7) ^ v3_swz(rr);
        int gr = (isA ? row0 : col0) + rr;
        const int lim = isA ? R : Cc;
        gr = gr < lim ? gr : lim - 1;
        voff[j] = (int)(((unsigned)gr * (unsigned)(isA ? lda : ldb) + (unsigned)(lc * 8)) * 2u);
    }
    const unsigned ra = (unsigned)((uint64_t)R * lda * 2u);
    const unsigned rb = (unsigned)((uint64_t)Cc * ldb * 2u);

    // fragment row addresses: a lane reads row lane % 16 of each 16-row block
    // and the 16-byte chunk 4 s + lane / 16 of sub-step s
    const int lr = lane & 15;
    const int lh = lane >> 4;
    const unsigned sbase =
        (unsigned)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)smem;
    const unsigned cs0 = (unsigned)((lh ^ v3_swz(lr)) * 16);
    const unsigned cs1 = cs0 ^ 64u;
    const unsigned arow = sbase + (unsigned)((wrow0 + lr) * V3_ROWB);
    const unsigned brow = sbase + (unsigned)((V3_BM + wcol0 + lr) * V3_ROWB);
    // addresses per [stage][sub-step]
    const unsigned aA00 = arow + cs0, aA01 = arow + cs1;
    const unsigned aA10 = arow + V3_STAGE + cs0, aA11 = arow + V3_STAGE + cs1;
    const unsigned aB00 = brow + cs0, aB01 = brow + cs1;
    const unsigned aB10 = brow + V3_STAGE + cs0, aB11 = brow + V3_STAGE + cs1;

    f32x4_t acc[V3_NB][V3_NB];
    bf16x8_t fa0[V3_NB], fb0[V3_NB], fa1[V3_NB], fb1[V3_NB];

    // prologue: steps kt0 and kt0+1 into stages 0 and 1, then the fragments
    // of step kt0's sub-step 0
    v3_load_any(smem, A, B, ra, rb, voff, wave, lane, kt0, 0, D);
    if (kt0 + 1 < kt_end) v3_load_any(smem, A, B, ra, rb, voff, wave, lane, kt0 + 1, 1, D);
    if (kt0 + 1 < nfull) {
        // both full-depth: step kt0's loads are the older half of vmcnt
        __builtin_amdgcn_s_waitcnt(0x0F70 | (V3_LPW & 15) | ((V3_LPW >> 4) << 14));
    } else {
        v3_wait_vm0();
        v3_wait_lgkm0();
    }
    __builtin_amdgcn_s_barrier();
    v3_read_all(fa0, fb0, aA00, aB00);
    v3_wait_lgkm0();

    int kt = kt0;
    int st = 0;
    // one step with the stage chosen at run time (the first one and the last
    // ones); FIRST: the accumulators start at zero
    auto generic_step = [&](auto first) {
        if constexpr (decltype(first)::value) {
            v3_sub0_first(acc, fa0, fb0, fa1, fb1, aA01, aB01);
        } else {
            v3_wait_lgkm0();
            v3_sub0(acc, fa0, fb0, fa1, fb1, st ? aA11 : aA01, st ? aB11 : aB01);
        }
        v3_wait_lgkm0();
        if (kt + 1 < kt_end) {
            v3_wait_vm0();
            __builtin_amdgcn_s_barrier();
            if (kt + 2 < kt_end) v3_load_any(smem, A, B, ra, rb, voff, wave, lane, kt + 2, st, D);
            v3_read_all(fa0, fb0, st ? aA00 : aA10, st ? aB00 : aB10);
        }
        v3_mfmas(acc, fa1, fb1);
        st ^= 1;
        ++kt;
    };
    generic_step(std::true_type{});
    // steady state, two steps per iteration (stages 1 and 0; the first step
    // used stage 0): the loads issued in them are full-depth steps below kt_end
    while (kt + 3 < nfull) {
        v3_wait_lgkm0();
        v3_sub0(acc, fa0, fb0, fa1, fb1, aA11, aB11);
        v3_wait_lgkm0();
        v3_wait_vm0();
        __builtin_amdgcn_s_barrier();
        v3_sub1_steady<1>(acc, fa1, fb1, fa0, fb0, aA00, aB00, smem, A, B, ra, rb, voff, wave, kt + 2);
        v3_wait_lgkm0();
        v3_sub0(acc, fa0, fb0, fa1, fb1, aA01, aB01);
        v3_wait_lgkm0();
        v3_wait_vm0();
        __builtin_amdgcn_s_barrier();
        v3_sub1_steady<0>(acc, fa1, fb1, fa0, fb0, aA10, aB10, smem, A, B, ra, rb, voff, wave, kt + 3);
        kt += 2;
    }
    while (kt < kt_end) generic_step(std::false_type{});

    // the accumulators are written by inline assembly the compiler does not
    // know as MFMAs: wait out the MFMA-to-VALU read hazard before any read
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    __syncthreads();

    // ---- epilogue ----------------------------------------------------------------
    // block (i, j): lane holds output row wrow0 + 16 i + lr and the 4 columns
    // wcol0 + 16 j + 4 lh + {0..3}
    if constexpr (MODE == V3_F32) {
        float* C = reinterpret_cast<float*>(Cout) + blockIdx.y * split_stride;
#pragma unroll
        for (int i = 0; i < V3_NB; ++i) {
            const int r = row0 + wrow0 + 16 * i + lr;
            if (r >= R) continue;
#pragma unroll
            for (int j = 0; j < V3_NB; ++j) {
                const int c = col0 + wcol0 + 16 * j + 4 * lh;
                float* p = C + (int64_t)r * ldc + c;
                const f32x4_t v = v3_acc_read(acc[i][j]);
                if (c + 4 <= Cc) {
                    *reinterpret_cast<f32x4_t*>(p) = v;
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e)
                        if (c + e < Cc) p[e] = v[e];
                }
            }
        }
    } else {
        unsigned char* ep = smem + wave * V3_WT * V3_EPI_LD;
#pragma unroll
        for (int i = 0; i < V3_NB; ++i)
#pragma unroll
            for (int j = 0; j < V3_NB; ++j) {
                const f32x4_t a = v3_acc_read(acc[i][j]);
                u32x2_t v;
                v[0] = pack_bf16x2(a[0], a[1]);
                v[1] = pack_bf16x2(a[2], a[3]);
                *reinterpret_cast<u32x2_t*>(ep + (16 * i + lr) * V3_EPI_LD + (16 * j + 4 * lh) * 2) = v;
            }
        __syncthreads();
        uint16_t* C = reinterpret_cast<uint16_t*>(Cout);
        // 16 chunks of 8 columns per wave-tile row, 4 rows per instruction
#pragma unroll 4
        for (int it = 0; it < V3_WT / 4; ++it) {
            const int rl = it * 4 + (lane >> 4);
            const int cl = (lane & 15) * 8;
            const int r = row0 + wrow0 + rl;
            const int c = col0 + wcol0 + cl;
            const u32x4_t v = *reinterpret_cast<const u32x4_t*>(ep + rl * V3_EPI_LD + cl * 2);
            if (r < R) {
                uint16_t* p = C + (int64_t)r * ldc + c;
                if (c + 8 <= Cc) {
                    *reinterpret_cast<u32x4_t*>(p) = v;
                } else if (c < Cc) {
#pragma unroll
                    for (int e = 0; e < 8; ++e)
                        if (c + e < Cc) p[e] = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
                }
            }
        }
    }
}

}  // namespace

// Tiled 256 x 256 product with the hand-ordered four-wave kernel; split-K
// partial sums are reduced by launch_splitk_reduce.  Returns
// hipErrorInvalidValue for shapes it does not take (the caller falls back).
hipError_t launch_gemm_tn_bf16_v3(const GemmArgs& g, hipStream_t stream) {
    const int64_t lim = (int64_t)1 << 31;
    if ((int64_t)g.R * g.lda >= lim || (int64_t)g.Cc * g.ldb >= lim || g.c_f32 || g.pair)
        return hipErrorInvalidValue;
    const int tiles_r = (g.R + V3_BM - 1) / V3_BM;
    const int tiles_c = (g.Cc + V3_BN - 1) / V3_BN;
    const int ktiles = (g.D + V3_BK - 1) / V3_BK;
    int S = g.splits < 1 ? 1 : g.splits;
    const int ktps = (ktiles + S - 1) / S;
    S = (ktiles + ktps - 1) / ktps;                 // no empty depth range
    dim3 grid(tiles_r * tiles_c, S);
    dim3 block(V3_NW * 64);
    const int map = g.variant >> 2;
    if (S == 1) {
        hipLaunchKernelGGL((gemm_tn_bf16_v3_kernel<V3_BF16>), grid, block, 0, stream, g.A, g.lda, g.B,
                           g.ldb, g.C, g.ldc, g.R, g.Cc, g.D, tiles_c, ktps, (int64_t)0, map);
        return hipGetLastError();
    }
    const int64_t ldp = splitk_ld(g.Cc);
    const int64_t split_stride = (int64_t)g.R * ldp;
    hipLaunchKernelGGL((gemm_tn_bf16_v3_kernel<V3_F32>), grid, block, 0, stream, g.A, g.lda, g.B,
                       g.ldb, (void*)g.partial, ldp, g.R, g.Cc, g.D, tiles_c, ktps, split_stride, map);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_splitk_reduce(g.partial, S, split_stride, ldp, g.C, g.ldc, g.R, g.Cc, 1, stream);
}

}  // namespace espace
