// Four-wave 256 x 256 bfloat16 "TN" GEMM for gfx950 with a hand-ordered
// main loop:
//
//     C[r][c] = sum_k A[r][k] * B[c][k]        (fp32 accumulation)
//
// A [R][D] and B [Cc][D] row-major with the reduced dimension contiguous.
//
// One wave per SIMD; wave (wr, wc) owns the 128 x 128 sub-tile at
// (128 wr, 128 wc) as 8 x 8 blocks of v_mfma_f32_16x16x32_bf16.  The MFMAs
// and the LDS fragment reads are inline assembly so that their order is
// exactly the one below (the compiler's scheduler otherwise groups a step's
// loads together and leaves the matrix pipe idle while they issue, and
// splits the accumulators between AGPRs and VGPRs with copies in the loop);
// the accumulators are pinned to the AGPRs.
//
// Depth step 64 as two sub-steps of 32, each with its own LDS half-stage of
// 32 KB (the 512 A|B rows of the tile, 64 bytes each; 16-byte chunk c of row
// r at slot c ^ ((r >> 2) & 3), which makes the fragment reads conflict
// free); four half-stages hold two steps.  Per sub-step h of step kt, each
// wave issues 64 MFMAs on the fragments in registers, with between them the
// 16 fragment reads of the following sub-step and its 8 buffer_load ... lds
// of half h of step kt + 2 into the half-stage this sub-step's fragments
// came from, and ends with a barrier.  A load thus has a step and a half to
// land, and the loads of a step are spread over all its MFMAs (the texture
// path that feeds the LDS cannot take a step's 64 KB in half a step).
#include <type_traits>

#include "common.hpp"
#include "kernels.hpp"

namespace espace {

namespace {

constexpr int V3_BM = 256, V3_BN = 256, V3_BK = 64;
constexpr int V3_NW = 4;                          // waves, 2 x 2
constexpr int V3_WT = 128;                        // wave tile edge
constexpr int V3_NB = 8;                          // 16 x 16 blocks per wave-tile edge
constexpr int V3_ROWB = 64;                       // bytes per half-stage row
constexpr int V3_HS = (V3_BM + V3_BN) * V3_ROWB;  // half-stage: 32 KB
constexpr int V3_LPH = (V3_BM + V3_BN) / 16 / V3_NW;   // 1 KB wave-loads per wave and half-stage (8)
constexpr int V3_SMEM = 4 * V3_HS;

__device__ __forceinline__ int v3_swz(int r) { return (r >> 2) & 3; }

// s_waitcnt with one counter and the others left free (gfx9 encoding)
__device__ __forceinline__ void v3_wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }
template <int N>
__device__ __forceinline__ void v3_wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}
// vmcnt(n) for n a multiple of 8 up to 56, chosen at run time
__device__ __forceinline__ void v3_wait_vm_n(int n) {
    if (n <= 0) v3_wait_vm<0>();
    else if (n <= 8) v3_wait_vm<8>();
    else if (n <= 16) v3_wait_vm<16>();
    else if (n <= 24) v3_wait_vm<24>();
    else if (n <= 32) v3_wait_vm<32>();
    else if (n <= 40) v3_wait_vm<40>();
    else if (n <= 48) v3_wait_vm<48>();
    else v3_wait_vm<56>();
}

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

// Fragment read x of a sub-step (block i of A at +1024 i from the lane's row
// address, of B at +1024 j), in the order the MFMAs use them: fa0, fb0..fb7,
// fa1..fa7.
template <int X>
__device__ __forceinline__ void v3_read(bf16x8_t* fa, bf16x8_t* fb, unsigned aa, unsigned ab) {
    if constexpr (X == 0) V3_READ(fa[0], aa, 0);
    else if constexpr (X <= 8) V3_READ(fb[X - 1], ab, (X - 1) * 1024);
    else V3_READ(fa[X - 8], aa, (X - 8) * 1024);
}

__device__ __forceinline__ void v3_read_dyn(int x, bf16x8_t* fa, bf16x8_t* fb, unsigned aa, unsigned ab) {
    // x is a constant after unrolling
#define V3_R(n) if (x == n) v3_read<n>(fa, fb, aa, ab);
    V3_R(0) V3_R(1) V3_R(2) V3_R(3) V3_R(4) V3_R(5) V3_R(6) V3_R(7)
    V3_R(8) V3_R(9) V3_R(10) V3_R(11) V3_R(12) V3_R(13) V3_R(14) V3_R(15)
#undef V3_R
}

// Wave-load j of half h of depth step kt into half-stage u (full depth): it
// covers rows 16q .. 16q+15 of the A|B tile, q = wave + 4j; j < 4 are A rows.
__device__ __forceinline__ void v3_load(unsigned char* smem, const uint16_t* A, const uint16_t* B,
                                        unsigned a_bytes, unsigned b_bytes, const int* voff,
                                        int wave, int kt, int h, int u, int j) {
    const int q = wave + 4 * j;
    const auto rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)(j < 4 ? A : B), (short)0,
                                                        (int)(j < 4 ? a_bytes : b_bytes), 0x00020000);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rsrc, (__attribute__((address_space(3))) void*)(smem + u * V3_HS + q * 1024), 16,
        voff[j], (kt * V3_BK + 32 * h) * 2, 0, 0);
}

// Half h of depth step kt into half-stage u for any step: full depth by
// buffer_load ... lds (8 per wave, returns 8), the depth tail through
// registers with the elements at or beyond D zeroed (returns 0: nothing of
// it stays in flight).
__device__ __forceinline__ int v3_load_half(unsigned char* smem, const uint16_t* A, const uint16_t* B,
                                            unsigned a_bytes, unsigned b_bytes, const int* voff,
                                            int wave, int lane, int kt, int h, int u, int D) {
    const int k0 = kt * V3_BK + 32 * h;
    if (k0 + 32 <= D) {
#pragma unroll
        for (int j = 0; j < V3_LPH; ++j) v3_load(smem, A, B, a_bytes, b_bytes, voff, wave, kt, h, u, j);
        return V3_LPH;
    }
#pragma unroll
    for (int j = 0; j < V3_LPH; ++j) {
        const int q = wave + 4 * j;
        const int rr = q * 16 + (lane >> 2) - (j < 4 ? 0 : V3_BM);
        const int lc = (lane & 3) ^ v3_swz(rr);
        const uint16_t* rowp = (j < 4 ? A : B) + ((unsigned)voff[j] >> 1) - lc * 8;
        const u32x4_t v = load_chunk_masked(rowp, k0 + lc * 8, D);
        *reinterpret_cast<u32x4_t*>(smem + u * V3_HS + q * 1024 + lane * 16) = v;
    }
    return 0;
}

// One sub-step: 64 MFMAs on (fa, fb); after MFMA 2x (x < 16) fragment read x
// into (ra, rb) from (aa, ab) when READS; after MFMA 8y + 4 (y < 8) wave-load
// y of half h of step kt into half-stage u when LOADS; FIRST: the
// accumulators start from zero (the inline constant 0 as the addend).
template <bool FIRST, bool READS, bool LOADS>
__device__ __forceinline__ void v3_substep(f32x4_t (&acc)[V3_NB][V3_NB], const bf16x8_t* fa,
                                           const bf16x8_t* fb, bf16x8_t* ra, bf16x8_t* rb,
                                           unsigned aa, unsigned ab, unsigned char* smem,
                                           const uint16_t* A, const uint16_t* B, unsigned a_bytes,
                                           unsigned b_bytes, const int* voff, int wave, int kt,
                                           int h, int u) {
#pragma unroll
    for (int i = 0; i < V3_NB; ++i)
#pragma unroll
        for (int j = 0; j < V3_NB; ++j) {
            if constexpr (FIRST)
                asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0"
                             : "=a"(acc[i][j]) : "v"(fb[j]), "v"(fa[i]));
            else
                V3_MFMA(acc[i][j], fb[j], fa[i]);
            const int x = i * V3_NB + j;
            if constexpr (READS)
                if (x < 32 && (x & 1) == 0) v3_read_dyn(x >> 1, ra, rb, aa, ab);
            if constexpr (LOADS)
                if ((x & 7) == 4) v3_load(smem, A, B, a_bytes, b_bytes, voff, wave, kt, h, u, x >> 3);
        }
}

enum { V3_BF16 = 0, V3_F32 = 1 };

// byte offsets of this lane's 16-byte chunk of each wave-load (depth offset
// excluded) for the tile at (row0, col0): row 16q + lane/4 of the A|B tile,
// logical chunk (lane % 4) ^ swz(row); rows past the matrix are clamped to
// its last row
__device__ __forceinline__ void v3_offsets(int* voff, int row0, int col0, int R, int Cc, int64_t lda,
                                           int64_t ldb, int wave, int lane) {
#pragma unroll
    for (int j = 0; j < V3_LPH; ++j) {
        const int q = wave + 4 * j;
        const bool isA = j < 4;
        const int rr = q * 16 + (lane >> 2) - (isA ? 0 : V3_BM);
        const int lc = (lane & 3) ^ v3_swz(rr);
        int gr = (isA ? row0 : col0) + rr;
        const int lim = isA ? R : Cc;
        gr = gr < lim ? gr : lim - 1;
        voff[j] = (int)(((unsigned)gr * (unsigned)(isA ? lda : ldb) + (unsigned)(lc * 8)) * 2u);
    }
}

// Matrices handed to this kernel hold fewer than 2^31 elements (the launcher
// checks), so byte offsets fit in 32 bits.  Every depth range is non-empty.
//
// Work items are the output tiles (and depth ranges, blockIdx.y); a
// workgroup takes items blockIdx.x, blockIdx.x + gridDim.x, ...  When the
// next item of a workgroup starts with two full-depth steps and this item's
// output is bf16 with a column count that is a multiple of 8, the last two
// steps of an item load the next item's first two steps, so they land while
// this item's results are written.  The results then take exactly 32 stores
// per wave (out-of-range lanes use an offset past the buffer, which the
// hardware drops), so the next item waits for its first step with
// vmcnt(16 + 32).
template <int MODE>
__global__ __launch_bounds__(256, 1)
void gemm_tn_bf16_v3_kernel(const uint16_t* __restrict__ A, int64_t lda,
                            const uint16_t* __restrict__ B, int64_t ldb,
                            void* __restrict__ Cout, int64_t ldc,
                            int R, int Cc, int D, int tiles_c, int ntiles, int ktiles_per_split,
                            int64_t split_stride, int map) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[V3_SMEM];

    const int ktiles = (D + V3_BK - 1) / V3_BK;
    const int kt0 = blockIdx.y * ktiles_per_split;
    const int kt_end = kt0 + ktiles_per_split < ktiles ? kt0 + ktiles_per_split : ktiles;
    const int nfull = D / V3_BK < kt_end ? D / V3_BK : kt_end;   // end of the full-depth steps
    const int nsteps = kt_end - kt0;
    // the next item's first two steps can be loaded ahead
    const bool ahead_ok = MODE == V3_BF16 && (Cc & 7) == 0 && kt0 + 2 <= nfull;

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wrow0 = (wave >> 1) * V3_WT;
    const int wcol0 = (wave & 1) * V3_WT;
    const unsigned ra = (unsigned)((uint64_t)R * lda * 2u);
    const unsigned rb = (unsigned)((uint64_t)Cc * ldb * 2u);

    // fragment row addresses: a lane reads row lane % 16 of each 16-row block
    // and depth chunk lane / 16 of the sub-step
    const int lr = lane & 15;
    const int lh = lane >> 4;
    const unsigned sbase =
        (unsigned)(uintptr_t)(__attribute__((address_space(3))) unsigned char*)smem;
    const unsigned slot = (unsigned)((lh ^ v3_swz(lr)) * 16);
    const unsigned arow = sbase + (unsigned)((wrow0 + lr) * V3_ROWB) + slot;
    const unsigned brow = sbase + (unsigned)((V3_BM + wcol0 + lr) * V3_ROWB) + slot;

    f32x4_t acc[V3_NB][V3_NB];
    bf16x8_t fa0[V3_NB], fb0[V3_NB], fa1[V3_NB], fb1[V3_NB];
    int voff[V3_LPH];

    int item = blockIdx.x;
    int tile_r, tile_c;
    tile_coords<4>(item, ntiles, tiles_c, map, tile_r, tile_c);
    bool ahead = false;     // this item's first two steps were loaded by the previous one
    int s0 = 0;             // stage of this item's first step (half-stages 2 s0, 2 s0 + 1)
    while (true) {
        const int row0 = tile_r * V3_BM;
        const int col0 = tile_c * V3_BN;
        const int next = item + (int)gridDim.x;
        const bool ahead_next = ahead_ok && next < ntiles;
        int ntr = 0, ntc = 0;
        if (next < ntiles) tile_coords<4>(next, ntiles, tiles_c, map, ntr, ntc);

        // half-stage of (stage relative to s0, half)
        auto hs = [&](int rel, int h) { return ((rel ^ s0) << 1) | h; };
        // fragment addresses of half-stage u
        const unsigned aA0 = arow + (unsigned)(hs(0, 0) * V3_HS), aB0 = brow + (unsigned)(hs(0, 0) * V3_HS);
        const unsigned aA1 = arow + (unsigned)(hs(0, 1) * V3_HS), aB1 = brow + (unsigned)(hs(0, 1) * V3_HS);
        const unsigned aA2 = arow + (unsigned)(hs(1, 0) * V3_HS), aB2 = brow + (unsigned)(hs(1, 0) * V3_HS);
        const unsigned aA3 = arow + (unsigned)(hs(1, 1) * V3_HS), aB3 = brow + (unsigned)(hs(1, 1) * V3_HS);

        if (ahead) {
            // this wave's loads of the first step, then 16 loads of the second
            // and 32 stores of the previous item's results were issued
            v3_wait_vm<48>();
        } else {
            // the half-stages may still be read by a wave finishing the previous item
            if (item != (int)blockIdx.x) __syncthreads();
            v3_offsets(voff, row0, col0, R, Cc, lda, ldb, wave, lane);
            int later = v3_load_half(smem, A, B, ra, rb, voff, wave, lane, kt0, 0, hs(0, 0), D);
            later = v3_load_half(smem, A, B, ra, rb, voff, wave, lane, kt0, 1, hs(0, 1), D);
            if (nsteps > 1) {
                later = v3_load_half(smem, A, B, ra, rb, voff, wave, lane, kt0 + 1, 0, hs(1, 0), D);
                later += v3_load_half(smem, A, B, ra, rb, voff, wave, lane, kt0 + 1, 1, hs(1, 1), D);
            } else {
                later = 0;
            }
            // the first step's loads are the older ones; register-path loads
            // completed where they were issued
            v3_wait_vm_n(later);
            v3_wait_lgkm0();
        }
        __builtin_amdgcn_s_barrier();
#pragma unroll
        for (int x = 0; x < 16; ++x) v3_read_dyn(x, fa0, fb0, aA0, aB0);
        v3_wait_lgkm0();

        int kt = kt0;
        int rel = 0;          // stage of step kt relative to s0
        // the loads issued in sub-step h of step kt: half h of step kt + 2 of
        // this item, or of the next item's first steps; returns how many stay
        // in flight
        auto issue_any = [&](int h) -> int {
            const int u = hs(rel, h);
            if (kt + 2 < kt_end) return v3_load_half(smem, A, B, ra, rb, voff, wave, lane, kt + 2, h, u, D);
            if (ahead_next) {
                if (kt + 2 == kt_end && h == 0)
                    v3_offsets(voff, ntr * V3_BM, ntc * V3_BN, R, Cc, lda, ldb, wave, lane);
#pragma unroll
                for (int j = 0; j < V3_LPH; ++j)
                    v3_load(smem, A, B, ra, rb, voff, wave, kt0 + (kt + 2 - kt_end), h, u, j);
                return V3_LPH;
            }
            return 0;
        };
        // one step with the stage chosen at run time (the first one and the
        // last ones); FIRST: the accumulators start at zero
        auto generic_step = [&](auto first) {
            constexpr bool F = decltype(first)::value;
            // after an item loaded ahead, its first step has the previous
            // item's 32 stores in flight behind the loads of its second step
            const int stores = (F && ahead) ? 32 : 0;
            // sub-step 0: fragments of sub-step 1 from the second half-stage
            v3_substep<F, true, false>(acc, fa0, fb0, fa1, fb1, rel ? aA3 : aA1, rel ? aB3 : aB1, smem,
                                       A, B, ra, rb, voff, wave, kt, 0, 0);
            const int n0 = issue_any(0);
            v3_wait_lgkm0();
            if (kt + 1 < kt_end || ahead_next) {
                // the next step's first half has landed (the loads just issued may stay in flight)
                if (kt + 1 < kt_end) v3_wait_vm_n(V3_LPH + stores + n0);
                __builtin_amdgcn_s_barrier();
            }
            // sub-step 1: fragments of the next step's sub-step 0 (after the
            // last step the reads are of no use but harmless: one code path
            // keeps the accumulators in place)
            v3_substep<false, true, false>(acc, fa1, fb1, fa0, fb0, rel ? aA0 : aA2, rel ? aB0 : aB2,
                                           smem, A, B, ra, rb, voff, wave, kt, 1, 0);
            const int n1 = issue_any(1);
            v3_wait_lgkm0();
            if (kt + 1 < kt_end) {
                // the next step's second half has landed
                v3_wait_vm_n(stores + n0 + n1);
                __builtin_amdgcn_s_barrier();
            }
            rel ^= 1;
            ++kt;
        };
        generic_step(std::true_type{});
        // steady state, two steps per iteration (relative stages 1 and 0):
        // the loads issued in them are full-depth halves of this item; each
        // barrier waits for the half-stage the next sub-step reads, with the
        // two newer half-steps of loads in flight
        while (kt + 3 < nfull) {
            v3_substep<false, true, true>(acc, fa0, fb0, fa1, fb1, aA3, aB3, smem, A, B, ra, rb, voff,
                                          wave, kt + 2, 0, hs(1, 0));
            v3_wait_lgkm0();
            v3_wait_vm<16>();
            __builtin_amdgcn_s_barrier();
            v3_substep<false, true, true>(acc, fa1, fb1, fa0, fb0, aA0, aB0, smem, A, B, ra, rb, voff,
                                          wave, kt + 2, 1, hs(1, 1));
            v3_wait_lgkm0();
            v3_wait_vm<16>();
            __builtin_amdgcn_s_barrier();
            v3_substep<false, true, true>(acc, fa0, fb0, fa1, fb1, aA1, aB1, smem, A, B, ra, rb, voff,
                                          wave, kt + 3, 0, hs(0, 0));
            v3_wait_lgkm0();
            v3_wait_vm<16>();
            __builtin_amdgcn_s_barrier();
            v3_substep<false, true, true>(acc, fa1, fb1, fa0, fb0, aA2, aB2, smem, A, B, ra, rb, voff,
                                          wave, kt + 3, 1, hs(0, 1));
            v3_wait_lgkm0();
            v3_wait_vm<16>();
            __builtin_amdgcn_s_barrier();
            kt += 2;
        }
        while (kt < kt_end) generic_step(std::false_type{});

        // the accumulators are written by inline assembly the compiler does
        // not know as MFMAs: wait out the MFMA-to-VALU read hazard
        __builtin_amdgcn_sched_barrier(0);
        asm volatile("s_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7\n\ts_nop 7" ::: "memory");
        __builtin_amdgcn_sched_barrier(0);

        // ---- epilogue ------------------------------------------------------------
        // block (i, j): lane holds output row wrow0 + 16 i + lr and the 4
        // columns wcol0 + 16 j + 4 lh + {0..3}
        if constexpr (MODE == V3_F32) {
            float* C = reinterpret_cast<float*>(Cout) + blockIdx.y * split_stride;
#pragma unroll
            for (int i = 0; i < V3_NB; ++i) {
                const int r = row0 + wrow0 + 16 * i + lr;
#pragma unroll
                for (int j = 0; j < V3_NB; ++j) {
                    const f32x4_t v = v3_acc_read(acc[i][j]);
                    const int c = col0 + wcol0 + 16 * j + 4 * lh;
                    if (r >= R) continue;
                    float* p = C + (int64_t)r * ldc + c;
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
            // straight from the registers: two column blocks of a row block
            // are converted to bf16 and half of each lane's values swapped
            // with the lane 16 away (v_permlane16_swap), after which every
            // lane holds 8 consecutive columns of its row: lane groups
            // lh = 0..3 hold columns 0-7 of block j, 0-7 of block j+1, 8-15
            // of block j, 8-15 of block j+1
            uint16_t* C = reinterpret_cast<uint16_t*>(Cout);
            const unsigned cbytes = (unsigned)((uint64_t)R * ldc * 2u);
            const auto crsrc = __builtin_amdgcn_make_buffer_rsrc((void*)C, (short)0, (int)cbytes, 0x00020000);
#pragma unroll
            for (int i = 0; i < V3_NB; ++i) {
                const int r = row0 + wrow0 + 16 * i + lr;
#pragma unroll
                for (int m = 0; m < V3_NB / 2; ++m) {
                    const f32x4_t a = v3_acc_read(acc[i][2 * m]);
                    const f32x4_t b = v3_acc_read(acc[i][2 * m + 1]);
                    const auto s0 = __builtin_amdgcn_permlane16_swap(pack_bf16x2(a[0], a[1]),
                                                                     pack_bf16x2(b[0], b[1]), false, false);
                    const auto s1 = __builtin_amdgcn_permlane16_swap(pack_bf16x2(a[2], a[3]),
                                                                     pack_bf16x2(b[2], b[3]), false, false);
                    const u32x4_t v = {s0[0], s1[0], s0[1], s1[1]};
                    const int c = col0 + wcol0 + 16 * (2 * m + (lh & 1)) + 8 * (lh >> 1);
                    if ((Cc & 7) == 0) {
                        // exactly one store instruction per lane group and
                        // block pair; lanes outside the matrix are dropped by
                        // the buffer's range check
                        const unsigned off = (r < R && c < Cc)
                                                 ? ((unsigned)r * (unsigned)ldc + (unsigned)c) * 2u
                                                 : 0xFFFFFFF0u;
                        __builtin_amdgcn_raw_buffer_store_b128(v, crsrc, (int)off, 0, 0);
                    } else if (r < R) {
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
        if (next >= ntiles) break;
        item = next;
        tile_r = ntr;
        tile_c = ntc;
        s0 = (s0 + nsteps) & 1;
        ahead = ahead_next;
    }
}

}  // namespace

// Tiled 256 x 256 product with the hand-ordered four-wave kernel; split-K
// partial sums are reduced by launch_splitk_reduce.  Returns
// hipErrorInvalidValue for products it does not take (the caller falls back).
hipError_t launch_gemm_tn_bf16_v3(const GemmArgs& g, hipStream_t stream) {
    const int64_t lim = (int64_t)1 << 31;
    if ((int64_t)g.R * g.lda >= lim || (int64_t)g.Cc * g.ldb >= lim || (int64_t)g.R * g.ldc >= lim ||
        g.c_f32 || g.pair)
        return hipErrorInvalidValue;
    const int tiles_r = (g.R + V3_BM - 1) / V3_BM;
    const int tiles_c = (g.Cc + V3_BN - 1) / V3_BN;
    const int ntiles = tiles_r * tiles_c;
    const int ktiles = (g.D + V3_BK - 1) / V3_BK;
    int S = g.splits < 1 ? 1 : g.splits;
    const int ktps = (ktiles + S - 1) / S;
    S = (ktiles + ktps - 1) / ktps;                 // no empty depth range
    dim3 block(V3_NW * 64);
    const int map = g.variant >> 2;
    if (S == 1) {
        // one workgroup per CU, each taking every 256th tile (variant bit 4:
        // one tile per workgroup)
        const int persistent = (g.variant & 16) ? ntiles : 256;
        dim3 grid(ntiles < persistent ? ntiles : persistent, 1);
        hipLaunchKernelGGL((gemm_tn_bf16_v3_kernel<V3_BF16>), grid, block, 0, stream, g.A, g.lda, g.B,
                           g.ldb, g.C, g.ldc, g.R, g.Cc, g.D, tiles_c, ntiles, ktps, (int64_t)0, map);
        return hipGetLastError();
    }
    dim3 grid(ntiles, S);
    const int64_t ldp = splitk_ld(g.Cc);
    const int64_t split_stride = (int64_t)g.R * ldp;
    hipLaunchKernelGGL((gemm_tn_bf16_v3_kernel<V3_F32>), grid, block, 0, stream, g.A, g.lda, g.B,
                       g.ldb, (void*)g.partial, ldp, g.R, g.Cc, g.D, tiles_c, ntiles, ktps, split_stride,
                       map);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_splitk_reduce(g.partial, S, split_stride, ldp, g.C, g.ldc, g.R, g.Cc, 1, stream);
}

}  // namespace espace
