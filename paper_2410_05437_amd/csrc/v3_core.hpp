// Building blocks of the hand-ordered four-wave 256 x BN bfloat16 MFMA GEMM
// (gfx950), shared by the plain GEMM kernel and the one-launch projected
// linear layer.  See gemm_bf16_v3.hip for the pipeline they implement.
#pragma once

#include "common.hpp"

namespace espace {

namespace {

constexpr int V3_BM = 256, V3_BK = 64;
constexpr int V3_NW = 4;                          // waves, 2 x 2
constexpr int V3_WT = 128;                        // wave tile rows
constexpr int V3_NB = 8;                          // 16-row blocks per wave tile
constexpr int V3_ROWB = 64;                       // bytes per half-stage row

// Tile 256 x BN (BN = 256 or 192): each wave owns 128 x BN/2 as 8 x NBJ blocks.
template <int BN>
struct V3Cfg {
    static constexpr int NBJ = BN / 32;                   // 16-column blocks per wave tile
    static constexpr int ROWS = V3_BM + BN;               // A|B rows of a half-stage
    static constexpr int HS = ROWS * V3_ROWB;             // half-stage bytes (32 or 28 KB)
    static constexpr int LPH = ROWS / 16 / V3_NW;         // 1 KB wave-loads per wave and half-stage
    static constexpr int NRD = V3_NB + NBJ;               // fragment reads per sub-step
    static constexpr int NMF = V3_NB * NBJ;               // MFMAs per sub-step
    static constexpr int NST = V3_NB * NBJ / 2;           // epilogue stores per wave
    static constexpr int SMEM = 4 * HS;
    // row blocks of the partner's sums in flight in the pair epilogue: all
    // of them where the registers allow (256 x 192), else one ahead
    static constexpr int PD = BN == 192 ? V3_NB - 1 : 1;
    static_assert(ROWS % (16 * V3_NW) == 0 && 2 * NRD <= NMF && NBJ % 2 == 0, "tile");
    // MFMA after which wave-load y of a sub-step is issued
    static constexpr int load_slot(int y) { return y * NMF / LPH + NMF / (2 * LPH); }
};

__device__ __forceinline__ int v3_swz(int r) { return (r >> 1) & 3; }

// s_waitcnt with one counter and the others left free (gfx9 encoding)
__device__ __forceinline__ void v3_wait_lgkm0() { __builtin_amdgcn_s_waitcnt(0xC07F); }
template <int N>
__device__ __forceinline__ void v3_wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}
// vmcnt(n) for the counts the generic steps need (k wave-loads of LPH,
// plus the previous item's NST stores); any other n waits for everything
template <class C>
__device__ __forceinline__ void v3_wait_vm_n(int n) {
    constexpr int L = C::LPH, S = C::NST;
    if (n == 0) v3_wait_vm<0>();
    else if (n == L) v3_wait_vm<L>();
    else if (n == 2 * L) v3_wait_vm<2 * L>();
    else if (n == 3 * L) v3_wait_vm<3 * L>();
    else if (n == S) v3_wait_vm<S>();
    else if (n == L + S) v3_wait_vm<L + S>();
    else if (n == 2 * L + S) v3_wait_vm<2 * L + S>();
    else if (n == 3 * L + S) v3_wait_vm<3 * L + S>();
    else v3_wait_vm<0>();
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
// address, of B at +1024 j), in the order the MFMAs use them: fa0,
// fb0..fb(NBJ-1), fa1..fa7.
template <int NBJ, int X>
__device__ __forceinline__ void v3_read(bf16x8_t* fa, bf16x8_t* fb, unsigned aa, unsigned ab) {
    if constexpr (X == 0) V3_READ(fa[0], aa, 0);
    else if constexpr (X <= NBJ) V3_READ(fb[X - 1], ab, (X - 1) * 1024);
    else V3_READ(fa[X - NBJ], aa, (X - NBJ) * 1024);
}

template <int NBJ>
__device__ __forceinline__ void v3_read_dyn(int x, bf16x8_t* fa, bf16x8_t* fb, unsigned aa, unsigned ab) {
    // x is a constant after unrolling
#define V3_R(n) if constexpr (n < V3_NB + NBJ) { if (x == n) v3_read<NBJ, n>(fa, fb, aa, ab); }
    V3_R(0) V3_R(1) V3_R(2) V3_R(3) V3_R(4) V3_R(5) V3_R(6) V3_R(7)
    V3_R(8) V3_R(9) V3_R(10) V3_R(11) V3_R(12) V3_R(13) V3_R(14) V3_R(15)
#undef V3_R
}

// Wave-load j of half h of depth step kt into half-stage u (full depth): it
// covers rows 16q .. 16q+15 of the A|B tile, q = wave + 4j; j < 4 are A rows.
// APAIR: A in the row-pair layout, where the 32-deep block of half h of step
// kt lies (2 kt + h) * 128 bytes into a row pair (twice the plain offset).
template <class C, bool APAIR = false>
__device__ __forceinline__ void v3_load(unsigned char* smem, const uint16_t* A, const uint16_t* B,
                                        unsigned a_bytes, unsigned b_bytes, const int* voff,
                                        int wave, int kt, int h, int u, int j) {
    const int q = wave + 4 * j;
    const auto rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)(j < 4 ? A : B), (short)0,
                                                        (int)(j < 4 ? a_bytes : b_bytes), 0x00020000);
    const int soff = (kt * V3_BK + 32 * h) * ((APAIR && j < 4) ? 4 : 2);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rsrc, (__attribute__((address_space(3))) void*)(smem + u * C::HS + q * 1024), 16,
        voff[j], soff, 0, 0);
}

// Half h of depth step kt into half-stage u for any step: full depth by
// buffer_load ... lds (8 per wave, returns 8), the depth tail through
// registers with the elements at or beyond D zeroed (returns 0: nothing of
// it stays in flight).
template <class C, bool APAIR = false>
__device__ __forceinline__ int v3_load_half(unsigned char* smem, const uint16_t* A, const uint16_t* B,
                                            unsigned a_bytes, unsigned b_bytes, const int* voff,
                                            int wave, int lane, int kt, int h, int u, int D) {
    const int k0 = kt * V3_BK + 32 * h;
    if (k0 + 32 <= D) {
#pragma unroll
        for (int j = 0; j < C::LPH; ++j)
            v3_load<C, APAIR>(smem, A, B, a_bytes, b_bytes, voff, wave, kt, h, u, j);
        return C::LPH;
    }
#pragma unroll
    for (int j = 0; j < C::LPH; ++j) {
        const int q = wave + 4 * j;
        const int rr = q * 16 + (lane >> 2) - (j < 4 ? 0 : V3_BM);
        const int lc = (lane & 3) ^ v3_swz(rr);
        // plain rows: the row start; row pairs: the row's 32-element block at
        // depth k0 sits 2 k0 elements past its first block, so the element at
        // depth k0 + e (e < 32) is at rowp + k0 + (k0 + e)
        const uint16_t* rowp = (j < 4 ? A : B) + ((unsigned)voff[j] >> 1) - lc * 8 + ((APAIR && j < 4) ? k0 : 0);
        const u32x4_t v = load_chunk_masked(rowp, k0 + lc * 8, D);
        *reinterpret_cast<u32x4_t*>(smem + u * C::HS + q * 1024 + lane * 16) = v;
    }
    return 0;
}

// One sub-step: NMF MFMAs on (fa, fb); after MFMA 2x (x < NRD) fragment read
// x into (ra, rb) from (aa, ab) when READS; after MFMA load_slot(y) wave-load
// y of half h of step kt into half-stage u when LOADS and do_load (uniform);
// FIRST: the accumulators start from zero (the inline constant 0 as the
// addend).
template <class C, bool FIRST, bool READS, bool LOADS, bool APAIR = false>
__device__ __forceinline__ void v3_substep(f32x4_t (&acc)[V3_NB][C::NBJ], const bf16x8_t* fa,
                                           const bf16x8_t* fb, bf16x8_t* ra, bf16x8_t* rb,
                                           unsigned aa, unsigned ab, unsigned char* smem,
                                           const uint16_t* A, const uint16_t* B, unsigned a_bytes,
                                           unsigned b_bytes, const int* voff, int wave, int kt,
                                           int h, int u, bool do_load = true) {
#pragma unroll
    for (int i = 0; i < V3_NB; ++i)
#pragma unroll
        for (int j = 0; j < C::NBJ; ++j) {
            if constexpr (FIRST)
                asm volatile("v_mfma_f32_16x16x32_bf16 %0, %1, %2, 0"
                             : "=a"(acc[i][j]) : "v"(fb[j]), "v"(fa[i]));
            else
                V3_MFMA(acc[i][j], fb[j], fa[i]);
            const int x = i * C::NBJ + j;
            if constexpr (READS)
                if (x < 2 * C::NRD && (x & 1) == 0) v3_read_dyn<C::NBJ>(x >> 1, ra, rb, aa, ab);
            if constexpr (LOADS) {
#pragma unroll
                for (int y = 0; y < C::LPH; ++y)
                    if (x == C::load_slot(y) && do_load)
                        v3_load<C, APAIR>(smem, A, B, a_bytes, b_bytes, voff, wave, kt, h, u, y);
            }
        }
}

enum { V3_BF16 = 0, V3_F32 = 1, V3_PAIR = 2 };

// byte offsets of this lane's 16-byte chunk of each wave-load (depth offset
// excluded) for the tile at (row0, col0): row 16q + lane/4 of the A|B tile,
// logical chunk (lane % 4) ^ swz(row), swz(row) = (row >> SH) & 3 (SH = 1
// is v3_swz, for the bf16 fragment reads of 16 rows; the fp8 kernel's reads
// of 32 rows take SH = 2); rows past the matrix are clamped to its last row.
// APAIR: A in the row-pair layout (lda its pair pitch); the four lanes of a
// row then read one half of a 128-byte block whose other half the next
// four lanes read for the row's partner, so a wave-load is 8 whole lines.
template <class C, int SH = 1, bool APAIR = false>
__device__ __forceinline__ void v3_offsets(int* voff, int row0, int col0, int R, int Cc, int64_t lda,
                                           int64_t ldb, int wave, int lane) {
#pragma unroll
    for (int j = 0; j < C::LPH; ++j) {
        const int q = wave + 4 * j;
        const bool isA = j < 4;
        const int rr = q * 16 + (lane >> 2) - (isA ? 0 : V3_BM);
        const int lc = (lane & 3) ^ ((rr >> SH) & 3);
        int gr = (isA ? row0 : col0) + rr;
        const int lim = isA ? R : Cc;
        gr = gr < lim ? gr : lim - 1;
        if (APAIR && isA)
            voff[j] = (int)(((unsigned)(gr >> 1) * (unsigned)lda + (unsigned)((gr & 1) * 32 + lc * 8)) * 2u);
        else
            voff[j] = (int)(((unsigned)gr * (unsigned)(isA ? lda : ldb) + (unsigned)(lc * 8)) * 2u);
    }
}

// Two depth halves of one output tile combined without a second kernel:
// the half whose workgroup arrives first (one compare-and-swap on the
// tile's state word) stores its fp32 sums; the second waits for them and adds
// them to its own while it writes the tile.  fp32 addition of two terms is
// commutative, so the result does not depend on which half comes first.  The
// state word is (48-bit call tag << 16 | state), state 1 = first arrived,
// 2 = its sums are ready, 3 = consumed; any other content (another call,
// uninitialised memory, the previous replay of a captured launch) makes the
// next arrival the first.  Sums move through agent-scope (L2-coherent)
// 64-bit atomic stores and loads; the waits are bounded.  The sums of a
// wave sit at [wave][row block][column block][pair e][lane] of the tile's
// area `part`, 8 bytes (values 2e and 2e + 1 of the lane's four) each, so
// that every 64-lane store or load covers 512 contiguous bytes (whole cache
// lines: these writes go through to memory, where partial lines cost a
// read-modify-write).  Returns the lane's pair-0 word; pair 1 is 64 words on.
__device__ inline unsigned long long* v3_part_at(float* part, int wave, int nbj, int i, int j, int lane) {
    return reinterpret_cast<unsigned long long*>(part) +
           (((size_t)wave * V3_NB + i) * nbj + j) * 128 + lane;
}

// Roles in the pair combine: the first to arrive stores its sums; the second
// adds them while writing the output, or writes NaN when its wait for them
// gave up.
enum { V3_FIRST = 0, V3_SECOND = 1, V3_SECOND_TIMED_OUT = 2 };

template <class C>
__device__ int v3_pair(const f32x4_t (&acc)[V3_NB][C::NBJ], unsigned long long* state, float* part,
                       unsigned long long epoch, int* role, int wave, int lane, const WaitCfg& wc) {
    const unsigned long long tag = (epoch & 0xFFFFFFFFFFFFull) << 16;
    if (threadIdx.x == 0) {
        unsigned long long old = __hip_atomic_load(state, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        int r = V3_SECOND_TIMED_OUT;
        for (unsigned it = 0; it < wc.spins; ++it) {
            const unsigned long long st = old & 0xFFFFull;
            if ((old & ~0xFFFFull) == tag && (st == 1 || st == 2)) {
                r = V3_SECOND;
                break;
            }
            if (__hip_atomic_compare_exchange_strong(state, &old, tag | 1ull, __ATOMIC_RELAXED,
                                                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
                r = V3_FIRST;
                break;
            }
        }
        *role = r;
    }
    __syncthreads();
    if (*role == V3_FIRST) {
#pragma unroll
        for (int i = 0; i < V3_NB; ++i)
#pragma unroll
            for (int j = 0; j < C::NBJ; ++j) {
                const f32x4_t v = v3_acc_read(acc[i][j]);
                unsigned long long* p = v3_part_at(part, wave, C::NBJ, i, j, lane);
                __hip_atomic_store(p, (unsigned long long)__float_as_uint(v[0]) |
                                          ((unsigned long long)__float_as_uint(v[1]) << 32),
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                __hip_atomic_store(p + 64, (unsigned long long)__float_as_uint(v[2]) |
                                              ((unsigned long long)__float_as_uint(v[3]) << 32),
                                   __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
        __builtin_amdgcn_s_waitcnt(0);           // this wave's stores are complete
        __syncthreads();
        if (threadIdx.x == 0) __hip_atomic_store(state, tag | 2ull, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        return V3_FIRST;
    }
    if (threadIdx.x == 0 && *role == V3_SECOND) {
        int r = V3_SECOND_TIMED_OUT;
        for (unsigned it = 0; it < wc.spins; ++it) {
            if (__hip_atomic_load(state, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (tag | 2ull)) {
                r = V3_SECOND;
                break;
            }
            __builtin_amdgcn_s_sleep(2);
        }
        *role = r;
    }
    if (threadIdx.x == 0 && *role == V3_SECOND_TIMED_OUT) note_timeout(wc);
    __syncthreads();
    return *role;
}

// the first half's sums of block (i, j) of this lane
__device__ inline f32x4_t v3_part_load(float* part, int wave, int nbj, int i, int j, int lane) {
    const unsigned long long* p = v3_part_at(part, wave, nbj, i, j, lane);
    const unsigned long long lo = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const unsigned long long hi = __hip_atomic_load(p + 64, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return f32x4_t{__uint_as_float((unsigned)lo), __uint_as_float((unsigned)(lo >> 32)),
                   __uint_as_float((unsigned)hi), __uint_as_float((unsigned)(hi >> 32))};
}

}  // namespace

}  // namespace espace
