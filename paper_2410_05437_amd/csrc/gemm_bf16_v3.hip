// Four-wave 256 x 256 (and 256 x 192) bfloat16 "TN" GEMM for gfx950 with a
// hand-ordered main loop:
//
//     C[r][c] = sum_k A[r][k] * B[c][k]        (fp32 accumulation)
//
// A [R][D] and B [Cc][D] row-major with the reduced dimension contiguous.
//
// One wave per SIMD; wave (wr, wc) owns the 128 x 128 sub-tile at
// (128 wr, 128 wc) as 8 x 8 blocks of v_mfma_f32_16x16x32_bf16 (128 x 96 as
// 8 x 6 blocks for the 256 x 192 tile).  The MFMAs
// and the LDS fragment reads are inline assembly so that their order is
// exactly the one below (the compiler's scheduler otherwise groups a step's
// loads together and leaves the matrix pipe idle while they issue, and
// splits the accumulators between AGPRs and VGPRs with copies in the loop);
// the accumulators are pinned to the AGPRs.
//
// Depth step 64 as two sub-steps of 32, each with its own LDS half-stage of
// 32 KB (the 512 A|B rows of the tile, 64 bytes each; 16-byte chunk c of row
// r at slot c ^ ((r >> 1) & 3): measured on gfx950 with eight waves reading,
// ds_read_b128 of 16 rows x 4 chunks runs at 231 B/clk with this slot
// order and at 152 B/clk with c ^ ((r >> 2) & 3), against 256 B/clk for
// contiguous reads); four half-stages hold two steps.  Per sub-step h of step kt, each
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
template <class C>
__device__ __forceinline__ void v3_load(unsigned char* smem, const uint16_t* A, const uint16_t* B,
                                        unsigned a_bytes, unsigned b_bytes, const int* voff,
                                        int wave, int kt, int h, int u, int j) {
    const int q = wave + 4 * j;
    const auto rsrc = __builtin_amdgcn_make_buffer_rsrc((void*)(j < 4 ? A : B), (short)0,
                                                        (int)(j < 4 ? a_bytes : b_bytes), 0x00020000);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(
        rsrc, (__attribute__((address_space(3))) void*)(smem + u * C::HS + q * 1024), 16,
        voff[j], (kt * V3_BK + 32 * h) * 2, 0, 0);
}

// Half h of depth step kt into half-stage u for any step: full depth by
// buffer_load ... lds (8 per wave, returns 8), the depth tail through
// registers with the elements at or beyond D zeroed (returns 0: nothing of
// it stays in flight).
template <class C>
__device__ __forceinline__ int v3_load_half(unsigned char* smem, const uint16_t* A, const uint16_t* B,
                                            unsigned a_bytes, unsigned b_bytes, const int* voff,
                                            int wave, int lane, int kt, int h, int u, int D) {
    const int k0 = kt * V3_BK + 32 * h;
    if (k0 + 32 <= D) {
#pragma unroll
        for (int j = 0; j < C::LPH; ++j) v3_load<C>(smem, A, B, a_bytes, b_bytes, voff, wave, kt, h, u, j);
        return C::LPH;
    }
#pragma unroll
    for (int j = 0; j < C::LPH; ++j) {
        const int q = wave + 4 * j;
        const int rr = q * 16 + (lane >> 2) - (j < 4 ? 0 : V3_BM);
        const int lc = (lane & 3) ^ v3_swz(rr);
        const uint16_t* rowp = (j < 4 ? A : B) + ((unsigned)voff[j] >> 1) - lc * 8;
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
template <class C, bool FIRST, bool READS, bool LOADS>
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
                        v3_load<C>(smem, A, B, a_bytes, b_bytes, voff, wave, kt, h, u, y);
            }
        }
}

enum { V3_BF16 = 0, V3_F32 = 1, V3_PAIR = 2 };

// byte offsets of this lane's 16-byte chunk of each wave-load (depth offset
// excluded) for the tile at (row0, col0): row 16q + lane/4 of the A|B tile,
// logical chunk (lane % 4) ^ swz(row); rows past the matrix are clamped to
// its last row
template <class C>
__device__ __forceinline__ void v3_offsets(int* voff, int row0, int col0, int R, int Cc, int64_t lda,
                                           int64_t ldb, int wave, int lane) {
#pragma unroll
    for (int j = 0; j < C::LPH; ++j) {
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

// true on the workgroup that writes the output (the second to arrive),
// after the first one's sums are ready; the first stores its sums and
// returns false
template <class C>
__device__ bool v3_pair(const f32x4_t (&acc)[V3_NB][C::NBJ], unsigned long long* state, float* part,
                        unsigned long long epoch, int* role, int wave, int lane) {
    const unsigned long long tag = (epoch & 0xFFFFFFFFFFFFull) << 16;
    if (threadIdx.x == 0) {
        unsigned long long old = __hip_atomic_load(state, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        int second = 0;
        for (int it = 0; it < (1 << 20); ++it) {
            const unsigned long long st = old & 0xFFFFull;
            if ((old & ~0xFFFFull) == tag && (st == 1 || st == 2)) {
                second = 1;
                break;
            }
            if (__hip_atomic_compare_exchange_strong(state, &old, tag | 1ull, __ATOMIC_RELAXED,
                                                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
                break;
        }
        *role = second;
    }
    __syncthreads();
    if (*role == 0) {
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
        return false;
    }
    if (threadIdx.x == 0) {
        for (int it = 0; it < (1 << 24); ++it) {
            if (__hip_atomic_load(state, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT) == (tag | 2ull)) break;
            __builtin_amdgcn_s_sleep(2);
        }
    }
    __syncthreads();
    return true;
}

// the first half's sums of block (i, j) of this lane
__device__ inline f32x4_t v3_part_load(float* part, int wave, int nbj, int i, int j, int lane) {
    const unsigned long long* p = v3_part_at(part, wave, nbj, i, j, lane);
    const unsigned long long lo = __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    const unsigned long long hi = __hip_atomic_load(p + 64, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    return f32x4_t{__uint_as_float((unsigned)lo), __uint_as_float((unsigned)(lo >> 32)),
                   __uint_as_float((unsigned)hi), __uint_as_float((unsigned)(hi >> 32))};
}

// Matrices handed to this kernel hold fewer than 2^31 elements (the launcher
// checks), so byte offsets fit in 32 bits.  Every depth range is non-empty.
//
// Work items are the output tiles (and depth ranges, blockIdx.y); a
// workgroup takes items blockIdx.x, blockIdx.x + gridDim.x, ...  When the
// next item of a workgroup starts with two full-depth steps and this item's
// output is bf16 with a column count that is a multiple of 8, the last two
// steps of an item load the next item's first two steps, so they land while
// this item's results are written.  The results then take exactly NST stores
// per wave (out-of-range lanes use an offset past the buffer, which the
// hardware drops), so the next item waits for its first step with
// vmcnt(2 LPH + NST).  MODE_PAIR: two depth ranges (blockIdx.y) of a tile
// meet in v3_pair; `tile_state` and `pair_part` as there.
template <int MODE, int BN>
__global__ __launch_bounds__(256, 1)
void gemm_tn_bf16_v3_kernel(const uint16_t* __restrict__ A, int64_t lda,
                            const uint16_t* __restrict__ B, int64_t ldb,
                            void* __restrict__ Cout, int64_t ldc,
                            int R, int Cc, int D, int tiles_c, int ntiles, int ktiles_per_split,
                            int64_t split_stride, int map, unsigned long long* tile_state,
                            float* pair_part, unsigned long long epoch) {
    using C = V3Cfg<BN>;
    constexpr int NBJ = C::NBJ;
    __shared__ __attribute__((aligned(1024))) unsigned char smem[C::SMEM];
    __shared__ int pair_role;

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
    const int wcol0 = (wave & 1) * (BN / 2);
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

    f32x4_t acc[V3_NB][NBJ];
    bf16x8_t fa0[V3_NB], fb0[NBJ], fa1[V3_NB], fb1[NBJ];
    int voff[C::LPH];

    int item = blockIdx.x;
    int tile_r, tile_c;
    tile_coords<4>(item, ntiles, tiles_c, map, tile_r, tile_c);
    bool ahead = false;     // this item's first two steps were loaded by the previous one
    int s0 = 0;             // stage of this item's first step (half-stages 2 s0, 2 s0 + 1)
    while (true) {
        const int row0 = tile_r * V3_BM;
        const int col0 = tile_c * BN;
        const int next = item + (int)gridDim.x;
        const bool ahead_next = ahead_ok && next < ntiles;
        int ntr = 0, ntc = 0;
        if (next < ntiles) tile_coords<4>(next, ntiles, tiles_c, map, ntr, ntc);

        // half-stage of (stage relative to s0, half)
        auto hs = [&](int rel, int h) { return ((rel ^ s0) << 1) | h; };
        // fragment addresses of half-stage u
        const unsigned aA0 = arow + (unsigned)(hs(0, 0) * C::HS), aB0 = brow + (unsigned)(hs(0, 0) * C::HS);
        const unsigned aA1 = arow + (unsigned)(hs(0, 1) * C::HS), aB1 = brow + (unsigned)(hs(0, 1) * C::HS);
        const unsigned aA2 = arow + (unsigned)(hs(1, 0) * C::HS), aB2 = brow + (unsigned)(hs(1, 0) * C::HS);
        const unsigned aA3 = arow + (unsigned)(hs(1, 1) * C::HS), aB3 = brow + (unsigned)(hs(1, 1) * C::HS);

        if (ahead) {
            // this wave's loads of the first step, then the loads of the second
            // and the previous item's stores were issued
            v3_wait_vm<2 * C::LPH + C::NST>();
        } else {
            // the half-stages may still be read by a wave finishing the previous item
            if (item != (int)blockIdx.x) __syncthreads();
            v3_offsets<C>(voff, row0, col0, R, Cc, lda, ldb, wave, lane);
            int later = v3_load_half<C>(smem, A, B, ra, rb, voff, wave, lane, kt0, 0, hs(0, 0), D);
            later = v3_load_half<C>(smem, A, B, ra, rb, voff, wave, lane, kt0, 1, hs(0, 1), D);
            if (nsteps > 1) {
                later = v3_load_half<C>(smem, A, B, ra, rb, voff, wave, lane, kt0 + 1, 0, hs(1, 0), D);
                later += v3_load_half<C>(smem, A, B, ra, rb, voff, wave, lane, kt0 + 1, 1, hs(1, 1), D);
            } else {
                later = 0;
            }
            // the first step's loads are the older ones; register-path loads
            // completed where they were issued
            v3_wait_vm_n<C>(later);
            v3_wait_lgkm0();
        }
        __builtin_amdgcn_s_barrier();
#pragma unroll
        for (int x = 0; x < C::NRD; ++x) v3_read_dyn<NBJ>(x, fa0, fb0, aA0, aB0);
        v3_wait_lgkm0();

        int kt = kt0;
        int rel = 0;          // stage of step kt relative to s0
        // the loads of sub-step h of step kt: half h of step kt + 2 of this
        // item, or of the next item's first steps once this item has none
        // left (step lkt of that item).  1: full depth, issued between the
        // sub-step's MFMAs like those of the steady state; 2: the depth tail,
        // through registers after the MFMAs; 0: none.
        auto load_kind = [&](int h, int& lkt) -> int {
            if (kt + 2 < kt_end) {
                lkt = kt + 2;
                return lkt * V3_BK + 32 * h + 32 <= D ? 1 : 2;
            }
            lkt = kt0 + (kt + 2 - kt_end);
            if (!ahead_next) return 0;
            if (kt + 2 == kt_end && h == 0)
                v3_offsets<C>(voff, ntr * V3_BM, ntc * BN, R, Cc, lda, ldb, wave, lane);
            return 1;
        };
        // one step with the stage chosen at run time (the first one and the
        // last ones); FIRST: the accumulators start at zero
        auto generic_step = [&](auto first) {
            constexpr bool F = decltype(first)::value;
            // after an item loaded ahead, its first step has the previous
            // item's stores in flight behind the loads of its second step
            const int stores = (F && ahead) ? C::NST : 0;
            // sub-step 0: fragments of sub-step 1 from the second half-stage
            int lkt;
            const int k0 = load_kind(0, lkt);
            v3_substep<C, F, true, true>(acc, fa0, fb0, fa1, fb1, rel ? aA3 : aA1, rel ? aB3 : aB1, smem,
                                         A, B, ra, rb, voff, wave, lkt, 0, hs(rel, 0), k0 == 1);
            if (k0 == 2) v3_load_half<C>(smem, A, B, ra, rb, voff, wave, lane, lkt, 0, hs(rel, 0), D);
            const int n0 = k0 == 1 ? C::LPH : 0;
            v3_wait_lgkm0();
            if (kt + 1 < kt_end || ahead_next) {
                // the next step's first half has landed (the loads just issued may stay in flight)
                if (kt + 1 < kt_end) v3_wait_vm_n<C>(C::LPH + stores + n0);
                __builtin_amdgcn_s_barrier();
            }
            // sub-step 1: fragments of the next step's sub-step 0 (after the
            // last step the reads are of no use but harmless: one code path
            // keeps the accumulators in place)
            const int k1 = load_kind(1, lkt);
            v3_substep<C, false, true, true>(acc, fa1, fb1, fa0, fb0, rel ? aA0 : aA2, rel ? aB0 : aB2,
                                             smem, A, B, ra, rb, voff, wave, lkt, 1, hs(rel, 1), k1 == 1);
            if (k1 == 2) v3_load_half<C>(smem, A, B, ra, rb, voff, wave, lane, lkt, 1, hs(rel, 1), D);
            const int n1 = k1 == 1 ? C::LPH : 0;
            v3_wait_lgkm0();
            if (kt + 1 < kt_end) {
                // the next step's second half has landed
                v3_wait_vm_n<C>(stores + n0 + n1);
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
            v3_substep<C, false, true, true>(acc, fa0, fb0, fa1, fb1, aA3, aB3, smem, A, B, ra, rb, voff,
                                             wave, kt + 2, 0, hs(1, 0));
            v3_wait_lgkm0();
            v3_wait_vm<2 * C::LPH>();
            __builtin_amdgcn_s_barrier();
            v3_substep<C, false, true, true>(acc, fa1, fb1, fa0, fb0, aA0, aB0, smem, A, B, ra, rb, voff,
                                             wave, kt + 2, 1, hs(1, 1));
            v3_wait_lgkm0();
            v3_wait_vm<2 * C::LPH>();
            __builtin_amdgcn_s_barrier();
            v3_substep<C, false, true, true>(acc, fa0, fb0, fa1, fb1, aA1, aB1, smem, A, B, ra, rb, voff,
                                             wave, kt + 3, 0, hs(0, 0));
            v3_wait_lgkm0();
            v3_wait_vm<2 * C::LPH>();
            __builtin_amdgcn_s_barrier();
            v3_substep<C, false, true, true>(acc, fa1, fb1, fa0, fb0, aA2, aB2, smem, A, B, ra, rb, voff,
                                             wave, kt + 3, 1, hs(0, 1));
            v3_wait_lgkm0();
            v3_wait_vm<2 * C::LPH>();
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
        float* tpart = nullptr;
        unsigned long long* tstate = nullptr;
        if constexpr (MODE == V3_PAIR) {
            const int tile = tile_r * tiles_c + tile_c;
            tpart = pair_part + (size_t)tile * (V3_BM * BN);
            tstate = tile_state + tile;
            if (!v3_pair<C>(acc, tstate, tpart, epoch, &pair_role, wave, lane)) return;
        }
        // the first half's sums of row blocks i .. i + C::PD - 1 are in
        // flight while row block i is written (pbuf[i % (C::PD + 1)]), so
        // that many device-scope round trips overlap
        f32x4_t pbuf[C::PD + 1][NBJ];
        auto part_row = [&](int i) {
            if constexpr (MODE == V3_PAIR) {
#pragma unroll
                for (int j = 0; j < NBJ; ++j)
                    pbuf[i % (C::PD + 1)][j] = v3_part_load(tpart, wave, NBJ, i, j, lane);
            }
        };
#pragma unroll
        for (int i = 0; i < C::PD; ++i) part_row(i);
        // the value of block (i, j) to write
        auto value = [&](int i, int j) -> f32x4_t {
            const f32x4_t a = v3_acc_read(acc[i][j]);
            if constexpr (MODE == V3_PAIR) return a + pbuf[i % (C::PD + 1)][j];
            return a;
        };
        if constexpr (MODE == V3_F32) {
            float* Cf = reinterpret_cast<float*>(Cout) + blockIdx.y * split_stride;
#pragma unroll
            for (int i = 0; i < V3_NB; ++i) {
                const int r = row0 + wrow0 + 16 * i + lr;
#pragma unroll
                for (int j = 0; j < NBJ; ++j) {
                    const f32x4_t v = value(i, j);
                    const int c = col0 + wcol0 + 16 * j + 4 * lh;
                    if (r >= R) continue;
                    float* p = Cf + (int64_t)r * ldc + c;
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
            uint16_t* Cb = reinterpret_cast<uint16_t*>(Cout);
            const int cl0 = col0 + wcol0 + 16 * (lh & 1) + 8 * (lh >> 1);   // + 32 m
            auto pair_row = [&](int i, int m) -> u32x4_t {
                const f32x4_t a = value(i, 2 * m);
                const f32x4_t b = value(i, 2 * m + 1);
                const auto s0 = __builtin_amdgcn_permlane16_swap(pack_bf16x2(a[0], a[1]),
                                                                 pack_bf16x2(b[0], b[1]), false, false);
                const auto s1 = __builtin_amdgcn_permlane16_swap(pack_bf16x2(a[2], a[3]),
                                                                 pack_bf16x2(b[2], b[3]), false, false);
                return u32x4_t{s0[0], s1[0], s0[1], s1[1]};
            };
            if ((Cc & 7) == 0) {
                // exactly one store instruction per lane group and block
                // pair, no branches; lanes outside the matrix get an offset
                // past the buffer, which its range check drops
                const unsigned cbytes = (unsigned)((uint64_t)R * ldc * 2u);
                const auto crsrc = __builtin_amdgcn_make_buffer_rsrc((void*)Cb, (short)0, (int)cbytes, 0x00020000);
#pragma unroll
                for (int i = 0; i < V3_NB; ++i) {
                    if (i + C::PD < V3_NB) part_row(i + C::PD);
                    const int r = row0 + wrow0 + 16 * i + lr;
                    const unsigned rowoff = (unsigned)r * (unsigned)ldc;
#pragma unroll
                    for (int m = 0; m < NBJ / 2; ++m) {
                        const u32x4_t v = pair_row(i, m);
                        const int c = cl0 + 32 * m;
                        const unsigned off = (r < R && c < Cc) ? (rowoff + (unsigned)c) * 2u : 0xFFFFFFF0u;
                        __builtin_amdgcn_raw_buffer_store_b128(v, crsrc, (int)off, 0, 0);
                    }
                }
            } else {
#pragma unroll
                for (int i = 0; i < V3_NB; ++i) {
                    if (i + C::PD < V3_NB) part_row(i + C::PD);
                    const int r = row0 + wrow0 + 16 * i + lr;
#pragma unroll
                    for (int m = 0; m < NBJ / 2; ++m) {
                        const u32x4_t v = pair_row(i, m);
                        const int c = cl0 + 32 * m;
                        if (r < R) {
                            uint16_t* p = Cb + (int64_t)r * ldc + c;
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
        }
        if constexpr (MODE == V3_PAIR) {
            // every wave has loaded the first half's sums
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            if (threadIdx.x == 0) __hip_atomic_store(tstate, ((epoch & 0xFFFFFFFFFFFFull) << 16) | 3ull,
                                                     __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        }
        if (next >= ntiles) break;
        item = next;
        tile_r = ntr;
        tile_c = ntc;
        s0 = (s0 + nsteps) & 1;
        ahead = ahead_next;
    }
}

// Tiled 256 x BN product with the hand-ordered four-wave kernel.  Depth
// ranges: two combined inside the kernel (pair), or fp32 partial sums
// reduced by launch_splitk_reduce.
template <int BN>
hipError_t launch_v3(const GemmArgs& g, hipStream_t stream) {
    const int tiles_r = (g.R + V3_BM - 1) / V3_BM;
    const int tiles_c = (g.Cc + BN - 1) / BN;
    const int ntiles = tiles_r * tiles_c;
    const int ktiles = (g.D + V3_BK - 1) / V3_BK;
    int S = g.splits < 1 ? 1 : g.splits;
    const int ktps = (ktiles + S - 1) / S;
    const bool pair = g.pair && S == 2 && (ktiles + ktps - 1) / ktps == 2;
    S = (ktiles + ktps - 1) / ktps;                 // no empty depth range
    dim3 block(V3_NW * 64);
    const int map = g.variant >> 2;
    if (S == 1) {
        // one workgroup per CU, each taking every 256th tile (variant bit 4:
        // one tile per workgroup)
        const int persistent = (g.variant & 16) ? ntiles : 256;
        dim3 grid(ntiles < persistent ? ntiles : persistent, 1);
        hipLaunchKernelGGL((gemm_tn_bf16_v3_kernel<V3_BF16, BN>), grid, block, 0, stream, g.A, g.lda, g.B,
                           g.ldb, g.C, g.ldc, g.R, g.Cc, g.D, tiles_c, ntiles, ktps, (int64_t)0, map,
                           nullptr, nullptr, 0ull);
        return hipGetLastError();
    }
    dim3 grid(ntiles, S);
    if (pair) {
        // partial: tiles x 256 x BN fp32, then one state word per tile
        unsigned long long* state =
            reinterpret_cast<unsigned long long*>(g.partial + (size_t)ntiles * V3_BM * BN);
        hipLaunchKernelGGL((gemm_tn_bf16_v3_kernel<V3_PAIR, BN>), grid, block, 0, stream, g.A, g.lda, g.B,
                           g.ldb, g.C, g.ldc, g.R, g.Cc, g.D, tiles_c, ntiles, ktps, (int64_t)0, map,
                           state, g.partial, g.epoch);
        return hipGetLastError();
    }
    const int64_t ldp = splitk_ld(g.Cc);
    const int64_t split_stride = (int64_t)g.R * ldp;
    hipLaunchKernelGGL((gemm_tn_bf16_v3_kernel<V3_F32, BN>), grid, block, 0, stream, g.A, g.lda, g.B,
                       g.ldb, (void*)g.partial, ldp, g.R, g.Cc, g.D, tiles_c, ntiles, ktps, split_stride,
                       map, nullptr, nullptr, 0ull);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_splitk_reduce(g.partial, S, split_stride, ldp, g.C, g.ldc, g.R, g.Cc, 1, stream);
}

template <int BN>
hipError_t launch_v3_ranges(const GemmArgs& g, bool upper, int* ranges, hipStream_t stream) {
    const int tiles_r = (g.R + V3_BM - 1) / V3_BM;
    const int tiles_c = (g.Cc + BN - 1) / BN;
    const int ntiles = upper ? tiles_c * (tiles_c + 1) / 2 : tiles_r * tiles_c;
    const int ktiles = (g.D + V3_BK - 1) / V3_BK;
    const int S0 = g.splits < 1 ? 1 : g.splits;
    const int ktps = (ktiles + S0 - 1) / S0;
    const int S = (ktiles + ktps - 1) / ktps;
    *ranges = S;
    const int64_t ldp = splitk_ld(g.Cc);
    hipLaunchKernelGGL((gemm_tn_bf16_v3_kernel<V3_F32, BN>), dim3(ntiles, S), dim3(V3_NW * 64), 0, stream, g.A,
                       g.lda, g.B, g.ldb, (void*)g.partial, ldp, g.R, g.Cc, g.D, tiles_c, ntiles, ktps,
                       (int64_t)g.R * ldp, (g.variant >> 2) | (upper ? 8 : 0), nullptr, nullptr, 0ull);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_tn_bf16_v3_ranges(const GemmArgs& g, bool upper, int* ranges, hipStream_t stream) {
    const int64_t lim = (int64_t)1 << 31;
    if ((int64_t)g.R * g.lda >= lim || (int64_t)g.Cc * g.ldb >= lim || g.D < 1 || !g.partial)
        return hipErrorInvalidValue;
    if (upper && (g.R != g.Cc || (g.tile != TILE_256x256 && g.tile != TILE_256x256_W8 &&
                                  g.tile != TILE_256x256_W8T)))
        return hipErrorInvalidValue;
    switch (g.tile) {
        case TILE_256x256:
        case TILE_256x256_W8:
        case TILE_256x256_W8T: return launch_v3_ranges<256>(g, upper, ranges, stream);
        case TILE_256x192_W8: return launch_v3_ranges<192>(g, upper, ranges, stream);
        default: return hipErrorInvalidValue;
    }
}

// 256 x 256 and 256 x 192 plans with the hand-ordered four-wave kernel;
// hipErrorInvalidValue for products it does not take (the caller falls back).
hipError_t launch_gemm_tn_bf16_v3(const GemmArgs& g, hipStream_t stream) {
    const int64_t lim = (int64_t)1 << 31;
    if ((int64_t)g.R * g.lda >= lim || (int64_t)g.Cc * g.ldb >= lim || (int64_t)g.R * g.ldc >= lim ||
        g.c_f32)
        return hipErrorInvalidValue;
    switch (g.tile) {
        case TILE_256x256:
        case TILE_256x256_W8:
        case TILE_256x256_W8T: return launch_v3<256>(g, stream);
        case TILE_256x192_W8: return launch_v3<192>(g, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace espace
