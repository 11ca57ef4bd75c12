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
#include "v3_core.hpp"

namespace espace {

namespace {

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
// meet in v3_pair; `tile_state` and `pair_part` as there.  APAIR: A is in
// the row-pair layout (pair_offset, lda its pair pitch); c_pairs: the bf16
// output is written in that layout (ldc its pair pitch).
template <int MODE, int BN, int APAIR = 0>
__global__ __launch_bounds__(256, 1)
void gemm_tn_bf16_v3_kernel(const uint16_t* __restrict__ A, int64_t lda,
                            const uint16_t* __restrict__ B, int64_t ldb,
                            void* __restrict__ Cout, int64_t ldc,
                            int R, int Cc, int D, int tiles_c, int ntiles, int ktiles_per_split,
                            int64_t split_stride, int map, unsigned long long* tile_state,
                            float* pair_part, unsigned long long epoch, WaitCfg wc, int c_pairs) {
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
    const unsigned ra = (unsigned)((uint64_t)(APAIR ? (R + 1) / 2 : R) * lda * 2u);
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
            v3_offsets<C, 1, APAIR != 0>(voff, row0, col0, R, Cc, lda, ldb, wave, lane);
            int later = v3_load_half<C, APAIR != 0>(smem, A, B, ra, rb, voff, wave, lane, kt0, 0, hs(0, 0), D);
            later = v3_load_half<C, APAIR != 0>(smem, A, B, ra, rb, voff, wave, lane, kt0, 1, hs(0, 1), D);
            if (nsteps > 1) {
                later = v3_load_half<C, APAIR != 0>(smem, A, B, ra, rb, voff, wave, lane, kt0 + 1, 0, hs(1, 0), D);
                later += v3_load_half<C, APAIR != 0>(smem, A, B, ra, rb, voff, wave, lane, kt0 + 1, 1, hs(1, 1), D);
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
        // the first sub-step loads step kt0 + 2 into the half-stage just read:
        // every wave's reads of it must be complete before any wave issues them
        __builtin_amdgcn_s_barrier();

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
                v3_offsets<C, 1, APAIR != 0>(voff, ntr * V3_BM, ntc * BN, R, Cc, lda, ldb, wave, lane);
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
            v3_substep<C, F, true, true, APAIR != 0>(acc, fa0, fb0, fa1, fb1, rel ? aA3 : aA1, rel ? aB3 : aB1, smem,
                                         A, B, ra, rb, voff, wave, lkt, 0, hs(rel, 0), k0 == 1);
            if (k0 == 2) v3_load_half<C, APAIR != 0>(smem, A, B, ra, rb, voff, wave, lane, lkt, 0, hs(rel, 0), D);
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
            v3_substep<C, false, true, true, APAIR != 0>(acc, fa1, fb1, fa0, fb0, rel ? aA0 : aA2, rel ? aB0 : aB2,
                                             smem, A, B, ra, rb, voff, wave, lkt, 1, hs(rel, 1), k1 == 1);
            if (k1 == 2) v3_load_half<C, APAIR != 0>(smem, A, B, ra, rb, voff, wave, lane, lkt, 1, hs(rel, 1), D);
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
            v3_substep<C, false, true, true, APAIR != 0>(acc, fa0, fb0, fa1, fb1, aA3, aB3, smem, A, B, ra, rb, voff,
                                             wave, kt + 2, 0, hs(1, 0));
            v3_wait_lgkm0();
            v3_wait_vm<2 * C::LPH>();
            __builtin_amdgcn_s_barrier();
            v3_substep<C, false, true, true, APAIR != 0>(acc, fa1, fb1, fa0, fb0, aA0, aB0, smem, A, B, ra, rb, voff,
                                             wave, kt + 2, 1, hs(1, 1));
            v3_wait_lgkm0();
            v3_wait_vm<2 * C::LPH>();
            __builtin_amdgcn_s_barrier();
            v3_substep<C, false, true, true, APAIR != 0>(acc, fa0, fb0, fa1, fb1, aA1, aB1, smem, A, B, ra, rb, voff,
                                             wave, kt + 3, 0, hs(0, 0));
            v3_wait_lgkm0();
            v3_wait_vm<2 * C::LPH>();
            __builtin_amdgcn_s_barrier();
            v3_substep<C, false, true, true, APAIR != 0>(acc, fa1, fb1, fa0, fb0, aA2, aB2, smem, A, B, ra, rb, voff,
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
        bool timed_out = false;
        if constexpr (MODE == V3_PAIR) {
            const int tile = tile_r * tiles_c + tile_c;
            tpart = pair_part + (size_t)tile * (V3_BM * BN);
            tstate = tile_state + tile;
            const int role = v3_pair<C>(acc, tstate, tpart, epoch, &pair_role, wave, lane, wc);
            if (role == V3_FIRST) return;
            timed_out = role == V3_SECOND_TIMED_OUT;
        }
        // the first half's sums of row blocks i .. i + C::PD - 1 are in
        // flight while row block i is written (pbuf[i % (C::PD + 1)]), so
        // that many device-scope round trips overlap
        f32x4_t pbuf[C::PD + 1][NBJ];
        auto part_row = [&](int i) {
            if constexpr (MODE == V3_PAIR) {
                if (timed_out) return;
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
            if constexpr (MODE == V3_PAIR) {
                if (timed_out) return f32x4_t{__builtin_nanf(""), __builtin_nanf(""), __builtin_nanf(""),
                                              __builtin_nanf("")};
                return a + pbuf[i % (C::PD + 1)][j];
            }
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
                const unsigned cbytes = (unsigned)((uint64_t)(c_pairs ? (R + 1) / 2 : R) * ldc * 2u);
                const auto crsrc = __builtin_amdgcn_make_buffer_rsrc((void*)Cb, (short)0, (int)cbytes, 0x00020000);
#pragma unroll
                for (int i = 0; i < V3_NB; ++i) {
                    if (i + C::PD < V3_NB) part_row(i + C::PD);
                    const int r = row0 + wrow0 + 16 * i + lr;
                    // row pairs: row r's 32-column blocks are 64 elements apart
                    const unsigned rowoff = c_pairs ? (unsigned)(r >> 1) * (unsigned)ldc + (unsigned)((r & 1) * 32)
                                                    : (unsigned)r * (unsigned)ldc;
#pragma unroll
                    for (int m = 0; m < NBJ / 2; ++m) {
                        const u32x4_t v = pair_row(i, m);
                        const int c = cl0 + 32 * m;
                        const unsigned cc = c_pairs ? (unsigned)((c >> 5) * 64 + (c & 31)) : (unsigned)c;
                        const unsigned off = (r < R && c < Cc) ? (rowoff + cc) * 2u : 0xFFFFFFF0u;
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
                            uint16_t* p = Cb + (c_pairs ? pair_offset(r, c, ldc) : (int64_t)r * ldc + c);
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
    const int map = 0;
    if (S == 1) {
        // one workgroup per CU, each taking every cus-th tile
        const int persistent = g.cus > 0 ? g.cus : 256;
        dim3 grid(ntiles < persistent ? ntiles : persistent, 1);
        if (g.a_pairs)
            hipLaunchKernelGGL((gemm_tn_bf16_v3_kernel<V3_BF16, BN, 1>), grid, block, 0, stream, g.A, g.lda, g.B,
                               g.ldb, g.C, g.ldc, g.R, g.Cc, g.D, tiles_c, ntiles, ktps, (int64_t)0, map,
                               nullptr, nullptr, 0ull, g.wait, g.c_pairs);
        else
            hipLaunchKernelGGL((gemm_tn_bf16_v3_kernel<V3_BF16, BN>), grid, block, 0, stream, g.A, g.lda, g.B,
                               g.ldb, g.C, g.ldc, g.R, g.Cc, g.D, tiles_c, ntiles, ktps, (int64_t)0, map,
                               nullptr, nullptr, 0ull, g.wait, g.c_pairs);
        return hipGetLastError();
    }
    dim3 grid(ntiles, S);
    if (pair) {
        // partial: tiles x 256 x BN fp32, then one state word per tile
        unsigned long long* state =
            reinterpret_cast<unsigned long long*>(g.partial + (size_t)ntiles * V3_BM * BN);
        hipLaunchKernelGGL((gemm_tn_bf16_v3_kernel<V3_PAIR, BN>), grid, block, 0, stream, g.A, g.lda, g.B,
                           g.ldb, g.C, g.ldc, g.R, g.Cc, g.D, tiles_c, ntiles, ktps, (int64_t)0, map,
                           state, g.partial, g.epoch, g.wait, g.c_pairs);
        return hipGetLastError();
    }
    const int64_t ldp = splitk_ld(g.Cc);
    const int64_t split_stride = (int64_t)g.R * ldp;
    hipLaunchKernelGGL((gemm_tn_bf16_v3_kernel<V3_F32, BN>), grid, block, 0, stream, g.A, g.lda, g.B,
                       g.ldb, (void*)g.partial, ldp, g.R, g.Cc, g.D, tiles_c, ntiles, ktps, split_stride,
                       map, nullptr, nullptr, 0ull, g.wait, 0);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_splitk_reduce(g.partial, S, split_stride, ldp, g.C, g.ldc, g.R, g.Cc, g.c_pairs ? 2 : 1, stream);
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
                       (int64_t)g.R * ldp, upper ? 8 : 0, nullptr, nullptr, 0ull, g.wait, 0);
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
    // row-pair A only on the single-range kernel; pair pitches are whole
    // 64-element blocks
    const int ktiles = (g.D + V3_BK - 1) / V3_BK;
    const int S = g.splits < 1 ? 1 : g.splits;
    const int nranges = (ktiles + (ktiles + S - 1) / S - 1) / ((ktiles + S - 1) / S);
    if ((g.a_pairs && (nranges != 1 || g.lda % 64)) || (g.c_pairs && g.ldc % 64))
        return hipErrorNotSupported;
    switch (g.tile) {
        case TILE_256x256:
        case TILE_256x256_W8:
        case TILE_256x256_W8T: return launch_v3<256>(g, stream);
        case TILE_256x192_W8: return launch_v3<192>(g, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace espace
