// Tiled bfloat16 "TN" GEMM for gfx950 with two alternating wave groups:
//
//     C[r][c] = sum_k A[r][k] * B[c][k]        (fp32 accumulation)
//
// A [R][D] and B [Cc][D] row-major with the reduced dimension contiguous.
//
// A 256 x 256 output tile per workgroup of 8 waves; wave w owns a 64 x 128
// sub-tile (rows 64*(w%4), columns 128*(w/4)) of 32x32 MFMA blocks.  Waves
// w and w+4 share a SIMD, and the two groups (waves 0-3, waves 4-7) take
// turns: while one group runs its MFMAs from registers (compute phase), the
// other reads the fragments of its next depth step from LDS (memory phase),
// and group 0 also issues the direct-to-LDS loads of a later step.  A
// barrier separates phases; group 1 starts one phase late, so each SIMD's
// matrix unit is fed by one wave while the other wave waits on memory, and
// a barrier costs only its own latency instead of draining the pipeline.
//
// LDS holds STAGES depth steps of 32 (64-byte rows, 32 KB per stage).  The
// loads of step t+STAGES-1 are issued in group 0's memory phase of step t
// and must land 2*(STAGES-1) phases later.  Chunk c of row r sits at slot
// c ^ ((r >> 2) & 3), which spreads the 16 rows read by 16 consecutive lanes
// over all 64 banks.
//
// Phase schedule (2 phases per step):
//     phase 2t   : group 0 memory(t),  group 1 compute(t-1)
//     phase 2t+1 : group 0 compute(t), group 1 memory(t)
// Before the barrier that opens phase 2t, group 0 has waited for its loads
// of step t; both groups finish their fragment reads (lgkmcnt 0) before the
// barrier that closes their memory phase, so a stage is free for reloading
// once both groups have read it.
#include "common.hpp"
#include "kernels.hpp"

namespace espace {

namespace {

constexpr int PP_BM = 256;
constexpr int PP_BN = 256;
constexpr int PP_BK = 32;               // depth per step
constexpr int PP_ROWB = PP_BK * 2;      // 64-byte LDS rows
constexpr int PP_CPR = PP_BK / 8;       // 4 chunks per row
constexpr int PP_RPL = 1024 / PP_ROWB;  // 16 rows per 1 KB wave-load
constexpr int PP_WTM = 64;
constexpr int PP_WTN = 128;
constexpr int PP_TM = PP_WTM / 32;      // 2
constexpr int PP_TN = PP_WTN / 32;      // 4
constexpr int PP_NSUB = PP_BK / 16;     // 2 MFMA sub-steps per step
constexpr int PP_STAGE = (PP_BM + PP_BN) * PP_ROWB;     // 32 KB
constexpr int PP_NLOAD = (PP_BM + PP_BN) / PP_RPL;      // 32 wave-loads per stage
constexpr int PP_LPW = PP_NLOAD / 4;                    // per group-0 wave
constexpr int PP_EPI_LD = PP_WTN * 2 + 16;
constexpr int PP_EPI = 8 * PP_WTM * PP_EPI_LD;

template <int STAGES>
struct PPSmem {
    static constexpr int SIZE = (STAGES * PP_STAGE > PP_EPI) ? STAGES * PP_STAGE : PP_EPI;
};

__device__ __forceinline__ int pp_swz(int r) { return (r >> 2) & 3; }

template <int N>
__device__ __forceinline__ void pp_wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

__device__ __forceinline__ void pp_wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

// at most n steps of this wave's loads outstanding (0 <= n <= 3)
__device__ __forceinline__ void pp_wait_steps(int n) {
    if (n <= 0) pp_wait_vmcnt<0>();
    else if (n == 1) pp_wait_vmcnt<PP_LPW>();
    else if (n == 2) pp_wait_vmcnt<2 * PP_LPW>();
    else pp_wait_vmcnt<3 * PP_LPW>();
}

// workgroup barrier that the compiler may not move memory operations across
__device__ __forceinline__ void pp_sync() {
    asm volatile("" ::: "memory");
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    asm volatile("" ::: "memory");
}

// Loads of step kt into stage st by group-0 wave gw (0..3).
__device__ __forceinline__ void pp_issue(unsigned char* smem, const uint16_t* __restrict__ A,
                                         const uint16_t* __restrict__ B, const int* off, int gw,
                                         int lane, int kt, int st, int D) {
    const int k0 = kt * PP_BK;
    unsigned char* sbase = smem + st * PP_STAGE;
    if (k0 + PP_BK <= D) {
#pragma unroll
        for (int j = 0; j < PP_LPW; ++j) {
            const int q = gw + j * 4;
            const uint16_t* base = (q * PP_RPL < PP_BM) ? A : B;
            __builtin_amdgcn_global_load_lds(base + off[j] + k0, sbase + q * 1024, 16, 0, 0);
        }
    } else {
#pragma unroll
        for (int j = 0; j < PP_LPW; ++j) {
            const int q = gw + j * 4;
            const bool isA = q * PP_RPL < PP_BM;
            const uint16_t* base = isA ? A : B;
            const int rr = q * PP_RPL + lane / PP_CPR - (isA ? 0 : PP_BM);
            const int lc = (lane % PP_CPR) ^ pp_swz(rr);
            const uint16_t* rowp = base + off[j] - lc * 8;
            const u32x4_t v = load_chunk_masked(rowp, k0 + lc * 8, D);
            *reinterpret_cast<u32x4_t*>(sbase + q * 1024 + lane * 16) = v;
        }
    }
}

template <int STAGES, bool OUT_F32>
__global__ __launch_bounds__(512, 2)
void gemm_tn_bf16_pp_kernel(const uint16_t* __restrict__ A, int64_t lda,
                            const uint16_t* __restrict__ B, int64_t ldb,
                            void* __restrict__ Cout, int64_t ldc,
                            int R, int Cc, int D, int tiles_c, int ktiles_per_split,
                            int64_t split_stride, int map) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[PPSmem<STAGES>::SIZE];

    int tile_r, tile_c;
    tile_coords<4>(blockIdx.x, gridDim.x, tiles_c, map, tile_r, tile_c);
    const int row0 = tile_r * PP_BM;
    const int col0 = tile_c * PP_BN;

    const int ktiles = (D + PP_BK - 1) / PP_BK;
    const int kt0 = blockIdx.y * ktiles_per_split;
    int kt_end = kt0 + ktiles_per_split;
    kt_end = kt_end < ktiles ? kt_end : ktiles;
    const int nsteps = kt_end > kt0 ? kt_end - kt0 : 0;

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int grp = wave >> 2;
    const int gw = wave & 3;
    const int wrow0 = gw * PP_WTM;
    const int wcol0 = grp * PP_WTN;

    // group-0 load descriptors
    int off[PP_LPW];
#pragma unroll
    for (int j = 0; j < PP_LPW; ++j) {
        const int q = gw + j * 4;
        const int rl = q * PP_RPL + lane / PP_CPR;
        const bool isA = q * PP_RPL < PP_BM;
        const int rr = isA ? rl : rl - PP_BM;
        const int lc = (lane % PP_CPR) ^ pp_swz(rr);
        int gr = (isA ? row0 : col0) + rr;
        const int lim = isA ? R : Cc;
        gr = gr < lim ? gr : lim - 1;
        off[j] = gr * (int)(isA ? lda : ldb) + lc * 8;
    }

    const int lr = lane & 31;
    const int lh = lane >> 5;
    const int sw = pp_swz(lr);
    const int a_off = (wrow0 + lr) * PP_ROWB;
    const int b_off = (PP_BM + wcol0 + lr) * PP_ROWB;

    f32x16_t acc[PP_TM][PP_TN];
#pragma unroll
    for (int i = 0; i < PP_TM; ++i)
#pragma unroll
        for (int j = 0; j < PP_TN; ++j)
#pragma unroll
            for (int v = 0; v < 16; ++v) acc[i][j][v] = 0.f;

    bf16x8_t fa[PP_NSUB][PP_TM];
    bf16x8_t fb[PP_NSUB][PP_TN];

    // prologue: group 0 loads steps 0 .. STAGES-2 and waits for step 0
    if (grp == 0) {
#pragma unroll
        for (int p = 0; p < STAGES - 1; ++p)
            if (p < nsteps) pp_issue(smem, A, B, off, gw, lane, kt0 + p, p, D);
        const int newer = (nsteps - 1) < (STAGES - 2) ? (nsteps - 1) : (STAGES - 2);
        pp_wait_steps(newer);
    }
    pp_sync();
    if (grp == 1) pp_sync();

    int st = 0;
    for (int s = 0; s < nsteps; ++s) {
        // ---- memory phase of step s ----
        if (grp == 0 && s + STAGES - 1 < nsteps) {
            int ist = st - 1;
            if (ist < 0) ist += STAGES;
            pp_issue(smem, A, B, off, gw, lane, kt0 + s + STAGES - 1, ist, D);
        }
        {
            const unsigned char* sbase = smem + st * PP_STAGE;
#pragma unroll
            for (int u = 0; u < PP_NSUB; ++u) {
                const int pc = ((2 * u + lh) ^ sw) * 16;
#pragma unroll
                for (int i = 0; i < PP_TM; ++i)
                    fa[u][i] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(
                        sbase + a_off + i * 32 * PP_ROWB + pc));
#pragma unroll
                for (int j = 0; j < PP_TN; ++j)
                    fb[u][j] = as_bf16x8(*reinterpret_cast<const u32x4_t*>(
                        sbase + b_off + j * 32 * PP_ROWB + pc));
            }
        }
        pp_wait_lgkmcnt0();
        pp_sync();
        // ---- compute phase of step s ----
#pragma unroll
        for (int u = 0; u < PP_NSUB; ++u)
#pragma unroll
            for (int i = 0; i < PP_TM; ++i)
#pragma unroll
                for (int j = 0; j < PP_TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fb[u][j], fa[u][i],
                                                                         acc[i][j], 0, 0, 0);
        if (grp == 0 && s + 1 < nsteps) {
            // loads issued after step s+1 that may stay in flight
            const int last = (s + STAGES - 1 < nsteps - 1) ? s + STAGES - 1 : nsteps - 1;
            pp_wait_steps(last - (s + 1));
        }
        pp_sync();
        st = (st + 1 == STAGES) ? 0 : st + 1;
    }
    if (grp == 0) pp_sync();
    __syncthreads();

    // ---- epilogue ----------------------------------------------------------------
    if constexpr (OUT_F32) {
        float* C = reinterpret_cast<float*>(Cout) + blockIdx.y * split_stride;
#pragma unroll
        for (int i = 0; i < PP_TM; ++i) {
            const int r = row0 + wrow0 + 32 * i + lr;
            if (r >= R) continue;
#pragma unroll
            for (int j = 0; j < PP_TN; ++j) {
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int c = col0 + wcol0 + 32 * j + 8 * q + 4 * lh;
                    f32x4_t v = {acc[i][j][4 * q], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                                 acc[i][j][4 * q + 3]};
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
        }
    } else {
        unsigned char* ep = smem + wave * PP_WTM * PP_EPI_LD;
#pragma unroll
        for (int i = 0; i < PP_TM; ++i)
#pragma unroll
            for (int j = 0; j < PP_TN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    u32x2_t v;
                    v[0] = pack_bf16x2(acc[i][j][4 * q], acc[i][j][4 * q + 1]);
                    v[1] = pack_bf16x2(acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]);
                    const int rl = 32 * i + lr;
                    const int cl = 32 * j + 8 * q + 4 * lh;
                    *reinterpret_cast<u32x2_t*>(ep + rl * PP_EPI_LD + cl * 2) = v;
                }
        __syncthreads();
        uint16_t* C = reinterpret_cast<uint16_t*>(Cout);
        constexpr int CPRO = PP_WTN / 8;
        constexpr int RPI = 64 / CPRO;
#pragma unroll 4
        for (int it = 0; it < PP_WTM / RPI; ++it) {
            const int rl = it * RPI + lane / CPRO;
            const int cl = (lane % CPRO) * 8;
            const int r = row0 + wrow0 + rl;
            const int c = col0 + wcol0 + cl;
            const u32x4_t v = *reinterpret_cast<const u32x4_t*>(ep + rl * PP_EPI_LD + cl * 2);
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

template <int STAGES>
hipError_t launch_pp(const GemmArgs& g, hipStream_t stream) {
    const int tiles_r = (g.R + PP_BM - 1) / PP_BM;
    const int tiles_c = (g.Cc + PP_BN - 1) / PP_BN;
    const int ktiles = (g.D + PP_BK - 1) / PP_BK;
    const int S = g.splits;
    const int ktps = (ktiles + S - 1) / S;
    dim3 grid(tiles_r * tiles_c, S);
    dim3 block(512);
    if (S == 1) {
        hipLaunchKernelGGL((gemm_tn_bf16_pp_kernel<STAGES, false>), grid, block, 0, stream, g.A,
                           g.lda, g.B, g.ldb, g.C, g.ldc, g.R, g.Cc, g.D, tiles_c, ktps,
                           (int64_t)0, g.variant >> 2);
        return hipGetLastError();
    }
    const int64_t ldp = splitk_ld(g.Cc);
    const int64_t split_stride = (int64_t)g.R * ldp;
    hipLaunchKernelGGL((gemm_tn_bf16_pp_kernel<STAGES, true>), grid, block, 0, stream, g.A,
                       g.lda, g.B, g.ldb, (void*)g.partial, ldp, g.R, g.Cc, g.D, tiles_c, ktps,
                       split_stride, g.variant >> 2);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_splitk_reduce(g.partial, S, split_stride, ldp, g.C, g.ldc, g.R, g.Cc,
                                g.c_f32 ? 0 : 1, stream);
}

}  // namespace

hipError_t launch_gemm_tn_bf16_pp(const GemmArgs& g0, hipStream_t stream) {
    GemmArgs g = g0;
    if (g.pair) {            // no in-kernel pair combine here: one depth range
        g.splits = 1;
        g.pair = 0;
    }
    const int64_t lim = (int64_t)1 << 31;
    if ((int64_t)g.R * g.lda >= lim || (int64_t)g.Cc * g.ldb >= lim || g.c_f32)
        return launch_gemm_tn_bf16(g, stream);
    return (g.variant & 1) ? launch_pp<3>(g, stream) : launch_pp<4>(g, stream);
}

}  // namespace espace
