// Bandwidth-oriented bfloat16 product for few tokens (decode):
//
//     C[n][j] = sum_k A[n][k] * B[j][k],   n < R <= 32 (tokens), j < Cc
//
// The many-row operand B (P, the folded weight, or W) is streamed from HBM
// exactly once; the few-row operand A (the tokens) is small and stays in L2.
// A workgroup owns 16*RG consecutive rows of B and one range of the reduced
// dimension; its WAVES waves take interleaved 32-element steps of that range,
// so at any moment the workgroup reads WAVES*64 contiguous bytes of each row,
// and each wave keeps UNROLL steps of loads in flight.
// The arithmetic is done by v_mfma_f32_16x16x32_bf16 with the B rows as the
// 16-row operand and up to 16 tokens as the 16-column operand, which keeps
// the ALU cost negligible next to the memory stream.  Per-wave partial sums
// are reduced through LDS in a fixed order; several depth ranges (split > 1)
// write fp32 partials that a second kernel sums in a fixed order, so results
// do not depend on scheduling.
//
// Depth segments (SEG = 2 or 4, 16/SEG tokens per token group, one or two
// groups).  With few rows of B
// (the projection, L rows) 16-row groups leave most CUs idle, and a depth
// split costs a second launch.  Instead the 16 rows of the MFMA operand are
// 16/SEG rows of B times SEG depth segments: operand row r is row r/SEG of
// the group over segment r%SEG, and token column c is token c/SEG over
// segment c%SEG.  The diagonal blocks (row segment = column segment) of the
// 16x16 result hold the per-segment partial dot products; the SEG of them
// for one (row, token) sit in SEG neighbouring lanes and are summed with
// lane exchanges in a fixed order.  A workgroup then owns 16/SEG rows, so
// SEG times as many workgroups share the stream, in one launch.  With two
// token groups both MFMAs of a step share the weight operand.
#include "common.hpp"
#include "kernels.hpp"

namespace espace {

namespace {

constexpr int STEP = 32;   // reduced elements per MFMA

template <int RG, int TG, int WAVES, int UNROLL, int SEG>
__global__ __launch_bounds__(WAVES * 64)
void skinny_tn_bf16_kernel(const uint16_t* __restrict__ A, int64_t lda,
                           const uint16_t* __restrict__ B, int64_t ldb,
                           void* __restrict__ Cout, int64_t ldc,
                           int R, int Cc, int D, int steps_per_split,
                           int out_f32, int64_t split_stride) {
    static_assert(SEG == 1 || (TG <= 2 && (SEG == 2 || SEG == 4)), "segments: 2 or 4, one or two token groups");
    constexpr int GROWS = 16 / SEG;    // rows of B per 16-row operand
    __shared__ f32x4_t red[WAVES - 1][RG * TG][64];

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int j0 = blockIdx.x * (GROWS * RG);
    // steps per depth segment (the whole depth when SEG == 1)
    const int nsteps = ((D + STEP - 1) / STEP + SEG - 1) / SEG;
    const int s_begin = blockIdx.y * steps_per_split;
    int s_end = s_begin + steps_per_split;
    s_end = s_end < nsteps ? s_end : nsteps;

    const int lr = lane & 15;          // operand row / token column inside a 16-wide group
    const int lk = (lane >> 4) * 8;    // element offset of this lane's chunk
    const int seg = lr % SEG;          // depth segment of this lane's row and column
    const int koff = seg * nsteps * STEP + lk;
    // steps whose 32 elements lie below D in every segment
    const int dlast = D - (SEG - 1) * nsteps * STEP;
    const int s_fast_end = dlast <= 0 ? 0 : (s_end < dlast / STEP ? s_end : dlast / STEP);

    const uint16_t* brow[RG];
#pragma unroll
    for (int g = 0; g < RG; ++g) {
        int j = j0 + g * GROWS + lr / SEG;
        j = j < Cc ? j : Cc - 1;
        brow[g] = B + (int64_t)j * ldb;
    }
    // token rows beyond R read row 0 and are zeroed with a mask; a token
    // group holds 16 / SEG tokens
    const uint16_t* arow[TG];
    uint32_t amask[TG];
#pragma unroll
    for (int t = 0; t < TG; ++t) {
        const int n = t * (16 / SEG) + lr / SEG;
        amask[t] = n < R ? 0xffffffffu : 0u;
        arow[t] = A + (int64_t)(n < R ? n : 0) * lda;
    }

    f32x4_t acc[RG][TG];
#pragma unroll
    for (int g = 0; g < RG; ++g)
#pragma unroll
        for (int t = 0; t < TG; ++t) acc[g][t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // Main loop: UNROLL whole steps per wave, every load unconditional, so
    // that all of them are in flight together.
    int s0 = s_begin + wave;
    for (; s0 + (UNROLL - 1) * WAVES < s_fast_end; s0 += WAVES * UNROLL) {
        u32x4_t vb[UNROLL][RG];
        u32x4_t va[UNROLL][TG];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            const int k = (s0 + u * WAVES) * STEP + koff;
#pragma unroll
            for (int g = 0; g < RG; ++g) vb[u][g] = *reinterpret_cast<const u32x4_t*>(brow[g] + k);
#pragma unroll
            for (int t = 0; t < TG; ++t) va[u][t] = *reinterpret_cast<const u32x4_t*>(arow[t] + k) & amask[t];
        }
        __builtin_amdgcn_sched_barrier(0);   // all loads issue before the first MFMA
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
#pragma unroll
            for (int g = 0; g < RG; ++g)
#pragma unroll
                for (int t = 0; t < TG; ++t)
                    acc[g][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        as_bf16x8(vb[u][g]), as_bf16x8(va[u][t]), acc[g][t], 0, 0, 0);
    }
    // Tail (at most one pass): steps past the range or the depth load from a
    // clamped address and are masked, without branches.
    for (; s0 < s_end; s0 += WAVES * UNROLL) {
        u32x4_t vb[UNROLL][RG];
        u32x4_t va[UNROLL][TG];
        int valid[UNROLL];
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
            const int s = s0 + u * WAVES;
            const int k = s * STEP + koff;
            valid[u] = s < s_end ? D - k : 0;
            const int kk = valid[u] > 0 ? k : 0;
#pragma unroll
            for (int g = 0; g < RG; ++g) vb[u][g] = *reinterpret_cast<const u32x4_t*>(brow[g] + kk);
#pragma unroll
            for (int t = 0; t < TG; ++t) va[u][t] = *reinterpret_cast<const u32x4_t*>(arow[t] + kk);
        }
        __builtin_amdgcn_sched_barrier(0);   // masks are applied once the loads are in flight
#pragma unroll
        for (int u = 0; u < UNROLL; ++u) {
#pragma unroll
            for (int g = 0; g < RG; ++g) vb[u][g] = mask_chunk(vb[u][g], valid[u]);
#pragma unroll
            for (int t = 0; t < TG; ++t) va[u][t] = mask_chunk(va[u][t], valid[u]) & amask[t];
        }
#pragma unroll
        for (int u = 0; u < UNROLL; ++u)
#pragma unroll
            for (int g = 0; g < RG; ++g)
#pragma unroll
                for (int t = 0; t < TG; ++t)
                    acc[g][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(
                        as_bf16x8(vb[u][g]), as_bf16x8(va[u][t]), acc[g][t], 0, 0, 0);
    }

    // reduce the waves' partial sums through LDS, in wave order
    if (wave > 0) {
#pragma unroll
        for (int g = 0; g < RG; ++g)
#pragma unroll
            for (int t = 0; t < TG; ++t) red[wave - 1][g * TG + t][lane] = acc[g][t];
    }
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int w = 0; w < WAVES - 1; ++w)
#pragma unroll
        for (int g = 0; g < RG; ++g)
#pragma unroll
            for (int t = 0; t < TG; ++t) acc[g][t] += red[w][g * TG + t][lane];

    if (SEG > 1) {
        // Lane l holds operand rows 4*(l/16) + i (i < 4), that is rows
        // 4*(l/16)/SEG + i/SEG of the group over segments i%SEG, and token
        // column l%16.  Its diagonal entries are i = seg + SEG*c, for the
        // 4/SEG consecutive rows c; the SEG lanes of one token add theirs.
        constexpr int OUTS = 4 / SEG;
#pragma unroll
        for (int gt = 0; gt < RG * TG; ++gt) {
            const int g = gt / TG, t = gt % TG;
            const int n = t * (16 / SEG) + lr / SEG;
            float d[OUTS];
#pragma unroll
            for (int c = 0; c < OUTS; ++c) {
                float v = acc[g][t][SEG * c];
#pragma unroll
                for (int h = 1; h < SEG; ++h) v = seg == h ? acc[g][t][SEG * c + h] : v;
                d[c] = v;
            }
#pragma unroll
            for (int m = 1; m < SEG; m <<= 1)
#pragma unroll
                for (int c = 0; c < OUTS; ++c) d[c] += __shfl_xor(d[c], m);
            if (seg != 0 || n >= R) continue;
            const int jb = j0 + g * GROWS + (lane >> 4) * OUTS;
            if (out_f32) {
                float* C = reinterpret_cast<float*>(Cout) + (int64_t)n * ldc;
#pragma unroll
                for (int c = 0; c < OUTS; ++c)
                    if (jb + c < Cc) C[jb + c] = d[c];
            } else {
                uint16_t* C = reinterpret_cast<uint16_t*>(Cout) + (int64_t)n * ldc;
                if (OUTS == 2 && jb + 1 < Cc) {
                    *reinterpret_cast<uint32_t*>(C + jb) = pack_bf16x2(d[0], d[OUTS - 1]);
                } else {
#pragma unroll
                    for (int c = 0; c < OUTS; ++c)
                        if (jb + c < Cc) C[jb + c] = (uint16_t)bf16_rne(d[c]);
                }
            }
        }
        return;
    }

    // accumulator i of lane l holds B row 4*(l/16) + i and token l%16 of its
    // 16x16 tile: four consecutive output columns of one token row
#pragma unroll
    for (int g = 0; g < RG; ++g) {
        const int jb = j0 + g * 16 + 4 * (lane >> 4);
#pragma unroll
        for (int t = 0; t < TG; ++t) {
            const int n = t * 16 + lr;
            if (n >= R) continue;
            if (out_f32) {
                float* C = reinterpret_cast<float*>(Cout) + blockIdx.y * split_stride + (int64_t)n * ldc;
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (jb + i < Cc) C[jb + i] = acc[g][t][i];
            } else {
                uint16_t* C = reinterpret_cast<uint16_t*>(Cout) + (int64_t)n * ldc;
                if (jb + 3 < Cc) {
                    u32x2_t v;
                    v[0] = pack_bf16x2(acc[g][t][0], acc[g][t][1]);
                    v[1] = pack_bf16x2(acc[g][t][2], acc[g][t][3]);
                    *reinterpret_cast<u32x2_t*>(C + jb) = v;
                } else {
#pragma unroll
                    for (int i = 0; i < 4; ++i)
                        if (jb + i < Cc) C[jb + i] = (uint16_t)bf16_rne(acc[g][t][i]);
                }
            }
        }
    }
}

template <int RG, int TG, int WAVES, int UNROLL, int SEG = 1>
hipError_t launch_skinny_cfg(const GemmArgs& g, hipStream_t stream) {
    const int nsteps = ((g.D + STEP - 1) / STEP + SEG - 1) / SEG;
    const int S = g.splits;
    if (SEG > 1 && (S != 1 || g.R > TG * (16 / SEG))) return hipErrorInvalidValue;
    const int sps = (nsteps + S - 1) / S;
    const int rows = 16 / SEG * RG;
    dim3 grid((g.Cc + rows - 1) / rows, S);
    dim3 block(WAVES * 64);
    if (S == 1) {
        hipLaunchKernelGGL((skinny_tn_bf16_kernel<RG, TG, WAVES, UNROLL, SEG>), grid, block, 0, stream,
                           g.A, g.lda, g.B, g.ldb, g.C, g.ldc, g.R, g.Cc, g.D, sps, g.c_f32,
                           (int64_t)0);
        return hipGetLastError();
    }
    const int64_t ldp = splitk_ld(g.Cc);
    const int64_t split_stride = (int64_t)g.R * ldp;
    hipLaunchKernelGGL((skinny_tn_bf16_kernel<RG, TG, WAVES, UNROLL, SEG>), grid, block, 0, stream,
                       g.A, g.lda, g.B, g.ldb, (void*)g.partial, ldp, g.R, g.Cc, g.D, sps, 1,
                       split_stride);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    return launch_splitk_reduce(g.partial, S, split_stride, ldp, g.C, g.ldc, g.R, g.Cc,
                                g.c_f32 ? 0 : 1, stream);
}

template <int RG, int WAVES, int UNROLL>
hipError_t launch_skinny_tg(const GemmArgs& g, hipStream_t stream) {
    if (g.R <= 16) return launch_skinny_cfg<RG, 1, WAVES, UNROLL>(g, stream);
    return launch_skinny_cfg<RG, 2, WAVES, UNROLL>(g, stream);
}

}  // namespace

hipError_t launch_skinny_tn_bf16(const GemmArgs& g, hipStream_t stream) {
    if (g.R > 32) return hipErrorInvalidValue;
    switch (g.tile) {
        case SKINNY_RG1_W4: return launch_skinny_tg<1, 4, 4>(g, stream);
        case SKINNY_RG2_W4: return launch_skinny_tg<2, 4, 4>(g, stream);
        case SKINNY_RG1_W8: return launch_skinny_tg<1, 8, 4>(g, stream);
        case SKINNY_RG2_W8: return launch_skinny_tg<2, 8, 4>(g, stream);
        case SKINNY_RG1_W4_U8: return launch_skinny_tg<1, 4, 8>(g, stream);
        case SKINNY_RG2_W4_U8: return launch_skinny_tg<2, 4, 8>(g, stream);
        case SKINNY_RG1_W8_U8: return launch_skinny_tg<1, 8, 8>(g, stream);
        case SKINNY_RG2_W8_U8: return launch_skinny_tg<2, 8, 8>(g, stream);
        case SKINNY_RG1_W8_U6: return launch_skinny_tg<1, 8, 6>(g, stream);
        case SKINNY_RG2_W4_U6: return launch_skinny_tg<2, 4, 6>(g, stream);
        case SKINNY_RG1_W16_U8: return launch_skinny_tg<1, 16, 8>(g, stream);
        case SKINNY_RG1_W16_U4: return launch_skinny_tg<1, 16, 4>(g, stream);
        case SKINNY_SEG2_W8_U8: return launch_skinny_cfg<1, 1, 8, 8, 2>(g, stream);
        case SKINNY_SEG2_W16_U4: return launch_skinny_cfg<1, 1, 16, 4, 2>(g, stream);
        case SKINNY_SEG2_TG2_W8_U8: return launch_skinny_cfg<1, 2, 8, 8, 2>(g, stream);
        case SKINNY_SEG2_TG2_W16_U4: return launch_skinny_cfg<1, 2, 16, 4, 2>(g, stream);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace espace
