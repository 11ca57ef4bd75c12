// The whole projected linear layer for few tokens (decode) in one launch:
//
//     phase 1   Z[n][l] = sum_k X[n][k] * Pt[l][k]      (projection)
//     phase 2   Y[n][m] = sum_l Z[n][l] * Wf[m][l]      (folded weight)
//
// N <= 16*TG tokens.  Both phases stream a many-row operand (Pt, then Wf)
// from HBM once; the tokens (X, then Z) are small.  A unit of work is 16
// rows of the streamed operand over a range of the reduced dimension, done
// by one workgroup of 8 waves: the waves take interleaved 32-element steps
// (v_mfma_f32_16x16x32_bf16, streamed rows as the 16-row operand, tokens as
// the 16-column operand) and are summed through LDS in wave order.
//
// Scheduling without a grid barrier.  Each workgroup takes a ticket from an
// atomic counter in the workspace.  The first P1 tickets are projection
// units (16 rows of Pt over one of S1 depth ranges); the others are phase-2
// workgroups, which load the Wf rows of their first unit into registers and
// then wait until every projection unit has finished.  A workgroup only ever
// waits for lower tickets, which were taken by workgroups already running,
// so the launch makes progress whatever the number of resident workgroups.
// With S1 > 1, the last of the S1 units of a row group (found with a per-row-
// group counter) adds the S1 fp32 partial sums in a fixed order, so the
// result does not depend on scheduling.  Z is rounded to bfloat16, as in the
// two-launch path.
//
// Cross-workgroup data (Z, the partial sums, the counters) only moves through
// agent-scope atomic loads and stores, which are coherent across the L2
// caches of the XCDs; a writer waits for its stores to complete before it
// signals.  No cache-wide write-back or invalidation is needed, which matters
// here: hundreds of workgroups issuing them at once stall every L2.
//
// The counters need no initialisation: a per-call tag (epoch) claims the
// block; the first workgroup of a call that does not find its tag there
// resets the counters and publishes the tag.  A replay of a captured launch
// (same tag) continues from where the previous replay stopped: tickets,
// row-group and completion counts advance by fixed amounts per launch.  All
// waits are bounded, so every workgroup finishes even if the block is
// overwritten meanwhile.
#include "common.hpp"
#include "kernels.hpp"

namespace espace {

namespace {

constexpr int DF_WAVES = 8;
constexpr int DF_STEP = 32;
constexpr int DF_UNROLL = 8;
constexpr int DF_LDS_MAX = 152 * 1024;        // dynamic LDS limit per workgroup
constexpr unsigned DF_SPIN_LIMIT = 1u << 22;  // bounded waits

// u64 word offsets in the counter block (hot words on separate 128-B lines)
constexpr int SYNC_TAG = 0, SYNC_TICKET = 16, SYNC_DONE = 32, SYNC_RG = 48;

template <int TG>
constexpr int red_bytes() { return (DF_WAVES - 1) * TG * 64 * 16; }

int zrow_bytes(int L) { return ((L + DF_STEP - 1) / DF_STEP) * DF_STEP * 2 + 16; }

__device__ __forceinline__ unsigned long long ld_agent(const unsigned long long* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ void st_agent(unsigned long long* p, unsigned long long v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ __forceinline__ unsigned long long add_agent(unsigned long long* p, unsigned long long v) {
    return __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
// Wait until this wave's earlier memory operations have completed.
__device__ __forceinline__ void wait_mem() { __builtin_amdgcn_s_waitcnt(0); }

// Take a ticket (thread 0 only); claims the counter block for this call first.
__device__ unsigned long long take_ticket(unsigned long long* sync, unsigned long long epoch, int nrg) {
    unsigned long long t = ld_agent(sync + SYNC_TAG);
    for (unsigned it = 0; t != epoch && it < DF_SPIN_LIMIT; ++it) {
        if (t != ~epoch && __hip_atomic_compare_exchange_strong(sync + SYNC_TAG, &t, ~epoch, __ATOMIC_RELAXED,
                                                                __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT)) {
            st_agent(sync + SYNC_TICKET, 0ull);
            st_agent(sync + SYNC_DONE, 0ull);
            for (int i = 0; i < nrg; ++i) st_agent(sync + SYNC_RG + i, 0ull);
            wait_mem();
            st_agent(sync + SYNC_TAG, epoch);
            wait_mem();
            break;
        }
        __builtin_amdgcn_s_sleep(1);
        t = ld_agent(sync + SYNC_TAG);
    }
    return add_agent(sync + SYNC_TICKET, 1ull);
}

// Row r0 + (lane & 15) of a row-major matrix, clamped to the last row.
__device__ __forceinline__ const uint16_t* unit_row(const uint16_t* W, int64_t ldw, int rows, int r0, int lr) {
    const int r = r0 + lr;
    return W + (int64_t)(r < rows ? r : rows - 1) * ldw;
}

// One wave's loads of a unit's streamed rows: steps s0, s0+8, ...
// (DF_UNROLL of them; steps >= s_end give zeros).
__device__ __forceinline__ void load_rows(u32x4_t (&vw)[DF_UNROLL], const uint16_t* wrow, int depth, int s0,
                                          int s_end, int lk) {
#pragma unroll
    for (int u = 0; u < DF_UNROLL; ++u) {
        const int s = s0 + u * DF_WAVES;
        const int k = s * DF_STEP + lk;
        vw[u] = (s < s_end) ? ((k + 8 <= depth) ? *reinterpret_cast<const u32x4_t*>(wrow + k)
                                                : load_chunk_masked(wrow, k, depth))
                            : u32x4_t{0u, 0u, 0u, 0u};
    }
}

// Partial sums of a unit: 16 streamed rows (this lane's row at wrow) x 16*TG
// tokens over the steps s_begin + wave, s_begin + wave + 8, ... < s_end.
// Tokens come from global memory (act, row stride lda, ntok rows) or from
// LDS (zlds, row stride zld bytes, zero beyond the depth).  When
// `preloaded`, vw already holds this wave's first DF_UNROLL steps.
template <int TG, bool ACT_LDS>
__device__ __forceinline__ void unit_dot(f32x4_t (&acc)[TG], u32x4_t (&vw)[DF_UNROLL], bool preloaded,
                                         const uint16_t* __restrict__ wrow, const uint16_t* __restrict__ act,
                                         int64_t lda, int ntok, const unsigned char* zlds, int zld, int depth,
                                         int s_begin, int s_end, int wave, int lane) {
    const int lr = lane & 15;
    const int lk = (lane >> 4) * 8;
    const uint16_t* arow[TG];
    bool aval[TG];
#pragma unroll
    for (int t = 0; t < TG; ++t) {
        const int n = t * 16 + lr;
        aval[t] = n < ntok;
        arow[t] = ACT_LDS ? nullptr : act + (int64_t)(aval[t] ? n : 0) * lda;
    }
#pragma unroll
    for (int t = 0; t < TG; ++t) acc[t] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    for (int s0 = s_begin + wave; s0 < s_end; s0 += DF_WAVES * DF_UNROLL) {
        if (!preloaded) load_rows(vw, wrow, depth, s0, s_end, lk);
        preloaded = false;
        u32x4_t va[DF_UNROLL][TG];
#pragma unroll
        for (int u = 0; u < DF_UNROLL; ++u) {
            const int s = s0 + u * DF_WAVES;
            const int k = s * DF_STEP + lk;
            const bool live = s < s_end;
#pragma unroll
            for (int t = 0; t < TG; ++t) {
                if constexpr (ACT_LDS) {
                    va[u][t] = live ? *reinterpret_cast<const u32x4_t*>(zlds + (t * 16 + lr) * zld + k * 2)
                                    : u32x4_t{0u, 0u, 0u, 0u};
                } else {
                    va[u][t] = (live && aval[t])
                                   ? ((k + 8 <= depth) ? *reinterpret_cast<const u32x4_t*>(arow[t] + k)
                                                       : load_chunk_masked(arow[t], k, depth))
                                   : u32x4_t{0u, 0u, 0u, 0u};
                }
            }
        }
#pragma unroll
        for (int u = 0; u < DF_UNROLL; ++u)
#pragma unroll
            for (int t = 0; t < TG; ++t)
                acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(vw[u]), as_bf16x8(va[u][t]),
                                                                 acc[t], 0, 0, 0);
    }
}

// Sum the 8 waves' partial sums into wave 0 (fixed order).  All threads of
// the workgroup call it; it returns true on wave 0.
template <int TG>
__device__ __forceinline__ bool reduce_waves(f32x4_t (&acc)[TG], f32x4_t* red, int wave, int lane) {
    if (wave > 0) {
#pragma unroll
        for (int t = 0; t < TG; ++t) red[((wave - 1) * TG + t) * 64 + lane] = acc[t];
    }
    __syncthreads();
    const bool w0 = wave == 0;
    if (w0) {
#pragma unroll
        for (int w = 0; w < DF_WAVES - 1; ++w)
#pragma unroll
            for (int t = 0; t < TG; ++t) acc[t] += red[(w * TG + t) * 64 + lane];
    }
    __syncthreads();
    return w0;
}

// Store 4 consecutive output columns c..c+3 of a token row (bf16).
__device__ __forceinline__ void store4_bf16(uint16_t* rowp, int c, int ncols, f32x4_t v) {
    if (c + 3 < ncols) {
        u32x2_t p;
        p[0] = pack_bf16x2(v[0], v[1]);
        p[1] = pack_bf16x2(v[2], v[3]);
        *reinterpret_cast<u32x2_t*>(rowp + c) = p;
    } else {
#pragma unroll
        for (int i = 0; i < 4; ++i)
            if (c + i < ncols) rowp[c + i] = (uint16_t)bf16_rne(v[i]);
    }
}

__device__ __forceinline__ unsigned long long pack4_bf16(f32x4_t v) {
    return (unsigned long long)pack_bf16x2(v[0], v[1]) | ((unsigned long long)pack_bf16x2(v[2], v[3]) << 32);
}
__device__ __forceinline__ unsigned long long pack2_f32(float a, float b) {
    return (unsigned long long)__float_as_uint(a) | ((unsigned long long)__float_as_uint(b) << 32);
}

template <int TG>
__global__ __launch_bounds__(DF_WAVES * 64) __attribute__((amdgpu_waves_per_eu(TG == 1 ? 4 : 2)))
void decode_fused_kernel(DecodeArgs a) {
    extern __shared__ __attribute__((aligned(16))) unsigned char dyn[];
    f32x4_t* red = reinterpret_cast<f32x4_t*>(dyn);
    unsigned char* zlds = dyn + red_bytes<TG>();
    __shared__ unsigned long long s_ticket;

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int lr = lane & 15;
    const int lq = lane >> 4;
    const int nrg1 = (a.L + 15) / 16;
    const unsigned G = gridDim.x;

    if (threadIdx.x == 0) s_ticket = take_ticket(a.sync, a.epoch, a.S1 > 1 ? nrg1 : 0);
    __syncthreads();
    const unsigned long long ticket = s_ticket;
    const unsigned long long launch = ticket / G;   // launches since the block was claimed
    const int id = (int)(ticket - launch * G);
    unsigned long long* done = a.sync + SYNC_DONE;

    if (id < a.P1) {
        // ---- phase 1: one projection unit -------------------------------------------
        const int ksteps = (a.K + DF_STEP - 1) / DF_STEP;
        const int rg = id / a.S1;
        const int s = id - rg * a.S1;
        const int sb = s * a.steps1;
        const int se = (sb + a.steps1 < ksteps) ? sb + a.steps1 : ksteps;
        f32x4_t acc[TG];
        u32x4_t vw[DF_UNROLL];
        unit_dot<TG, false>(acc, vw, false, unit_row(a.Pt, a.ldp, a.L, rg * 16, lr), a.X, a.ldx, a.N, nullptr,
                            0, a.K, sb, se, wave, lane);
        if (!reduce_waves<TG>(acc, red, wave, lane)) return;
        const int c = rg * 16 + 4 * lq;    // < ldz; Z columns >= L are never read
        if (a.S1 == 1) {
#pragma unroll
            for (int t = 0; t < TG; ++t) {
                const int n = t * 16 + lr;
                if (n < a.N)
                    st_agent(reinterpret_cast<unsigned long long*>(a.Z + (int64_t)n * a.ldz + c),
                             pack4_bf16(acc[t]));
            }
            wait_mem();
            if (lane == 0) add_agent(done, 1ull);
            return;
        }
#pragma unroll
        for (int t = 0; t < TG; ++t) {
            const int n = t * 16 + lr;
            if (n < a.N && c < a.L) {
                unsigned long long* p =
                    reinterpret_cast<unsigned long long*>(a.part + ((int64_t)s * a.N + n) * a.ldpart + c);
                st_agent(p, pack2_f32(acc[t][0], acc[t][1]));
                st_agent(p + 1, pack2_f32(acc[t][2], acc[t][3]));
            }
        }
        wait_mem();
        unsigned long long prev = 0;
        if (lane == 0) prev = add_agent(a.sync + SYNC_RG + rg, 1ull);
        prev = __shfl(prev, 0);
        if (prev % (unsigned long long)a.S1 != (unsigned long long)(a.S1 - 1)) return;
        // last unit of this row group: add the S1 partial sums in split order
#pragma unroll
        for (int t = 0; t < TG; ++t) {
            const int n = t * 16 + lr;
            if (n < a.N && c < a.L) {
                f32x4_t sum = {0.f, 0.f, 0.f, 0.f};
                for (int q = 0; q < a.S1; ++q) {
                    const unsigned long long* p = reinterpret_cast<const unsigned long long*>(
                        a.part + ((int64_t)q * a.N + n) * a.ldpart + c);
                    const unsigned long long v0 = ld_agent(p), v1 = ld_agent(p + 1);
                    sum[0] += __uint_as_float((unsigned)v0);
                    sum[1] += __uint_as_float((unsigned)(v0 >> 32));
                    sum[2] += __uint_as_float((unsigned)v1);
                    sum[3] += __uint_as_float((unsigned)(v1 >> 32));
                }
                st_agent(reinterpret_cast<unsigned long long*>(a.Z + (int64_t)n * a.ldz + c), pack4_bf16(sum));
            }
        }
        wait_mem();
        if (lane == 0) add_agent(done, 1ull);
        return;
    }

    // ---- phase 2: folded weight ------------------------------------------------------
    const int p2 = id - a.P1;
    const int nrg2 = (a.M + 15) / 16;
    if (p2 >= nrg2) return;
    const int lsteps = (a.L + DF_STEP - 1) / DF_STEP;
    u32x4_t vw[DF_UNROLL];
    load_rows(vw, unit_row(a.Wf, a.ldwf, a.M, p2 * 16, lr), a.L, wave, lsteps, lq * 8);   // before Z is ready

    if (threadIdx.x == 0) {
        const unsigned long long target = (launch + 1) * (unsigned long long)nrg1;
        for (unsigned it = 0; it < DF_SPIN_LIMIT; ++it) {
            if (ld_agent(done) >= target) break;
            __builtin_amdgcn_s_sleep(2);
        }
    }
    __syncthreads();

    // Z -> LDS: token rows n < N (zero beyond L), zero rows for the other tokens
    const int zld = lsteps * DF_STEP * 2 + 16;
    const int zq = lsteps * DF_STEP / 4;          // 8-byte quads per row
    for (int i = threadIdx.x; i < 16 * TG * zq; i += blockDim.x) {
        const int n = i / zq;
        const int q = i - n * zq;
        const int l = q * 4;
        unsigned long long v = 0ull;
        if (n < a.N && l < a.L) {
            v = ld_agent(reinterpret_cast<const unsigned long long*>(a.Z + (int64_t)n * a.ldz + l));
            const int nv = a.L - l;
            if (nv < 4) v &= (1ull << (16 * nv)) - 1ull;
        }
        *reinterpret_cast<unsigned long long*>(zlds + n * zld + q * 8) = v;
    }
    __syncthreads();

    bool pre = true;
    for (int u = p2; u < nrg2; u += a.P2) {
        f32x4_t acc[TG];
        unit_dot<TG, true>(acc, vw, pre, unit_row(a.Wf, a.ldwf, a.M, u * 16, lr), nullptr, 0, a.N, zlds, zld,
                           a.L, 0, lsteps, wave, lane);
        pre = false;
        if (reduce_waves<TG>(acc, red, wave, lane)) {
            const int c = u * 16 + 4 * lq;
#pragma unroll
            for (int t = 0; t < TG; ++t) {
                const int n = t * 16 + lr;
                if (n < a.N) store4_bf16(a.Y + (int64_t)n * a.ldy, c, a.M, acc[t]);
            }
        }
    }
}

template <int TG>
int dyn_bytes(int L) { return red_bytes<TG>() + 16 * TG * zrow_bytes(L); }

template <int TG>
bool set_lds_limit() {
    static const bool ok = hipFuncSetAttribute(reinterpret_cast<const void*>(&decode_fused_kernel<TG>),
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               DF_LDS_MAX) == hipSuccess;
    return ok;
}

template <int TG>
hipError_t launch_df(const DecodeArgs& a, hipStream_t stream) {
    if (!set_lds_limit<TG>()) return hipErrorLaunchFailure;
    hipLaunchKernelGGL(decode_fused_kernel<TG>, dim3(a.P1 + a.P2), dim3(DF_WAVES * 64),
                       (unsigned)dyn_bytes<TG>(a.L), stream, a);
    return hipGetLastError();
}

}  // namespace

bool decode_fused_supported(int N, int L) {
    if (N < 1 || N > 32 || L < 1) return false;
    const int dyn = N <= 16 ? dyn_bytes<1>(L) : dyn_bytes<2>(L);
    return dyn <= DF_LDS_MAX;
}

size_t decode_fused_sync_bytes(int L) {
    const size_t words = SYNC_RG + (L + 15) / 16;
    return (words * 8 + 255) / 256 * 256;
}

// Work split for a device of `cus` compute units.  Projection units are
// sized to about 64 KB of Pt each (S1 depth ranges per 16-row group) while
// they take at most half of the resident workgroups; the phase-2 workgroups
// fill the rest, with the same number of Wf units each.
void decode_fused_plan(int N, int K, int L, int M, int cus, int* S1, int* steps1, int* P1, int* P2) {
    int per_cu = 1;                 // two token groups: 141 VGPRs, one workgroup per CU
    if (N <= 16) {
        per_cu = (160 * 1024) / dyn_bytes<1>(L);
        per_cu = per_cu < 1 ? 1 : (per_cu > 2 ? 2 : per_cu);
    }
    const int cap = cus * per_cu;
    const int ksteps = (K + DF_STEP - 1) / DF_STEP;
    const int nrg1 = (L + 15) / 16;
    const int nrg2 = (M + 15) / 16;
    const int unit_target_steps = 65536 / (16 * DF_STEP * 2);   // 64 KB of Pt
    int s1 = (ksteps + unit_target_steps - 1) / unit_target_steps;
    const int s1_cap = (cap / 2) / nrg1;
    if (s1 > s1_cap) s1 = s1_cap;
    if (s1 > ksteps) s1 = ksteps;
    if (s1 < 1) s1 = 1;
    *steps1 = (ksteps + s1 - 1) / s1;
    *S1 = (ksteps + *steps1 - 1) / *steps1;
    *P1 = nrg1 * *S1;
    int p2 = cap - *P1;
    if (p2 < cap / 2) p2 = cap / 2;
    if (p2 > nrg2) p2 = nrg2;
    const int rounds = (nrg2 + p2 - 1) / p2;
    *P2 = (nrg2 + rounds - 1) / rounds;
}

hipError_t launch_decode_fused(const DecodeArgs& a, hipStream_t stream) {
    if (a.N <= 16) return launch_df<1>(a, stream);
    return launch_df<2>(a, stream);
}

}  // namespace espace
