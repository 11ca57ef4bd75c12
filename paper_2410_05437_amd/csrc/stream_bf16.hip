// Persistent streaming bfloat16 product for 3 to 16 tokens (decode):
//
//     C[n][j] = sum_k A[n][k] * B[j][k],   n < R <= 16 (tokens), j < Cc
//
// The many-row operand B (the folded weight, P or W) is streamed from HBM
// once, the way the one- and two-token kernel streams it: every load
// instruction of a wave moves one 1 KB piece of one row (512 elements).  The
// loads go straight to LDS (buffer_load ... lds) into a ring of six 16 KB
// stages, five of them in flight, so the stream does not depend on how many
// loads the compiler keeps in registers.  A stage holds 16 rows (one group)
// x 512 of depth; chunk c of row r sits at chunk c ^ r, so that the 16 rows
// one fragment read touches fall on distinct banks.
//
// Workgroups are persistent (one per CU) and take groups blockIdx.x,
// blockIdx.x + gridDim.x, ...: at any moment the workgroups stream
// neighbouring rows (an equal contiguous share of the rows per workgroup,
// 256 places in memory at once, was 15-20% slower).  Its eight waves split
// the depth of every stage (64 elements each, two v_mfma_f32_16x16x32_bf16
// with the group's 16 rows as one operand and the tokens as the other); each
// wave keeps its
// slices of the tokens in registers for the whole call, loaded once.  At the
// end of a group the eight partial sums are added in wave order through LDS
// (fixed order: results do not depend on scheduling) and written.
//
// The depth tail: pieces starting at or beyond D are read from an offset
// past the buffer (the load returns zeros), the piece that straddles D is
// masked in registers, and the tokens are zero beyond D.
#include "common.hpp"
#include "kernels.hpp"

namespace espace {

namespace {

constexpr int ST_WAVES = 8;                       // waves per workgroup
constexpr int ST_SD = 512;                        // depth of a stage (elements)
constexpr int ST_RING = 6;                        // LDS stages
constexpr int ST_STAGE = 16 * ST_SD * 2;          // 16 rows x 1 KB
constexpr int ST_LPW = 16 / ST_WAVES;             // 1 KB row loads per wave and stage
constexpr int ST_MAX_NS = 12;                     // stages per group: depth up to 6144

// s_barrier that the compiler moves no memory access across (the loads of
// other waves into LDS are invisible to it); unlike __syncthreads() it does
// not wait for this wave's loads still in flight
__device__ __forceinline__ void st_barrier() { asm volatile("s_barrier" ::: "memory"); }

template <int N>
__device__ __forceinline__ void st_wait_vm() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt(0x0F70 | (N & 15) | ((N >> 4) << 14));
}

// vmcnt for at most `stages` newer stages of this wave's loads in flight
__device__ __forceinline__ void st_wait_stages(int stages) {
    switch (stages) {
        case 0: st_wait_vm<0>(); break;
        case 1: st_wait_vm<1 * ST_LPW>(); break;
        case 2: st_wait_vm<2 * ST_LPW>(); break;
        case 3: st_wait_vm<3 * ST_LPW>(); break;
        default: st_wait_vm<4 * ST_LPW>(); break;
    }
    static_assert(ST_RING - 2 == 4, "waits cover the ring");
}

template <int NS>
__global__ __launch_bounds__(ST_WAVES * 64, 1)
void stream_tn_bf16_kernel(const uint16_t* __restrict__ A, int64_t lda, const uint16_t* __restrict__ B,
                           int64_t ldb, void* __restrict__ Cout, int64_t ldc, int R, int Cc, int D, int out_f32) {
    __shared__ __attribute__((aligned(1024))) unsigned char smem[ST_RING * ST_STAGE + ST_WAVES * 64 * 16];
    f32x4_t* red = reinterpret_cast<f32x4_t*>(smem + ST_RING * ST_STAGE);
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int G = gridDim.x;
    const int ngroups = (Cc + 15) / 16;
    const int my_groups = (ngroups - (int)blockIdx.x + G - 1) / G;
    const int Q = my_groups * NS;                 // stages of this workgroup

    // this wave's slices of the tokens: token lane % 16, elements
    // 512 s + 64 wave + 32 t + 8 (lane / 16) .. + 7 (zero past D and for
    // token rows past R)
    u32x4_t tok[NS][2];
    {
        const int n = lane & 15;
        const uint16_t* arow = A + (int64_t)(n < R ? n : 0) * lda;
        const uint32_t m = n < R ? 0xffffffffu : 0u;
#pragma unroll
        for (int s = 0; s < NS; ++s)
#pragma unroll
            for (int t = 0; t < 2; ++t)
                tok[s][t] = load_chunk_masked(arow, ST_SD * s + 64 * wave + 32 * t + 8 * (lane >> 4), D) & m;
    }

    const auto brsrc = __builtin_amdgcn_make_buffer_rsrc((void*)B, (short)0, (int)((uint64_t)Cc * ldb * 2u),
                                                         0x00020000);
    // the loads of stage q (group blockIdx.x + (q / NS) G, depth piece q % NS)
    // into its ring slot: this wave's rows r = ST_LPW wave + j, lane l
    // fetching chunk l ^ r of the piece
    auto issue = [&](int q) {
        const int i = q / NS, s = q - i * NS;
        const int g = (int)blockIdx.x + i * G;
        unsigned char* slot = smem + (q % ST_RING) * ST_STAGE;
#pragma unroll
        for (int j = 0; j < ST_LPW; ++j) {
            const int r = ST_LPW * wave + j;
            int row = 16 * g + r;
            row = row < Cc ? row : Cc - 1;
            const int k = ST_SD * s + 8 * (lane ^ r);
            const unsigned off = k < D ? (unsigned)(((uint64_t)row * ldb + k) * 2u) : 0x7FFFFFF0u;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                brsrc, (__attribute__((address_space(3))) void*)(slot + r * 1024), 16, (int)off, 0, 0, 0);
        }
    };

    const int pre = Q < ST_RING - 1 ? Q : ST_RING - 1;
    for (int q = 0; q < pre; ++q) issue(q);

    // fragment of depth step t of a stage: row lane % 16, chunk
    // 8 wave + 4 t + lane / 16 of the piece (physical chunk ^ row)
    const int fr = lane & 15;
    int foff[2];
#pragma unroll
    for (int t = 0; t < 2; ++t) {
        const int c = 8 * wave + 4 * t + (lane >> 4);
        foff[t] = fr * 1024 + ((c ^ fr) << 4);
    }
    // the piece of the last stage that straddles D: mask its lanes' chunks
    const int dlast = D - ST_SD * (NS - 1);       // depth in the last stage (1 .. 512)

    int q = 0;
    for (int i = 0; i < my_groups; ++i) {
        f32x4_t acc = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int s = 0; s < NS; ++s, ++q) {
            // stage q has landed (newer stages may stay in flight), and every
            // wave is done reading stage q - 1, whose slot receives stage q + 5
            const int newer = (Q - 1 - q) < (ST_RING - 2) ? (Q - 1 - q) : (ST_RING - 2);
            st_wait_stages(newer);
            st_barrier();
            if (q + ST_RING - 1 < Q) issue(q + ST_RING - 1);
            const unsigned char* slot = smem + (q % ST_RING) * ST_STAGE;
            u32x4_t w[2];
#pragma unroll
            for (int t = 0; t < 2; ++t) w[t] = *reinterpret_cast<const u32x4_t*>(slot + foff[t]);
            if (s == NS - 1) {
#pragma unroll
                for (int t = 0; t < 2; ++t) {
                    const int k = 64 * wave + 32 * t + 8 * (lane >> 4);   // depth inside the last piece
                    w[t] = mask_chunk(w[t], dlast - k < 0 ? 0 : (dlast - k > 8 ? 8 : dlast - k));
                }
            }
#pragma unroll
            for (int t = 0; t < 2; ++t)
                acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(w[t]), as_bf16x8(tok[s][t]), acc, 0, 0, 0);
        }
        // the group's sums: the eight waves' partial sums in wave order
        red[wave * 64 + lane] = acc;
        asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        st_barrier();
        if (wave == 0) {
            f32x4_t v = red[lane];
#pragma unroll
            for (int u = 1; u < ST_WAVES; ++u) v += red[u * 64 + lane];
            // lane l: token l % 16, rows 4 (l / 16) .. + 3 of the group
            const int n = lane & 15;
            const int j = 16 * ((int)blockIdx.x + i * G) + 4 * (lane >> 4);
            if (n < R && j < Cc) {
                if (out_f32) {
                    float* p = reinterpret_cast<float*>(Cout) + (int64_t)n * ldc + j;
                    if (j + 4 <= Cc) {
                        *reinterpret_cast<f32x4_t*>(p) = v;
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (j + e < Cc) p[e] = v[e];
                    }
                } else {
                    uint16_t* p = reinterpret_cast<uint16_t*>(Cout) + (int64_t)n * ldc + j;
                    if (j + 4 <= Cc) {
                        *reinterpret_cast<u32x2_t*>(p) = u32x2_t{pack_bf16x2(v[0], v[1]), pack_bf16x2(v[2], v[3])};
                    } else {
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (j + e < Cc) p[e] = (uint16_t)bf16_rne(v[e]);
                    }
                }
            }
        }
        // red is rewritten NS stages (and as many barriers) later
    }
}

template <int NS>
hipError_t launch_ns(const GemmArgs& g, hipStream_t stream) {
    const int ngroups = (g.Cc + 15) / 16;
    const int cus = g.cus > 0 ? g.cus : 256;
    const int grid = ngroups < cus ? ngroups : cus;
    hipLaunchKernelGGL((stream_tn_bf16_kernel<NS>), dim3(grid), dim3(ST_WAVES * 64), 0, stream, g.A, g.lda, g.B,
                       g.ldb, g.C, g.ldc, g.R, g.Cc, g.D, g.c_f32);
    return hipGetLastError();
}

}  // namespace

bool stream_supported(int R, int D) { return R >= 1 && R <= 16 && D >= 1 && D <= ST_SD * ST_MAX_NS; }

hipError_t launch_stream_tn_bf16(const GemmArgs& g, hipStream_t stream) {
    if (!stream_supported(g.R, g.D) || g.Cc < 1 || (int64_t)g.Cc * g.ldb * 2 >= ((int64_t)1 << 31))
        return hipErrorInvalidValue;
    switch ((g.D + ST_SD - 1) / ST_SD) {
        case 1: return launch_ns<1>(g, stream);
        case 2: return launch_ns<2>(g, stream);
        case 3: return launch_ns<3>(g, stream);
        case 4: return launch_ns<4>(g, stream);
        case 5: return launch_ns<5>(g, stream);
        case 6: return launch_ns<6>(g, stream);
        case 7: return launch_ns<7>(g, stream);
        case 8: return launch_ns<8>(g, stream);
        case 9: return launch_ns<9>(g, stream);
        case 10: return launch_ns<10>(g, stream);
        case 11: return launch_ns<11>(g, stream);
        default: return launch_ns<12>(g, stream);
    }
}

}  // namespace espace
