// C ABI of the projected linear layer: argument validation, the choice of
// kernel configuration for each product, and the launches.
//
// Every entry point validates all of its arguments before touching the device,
// so an error status guarantees that nothing was enqueued or written.
#include "espace.h"

#include <hip/hip_runtime.h>

#include <cstdarg>
#include <cstdio>
#include <atomic>
#include <cstdlib>
#include <cstring>
#include <algorithm>
#include <mutex>
#include <random>
#include <string>

#include "kernels.hpp"

// Scratch of espace_projected_linear_noalloc: Z and the partial sums of one
// call, held by every device the library runs on until the process ends.
// Calls on one device share it.
static __device__ __align__(256) unsigned char scratch[ESPACE_NOALLOC_SCRATCH_BYTES];

// Count of the bounded cross-workgroup waits that gave up (one per device;
// the kernels add to it through the address hipGetSymbolAddress gives).
__device__ unsigned long long g_wait_timeouts;

namespace {

using espace::GemmArgs;

constexpr unsigned kDefaultWaitSpins = 1u << 22;
std::atomic<unsigned> g_wait_spins{kDefaultWaitSpins};

thread_local std::string g_last_error;

espace_status fail(espace_status s, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof buf, fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return s;
}

espace_status ok() {
    g_last_error.clear();
    return ESPACE_OK;
}

constexpr int64_t kMaxDim = (int64_t)1 << 30;
constexpr int kDefaultCUs = 256;      // MI355X, for queries made without a device
constexpr size_t kWsAlign = 256;

size_t elem_size(espace_dtype dt) { return dt == ESPACE_BF16 ? 2 : 4; }
int64_t ld_align(espace_dtype dt) { return dt == ESPACE_BF16 ? 8 : 4; }
int64_t round_up(int64_t x, int64_t m) { return (x + m - 1) / m * m; }
size_t align_ws(size_t x) { return (x + kWsAlign - 1) / kWsAlign * kWsAlign; }

// Compute units of the current device (read once per device); configurations
// are planned for this count.  Without a usable device (a workspace query on a
// host with no GPU) the full MI355X count.
int device_cus() {
    static std::mutex mu;
    static int cus[64] = {0};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
        (void)hipGetLastError();
        return kDefaultCUs;
    }
    std::lock_guard<std::mutex> lk(mu);
    if (cus[dev] == 0) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1) {
            (void)hipGetLastError();
            n = kDefaultCUs;
        }
        cus[dev] = n;
    }
    return cus[dev];
}

// Device address of this device's g_wait_timeouts (looked up once per device;
// the array's name is a host-side stand-in and must not reach a kernel).
unsigned long long* timeout_counter() {
    static std::mutex mu;
    static unsigned long long* ptr[64] = {nullptr};
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) {
        (void)hipGetLastError();
        return nullptr;
    }
    std::lock_guard<std::mutex> lk(mu);
    if (!ptr[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(g_wait_timeouts)) != hipSuccess) {
            (void)hipGetLastError();
            return nullptr;
        }
        ptr[dev] = static_cast<unsigned long long*>(p);
    }
    return ptr[dev];
}

espace::WaitCfg wait_cfg() {
    espace::WaitCfg w;
    w.spins = g_wait_spins.load(std::memory_order_relaxed);
    w.timeouts = timeout_counter();
    return w;
}

// ---- planning ---------------------------------------------------------------

enum Kind { KIND_TILED = 0, KIND_SKINNY = 1, KIND_F32 = 2, KIND_GEMV = 3, KIND_STREAM = 4 };

struct Plan {
    int kind = KIND_F32;
    int tile = 0;
    int splits = 1;
    int pair = 0;               // splits == 2 combined inside the GEMM kernel
    size_t partial_bytes = 0;   // fp32 partial sums for splits > 1 (and pair state words)
    // tiled products in two launches by rows: rows [0, rows1) as above, the
    // rest with (tile2, splits2, pair2); 0: one launch
    int rows1 = 0;
    int tile2 = 0, splits2 = 1, pair2 = 0;
};

int ceil_div(int64_t a, int64_t b) { return (int)((a + b - 1) / b); }

Plan plan_skinny(int R, int Cc, int D, int cus) {
    // Measured on the decode layers (N <= 32): a launch costs a few µs
    // whatever its size, so the depth is split only when the tokens make
    // each workgroup's loads heavy or the depth is very large; 8 waves with
    // 6 loads in flight fit 48-step depths exactly; 32-row groups halve the
    // token re-reads from L2 when there are 9 or more tokens.  With fewer
    // 16-row groups than half the CUs (the projection,
    // L = 1536 rows), two depth segments per MFMA operand double the
    // workgroups in one launch (K = 4096: 5.6 against 7.5 µs; K = 11008:
    // 12.5 against 17.6 µs with a three-way split), and with 9 to 16 tokens
    // as two token groups of 8 sharing the weight operand (K = 4096: 7.9
    // against 8.1 µs at 16 tokens, 7.4 against 7.8 at 12, with a two-way
    // split and its reduction launch); with 128 or more groups
    // one depth range is fastest up to 256 steps (K = 6144, L = 3686: 12.3
    // against 17.6 µs with two ranges).
    Plan p;
    p.kind = KIND_SKINNY;
    const int nb1 = ceil_div(Cc, 16);
    const int steps = ceil_div(D, 32);
    const int target = 2 * cus;
    if (nb1 >= target) {
        if (R > 8) p.tile = espace::SKINNY_RG2_W4;
        else p.tile = (steps <= 48) ? espace::SKINNY_RG1_W8_U6 : espace::SKINNY_RG1_W8_U8;
    } else if (R <= 16 && nb1 < cus / 2 && steps <= 384) {
        if (R <= 8) p.tile = steps <= 128 ? espace::SKINNY_SEG2_W8_U8 : espace::SKINNY_SEG2_W16_U4;
        else p.tile = steps <= 128 ? espace::SKINNY_SEG2_TG2_W8_U8 : espace::SKINNY_SEG2_TG2_W16_U4;
    } else {
        p.tile = espace::SKINNY_RG1_W8_U8;
        int s = R > 8 ? 2 : 1;
        // at most 128 KB of each 16 rows per workgroup beyond 256 steps
        const int by_depth = (R > 8 || steps > 256) ? ceil_div(steps, 128) : 1;
        if (by_depth > s) s = by_depth;
        if (s > 1 && steps / s < 32) s = steps / 32 > 1 ? steps / 32 : 1;   // >= 4 steps per wave
        p.splits = s;
    }
    if (p.splits > 1) p.partial_bytes = (size_t)p.splits * R * espace::splitk_ld(Cc) * sizeof(float);
    return p;
}

struct TileShape { int tile, bm, bn, per_cu; double eff; };

// Per-call tags of the state words in workspaces (decode counters, pair
// states): a counter started from a random 64-bit value, so that leftover
// workspace contents match a tag with negligible probability.
unsigned long long next_epoch() {
    static std::atomic<unsigned long long> next{[] {
        std::random_device rd;
        return ((unsigned long long)rd() << 32) ^ (unsigned long long)rd();
    }()};
    return next.fetch_add(1, std::memory_order_relaxed);
}

// Workspace of a tiled plan: pair state words after the pair tiles, or the
// split-K partial sums.
void set_partial_bytes(Plan& p, int64_t R, int64_t Cc) {
    p.partial_bytes = 0;
    if (p.pair) {
        int bm = 0, bn = 0;
        espace::tile_dims(p.tile, &bm, &bn);
        const size_t tiles = (size_t)ceil_div(R, bm) * ceil_div(Cc, bn);
        p.partial_bytes = tiles * bm * bn * sizeof(float) + tiles * 8;
    } else if (p.splits > 1) {
        p.partial_bytes = (size_t)p.splits * R * espace::splitk_ld(Cc) * sizeof(float);
    }
}

Plan plan_tiled_one(int R, int Cc, int D, int cus, double* cost_out) {
    // Estimated time of each tile shape (and depth split) from the number of
    // rounds of workgroups the chip needs, the per-tile work and a relative
    // efficiency of the tile shape; the cheapest wins.  Two depth halves can
    // also be combined inside the kernel ("pair"), which costs one fp32 tile
    // written and read per output tile instead of a reduction pass.
    static const TileShape shapes[] = {
        {espace::TILE_256x256_W8T, 256, 256, 1, 1.00},
        {espace::TILE_256x192_W8, 256, 192, 1, 0.97},
        {espace::TILE_256x128, 256, 128, 1, 0.85},
        {espace::TILE_128x256, 128, 256, 1, 0.85},
        {espace::TILE_128x128, 128, 128, 2, 0.70},
        {espace::TILE_128x192, 128, 192, 1, 0.70},
    };
    const int ktiles = ceil_div(D, 64);
    const double byte_cost = 315.0 / (2.0 * 64 * cus);   // bytes priced against the MFMA rate
    Plan best;
    best.kind = KIND_TILED;
    double best_cost = 1e300;
    for (const TileShape& s : shapes) {
        const int64_t tiles = (int64_t)ceil_div(R, s.bm) * ceil_div(Cc, s.bn);
        const int64_t slots = (int64_t)cus * s.per_cu;
        for (int splits = 1; splits <= 4; ++splits) {
            if (splits > 1 && ktiles / splits < 8) break;
            for (int pair = 0; pair <= (splits == 2 ? 1 : 0); ++pair) {
                const int64_t blocks = tiles * splits;
                const int64_t rounds = (blocks + slots - 1) / slots;
                // a round runs per_cu blocks on every CU
                const double per_round = (double)s.bm * s.bn * ceil_div(ktiles, splits) * s.per_cu;
                double cost = rounds * per_round / s.eff;
                // the pair hand-off prices at 1.6x its bytes (measured: the
                // second half waits for the first's stores)
                if (pair) cost += 3.2 * tiles * s.bm * s.bn * 4.0 * byte_cost;
                else if (splits > 1) cost += 2.0 * splits * (double)R * Cc * 4.0 * byte_cost;
                if (cost < best_cost) {
                    best_cost = cost;
                    best.tile = s.tile;
                    best.splits = splits;
                    best.pair = pair;
                }
            }
        }
    }
    set_partial_bytes(best, R, Cc);
    if (cost_out) *cost_out = best_cost;
    return best;
}

Plan plan_tiled(int R, int Cc, int D, int cus) {
    // A product whose tiles leave the last round of workgroups partly empty
    // can run as two launches split by rows, each with whole rounds.  Taken
    // when the model prices it at least 3% cheaper, a launch counted as 3 µs
    // (110 000 of its units at the expand GEMM's measured rate).  Measured
    // (operands rotated through HBM): the Llama2-7B FFN up+gate fold, 22016 x
    // 1536 at depth 4096, 271 -> 247 µs; the GPT3-22B FFN up projection at
    // L = 2458, 8192 x 2458 at depth 6144, 258 -> 240 µs, and the down one,
    // depth 24576, 1039 -> 1027 µs; the up+gate dense product (4096 x 22016 x
    // 4096) 593 -> 597 µs, within the noise; the QKV fold,
    // 12288 x 1536 (1.5 rounds of 256 x 192 tiles, split as 4096 rows on 128 x
    // 192 tiles and 8192 on 256 x 192), 162 -> 167 µs, no gain: a half-empty
    // last round runs at higher clocks than the model assumes.
    double cost = 0;
    Plan best = plan_tiled_one(R, Cc, D, cus, &cost);
    if (R > 32768) return best;   // many rounds: the last one's share is small
    constexpr double kLaunch = 110e3;
    double best_split = 0.97 * cost;
    for (int r1 = 256; r1 < R; r1 += 256) {
        double c1 = 0, c2 = 0;
        const Plan p1 = plan_tiled_one(r1, Cc, D, cus, &c1);
        const Plan p2 = plan_tiled_one(R - r1, Cc, D, cus, &c2);
        if (c1 + c2 + kLaunch < best_split) {
            best_split = c1 + c2 + kLaunch;
            best = p1;
            best.rows1 = r1;
            best.tile2 = p2.tile;
            best.splits2 = p2.splits;
            best.pair2 = p2.pair;
            best.partial_bytes = std::max(p1.partial_bytes, p2.partial_bytes);
        }
    }
    return best;
}

// 3 to 16 tokens on a weight of at least 16 rows per CU: the persistent
// streaming kernel.  Measured on the Llama2-7B FFN up+gate layer (22016 x
// 1536 folded weight, 22016 x 4096 dense weight) against the skinny MFMA
// kernel: expansion 19.6 -> 14.6 µs at 8 tokens, 19.9 -> 15.1 at 16; dense
// 45.2 -> 34.2 and 57.3 -> 36.0 µs.  The projections (1536 rows) stay on the
// skinny kernel (5.8 against 6.6 µs at 8 tokens), one and two tokens on the
// whole-row kernel (the streaming kernel: 12.9 -> 16.8 µs on the expansion).
bool use_stream(int R, int Cc, int D) {
    return R >= 3 && espace::stream_supported(R, D) && (int64_t)Cc >= 16 * (int64_t)device_cus();
}

Plan plan_tn(int64_t R, int64_t Cc, int64_t D, espace_dtype dt) {
    if (dt == ESPACE_F32) return Plan{};
    if (R <= 32) {
        // One or two tokens: whole-row streaming with bf16 dot products
        // (measured at N = 1 on every decode layer of the workloads: 2-22%
        // faster than the MFMA kernel, e.g. the Llama2-7B up+gate expansion
        // 15.5 -> 14.2 µs, its dense W 38.1 -> 33.6 µs, the GPT3-22B
        // expansion at L = 2458 31.1 -> 24.4 µs; at N = 2 faster or within
        // 0.5 µs; slower from 3 tokens on).
        if (espace::gemv_supported((int)R, (int)D)) {
            Plan g;
            g.kind = KIND_GEMV;
            return g;
        }
        if (use_stream((int)R, (int)Cc, (int)D)) {
            Plan g;
            g.kind = KIND_STREAM;
            return g;
        }
        return plan_skinny((int)R, (int)Cc, (int)D, device_cus());
    }
    return plan_tiled((int)R, (int)Cc, (int)D, device_cus());
}

// ESPACE_PLAN_LOG=1 prints each product's plan to stderr (read once per process).
Plan plan_tn_logged(int64_t R, int64_t Cc, int64_t D, espace_dtype dt) {
    static const bool log = [] {
        const char* s = std::getenv("ESPACE_PLAN_LOG");
        return s && std::atoi(s) != 0;
    }();
    const Plan p = plan_tn(R, Cc, D, dt);
    if (log)
        std::fprintf(stderr,
                     "espace plan R=%lld Cc=%lld D=%lld: kind=%d tile=%d splits=%d pair=%d partial=%zu rows1=%d "
                     "tile2=%d splits2=%d pair2=%d\n",
                     (long long)R, (long long)Cc, (long long)D, (int)p.kind, p.tile, p.splits, p.pair,
                     p.partial_bytes, p.rows1, p.tile2, p.splits2, p.pair2);
    return p;
}

// Leading dimension of Z in the workspace.  For decode (N <= 32, bf16) the
// rows are offset by a further 64 bytes: every workgroup of the expansion
// reads the same few Z rows at the same depth, and rows 3 KB apart (L = 1536)
// meet in the same memory channels (measured on the Llama2-7B up+gate
// expansion: 19.9 -> 19.1 µs at 16 tokens, 24.3 -> 22.5 µs at 32).
int64_t z_ld(int64_t L, int64_t N, espace_dtype dt) {
    if (dt != ESPACE_BF16) return round_up(L, 32);
    return round_up(L, 64) + (N <= 32 ? 32 : 0);
}

// Bytes of Z in the workspace: N rows of z_ld elements, or for prefill
// (N > 32) as many row pairs of 2 z_ld elements (the row-pair layout, below)
size_t z_bytes(int64_t N, int64_t L, espace_dtype dt) {
    const int64_t rows = N > 32 ? round_up(N, 2) : N;
    return align_ws((size_t)rows * z_ld(L, N, dt) * elem_size(dt));
}

// Workspace of the training-view gradients: transposed operands (the GEMM
// kernels reduce over the contiguous dimension of both operands), the
// intermediate products, and the GEMMs' partial sums (used one after the
// other).  Leading dimensions: multiples of 8 elements.
struct BwdLayout {
    size_t a, b, c, d, e, f, part, total;
};

int64_t ld8(int64_t c) { return (c + 7) / 8 * 8; }

BwdLayout bwd_layout(int64_t M, int64_t K, int64_t L, int64_t N, espace_dtype dt) {
    const size_t es = elem_size(dt);
    BwdLayout b{};
    size_t o = 0;
    b.a = o; o = align_ws(o + (size_t)L * ld8(M) * es);   // Wfᵀ  [L][M]
    b.b = o; o = align_ws(o + (size_t)K * ld8(L) * es);   // P    [K][L]
    b.c = o; o = align_ws(o + (size_t)M * ld8(N) * es);   // dYᵀ  [M][N]
    b.d = o; o = align_ws(o + (size_t)L * ld8(N) * es);   // Zᵀ   [L][N]
    b.e = o; o = align_ws(o + (size_t)N * ld8(L) * es);   // dZ   [N][L]
    b.f = o; o = align_ws(o + (size_t)M * ld8(L) * es);   // G    [M][L]
    b.part = o;
    size_t part = plan_tn(N, L, M, dt).partial_bytes;
    part = std::max(part, plan_tn(N, K, L, dt).partial_bytes);
    part = std::max(part, plan_tn(M, L, N, dt).partial_bytes);
    part = std::max(part, plan_tn(M, K, L, dt).partial_bytes);
    b.total = align_ws(o + part);
    return b;
}

BwdLayout dense_bwd_layout(int64_t M, int64_t K, int64_t N, espace_dtype dt) {
    const size_t es = elem_size(dt);
    BwdLayout b{};
    size_t o = 0;
    b.a = o; o = align_ws(o + (size_t)K * ld8(M) * es);   // Wᵀ   [K][M]
    b.c = o; o = align_ws(o + (size_t)M * ld8(N) * es);   // dYᵀ  [M][N]
    b.d = o; o = align_ws(o + (size_t)K * ld8(N) * es);   // Xᵀ   [K][N]
    b.part = o;
    const size_t part = std::max(plan_tn(N, K, M, dt).partial_bytes, plan_tn(M, K, N, dt).partial_bytes);
    b.total = align_ws(o + part);
    return b;
}

size_t ws_bytes(espace_op op, int64_t M, int64_t K, int64_t L, int64_t N, espace_dtype dt) {
    switch (op) {
        case ESPACE_OP_FOLD: return M ? align_ws(plan_tn(M, L, K, dt).partial_bytes) : 0;
        case ESPACE_OP_PROJECT: return N ? align_ws(plan_tn(N, L, K, dt).partial_bytes) : 0;
        case ESPACE_OP_EXPAND: return (N && M) ? align_ws(plan_tn(N, M, L, dt).partial_bytes) : 0;
        case ESPACE_OP_DENSE: return (N && M) ? align_ws(plan_tn(N, M, K, dt).partial_bytes) : 0;
        case ESPACE_OP_AUTOCORR: return N ? align_ws(espace::autocorr_workspace_bytes(N, K, dt == ESPACE_F32)) : 0;
        case ESPACE_OP_PCA: return align_ws(espace::pca_workspace_bytes(K));
        case ESPACE_OP_SYMPRODUCT: return align_ws(espace::symprod_workspace_bytes(K));
        case ESPACE_OP_BACKWARD: return (N && M) ? bwd_layout(M, K, L, N, dt).total : 0;
        case ESPACE_OP_DENSE_BACKWARD: return (N && M) ? dense_bwd_layout(M, K, N, dt).total : 0;
        case ESPACE_OP_PROJECTED_LINEAR: {
            if (!N || !M) return 0;
            const size_t a = plan_tn(N, L, K, dt).partial_bytes;
            const size_t b = plan_tn(N, M, L, dt).partial_bytes;
            return z_bytes(N, L, dt) + align_ws(a > b ? a : b);
        }
    }
    return SIZE_MAX;
}

// ---- MX-FP8 sizes -------------------------------------------------------------

// Columns of an MX-FP8 matrix as stored: whole 128-column steps of the MFMA.
int64_t mx_cols(int64_t cols) { return (cols + 127) / 128 * 128; }

// Workspace of the MX-FP8 layer: Z's codes in row pairs (round_up(N, 2) / 2
// pairs of 2 mx_cols(L) bytes: each 128-byte block holds 64 consecutive codes
// of two neighbouring tokens, so the expansion's 64-byte half-rows of Z are
// read as whole cache lines) and its scale bytes [N][mx_cols(L) / 32].
size_t mx_ws_bytes(int64_t M, int64_t L, int64_t N) {
    if (!N || !M) return 0;
    return align_ws((size_t)round_up(N, 2) * mx_cols(L)) + align_ws((size_t)N * mx_cols(L) / 32);
}


// ---- validation -------------------------------------------------------------

struct Range { const char* name; uintptr_t lo, hi; };

Range mat_range(const char* name, const void* p, int64_t rows, int64_t ld, espace_dtype dt) {
    const uintptr_t lo = (uintptr_t)p;
    return Range{name, lo, lo + (uintptr_t)(rows * ld) * elem_size(dt)};
}

espace_status check_dtype(espace_dtype dt) {
    if (dt != ESPACE_F32 && dt != ESPACE_BF16)
        return fail(ESPACE_ERR_DTYPE, "unknown dtype %d", (int)dt);
    return ESPACE_OK;
}

espace_status check_dims(int64_t M, int64_t K, int64_t L, int64_t N, bool has_L) {
    if (M < 0 || N < 0) return fail(ESPACE_ERR_SHAPE, "negative size (M=%lld, N=%lld)", (long long)M, (long long)N);
    if (K < 1) return fail(ESPACE_ERR_SHAPE, "K must be >= 1 (got %lld)", (long long)K);
    if (M > kMaxDim || N > kMaxDim || K > kMaxDim)
        return fail(ESPACE_ERR_SHAPE, "size above 2^30");
    if (has_L && (L < 1 || L > K))
        return fail(ESPACE_ERR_SHAPE, "need 1 <= L <= K (L=%lld, K=%lld)", (long long)L, (long long)K);
    return ESPACE_OK;
}

espace_status check_mat(const char* name, const void* p, int64_t rows, int64_t cols, int64_t ld,
                        espace_dtype dt) {
    if (!p) return fail(ESPACE_ERR_NULL, "%s is NULL", name);
    if (ld < cols || ld > kMaxDim * 4)
        return fail(ESPACE_ERR_SHAPE, "%s: leading dimension %lld < %lld columns", name,
                    (long long)ld, (long long)cols);
    if (ld % ld_align(dt))
        return fail(ESPACE_ERR_ALIGN, "%s: leading dimension %lld not a multiple of %lld elements",
                    name, (long long)ld, (long long)ld_align(dt));
    if ((uintptr_t)p % 16)
        return fail(ESPACE_ERR_ALIGN, "%s: pointer not 16-byte aligned", name);
    if (rows * ld > ((int64_t)1 << 40)) return fail(ESPACE_ERR_SHAPE, "%s too large", name);
    return ESPACE_OK;
}

bool overlaps(const Range& a, const Range& b) { return a.lo < b.hi && b.lo < a.hi; }

espace_status check_alias(const Range& out, const Range* ins, int n) {
    for (int i = 0; i < n; ++i)
        if (ins[i].lo != ins[i].hi && overlaps(out, ins[i]))
            return fail(ESPACE_ERR_ALIAS, "output %s overlaps %s", out.name, ins[i].name);
    return ESPACE_OK;
}

espace_status check_workspace(void* ws, size_t have, size_t need) {
    if (need == 0) return ESPACE_OK;
    if (!ws) return fail(ESPACE_ERR_WORKSPACE, "workspace of %zu bytes needed, got NULL", need);
    if (have < need) return fail(ESPACE_ERR_WORKSPACE, "workspace of %zu bytes needed, got %zu", need, have);
    if ((uintptr_t)ws % kWsAlign) return fail(ESPACE_ERR_ALIGN, "workspace not 256-byte aligned");
    return ESPACE_OK;
}

// An MX-FP8 operand: codes [rows][ldq] and scale bytes [rows][lds] covering
// mx_cols(cols) columns, each spanning less than 2^31 bytes.
espace_status check_mx(const char* name, const void* Q, int64_t ldq, const void* S, int64_t lds, int64_t rows,
                       int64_t cols) {
    if (!Q || !S) return fail(ESPACE_ERR_NULL, "%s: codes or scales NULL", name);
    const int64_t cp = mx_cols(cols);
    if (ldq < cp || lds < cp / 32)
        return fail(ESPACE_ERR_SHAPE, "%s: leading dimensions %lld (codes) / %lld (scales) below %lld / %lld", name,
                    (long long)ldq, (long long)lds, (long long)cp, (long long)(cp / 32));
    if (ldq % 16 || lds % 4)
        return fail(ESPACE_ERR_ALIGN, "%s: leading dimensions must be multiples of 16 (codes) and 4 (scales)", name);
    if ((uintptr_t)Q % 16 || (uintptr_t)S % 4)
        return fail(ESPACE_ERR_ALIGN, "%s: codes not 16-byte or scales not 4-byte aligned", name);
    if (rows * ldq >= ((int64_t)1 << 31) || rows * lds >= ((int64_t)1 << 31))
        return fail(ESPACE_ERR_SHAPE, "%s spans 2^31 bytes or more", name);
    return ESPACE_OK;
}

Range byte_range(const char* name, const void* p, int64_t rows, int64_t ld) {
    return Range{name, (uintptr_t)p, (uintptr_t)p + (uintptr_t)(rows * ld)};
}

std::mutex g_dev_mu;
int g_dev_ok[64];   // 0 unknown, 1 gfx950, -1 other

espace_status check_device() {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= 64) return fail(ESPACE_ERR_DEVICE, "device id %d out of range", dev);
    std::lock_guard<std::mutex> lk(g_dev_mu);
    if (g_dev_ok[dev] == 0) {
        hipDeviceProp_t prop;
        e = hipGetDeviceProperties(&prop, dev);
        if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "hipGetDeviceProperties: %s", hipGetErrorString(e));
        g_dev_ok[dev] = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : -1;
    }
    if (g_dev_ok[dev] != 1) return fail(ESPACE_ERR_DEVICE, "device %d is not gfx950", dev);
    return ESPACE_OK;
}

// the calibration GEMM indexes Xt [K][round_up(N, 8)] and the fp32 sums
// [K][round_up(K, 8)] with 32-bit offsets
bool autocorr_fits(int64_t K, int64_t N) {
    const int64_t lim = (int64_t)1 << 31;
    return K * ((N + 7) / 8 * 8) < lim && K * ((K + 7) / 8 * 8) < lim;
}

constexpr int64_t kMaxPcaDim = 32768;
constexpr int64_t kMaxSymDim = 46340;        // K·round_up(K, 8) < 2^31

#define ESPACE_TRY(x)                       \
    do {                                    \
        espace_status _s = (x);             \
        if (_s != ESPACE_OK) return _s;     \
    } while (0)

// ---- launch -----------------------------------------------------------------

// One tiled launch of the plan in g.
hipError_t launch_tiled(const GemmArgs& g, hipStream_t stream) {
    if (g.tile == espace::TILE_256x256_W8T || g.tile == espace::TILE_256x192_W8) {
        // the four-wave kernel; matrices of 2^31 elements or more take the
        // register-staged kernel with 64-bit offsets (plain layouts only)
        const hipError_t e = espace::launch_gemm_tn_bf16_v3(g, stream);
        if (e == hipErrorInvalidValue && !g.a_pairs && !g.c_pairs) return espace::launch_gemm_tn_bf16(g, stream);
        return e;
    }
    return espace::launch_gemm_tn_bf16_v2(g, stream);
}

// a_pairs / c_pairs: A is read, C written in the row-pair layout (GemmArgs);
// only for the tiled plans z_pairs admits
espace_status run_tn(const void* A, int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc,
                     int64_t R, int64_t Cc, int64_t D, espace_dtype dt, void* partial,
                     hipStream_t stream, int a_pairs = 0, int c_pairs = 0) {
    hipError_t e;
    if (dt == ESPACE_F32) {
        e = espace::launch_gemm_tn_f32((const float*)A, lda, (const float*)B, ldb, (float*)C, ldc,
                                       (int)R, (int)Cc, (int)D, stream);
    } else {
        const Plan p = plan_tn_logged(R, Cc, D, dt);
        GemmArgs g;
        g.A = (const uint16_t*)A;
        g.lda = lda;
        g.B = (const uint16_t*)B;
        g.ldb = ldb;
        g.C = C;
        g.ldc = ldc;
        g.R = (int)R;
        g.Cc = (int)Cc;
        g.D = (int)D;
        g.c_f32 = 0;
        g.tile = p.tile;
        g.splits = p.splits;
        g.partial = (float*)partial;
        g.pair = p.pair;
        g.cus = device_cus();
        g.wait = wait_cfg();
        g.a_pairs = a_pairs;
        g.c_pairs = c_pairs;
        if (p.pair) g.epoch = next_epoch();
        if ((a_pairs || c_pairs) && p.kind != KIND_TILED)
            return fail(ESPACE_ERR_HIP, "row-pair layout on a plan that does not take it");
        if (p.kind == KIND_TILED && p.rows1 > 0) {
            // rows [0, rows1), then the rest with its own tile plan (and its
            // own tag for pair states: the workspace serves both)
            g.R = p.rows1;
            e = launch_tiled(g, stream);
            if (e == hipSuccess) {
                // rows1 is a multiple of 256: row pairs start on a pair
                g.A = (const uint16_t*)A + (int64_t)(a_pairs ? p.rows1 / 2 : p.rows1) * lda;
                g.C = (uint16_t*)C + (int64_t)(c_pairs ? p.rows1 / 2 : p.rows1) * ldc;
                g.R = (int)(R - p.rows1);
                g.tile = p.tile2;
                g.splits = p.splits2;
                g.pair = p.pair2;
                if (p.pair2) g.epoch = next_epoch();
                e = launch_tiled(g, stream);
            }
        } else if (p.kind == KIND_SKINNY) {
            e = espace::launch_skinny_tn_bf16(g, stream);
        } else if (p.kind == KIND_GEMV) {
            e = espace::launch_gemv_tn_bf16(g, stream);
        } else if (p.kind == KIND_STREAM) {
            e = espace::launch_stream_tn_bf16(g, stream);
        } else {
            e = launch_tiled(g, stream);
        }
    }
    if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "kernel launch: %s", hipGetErrorString(e));
    return ESPACE_OK;
}

// Whether the layer keeps Z in the row-pair layout (GemmArgs): every 128-byte
// line then holds the 32-deep blocks of two tokens, so the expand GEMM's
// 64-byte half-rows of Z arrive as whole lines, half the L2 requests for
// that operand (the load path of the CUs bounds these GEMMs; measured on the
// Llama2-7B QKV layer with operands rotated through HBM: 196.7 -> 191.0 µs,
// the GPT3-22B FFN-up layer at L = 2458: 1180 -> 1117 µs).
// Taken for prefill when the projection is tiled (any depth split; its
// output is written by the GEMM kernel, the pair combine or the reduction
// pass) and every launch of the expand GEMM is a single-range launch of the
// four-wave kernel.
bool z_pairs(int64_t N, int64_t L, int64_t K, int64_t M, int64_t ldx, int64_t ldp, int64_t ldwf, int64_t ldy,
             espace_dtype dt) {
    if (dt != ESPACE_BF16 || N <= 32) return false;
    const Plan a = plan_tn(N, L, K, dt);
    const Plan b = plan_tn(N, M, L, dt);
    auto v3_single = [](int tile, int splits) {
        return splits == 1 && (tile == espace::TILE_256x256_W8T || tile == espace::TILE_256x192_W8);
    };
    if (a.kind != KIND_TILED || b.kind != KIND_TILED) return false;
    if (!v3_single(b.tile, b.splits) || (b.rows1 > 0 && !v3_single(b.tile2, b.splits2))) return false;
    // the kernels' 32-bit offsets (the register-staged fallback keeps plain layouts)
    const int64_t lim = (int64_t)1 << 31;
    const int64_t ldzp = 2 * z_ld(L, N, dt);
    return N * ldx < lim && L * ldp < lim && N * ldzp < lim && M * ldwf < lim && N * ldy < lim;
}

// The layer's launches after validation: Z and the partial sums in
// `workspace` (ws_bytes(ESPACE_OP_PROJECTED_LINEAR, ...) bytes).
espace_status projected_linear_launch(const void* X, int64_t ldx, const void* Pt, int64_t ldp, const void* Wf,
                                      int64_t ldwf, void* Y, int64_t ldy, int64_t M, int64_t K, int64_t L,
                                      int64_t N, espace_dtype dt, void* workspace, hipStream_t stream) {
    void* Z = workspace;
    void* partial = (char*)workspace + z_bytes(N, L, dt);
    if (z_pairs(N, L, K, M, ldx, ldp, ldwf, ldy, dt)) {
        const int64_t ldzp = 2 * z_ld(L, N, dt);   // elements per row pair
        ESPACE_TRY(run_tn(X, ldx, Pt, ldp, Z, ldzp, N, L, K, dt, partial, stream, 0, 1));
        ESPACE_TRY(run_tn(Z, ldzp, Wf, ldwf, Y, ldy, N, M, L, dt, partial, stream, 1, 0));
        return ESPACE_OK;
    }
    const int64_t ldz = z_ld(L, N, dt);
    ESPACE_TRY(run_tn(X, ldx, Pt, ldp, Z, ldz, N, L, K, dt, partial, stream));
    ESPACE_TRY(run_tn(Z, ldz, Wf, ldwf, Y, ldy, N, M, L, dt, partial, stream));
    return ESPACE_OK;
}

// Device address of this device's copy of `scratch`, looked up once per
// device with that device current (the array's name in host code is a
// host-side stand-in, never passed to a kernel).
espace_status noalloc_scratch(void** out) {
    static std::mutex mu;
    static void* ptr[64] = {nullptr};
    int dev = 0;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= 64) return fail(ESPACE_ERR_DEVICE, "device id %d out of range", dev);
    std::lock_guard<std::mutex> lk(mu);
    if (!ptr[dev]) {
        void* p = nullptr;
        const hipError_t g = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (g != hipSuccess || !p)
            return fail(ESPACE_ERR_HIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(g));
        if ((uintptr_t)p % kWsAlign) return fail(ESPACE_ERR_ALIGN, "scratch not 256-byte aligned");
        ptr[dev] = p;
    }
    *out = ptr[dev];
    return ESPACE_OK;
}

}  // namespace

// The MX-FP8 products after validation.
// z_pairs: Z's codes in row pairs (ldzq bytes per pair)
espace_status mx_project_launch(const void* Ptq, int64_t ldpq, const void* Pts, int64_t ldps, const void* Xq,
                                int64_t ldxq, const void* Xs, int64_t ldxs, void* Zq, int64_t ldzq, void* Zs,
                                int64_t ldzs, int64_t K, int64_t L, int64_t N, hipStream_t stream,
                                int z_pairs = 0) {
    espace::MxGemmArgs a{};
    a.out_pairs = z_pairs;
    a.T = (const uint8_t*)Xq; a.ldt = ldxq; a.Ts = (const uint8_t*)Xs; a.ldts = ldxs;
    a.W = (const uint8_t*)Ptq; a.ldw = ldpq; a.Ws = (const uint8_t*)Pts; a.ldws = ldps;
    a.out = Zq; a.ldo = ldzq; a.outs = (uint8_t*)Zs; a.ldos = ldzs;
    a.R = (int)N; a.C = (int)L; a.D = (int)K; a.cpad = (int)mx_cols(L);
    const hipError_t e = espace::launch_gemm_mx(a, 1, device_cus(), stream);
    if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "MX-FP8 projection launch: %s", hipGetErrorString(e));
    return ESPACE_OK;
}

espace_status mx_expand_launch(const void* Zq, int64_t ldzq, const void* Zs, int64_t ldzs, const void* Wfq,
                               int64_t ldwq, const void* Wfs, int64_t ldws, void* Y, int64_t ldy, int64_t M,
                               int64_t L, int64_t N, hipStream_t stream, int z_pairs = 0) {
    espace::MxGemmArgs a{};
    a.t_pairs = z_pairs;
    a.T = (const uint8_t*)Zq; a.ldt = ldzq; a.Ts = (const uint8_t*)Zs; a.ldts = ldzs;
    a.W = (const uint8_t*)Wfq; a.ldw = ldwq; a.Ws = (const uint8_t*)Wfs; a.ldws = ldws;
    a.out = Y; a.ldo = ldy;
    a.R = (int)N; a.C = (int)M; a.D = (int)L; a.cpad = (int)mx_cols(M);
    const hipError_t e = espace::launch_gemm_mx(a, 0, device_cus(), stream);
    if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "MX-FP8 expansion launch: %s", hipGetErrorString(e));
    return ESPACE_OK;
}


extern "C" {

int espace_abi_version(void) { return ESPACE_ABI_VERSION; }

espace_status espace_set_wait_limit(unsigned spins) {
    g_wait_spins.store(spins ? spins : kDefaultWaitSpins, std::memory_order_relaxed);
    return ok();
}

espace_status espace_wait_timeouts(unsigned long long* count) {
    if (!count) return fail(ESPACE_ERR_NULL, "count is NULL");
    ESPACE_TRY(check_device());
    unsigned long long* p = timeout_counter();
    if (!p) return fail(ESPACE_ERR_HIP, "device counter not available");
    const hipError_t e = hipMemcpy(count, p, sizeof *count, hipMemcpyDeviceToHost);
    if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "reading the counter: %s", hipGetErrorString(e));
    return ok();
}

const char* espace_last_error(void) { return g_last_error.c_str(); }

const char* espace_status_string(espace_status s) {
    switch (s) {
        case ESPACE_OK: return "ok";
        case ESPACE_ERR_NULL: return "null pointer";
        case ESPACE_ERR_SHAPE: return "invalid shape";
        case ESPACE_ERR_ALIGN: return "misaligned pointer or leading dimension";
        case ESPACE_ERR_DTYPE: return "invalid dtype";
        case ESPACE_ERR_ALIAS: return "output overlaps an input";
        case ESPACE_ERR_WORKSPACE: return "workspace missing or too small";
        case ESPACE_ERR_HIP: return "HIP runtime error";
        case ESPACE_ERR_DEVICE: return "unsupported device";
    }
    return "unknown status";
}

size_t espace_workspace_bytes(espace_op op, int64_t M, int64_t K, int64_t L, int64_t N,
                              espace_dtype dt) {
    if (dt != ESPACE_F32 && dt != ESPACE_BF16) return SIZE_MAX;
    if (op == ESPACE_OP_AUTOCORR) {
        if (K < 1 || N < 0 || K > kMaxDim || N > kMaxDim || !autocorr_fits(K, N)) return SIZE_MAX;
        return ws_bytes(op, 0, K, 0, N, dt);
    }
    if (op == ESPACE_OP_PCA) {
        if (K < 1 || K > kMaxPcaDim || L < 1 || L > K) return SIZE_MAX;
        return ws_bytes(op, 0, K, L, 0, dt);
    }
    if (op == ESPACE_OP_SYMPRODUCT) {
        if (K < 1 || K > kMaxSymDim) return SIZE_MAX;
        return ws_bytes(op, 0, K, 0, 0, dt);
    }
    if (op == ESPACE_OP_BACKWARD || op == ESPACE_OP_DENSE_BACKWARD) {
        const bool hl = op == ESPACE_OP_BACKWARD;
        if (M < 0 || N < 0 || K < 1 || M > kMaxDim || N > kMaxDim || K > kMaxDim) return SIZE_MAX;
        if (hl && (L < 1 || L > K)) return SIZE_MAX;
        return ws_bytes(op, M, K, hl ? L : 0, N, dt);
    }
    if (op == ESPACE_OP_PROJECTED_LINEAR_MXFP8) {
        if (M < 0 || N < 0 || K < 1 || M > kMaxDim || N > kMaxDim || K > kMaxDim || L < 1 || L > K)
            return SIZE_MAX;
        return mx_ws_bytes(M, L, N);
    }
    const bool has_L = op != ESPACE_OP_DENSE;
    int64_t Kc = K;
    if (op == ESPACE_OP_EXPAND) Kc = L;       // expand has no K; L bounds itself
    if (M < 0 || N < 0 || Kc < 1 || M > kMaxDim || N > kMaxDim || Kc > kMaxDim) return SIZE_MAX;
    if (has_L && (L < 1 || L > Kc)) return SIZE_MAX;
    if (op < ESPACE_OP_FOLD || op > ESPACE_OP_DENSE) return SIZE_MAX;
    return ws_bytes(op, M, K, L, N, dt);
}

espace_status espace_fold_weights(const void* W, int64_t ldw, const void* Pt, int64_t ldp,
                                  void* Wf, int64_t ldwf, int64_t M, int64_t K, int64_t L,
                                  espace_dtype dt, void* workspace, size_t workspace_bytes,
                                  hipStream_t stream) {
    ESPACE_TRY(check_dtype(dt));
    ESPACE_TRY(check_dims(M, K, L, 0, true));
    if (M == 0) return ok();
    ESPACE_TRY(check_mat("W", W, M, K, ldw, dt));
    ESPACE_TRY(check_mat("Pt", Pt, L, K, ldp, dt));
    ESPACE_TRY(check_mat("Wf", Wf, M, L, ldwf, dt));
    const size_t need = ws_bytes(ESPACE_OP_FOLD, M, K, L, 0, dt);
    ESPACE_TRY(check_workspace(workspace, workspace_bytes, need));
    const Range ins[] = {mat_range("W", W, M, ldw, dt), mat_range("Pt", Pt, L, ldp, dt),
                         Range{"workspace", (uintptr_t)workspace, (uintptr_t)workspace + (need ? workspace_bytes : 0)}};
    ESPACE_TRY(check_alias(mat_range("Wf", Wf, M, ldwf, dt), ins, 3));
    ESPACE_TRY(check_device());
    ESPACE_TRY(run_tn(W, ldw, Pt, ldp, Wf, ldwf, M, L, K, dt, workspace, stream));
    return ok();
}

espace_status espace_project(const void* Pt, int64_t ldp, const void* X, int64_t ldx, void* Z,
                             int64_t ldz, int64_t K, int64_t L, int64_t N, espace_dtype dt,
                             void* workspace, size_t workspace_bytes, hipStream_t stream) {
    ESPACE_TRY(check_dtype(dt));
    ESPACE_TRY(check_dims(0, K, L, N, true));
    if (N == 0) return ok();
    ESPACE_TRY(check_mat("Pt", Pt, L, K, ldp, dt));
    ESPACE_TRY(check_mat("X", X, N, K, ldx, dt));
    ESPACE_TRY(check_mat("Z", Z, N, L, ldz, dt));
    const size_t need = ws_bytes(ESPACE_OP_PROJECT, 0, K, L, N, dt);
    ESPACE_TRY(check_workspace(workspace, workspace_bytes, need));
    const Range ins[] = {mat_range("Pt", Pt, L, ldp, dt), mat_range("X", X, N, ldx, dt),
                         Range{"workspace", (uintptr_t)workspace, (uintptr_t)workspace + (need ? workspace_bytes : 0)}};
    ESPACE_TRY(check_alias(mat_range("Z", Z, N, ldz, dt), ins, 3));
    ESPACE_TRY(check_device());
    ESPACE_TRY(run_tn(X, ldx, Pt, ldp, Z, ldz, N, L, K, dt, workspace, stream));
    return ok();
}

espace_status espace_expand(const void* Z, int64_t ldz, const void* Wf, int64_t ldwf, void* Y,
                            int64_t ldy, int64_t M, int64_t L, int64_t N, espace_dtype dt,
                            void* workspace, size_t workspace_bytes, hipStream_t stream) {
    ESPACE_TRY(check_dtype(dt));
    ESPACE_TRY(check_dims(M, L, L, N, true));
    if (M == 0 || N == 0) return ok();
    ESPACE_TRY(check_mat("Z", Z, N, L, ldz, dt));
    ESPACE_TRY(check_mat("Wf", Wf, M, L, ldwf, dt));
    ESPACE_TRY(check_mat("Y", Y, N, M, ldy, dt));
    const size_t need = ws_bytes(ESPACE_OP_EXPAND, M, L, L, N, dt);
    ESPACE_TRY(check_workspace(workspace, workspace_bytes, need));
    const Range ins[] = {mat_range("Z", Z, N, ldz, dt), mat_range("Wf", Wf, M, ldwf, dt),
                         Range{"workspace", (uintptr_t)workspace, (uintptr_t)workspace + (need ? workspace_bytes : 0)}};
    ESPACE_TRY(check_alias(mat_range("Y", Y, N, ldy, dt), ins, 3));
    ESPACE_TRY(check_device());
    ESPACE_TRY(run_tn(Z, ldz, Wf, ldwf, Y, ldy, N, M, L, dt, workspace, stream));
    return ok();
}

espace_status espace_projected_linear(const void* X, int64_t ldx, const void* Pt, int64_t ldp,
                                      const void* Wf, int64_t ldwf, void* Y, int64_t ldy,
                                      int64_t M, int64_t K, int64_t L, int64_t N, espace_dtype dt,
                                      void* workspace, size_t workspace_bytes, hipStream_t stream) {
    ESPACE_TRY(check_dtype(dt));
    ESPACE_TRY(check_dims(M, K, L, N, true));
    if (M == 0 || N == 0) return ok();
    ESPACE_TRY(check_mat("X", X, N, K, ldx, dt));
    ESPACE_TRY(check_mat("Pt", Pt, L, K, ldp, dt));
    ESPACE_TRY(check_mat("Wf", Wf, M, L, ldwf, dt));
    ESPACE_TRY(check_mat("Y", Y, N, M, ldy, dt));
    const size_t need = ws_bytes(ESPACE_OP_PROJECTED_LINEAR, M, K, L, N, dt);
    ESPACE_TRY(check_workspace(workspace, workspace_bytes, need));
    const Range ws{"workspace", (uintptr_t)workspace, (uintptr_t)workspace + workspace_bytes};
    const Range ins[] = {mat_range("X", X, N, ldx, dt), mat_range("Pt", Pt, L, ldp, dt),
                         mat_range("Wf", Wf, M, ldwf, dt), ws};
    ESPACE_TRY(check_alias(mat_range("Y", Y, N, ldy, dt), ins, 4));
    // the workspace holds Z and must not overlap the inputs either
    const Range wsr{"workspace", ws.lo, ws.lo + need};
    ESPACE_TRY(check_alias(wsr, ins, 3));
    ESPACE_TRY(check_device());
    ESPACE_TRY(projected_linear_launch(X, ldx, Pt, ldp, Wf, ldwf, Y, ldy, M, K, L, N, dt, workspace, stream));
    return ok();
}

espace_status espace_projected_linear_noalloc(const void* X, int64_t ldx, const void* Pt, int64_t ldp,
                                              const void* Wf, int64_t ldwf, void* Y, int64_t ldy,
                                              int64_t M, int64_t K, int64_t L, int64_t N, espace_dtype dt,
                                              hipStream_t stream) {
    ESPACE_TRY(check_dtype(dt));
    ESPACE_TRY(check_dims(M, K, L, N, true));
    if (M == 0 || N == 0) return ok();
    ESPACE_TRY(check_mat("X", X, N, K, ldx, dt));
    ESPACE_TRY(check_mat("Pt", Pt, L, K, ldp, dt));
    ESPACE_TRY(check_mat("Wf", Wf, M, L, ldwf, dt));
    ESPACE_TRY(check_mat("Y", Y, N, M, ldy, dt));
    const size_t need = ws_bytes(ESPACE_OP_PROJECTED_LINEAR, M, K, L, N, dt);
    if (need > (size_t)ESPACE_NOALLOC_SCRATCH_BYTES)
        return fail(ESPACE_ERR_WORKSPACE,
                    "these sizes need %zu bytes of scratch, above the %zu bytes the allocation-free call holds "
                    "(use espace_projected_linear with a workspace)",
                    need, (size_t)ESPACE_NOALLOC_SCRATCH_BYTES);
    const Range ins[] = {mat_range("X", X, N, ldx, dt), mat_range("Pt", Pt, L, ldp, dt),
                         mat_range("Wf", Wf, M, ldwf, dt)};
    ESPACE_TRY(check_alias(mat_range("Y", Y, N, ldy, dt), ins, 3));
    ESPACE_TRY(check_device());
    void* ws = nullptr;
    ESPACE_TRY(noalloc_scratch(&ws));
    ESPACE_TRY(projected_linear_launch(X, ldx, Pt, ldp, Wf, ldwf, Y, ldy, M, K, L, N, dt, ws, stream));
    return ok();
}

espace_status espace_dense_linear(const void* X, int64_t ldx, const void* W, int64_t ldw, void* Y,
                                  int64_t ldy, int64_t M, int64_t K, int64_t N, espace_dtype dt,
                                  void* workspace, size_t workspace_bytes, hipStream_t stream) {
    ESPACE_TRY(check_dtype(dt));
    ESPACE_TRY(check_dims(M, K, 1, N, false));
    if (M == 0 || N == 0) return ok();
    ESPACE_TRY(check_mat("X", X, N, K, ldx, dt));
    ESPACE_TRY(check_mat("W", W, M, K, ldw, dt));
    ESPACE_TRY(check_mat("Y", Y, N, M, ldy, dt));
    const size_t need = ws_bytes(ESPACE_OP_DENSE, M, K, 0, N, dt);
    ESPACE_TRY(check_workspace(workspace, workspace_bytes, need));
    const Range ins[] = {mat_range("X", X, N, ldx, dt), mat_range("W", W, M, ldw, dt),
                         Range{"workspace", (uintptr_t)workspace, (uintptr_t)workspace + (need ? workspace_bytes : 0)}};
    ESPACE_TRY(check_alias(mat_range("Y", Y, N, ldy, dt), ins, 3));
    ESPACE_TRY(check_device());
    ESPACE_TRY(run_tn(X, ldx, W, ldw, Y, ldy, N, M, K, dt, workspace, stream));
    return ok();
}

espace_status espace_projected_linear_backward(const void* dY, int64_t lddy, const void* Z, int64_t ldz,
                                               const void* Pt, int64_t ldp, const void* Wf, int64_t ldwf, void* dX,
                                               int64_t lddx, void* dW, int64_t lddw, int64_t M, int64_t K,
                                               int64_t L, int64_t N, espace_dtype dt, void* workspace,
                                               size_t workspace_bytes, hipStream_t stream) {
    ESPACE_TRY(check_dtype(dt));
    ESPACE_TRY(check_dims(M, K, L, N, true));
    if (M == 0 || N == 0 || (!dX && !dW)) return ok();
    ESPACE_TRY(check_mat("dY", dY, N, M, lddy, dt));
    ESPACE_TRY(check_mat("Pt", Pt, L, K, ldp, dt));
    if (dX) {
        ESPACE_TRY(check_mat("Wf", Wf, M, L, ldwf, dt));
        ESPACE_TRY(check_mat("dX", dX, N, K, lddx, dt));
    }
    if (dW) {
        ESPACE_TRY(check_mat("Z", Z, N, L, ldz, dt));
        ESPACE_TRY(check_mat("dW", dW, M, K, lddw, dt));
    }
    const BwdLayout b = bwd_layout(M, K, L, N, dt);
    ESPACE_TRY(check_workspace(workspace, workspace_bytes, b.total));
    const Range ws{"workspace", (uintptr_t)workspace, (uintptr_t)workspace + workspace_bytes};
    const Range ins[] = {mat_range("dY", dY, N, lddy, dt), mat_range("Pt", Pt, L, ldp, dt),
                         dX ? mat_range("Wf", Wf, M, ldwf, dt) : Range{"Wf", 0, 0},
                         dW ? mat_range("Z", Z, N, ldz, dt) : Range{"Z", 0, 0}, ws};
    if (dX) ESPACE_TRY(check_alias(mat_range("dX", dX, N, lddx, dt), ins, 5));
    if (dW) ESPACE_TRY(check_alias(mat_range("dW", dW, M, lddw, dt), ins, 5));
    if (dX && dW) {
        const Range o[] = {mat_range("dX", dX, N, lddx, dt)};
        ESPACE_TRY(check_alias(mat_range("dW", dW, M, lddw, dt), o, 1));
    }
    ESPACE_TRY(check_device());
    unsigned char* w = static_cast<unsigned char*>(workspace);
    const bool f32 = dt == ESPACE_F32;
    void* P = w + b.b;
    void* part = w + b.part;
    hipError_t e = espace::launch_transpose(Pt, ldp, (int)L, (int)K, P, ld8(L), f32, stream);
    if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "transpose: %s", hipGetErrorString(e));
    if (dX) {
        // dZ = dY·Wf (reduced over M), dX = dZ·Pt (reduced over L)
        void* WfT = w + b.a;
        void* dZ = w + b.e;
        e = espace::launch_transpose(Wf, ldwf, (int)M, (int)L, WfT, ld8(M), f32, stream);
        if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "transpose: %s", hipGetErrorString(e));
        ESPACE_TRY(run_tn(dY, lddy, WfT, ld8(M), dZ, ld8(L), N, L, M, dt, part, stream));
        ESPACE_TRY(run_tn(dZ, ld8(L), P, ld8(L), dX, lddx, N, K, L, dt, part, stream));
    }
    if (dW) {
        // G = dYᵀ·Z (reduced over N), dW = G·Pt (reduced over L)
        void* dYT = w + b.c;
        void* ZT = w + b.d;
        void* G = w + b.f;
        e = espace::launch_transpose(dY, lddy, (int)N, (int)M, dYT, ld8(N), f32, stream);
        if (e == hipSuccess) e = espace::launch_transpose(Z, ldz, (int)N, (int)L, ZT, ld8(N), f32, stream);
        if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "transpose: %s", hipGetErrorString(e));
        ESPACE_TRY(run_tn(dYT, ld8(N), ZT, ld8(N), G, ld8(L), M, L, N, dt, part, stream));
        ESPACE_TRY(run_tn(G, ld8(L), P, ld8(L), dW, lddw, M, K, L, dt, part, stream));
    }
    return ok();
}

espace_status espace_dense_linear_backward(const void* dY, int64_t lddy, const void* X, int64_t ldx, const void* W,
                                           int64_t ldw, void* dX, int64_t lddx, void* dW, int64_t lddw, int64_t M,
                                           int64_t K, int64_t N, espace_dtype dt, void* workspace,
                                           size_t workspace_bytes, hipStream_t stream) {
    ESPACE_TRY(check_dtype(dt));
    ESPACE_TRY(check_dims(M, K, 1, N, false));
    if (M == 0 || N == 0 || (!dX && !dW)) return ok();
    ESPACE_TRY(check_mat("dY", dY, N, M, lddy, dt));
    if (dX) {
        ESPACE_TRY(check_mat("W", W, M, K, ldw, dt));
        ESPACE_TRY(check_mat("dX", dX, N, K, lddx, dt));
    }
    if (dW) {
        ESPACE_TRY(check_mat("X", X, N, K, ldx, dt));
        ESPACE_TRY(check_mat("dW", dW, M, K, lddw, dt));
    }
    const BwdLayout b = dense_bwd_layout(M, K, N, dt);
    ESPACE_TRY(check_workspace(workspace, workspace_bytes, b.total));
    const Range ws{"workspace", (uintptr_t)workspace, (uintptr_t)workspace + workspace_bytes};
    const Range ins[] = {mat_range("dY", dY, N, lddy, dt), dX ? mat_range("W", W, M, ldw, dt) : Range{"W", 0, 0},
                         dW ? mat_range("X", X, N, ldx, dt) : Range{"X", 0, 0}, ws};
    if (dX) ESPACE_TRY(check_alias(mat_range("dX", dX, N, lddx, dt), ins, 4));
    if (dW) ESPACE_TRY(check_alias(mat_range("dW", dW, M, lddw, dt), ins, 4));
    if (dX && dW) {
        const Range o[] = {mat_range("dX", dX, N, lddx, dt)};
        ESPACE_TRY(check_alias(mat_range("dW", dW, M, lddw, dt), o, 1));
    }
    ESPACE_TRY(check_device());
    unsigned char* w = static_cast<unsigned char*>(workspace);
    const bool f32 = dt == ESPACE_F32;
    void* part = w + b.part;
    hipError_t e;
    if (dX) {
        // dX = dY·W (reduced over M)
        void* WT = w + b.a;
        e = espace::launch_transpose(W, ldw, (int)M, (int)K, WT, ld8(M), f32, stream);
        if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "transpose: %s", hipGetErrorString(e));
        ESPACE_TRY(run_tn(dY, lddy, WT, ld8(M), dX, lddx, N, K, M, dt, part, stream));
    }
    if (dW) {
        // dW = dYᵀ·X (reduced over N)
        void* dYT = w + b.c;
        void* XT = w + b.d;
        e = espace::launch_transpose(dY, lddy, (int)N, (int)M, dYT, ld8(N), f32, stream);
        if (e == hipSuccess) e = espace::launch_transpose(X, ldx, (int)N, (int)K, XT, ld8(N), f32, stream);
        if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "transpose: %s", hipGetErrorString(e));
        ESPACE_TRY(run_tn(dYT, ld8(N), XT, ld8(N), dW, lddw, M, K, N, dt, part, stream));
    }
    return ok();
}

espace_status espace_autocorrelation_update(const void* X, int64_t ldx, float* C, int64_t ldc, int64_t K,
                                            int64_t N, int normalize, float alpha, espace_dtype dt,
                                            void* workspace, size_t workspace_bytes, hipStream_t stream) {
    ESPACE_TRY(check_dtype(dt));
    ESPACE_TRY(check_dims(0, K, 1, N, false));
    if (N == 0) return ok();
    if (!autocorr_fits(K, N))
        return fail(ESPACE_ERR_SHAPE, "K=%lld, N=%lld too large for one update (split the batch)", (long long)K,
                    (long long)N);
    ESPACE_TRY(check_mat("X", X, N, K, ldx, dt));
    ESPACE_TRY(check_mat("C", C, K, K, ldc, ESPACE_F32));
    const size_t need = ws_bytes(ESPACE_OP_AUTOCORR, 0, K, 0, N, dt);
    ESPACE_TRY(check_workspace(workspace, workspace_bytes, need));
    const Range ins[] = {mat_range("X", X, N, ldx, dt),
                         Range{"workspace", (uintptr_t)workspace, (uintptr_t)workspace + workspace_bytes}};
    ESPACE_TRY(check_alias(mat_range("C", C, K, ldc, ESPACE_F32), ins, 2));
    ESPACE_TRY(check_device());
    const hipError_t e = espace::launch_autocorr_update(X, ldx, (int)N, (int)K, dt == ESPACE_F32, normalize != 0,
                                                        alpha, C, ldc, workspace, stream);
    if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "autocorrelation update: %s", hipGetErrorString(e));
    return ok();
}

espace_status espace_symmetrized_product(const float* A, int64_t lda, const float* B, int64_t ldb, float* C,
                                         int64_t ldc, int64_t K, float alpha, float beta, void* workspace,
                                         size_t workspace_bytes, hipStream_t stream) {
    ESPACE_TRY(check_dims(0, K, 1, 0, false));
    if (K > kMaxSymDim) return fail(ESPACE_ERR_SHAPE, "K=%lld above %lld", (long long)K, (long long)kMaxSymDim);
    ESPACE_TRY(check_mat("A", A, K, K, lda, ESPACE_F32));
    ESPACE_TRY(check_mat("B", B, K, K, ldb, ESPACE_F32));
    ESPACE_TRY(check_mat("C", C, K, K, ldc, ESPACE_F32));
    const size_t need = ws_bytes(ESPACE_OP_SYMPRODUCT, 0, K, 0, 0, ESPACE_F32);
    ESPACE_TRY(check_workspace(workspace, workspace_bytes, need));
    const Range ins[] = {mat_range("A", A, K, lda, ESPACE_F32), mat_range("B", B, K, ldb, ESPACE_F32),
                         Range{"workspace", (uintptr_t)workspace, (uintptr_t)workspace + workspace_bytes}};
    ESPACE_TRY(check_alias(mat_range("C", C, K, ldc, ESPACE_F32), ins, 3));
    ESPACE_TRY(check_device());
    const hipError_t e =
        espace::launch_symmetrized_product(A, lda, B, ldb, C, ldc, (int)K, alpha, beta, workspace, stream);
    if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "symmetrized product: %s", hipGetErrorString(e));
    return ok();
}

espace_status espace_principal_components(const float* C, int64_t ldc, void* Pt, int64_t ldp, float* eigenvalues,
                                          int* info, int64_t K, int64_t L, int by_magnitude, espace_dtype dt,
                                          void* workspace, size_t workspace_bytes, hipStream_t stream) {
    ESPACE_TRY(check_dtype(dt));
    ESPACE_TRY(check_dims(0, K, L, 0, true));
    if (K > kMaxPcaDim) return fail(ESPACE_ERR_SHAPE, "K=%lld above %lld", (long long)K, (long long)kMaxPcaDim);
    ESPACE_TRY(check_mat("C", C, K, K, ldc, ESPACE_F32));
    ESPACE_TRY(check_mat("Pt", Pt, L, K, ldp, dt));
    if ((uintptr_t)eigenvalues % 4) return fail(ESPACE_ERR_ALIGN, "eigenvalues: pointer not 4-byte aligned");
    if ((uintptr_t)info % 4) return fail(ESPACE_ERR_ALIGN, "info: pointer not 4-byte aligned");
    const size_t need = ws_bytes(ESPACE_OP_PCA, 0, K, L, 0, dt);
    ESPACE_TRY(check_workspace(workspace, workspace_bytes, need));
    const Range ws{"workspace", (uintptr_t)workspace, (uintptr_t)workspace + workspace_bytes};
    const Range cr = mat_range("C", C, K, ldc, ESPACE_F32);
    const Range pr = mat_range("Pt", Pt, L, ldp, dt);
    const Range er{"eigenvalues", (uintptr_t)eigenvalues, (uintptr_t)eigenvalues + (eigenvalues ? K * 4 : 0)};
    const Range ir{"info", (uintptr_t)info, (uintptr_t)info + (info ? 4 : 0)};
    const Range for_pt[] = {cr, ws, er, ir};
    ESPACE_TRY(check_alias(pr, for_pt, 4));
    if (eigenvalues) {
        const Range for_ev[] = {cr, ws, ir};
        ESPACE_TRY(check_alias(er, for_ev, 3));
    }
    if (info) {
        const Range for_info[] = {cr, ws};
        ESPACE_TRY(check_alias(ir, for_info, 2));
    }
    ESPACE_TRY(check_device());
    if (!espace::pca_available()) return fail(ESPACE_ERR_HIP, "rocSOLVER (librocsolver.so.0) could not be loaded");
    const hipError_t e = espace::launch_principal_components(C, ldc, (int)K, (int)L, by_magnitude != 0, Pt, ldp,
                                                             dt == ESPACE_F32, eigenvalues, info, workspace, stream);
    if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "principal components: %s", hipGetErrorString(e));
    return ok();
}

espace_status espace_quantize_mxfp8(const void* A, int64_t lda, int64_t R, int64_t C, void* Q, int64_t ldq, void* S,
                                    int64_t lds, hipStream_t stream) {
    if (R < 0 || C < 1 || R > kMaxDim || C > kMaxDim)
        return fail(ESPACE_ERR_SHAPE, "need R >= 0 and C >= 1 (R=%lld, C=%lld)", (long long)R, (long long)C);
    if (R == 0) return ok();
    ESPACE_TRY(check_mat("A", A, R, C, lda, ESPACE_BF16));
    ESPACE_TRY(check_mx("Q/S", Q, ldq, S, lds, R, C));
    const Range ar = mat_range("A", A, R, lda, ESPACE_BF16);
    const Range qr = byte_range("Q", Q, R, ldq), sr = byte_range("S", S, R, lds);
    const Range for_q[] = {ar, sr};
    ESPACE_TRY(check_alias(qr, for_q, 2));
    ESPACE_TRY(check_alias(sr, &ar, 1));
    ESPACE_TRY(check_device());
    const hipError_t e = espace::launch_mx_quantize((const uint16_t*)A, lda, (int)R, (int)C, (uint8_t*)Q, ldq,
                                                    (uint8_t*)S, lds, stream);
    if (e != hipSuccess) return fail(ESPACE_ERR_HIP, "MX-FP8 quantisation launch: %s", hipGetErrorString(e));
    return ok();
}

espace_status espace_project_mxfp8(const void* Ptq, int64_t ldpq, const void* Pts, int64_t ldps, const void* Xq,
                                   int64_t ldxq, const void* Xs, int64_t ldxs, void* Zq, int64_t ldzq, void* Zs,
                                   int64_t ldzs, int64_t K, int64_t L, int64_t N, hipStream_t stream) {
    ESPACE_TRY(check_dims(0, K, L, N, true));
    if (N == 0) return ok();
    ESPACE_TRY(check_mx("Pt", Ptq, ldpq, Pts, ldps, L, K));
    ESPACE_TRY(check_mx("X", Xq, ldxq, Xs, ldxs, N, K));
    ESPACE_TRY(check_mx("Z", Zq, ldzq, Zs, ldzs, N, L));
    const Range ins[] = {byte_range("Pt codes", Ptq, L, ldpq), byte_range("Pt scales", Pts, L, ldps),
                         byte_range("X codes", Xq, N, ldxq), byte_range("X scales", Xs, N, ldxs),
                         byte_range("Z scales", Zs, N, ldzs)};
    ESPACE_TRY(check_alias(byte_range("Z codes", Zq, N, ldzq), ins, 5));
    ESPACE_TRY(check_alias(byte_range("Z scales", Zs, N, ldzs), ins, 4));
    ESPACE_TRY(check_device());
    ESPACE_TRY(mx_project_launch(Ptq, ldpq, Pts, ldps, Xq, ldxq, Xs, ldxs, Zq, ldzq, Zs, ldzs, K, L, N, stream));
    return ok();
}

espace_status espace_expand_mxfp8(const void* Zq, int64_t ldzq, const void* Zs, int64_t ldzs, const void* Wfq,
                                  int64_t ldwq, const void* Wfs, int64_t ldws, void* Y, int64_t ldy, int64_t M,
                                  int64_t L, int64_t N, hipStream_t stream) {
    ESPACE_TRY(check_dims(M, L, L, N, true));
    if (M == 0 || N == 0) return ok();
    ESPACE_TRY(check_mx("Z", Zq, ldzq, Zs, ldzs, N, L));
    ESPACE_TRY(check_mx("Wf", Wfq, ldwq, Wfs, ldws, M, L));
    ESPACE_TRY(check_mat("Y", Y, N, M, ldy, ESPACE_BF16));
    const Range ins[] = {byte_range("Z codes", Zq, N, ldzq), byte_range("Z scales", Zs, N, ldzs),
                         byte_range("Wf codes", Wfq, M, ldwq), byte_range("Wf scales", Wfs, M, ldws)};
    ESPACE_TRY(check_alias(mat_range("Y", Y, N, ldy, ESPACE_BF16), ins, 4));
    ESPACE_TRY(check_device());
    ESPACE_TRY(mx_expand_launch(Zq, ldzq, Zs, ldzs, Wfq, ldwq, Wfs, ldws, Y, ldy, M, L, N, stream));
    return ok();
}

espace_status espace_projected_linear_mxfp8(const void* Xq, int64_t ldxq, const void* Xs, int64_t ldxs,
                                            const void* Ptq, int64_t ldpq, const void* Pts, int64_t ldps,
                                            const void* Wfq, int64_t ldwq, const void* Wfs, int64_t ldws, void* Y,
                                            int64_t ldy, int64_t M, int64_t K, int64_t L, int64_t N, void* workspace,
                                            size_t workspace_bytes, hipStream_t stream) {
    ESPACE_TRY(check_dims(M, K, L, N, true));
    if (M == 0 || N == 0) return ok();
    ESPACE_TRY(check_mx("X", Xq, ldxq, Xs, ldxs, N, K));
    ESPACE_TRY(check_mx("Pt", Ptq, ldpq, Pts, ldps, L, K));
    ESPACE_TRY(check_mx("Wf", Wfq, ldwq, Wfs, ldws, M, L));
    ESPACE_TRY(check_mat("Y", Y, N, M, ldy, ESPACE_BF16));
    const size_t need = mx_ws_bytes(M, L, N);
    ESPACE_TRY(check_workspace(workspace, workspace_bytes, need));
    const Range ins[] = {byte_range("X codes", Xq, N, ldxq), byte_range("X scales", Xs, N, ldxs),
                         byte_range("Pt codes", Ptq, L, ldpq), byte_range("Pt scales", Pts, L, ldps),
                         byte_range("Wf codes", Wfq, M, ldwq), byte_range("Wf scales", Wfs, M, ldws),
                         Range{"workspace", (uintptr_t)workspace, (uintptr_t)workspace + workspace_bytes}};
    ESPACE_TRY(check_alias(mat_range("Y", Y, N, ldy, ESPACE_BF16), ins, 7));
    ESPACE_TRY(check_alias(ins[6], ins, 6));
    ESPACE_TRY(check_device());
    // Z's codes in row pairs (2 mx_cols(L) bytes per pair), then its scales
    const int64_t ldzq = 2 * mx_cols(L), ldzs = mx_cols(L) / 32;
    unsigned char* Zq = static_cast<unsigned char*>(workspace);
    unsigned char* Zs = Zq + align_ws((size_t)round_up(N, 2) * mx_cols(L));
    ESPACE_TRY(mx_project_launch(Ptq, ldpq, Pts, ldps, Xq, ldxq, Xs, ldxs, Zq, ldzq, Zs, ldzs, K, L, N, stream, 1));
    ESPACE_TRY(mx_expand_launch(Zq, ldzq, Zs, ldzs, Wfq, ldwq, Wfs, ldws, Y, ldy, M, L, N, stream, 1));
    return ok();
}

}  // extern "C"
