// C ABI of the W4A16 linear layer: argument checks, handle ownership, the
// M-dispatch / work planner and the launches.  Declared in include/qlin.h.

#include "../../include/qlin.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <vector>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>

#include "qlin_internal.h"

using namespace qlin;

struct CachedPlan;

struct qlin_s {
    int device = -1;
    int num_cu = 0;
    int64_t K = 0, N = 0;
    int Kb = 0, Nt = 0;
    bool symmetric = false;
    uint4 *codes = nullptr;      // Nt * Kb blocks of 1 KiB
    void *sz = nullptr;          // Nt * Kb * 16 entries (u32 s|z<<16, or u16 s)
    // Workspace of qlin_forward / qlin_forward_path: arrival counters, then
    // fp32 split-K partials, sized at creation for the plans qlin_forward
    // runs at M <= 16 (zero bytes when none of them cuts the K range).
    void *ws = nullptr;
    size_t ws_bytes = 0;
    int cap_rows = 0;            // S * M the full workspace capacity covers (depends on K only)
    // the automatic plans for M = 1 .. 64 with the handle's workspace,
    // computed at creation (qlin_forward then plans nothing per call)
    CachedPlan *auto_plans = nullptr;
};

namespace qlin {

namespace {
thread_local char g_err[512] = "";
thread_local int g_status = QLIN_OK;
}  // namespace

int fail(int code, const char *fmt, ...) {
    g_status = code;
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

void clear_err() {
    g_err[0] = 0;
    g_status = QLIN_OK;
}

int hip_fail(hipError_t e, const char *what) {
    return fail(QLIN_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

int last_status() { return g_status; }

}  // namespace qlin

namespace {

constexpr int64_t kMaxK = 65536, kMaxN = 1 << 20, kMaxM = 65536;
constexpr int kCapRowsMin = 128;       // S * M the full workspace capacity always covers
constexpr size_t kMaxWsBytes = 0xFFFFFF00u;   // buffer-descriptor range of the partial sums
// Every workspace (a handle's, a caller's) starts with the arrival counters
// of the K-split launches, at fixed offsets, then the fp32 partial sums.
// Each launch leaves its counters at zero, so launches of different plans
// and handles can share one workspace in stream order.
constexpr int kMaxCounters = 4096;
constexpr size_t kCounterBytes = (size_t)kMaxCounters * 4;
static_assert(kCounterBytes == kScratchCounterBytes, "the static scratch has the workspace layout");

// Test hook: QLIN_FAULT=alloc makes every device allocation of this library fail.
hipError_t dev_alloc(void **p, size_t bytes) {
    const char *f = getenv("QLIN_FAULT");
    if (f && strcmp(f, "alloc") == 0) {
        *p = nullptr;
        return hipErrorOutOfMemory;
    }
    return hipMalloc(p, bytes);
}

float bf16_value(uint16_t b) {
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return f;
}

int check_shape(int64_t K, int64_t N, int64_t group) {
    if (K <= 0 || N <= 0 || group <= 0) return fail(QLIN_ERR_INVALID, "K, N and group must be positive");
    if (group != kGroup) return fail(QLIN_ERR_UNSUPPORTED, "group must be 128 (got %lld)", (long long)group);
    if (K % group) return fail(QLIN_ERR_INVALID, "K (%lld) must be a multiple of the group size", (long long)K);
    if (N % kTileN) return fail(QLIN_ERR_UNSUPPORTED, "N (%lld) must be a multiple of 16", (long long)N);
    if (K > kMaxK || N > kMaxN) return fail(QLIN_ERR_UNSUPPORTED, "K <= 65536 and N <= 1048576 required");
    return QLIN_OK;
}

// Is p device memory?  Pageable host memory is not known to the runtime
// (the query fails, its error is cleared) and counts as host.
bool is_device_ptr(const void *p) {
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, p) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    return attr.type == hipMemoryTypeDevice;
}

// Scales must be positive normal bf16 numbers in [2^-100, 2^100]: inside that
// range every (128 + q) * s and (q - z) * s is an exact binary32 number, which
// is what makes the matrix-core dequantization exact.
int check_scales(const uint16_t *s, size_t n) {
    for (size_t i = 0; i < n; ++i) {
        const int e = (s[i] >> 7) & 0xFF;
        if ((s[i] & 0x8000) || e < 127 - 100 || e > 127 + 99)
            return fail(QLIN_ERR_UNSUPPORTED, "scale %zu (0x%04x) outside [2^-100, 2^100] or not positive", i,
                        (unsigned)s[i]);
    }
    return QLIN_OK;
}

int check_zeros(const uint16_t *z, size_t n) {
    for (size_t i = 0; i < n; ++i) {
        const float v = bf16_value(z[i]);
        if (!(v >= 0.0f && v <= 15.0f) || v != std::floor(v))
            return fail(QLIN_ERR_INVALID, "zero-point %zu (0x%04x) is not an integer in [0, 15]", i, (unsigned)z[i]);
    }
    return QLIN_OK;
}

// Does a K chunk of Kc groups fit one SKINNY workgroup with M rows (staged x
// + one column tile)?
bool chunk_fits(int M, int Kc) { return lds_bytes(M, Kc, 1) <= kLdsMax; }

// Smallest number of K chunks whose chunks fit a SKINNY workgroup.
int min_split(int M, int Kb) {
    for (int S = 1; S <= Kb; ++S)
        if (chunk_fits(M, (Kb + S - 1) / S)) return S;
    return Kb + 1;   // not even one group fits (cannot happen for M <= 64)
}

// ------------------------------------------------------------------ planning
//
// A launch is planned for a Target: one linear, or a group of linears that
// share their input x (same K, same format) and run as one launch of the
// decode kernels.  The workspace the launch may use bounds the K splits:
// `cap_floats` fp32 partial sums and `cap_counters` arrival counters.

struct Target {
    int64_t K = 0, N = 0;        // N: columns over all members
    int Kb = 0, Nt = 0;          // Nt: column tiles over all members
    int num_cu = 0;
    bool symmetric = false;
    int nmem = 1;
    const qlin_s *mem[kMaxMembers] = {};
    size_t cap_floats = 0;
    int cap_counters = 0;
};

struct Plan {
    int path = 0;
    int kern = 0;
    int mrows = 0;     // template row count (GEMV: M; MFMA kernels: 16 * m-tiles)
    int S = 1, Gn = 1, grid = 1;
    int tn = 0;        // REGS/GEMV: tile slots (max tiles per range); SKINNY: staged x rows; TILED: NT
    size_t lds = 0;
    int TnMax = 1;     // tiles of the widest column range
    int gn[kMaxMembers] = {};   // column ranges of each member
    int rows = 0;      // rows per launch (decode kernels: M, or 16-row slices)
    size_t floats = 0; // fp32 partial sums the plan writes (K split)
    int counters = 0;  // arrival counters it uses (K split)
};

// S * M the full capacity covers for K = 128 Kb: the larger of 128 and the
// smallest feasible split of a 64-row chunk times its rows.
int capacity_rows(int Kb) {
    int rows = kCapRowsMin;
    for (int M = 1; M <= kMaxSkinnyM; ++M) {
        const int s_min = min_split(M, Kb);
        if (s_min > 1) rows = std::max(rows, s_min * M);
    }
    return rows;
}

}  // namespace

struct CachedPlan {
    Plan p;
    bool ok = false;
};

namespace {

// The workspace capacity a plan may assume when nothing limits it: partial
// sums for any split the decode planner considers (S * M up to the handle's
// cap_rows), and four 64 x 128 fp32 blocks per compute unit for a K-split
// tiled launch (32 MiB with 256 CUs: the measured splits of the deep layers
// at M = 512 .. 1024 need up to 31.5 MB).
void full_capacity(Target &t) {
    const int rows = t.mem[0]->cap_rows;
    const size_t dec = std::min(2 * (size_t)rows * (size_t)t.N, kMaxWsBytes / 4);
    t.cap_floats = std::max(dec, std::min((size_t)t.num_cu * 4 * 64 * 128, kMaxWsBytes / 4));
    t.cap_counters = std::min(std::max(t.Nt, t.num_cu), kMaxCounters);
}

Target target_of(const qlin_s *h) {
    Target t;
    t.K = h->K;
    t.N = h->N;
    t.Kb = h->Kb;
    t.Nt = h->Nt;
    t.num_cu = h->num_cu;
    t.symmetric = h->symmetric;
    t.nmem = 1;
    t.mem[0] = h;
    return t;
}

// Workspace bytes of a plan: the counter region and its partial sums, or
// nothing when it does not cut the K range.
size_t plan_ws_bytes(const Plan &p) { return p.floats ? kCounterBytes + p.floats * 4 : 0; }

// Narrows the full capacity (set first) to a workspace of `bytes`.
void set_capacity(Target &t, size_t bytes) {
    if (bytes <= kCounterBytes) {
        t.cap_floats = 0;
        t.cap_counters = 0;
        return;
    }
    t.cap_floats = std::min(t.cap_floats, (bytes - kCounterBytes) / 4);
}

// Partial sums and counters of a workspace (NULL without one).
float *ws_partials(void *ws) { return ws ? (float *)((char *)ws + kCounterBytes) : nullptr; }
uint32_t ws_partial_bytes(void *ws, size_t bytes) {
    return ws && bytes > kCounterBytes ? (uint32_t)std::min(bytes - kCounterBytes, kMaxWsBytes) : 0u;
}

int ceil_div(int a, int b) { return (a + b - 1) / b; }

// Widest column range when Gn ranges are spread over the members (each
// member gets at least one, at most one per tile): the smallest T with
// sum_i ceil(Nt_i / T) <= Gn.  -1 if Gn is outside [members, tiles].
int ranges_tnmax(const Target &t, int Gn) {
    if (Gn < t.nmem || Gn > t.Nt) return -1;
    if (t.nmem == 1) return ceil_div(t.Nt, Gn);
    int lo = 1, hi = 0;
    for (int i = 0; i < t.nmem; ++i) hi = std::max(hi, t.mem[i]->Nt);
    while (lo < hi) {
        const int T = (lo + hi) / 2;
        int need = 0;
        for (int i = 0; i < t.nmem; ++i) need += ceil_div(t.mem[i]->Nt, T);
        if (need <= Gn) hi = T;
        else lo = T + 1;
    }
    return lo;
}

// The ranges of each member for Gn in all: ceil(Nt_i / TnMax) each, then the
// ranges left over one at a time to the member whose ranges are the most
// loaded (fewer tiles per range for it, every compute unit busy).
void split_ranges(const Target &t, int Gn, int TnMax, int gn[]) {
    int left = Gn;
    for (int i = 0; i < t.nmem; ++i) {
        gn[i] = ceil_div(t.mem[i]->Nt, TnMax);
        left -= gn[i];
    }
    while (left > 0) {
        int best = -1;
        double load = 0.0;
        for (int i = 0; i < t.nmem; ++i) {
            const double l = (double)t.mem[i]->Nt / gn[i];
            if (gn[i] < t.mem[i]->Nt && l > load) { load = l; best = i; }
        }
        if (best < 0) break;
        ++gn[best];
        --left;
    }
}

// Auto M-dispatch uses the vector-ALU GEMV kernel up to this M (default 0:
// the matrix-core kernels were measured faster even at M = 1; the GEMV path
// stays available as an explicit choice).
int gemv_max_auto() {
    static int v = [] {
        const char *e = getenv("QLIN_GEMV_MAX_M");
        return e ? std::max(0, std::min(kMaxGemvM, atoi(e))) : 0;
    }();
    return v;
}

// Estimated time (ns) of one launch, fitted to measurements on MI355X:
// a fixed part (launch, first HBM round trip, the staged kernel's x
// staging barrier), the blocks of the busiest workgroup, the staged x
// chunk, and a fixed cost for the cross-workgroup reduction when the K
// range is cut.  The register-resident kernel reloads x per group and
// wave, which costs more per block as M grows.
double plan_cost(const Target &t, int kern, int M, int S, int Gn, int Tn) {
    const int Kc = (t.Kb + S - 1) / S;
    const int rounds = (S * Gn + t.num_cu - 1) / t.num_cu;
    const double blocks = (double)rounds * Tn * Kc;
    double c;
    if (kern == kKernStaged) {
        const double x_kib = (double)M * Kc * 256.0 / 1024.0;
        c = 4200.0 + 60.0 * blocks + 12.0 * rounds * x_kib;
    } else {
        c = 3300.0 + (60.0 + 3.5 * M) * blocks;
    }
    // never faster than streaming the weights at 6 TB/s
    const double blk = 1024.0 + (t.symmetric ? 32.0 : 64.0);
    c = std::max(c, (double)t.Nt * t.Kb * blk / 6.0e3);
    if (S > 1) c += 2500.0 + 100.0 * S;
    return c;
}

// Plans measured on MI355X (256 compute units) for the 4B decoder's linears
// where the cost model below picks a slower one: every kernel family and
// split from 1 to 8 was timed (HIP-graph replays over > 1 GiB of rotating
// weight copies) at M = 1, 2, 4, 8, 12 .. 16, and these won by 4-12%.  A
// group of linears sharing x is looked up by its total width (q|k|v: 6144).
struct TunedPlan { int m_lo, m_hi, K, N, kern, S; };
constexpr TunedPlan kTunedPlans[] = {
    {1, 2, 2560, 19456, kKernStaged, 1},    // gate|up at one or two rows (20% ahead of the register kernel)
    {13, 16, 2560, 1024, kKernStaged, 1},   // k and v projections
    {13, 16, 2560, 2560, kKernStaged, 1},
    {13, 16, 2560, 4096, kKernStaged, 1},   // q projection
    {14, 16, 4096, 2560, kKernStaged, 1},   // o projection
    {1, 4, 9728, 2560, kKernStaged, 1},     // down projection
    {8, 15, 9728, 2560, kKernMfma16, 3},
    {16, 16, 9728, 2560, kKernStaged, 3},
};

const TunedPlan *tuned_plan(const Target &t, int M) {
    if (t.num_cu != 256) return nullptr;
    for (const TunedPlan &e : kTunedPlans)
        if (M >= e.m_lo && M <= e.m_hi && t.K == e.K && t.N == e.N) return &e;
    return nullptr;
}

// Column blocks of a tiled launch with blocks of 4 nt tiles: each member's
// tiles are cut on their own.
int64_t tiled_col_blocks(const Target &t, int nt) {
    int64_t g = 0;
    for (int i = 0; i < t.nmem; ++i) g += (t.mem[i]->Nt + 4 * nt - 1) / (4 * nt);
    return g;
}

// Tiled plans measured on MI355X (256 compute units) for the 4B decoder's
// deep and narrow layers where the model below picks a slower one: every
// block shape with every K split from 1 to 6 was timed (HIP-graph replays
// over > 0.8 GB of rotating weight copies) at M = 128, 512, 1024 and 2048.
// Down (9728 -> 2560): 53.9 -> 42.4 us at M = 512, 85.3 -> 62.8 us at
// M = 1024; o (4096 -> 2560): 25.1 -> 23.8 us and 39.1 -> 35.1 us.  At
// M = 2048 the model's choices were the fastest; at M = 128 the one
// candidate that won alone (gate|up as 128 x 256 blocks in 3 K chunks,
// 28.1 against 29.1 us) made the whole pass 2% slower.  Each entry is used
// only where the workspace holds its partial blocks.
struct TunedTiled { int m_lo, m_hi, K, N, shape, S; };
constexpr TunedTiled kTunedTiled[] = {
    {385, 640, 9728, 2560, 1, 3},     // down: 64 x 128 blocks, 3 K chunks
    {385, 640, 4096, 2560, 1, 3},     // o
    {769, 1280, 9728, 2560, 0, 3},    // down: 128 x 256 blocks, 3 K chunks
    {769, 1280, 4096, 2560, 2, 2},    // o: 96 x 256 blocks, 2 K chunks
};

// TILED plan: one launch over all M rows and all members.  The block shape
// minimises (blocks per compute unit, rounded up) x (time of one block), with
// the block times measured on MI355X relative to the 128 x 256 shape (same
// K): 96 x 256 0.95, 64 x 128 0.42.  Ranked this way the three shapes come
// out in the measured order for every decoder linear at M = 512 .. 2048 (or
// within 2%): small blocks for narrow layers at small M, 96 x 256 where 128
// rows would leave part of the chip idle, 128 x 256 otherwise.
int make_tiled_plan(const Target &t, int64_t split_k, int64_t M, Plan *p) {
    if (split_k < 0 || split_k > t.Kb) return fail(QLIN_ERR_INVALID, "split_k must be in [0, K/128]");
    // one launch addresses x with 32-bit byte offsets: more rows than M * K
    // < 2^31 allows run as launches of that many rows each
    const int64_t rows = std::min<int64_t>(M, (((int64_t)1 << 31) - 1) / t.K);
    if (rows < M) {
        const int rc = make_tiled_plan(t, split_k, rows, p);
        p->rows = (int)rows;
        return rc;
    }
    constexpr int kShapes = (int)(sizeof kTiledShapes / sizeof kTiledShapes[0]);
    static const int forced = [] {                   // tuning knob: QLIN_TILED_SHAPE = index into kTiledShapes
        const char *e = getenv("QLIN_TILED_SHAPE");
        return e ? atoi(e) : -1;
    }();
    auto allowed = [&](int i) { return forced < 0 || forced >= kShapes || i == forced; };
    auto blocks_of = [&](int i) {
        const TiledShape c = kTiledShapes[i];
        return ((M + 16 * c.msw - 1) / (16 * c.msw)) * tiled_col_blocks(t, c.nt);
    };
    // Whole K range: the shape that minimises (blocks per compute unit,
    // rounded up) x (block time relative to 128 x 256).
    constexpr double kBlockTime[] = {1.0, 0.42, 0.95};
    static_assert(sizeof kBlockTime / sizeof kBlockTime[0] == kShapes, "");
    int best_i = -1, best_s = 1;
    double best = 1e300;
    for (int i = 0; i < kShapes; ++i) {
        if (!allowed(i)) continue;
        const double c = (double)((blocks_of(i) + t.num_cu - 1) / t.num_cu) * kBlockTime[i];
        if (c < best) { best = c; best_i = i; }
    }
    const TunedTiled *tuned = nullptr;
    if (split_k == 0 && forced < 0 && t.num_cu == 256)
        for (const TunedTiled &e : kTunedTiled)
            if (M >= e.m_lo && M <= e.m_hi && t.K == e.K && t.N == e.N) {
                const TiledShape c = kTiledShapes[e.shape];
                const int64_t blocks = blocks_of(e.shape);
                if (blocks <= t.cap_counters && (double)e.S * blocks * 16 * c.msw * 64 * c.nt <= (double)t.cap_floats)
                    tuned = &e;
            }
    // A measured plan if one fits; else a K split, when that leaves more than
    // half the CUs idle (or when one is asked for) and the workspace holds
    // its partial blocks.  Time model in us: a pipeline ramp plus a time per
    // 128-wide group of K per block with every CU busy (128 x 256: 2.28,
    // 64 x 128: 0.97, 96 x 256: 2.17), times the rounds of work items over the
    // CUs; a split adds the exchange: ~3 us of latency plus the partial
    // blocks written and read back at ~4 TB/s.
    if (tuned) {
        best_i = tuned->shape;
        best_s = tuned->S;
    } else if (split_k > 1 || (split_k == 0 && blocks_of(best_i) * 2 <= t.num_cu)) {
        constexpr double kRamp = 2.0, kGroupTime[] = {2.28, 0.97, 2.17}, kExchange = 3.0, kPartialBw = 4.0e6;
        static_assert(sizeof kGroupTime / sizeof kGroupTime[0] == kShapes, "");
        best_i = -1;
        best = 1e300;
        for (int i = 0; i < kShapes; ++i) {
            if (!allowed(i)) continue;
            const TiledShape c = kTiledShapes[i];
            const double bm = 16.0 * c.msw, bn = 64.0 * c.nt;
            const int64_t blocks = blocks_of(i);
            const int s_lo = split_k > 0 ? (int)split_k : 1;
            const int s_hi = split_k > 0 ? (int)split_k : std::min(16, t.Kb);
            for (int S = s_lo; S <= s_hi; ++S) {
                if (S > 1) {   // partial blocks and arrival counters must fit the workspace
                    if (blocks > t.cap_counters) continue;
                    if ((double)S * blocks * bm * bn > (double)t.cap_floats) continue;
                }
                const int Kc = (t.Kb + S - 1) / S;
                const double rounds = (double)((blocks * S + t.num_cu - 1) / t.num_cu);
                double c2 = rounds * (kRamp + kGroupTime[i] * Kc);
                if (S > 1) c2 += kExchange + 2.0 * S * blocks * bm * bn * 4.0 / kPartialBw;
                if (c2 < best) { best = c2; best_i = i; best_s = S; }
            }
        }
    }
    if (best_i < 0) return fail(QLIN_ERR_UNSUPPORTED, "split_k=%d does not fit (workspace or counters)", (int)split_k);
    const TiledShape sh = kTiledShapes[best_i];
    const int Mt = (int)((M + 16 * sh.msw - 1) / (16 * sh.msw));
    const int Gn = (int)tiled_col_blocks(t, sh.nt);
    p->path = kTiled;
    p->kern = kKernTiled;
    p->mrows = 16 * sh.msw;
    p->S = best_s;
    p->Gn = Gn;
    p->tn = sh.nt;
    p->grid = 8 * ((Gn * Mt * best_s + 7) / 8);
    p->lds = 0;
    p->rows = (int)M;
    p->floats = best_s > 1 ? (size_t)best_s * Gn * Mt * 16 * sh.msw * 64 * sh.nt : 0;
    p->counters = best_s > 1 ? Gn * Mt : 0;
    return QLIN_OK;
}

// Does the automatic choice run M rows through the TILED kernel (one
// launch) rather than the decode kernels?  Above 64 rows, always: with its K
// split the tiled kernel also covers the narrow, deep layers at small M
// (measured on MI355X at M = 128: o projection 14.5 us against 35.9 us as two
// 64-row launches, down projection 21.8 us against 74.2 us).
bool auto_tiled(int64_t M) { return M > kMaxSkinnyM; }

// Decode-kernel plan (M <= 64) for the target.  The automatic choice (AUTO)
// searches the kernel families and K splits that fit LDS and the workspace;
// when none fits (a caller workspace too small for the split a 17..64-row
// x chunk needs) it runs 16-row slices, whose plans never need more than a
// register-kernel launch without a split.
int make_decode_plan(const Target &t, int path, int64_t split_k, int Mi, Plan *p) {
    const bool auto_pick = path == kAuto;
    if (path == kAuto) path = (Mi <= gemv_max_auto()) ? kGemv : kSkinny;
    if (path == kGemv && Mi > kMaxGemvM) return fail(QLIN_ERR_UNSUPPORTED, "GEMV path needs M <= %d", kMaxGemvM);
    if (path == kRegs && Mi > 16) return fail(QLIN_ERR_UNSUPPORTED, "REGS path needs M <= 16");
    if (path == kSkinny && Mi > kMaxSkinnyM) return fail(QLIN_ERR_UNSUPPORTED, "SKINNY path needs M <= 64");
    if (split_k < 0 || split_k > t.Kb) return fail(QLIN_ERR_INVALID, "split_k must be in [0, K/128]");
    p->path = path;
    // candidate kernel families: the forced one, or for the automatic choice
    // (path SKINNY reached from AUTO) both matrix-core kernels when M <= 16
    int kerns[2], nk = 0;
    if (path == kGemv) kerns[nk++] = kKernGemv;
    else if (path == kRegs) kerns[nk++] = kKernMfma16;
    else if (auto_pick && Mi <= 16) { kerns[nk++] = kKernMfma16; kerns[nk++] = kKernStaged; }
    else kerns[nk++] = kKernStaged;

    auto tn_max_of = [&](int kern) {
        return kern == kKernGemv ? kTnMaxGemv : kern == kKernMfma16 ? kTnMax : t.Nt;
    };
    auto rows_of = [&](int kern) { return kern == kKernGemv ? Mi : 16 * ((Mi + 15) / 16); };
    // widest range of (kern, S, Gn) if the split fits, else -1
    auto fits = [&](int kern, int S, int Gn) {
        const int Tn = ranges_tnmax(t, Gn);
        if (Tn < 0) return -1;
        const int Kc = (t.Kb + S - 1) / S;
        if (S > 1 && ((size_t)S * Gn * Tn * Mi * 16 > t.cap_floats || Gn > t.cap_counters)) return -1;
        if (Tn > tn_max_of(kern)) return -1;
        if (kern != kKernStaged) return lds_bytes_regs(rows_of(kern), Tn) <= kLdsMax ? Tn : -1;
        if (!chunk_fits(Mi, Kc)) return -1;
        if ((int64_t)Tn * Kc >= 65536) return -1;   // the kernel's block walk divides u < 2^16 by Kc
        if ((int64_t)Tn * t.Kb * 1024 >= ((int64_t)1 << 31)) return -1;   // span of its buffer descriptors
        return lds_bytes(Mi, Kc, Tn) <= kLdsMax ? Tn : -1;
    };
    // column ranges for S chunks: one workgroup per CU (never more: a second
    // round of workgroups would double the time), but no range wider than the
    // kernel's tile limit (and more ranges if LDS demands).  Uneven ranges are
    // fine: splitting the columns over fewer, equal ranges leaves CUs idle,
    // and was measured slower.
    auto gn_for = [&](int kern, int S) {
        const int tm = tn_max_of(kern);
        int lo = t.nmem, need = 0;
        for (int i = 0; i < t.nmem; ++i) need += ceil_div(t.mem[i]->Nt, tm);
        lo = std::max(lo, need);
        int Gn = std::max(lo, std::min(t.Nt, std::max(1, t.num_cu / S)));
        Gn = std::min(Gn, t.Nt);
        while (Gn < t.Nt && fits(kern, S, Gn) < 0) ++Gn;
        return Gn;
    };

    int bestK = -1, bestS = -1, bestGn = 1, bestTn = 1;
    // a measured plan for this shape, if it fits; otherwise the cost model
    bool tuned = false;
    if (auto_pick && path == kSkinny && split_k == 0) {
        if (const TunedPlan *e = tuned_plan(t, Mi)) {
            const int Gn = gn_for(e->kern, e->S);
            const int Tn = fits(e->kern, e->S, Gn);
            if (Tn > 0) { bestK = e->kern; bestS = e->S; bestGn = Gn; bestTn = Tn; tuned = true; }
        }
    }
    double best = 1e300;
    for (int ki = 0; ki < nk && !tuned; ++ki) {
        const int kern = kerns[ki];
        const int s_lo = split_k > 0 ? (int)split_k : 1;
        const int s_hi = split_k > 0 ? (int)split_k : std::min(t.Kb, 64);
        for (int S = s_lo; S <= s_hi; ++S) {
            const int Gn = gn_for(kern, S);
            const int Tn = fits(kern, S, Gn);
            if (Tn < 0) continue;
            const double c = plan_cost(t, kern, Mi, S, Gn, Tn);
            if (c < best) { best = c; bestK = kern; bestS = S; bestGn = Gn; bestTn = Tn; }
        }
    }
    if (bestS < 0) {
        // nothing fits the workspace at this M: 16-row slices (the automatic
        // choice, or the staged kernel with the planner's split)
        if ((auto_pick || (path == kSkinny && split_k == 0)) && Mi > 16)
            return make_decode_plan(t, auto_pick ? kAuto : kSkinny, 0, 16, p);
        if (split_k > 0) return fail(QLIN_ERR_UNSUPPORTED, "split_k=%d does not fit (LDS or workspace)", (int)split_k);
        return fail(QLIN_ERR_UNSUPPORTED, "no work split fits this shape and workspace");
    }
    p->kern = bestK;
    p->mrows = rows_of(bestK);
    p->S = bestS;
    p->Gn = bestGn;
    p->TnMax = bestTn;
    p->grid = bestS * bestGn;
    split_ranges(t, bestGn, bestTn, p->gn);
    const bool regs = bestK != kKernStaged;
    const int Kc = (t.Kb + bestS - 1) / bestS;
    p->tn = regs ? bestTn : staged_rows(Mi);
    const size_t need = regs ? lds_bytes_regs(p->mrows, bestTn) : lds_bytes(Mi, Kc, bestTn);
    // at least 80 KiB + 1 of LDS per workgroup keeps one workgroup per CU, so
    // the grid spreads over all CUs
    p->lds = std::max(need, (size_t)80 * 1024 + 256);
    p->rows = Mi;
    p->floats = bestS > 1 ? (size_t)bestS * bestGn * bestTn * Mi * 16 : 0;
    p->counters = bestS > 1 ? bestGn : 0;
    return QLIN_OK;
}

// The plan of a launch of M rows: TILED (forced, or AUTO above 64 rows) is
// planned per member (one launch each); the decode kernels cover all members
// in one launch per slice of p->rows rows.
int make_plan(const Target &t, int path, int64_t split_k, int64_t M, Plan *p) {
    if (path < kAuto || path > kRegs) return fail(QLIN_ERR_INVALID, "unknown path %d", path);
    if (split_k < 0 || split_k > t.Kb) return fail(QLIN_ERR_INVALID, "split_k must be in [0, K/128]");
    if (path == kTiled || (path == kAuto && auto_tiled(M))) return make_tiled_plan(t, split_k, M, p);
    return make_decode_plan(t, path, split_k, (int)std::min<int64_t>(M, kMaxSkinnyM), p);
}

// Workspace bytes the launch needs for M rows under the target's capacity.
int workspace_need(const Target &t, int path, int64_t split_k, int64_t M, size_t *bytes) {
    *bytes = 0;
    Plan p;
    const int rc = make_plan(t, path, split_k, M, &p);
    if (rc == QLIN_OK) *bytes = plan_ws_bytes(p);
    return rc;
}

// Launch arguments of a decode-kernel plan for M rows (M <= 64) at x, with
// member i writing ys[i]; the workspace holds counters then partials.
FwdArgs fwd_args(const Target &t, const Plan &p, int64_t M, const uint16_t *x, uint16_t *const *ys,
                 void *ws, size_t ws_bytes, int64_t row0) {
    FwdArgs a;
    a.x = x + row0 * t.K;
    a.counters = (uint32_t *)ws;
    a.ws = ws_partials(ws);
    a.ws_bytes = ws_partial_bytes(ws, ws_bytes);
    a.M = (int)M;
    a.K = (int)t.K;
    a.Kb = t.Kb;
    a.S = p.S;
    a.Gn = p.Gn;
    a.inv_gn = p.Gn > 1 ? (uint32_t)((((uint64_t)1 << 32) + p.Gn - 1) / p.Gn) : 0u;
    a.Kq = t.Kb / p.S;
    a.Kr = t.Kb % p.S;
    a.TnMax = p.TnMax;
    a.nmem = t.nmem;
    int gn0 = 0;
    for (int i = 0; i < kMaxMembers; ++i) {
        FwdMember &f = a.mem[i];
        if (i >= t.nmem) {             // absent: starts past the last range, never selected
            f = a.mem[0];
            a.gn0[i] = p.Gn;
            continue;
        }
        const qlin_s *h = t.mem[i];
        f.codes = h->codes;
        f.sz = h->sz;
        f.y = ys[i] + row0 * h->N;
        f.N = (int)h->N;
        f.Nq = h->Nt / p.gn[i];
        f.Nr = h->Nt % p.gn[i];
        a.gn0[i] = gn0;
        gn0 += p.gn[i];
    }
    return a;
}

int check_rows(int64_t M) {
    if (M < 0) return fail(QLIN_ERR_INVALID, "M must be >= 0");
    if (M > kMaxM) return fail(QLIN_ERR_UNSUPPORTED, "M must be <= 65536");
    return QLIN_OK;
}

bool overlaps(uintptr_t a, size_t an, uintptr_t b, size_t bn) { return a < b + bn && b < a + an; }

// Checks of a forward over the members of t (x shared, outputs ys[i]), all
// before any HIP call: sizes, NULLs, alignment, the outputs overlapping x,
// each other or the workspace, and the device.
int check_launch(const Target &t, int64_t M, const uint16_t *x, uint16_t *const *ys, const void *ws,
                 size_t ws_bytes) {
    if (check_rows(M) != QLIN_OK || M == 0) return last_status();
    if (!x) return fail(QLIN_ERR_INVALID, "NULL x");
    if ((uintptr_t)x & 15) return fail(QLIN_ERR_ALIGN, "x must be 16-byte aligned");
    if ((uintptr_t)ws & 15) return fail(QLIN_ERR_ALIGN, "workspace must be 16-byte aligned");
    const size_t xb = (size_t)M * t.K * 2;
    for (int i = 0; i < t.nmem; ++i) {
        if (!ys[i]) return fail(QLIN_ERR_INVALID, "NULL y");
        if ((uintptr_t)ys[i] & 15) return fail(QLIN_ERR_ALIGN, "y must be 16-byte aligned");
        const size_t yb = (size_t)M * t.mem[i]->N * 2;
        if (overlaps((uintptr_t)x, xb, (uintptr_t)ys[i], yb)) return fail(QLIN_ERR_INVALID, "y overlaps x");
        if (ws && overlaps((uintptr_t)ws, ws_bytes, (uintptr_t)ys[i], yb))
            return fail(QLIN_ERR_INVALID, "y overlaps the workspace");
        for (int j = 0; j < i; ++j)
            if (overlaps((uintptr_t)ys[j], (size_t)M * t.mem[j]->N * 2, (uintptr_t)ys[i], yb))
                return fail(QLIN_ERR_INVALID, "two outputs overlap");
    }
    if (ws && overlaps((uintptr_t)ws, ws_bytes, (uintptr_t)x, xb)) return fail(QLIN_ERR_INVALID, "x overlaps the workspace");
    int dev = -1;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != t.mem[0]->device)
        return fail(QLIN_ERR_INVALID, "handle belongs to device %d, current is %d", t.mem[0]->device, dev);
    return QLIN_OK;
}

// One tiled launch of plan p over M rows (M * K < 2^31) at x, member i
// writing ys[i].
int launch_tiled_rows(const Target &t, const Plan &p, int64_t M, const uint16_t *x, uint16_t *const *ys,
                      void *ws, size_t ws_bytes, hipStream_t st) {
    TiledArgs a;
    a.x = x;
    a.M = (int)M;
    a.K = (int)t.K;
    a.Kb = t.Kb;
    a.Mt = (int)((M + p.mrows - 1) / p.mrows);
    a.Gn = p.Gn;
    a.S = p.S;
    a.Kq = t.Kb / p.S;
    a.Kr = t.Kb % p.S;
    a.counters = (uint32_t *)ws;
    a.ws = ws_partials(ws);
    a.ws_bytes = ws_partial_bytes(ws, ws_bytes);
    a.nmem = t.nmem;
    int gb0 = 0;
    for (int i = 0; i < kMaxMembers; ++i) {
        TiledMember &f = a.mem[i];
        if (i >= t.nmem) {             // absent: starts past the last column block, never selected
            f = a.mem[0];
            a.gb0[i] = p.Gn;
            continue;
        }
        const qlin_s *h = t.mem[i];
        f.codes = h->codes;
        f.sz = h->sz;
        f.y = ys[i];
        f.N = (int)h->N;
        f.Nt = h->Nt;
        a.gb0[i] = gb0;
        gb0 += (h->Nt + 4 * p.tn - 1) / (4 * p.tn);
    }
    const hipError_t e = launch_tiled(t.symmetric, TiledShape{p.mrows / 16, p.tn}, a, p.grid, st);
    return e == hipSuccess ? QLIN_OK : hip_fail(e, "tiled launch");
}

// Runs M rows through the members of t with the workspace (ws, ws_bytes)
// (capacity already set in t), in launches of the plan's rows each (a
// shorter last one has a plan of its own).  Arguments are checked by the
// caller.
int launch_all(const Target &t, int path, int64_t split_k, int64_t M, const uint16_t *x, uint16_t *const *ys,
               void *ws, size_t ws_bytes, hipStream_t st) {
    const bool tiled = path == kTiled || (path == kAuto && auto_tiled(M));
    for (int64_t m0 = 0; m0 < M;) {
        Plan p;
        int rc = tiled ? make_tiled_plan(t, split_k, M - m0, &p) : make_plan(t, path, split_k, M - m0, &p);
        if (rc != QLIN_OK) return rc;
        const int64_t Ms = std::min<int64_t>(p.rows, M - m0);
        if (Ms != p.rows) {
            rc = tiled ? make_tiled_plan(t, split_k, Ms, &p) : make_plan(t, path, split_k, Ms, &p);
            if (rc != QLIN_OK) return rc;
        }
        if (tiled) {
            uint16_t *yk[kMaxMembers];
            for (int i = 0; i < t.nmem; ++i) yk[i] = ys[i] + m0 * t.mem[i]->N;
            if ((rc = launch_tiled_rows(t, p, Ms, x + m0 * t.K, yk, ws, ws_bytes, st)) != QLIN_OK) return rc;
        } else {
            const FwdArgs a = fwd_args(t, p, Ms, x, ys, ws, ws_bytes, m0);
            const hipError_t e = launch_forward(p.kern, p.mrows, p.tn, t.symmetric, p.grid, p.lds, a, st);
            if (e != hipSuccess) return hip_fail(e, "forward launch");
        }
        m0 += Ms;
    }
    return QLIN_OK;
}

// The handle's own workspace: what the automatic plans at M = 1 .. 16 use
// with nothing limiting them.
size_t handle_ws_bytes(const qlin_s *h) {
    Target t = target_of(h);
    full_capacity(t);
    size_t bytes = 0;
    for (int M = 1; M <= 16; ++M) {
        Plan p;
        if (make_plan(t, kAuto, 0, M, &p) == QLIN_OK) bytes = std::max(bytes, plan_ws_bytes(p));
    }
    clear_err();
    return bytes;
}

void free_handle(qlin_s *h) {
    if (!h) return;
    if (h->codes) (void)hipFree(h->codes);
    if (h->sz) (void)hipFree(h->sz);
    if (h->ws) (void)hipFree(h->ws);
    delete[] h->auto_plans;
    delete h;
}

qlin_t create_impl(int64_t K, int64_t N, int64_t group, const uint32_t *packed, const uint16_t *scales,
                   const uint16_t *zeros, bool symmetric) {
    clear_err();
    if (check_shape(K, N, group) != QLIN_OK) return nullptr;
    if (!packed || !scales || (!symmetric && !zeros)) {
        fail(QLIN_ERR_INVALID, "NULL weight pointer");
        return nullptr;
    }
    const size_t ngroups = (size_t)N * (K / kGroup);
    // inputs may live in device memory (e.g. written by qlin_quantize): the
    // scale and zero-point checks then run on host copies
    std::vector<uint16_t> s_host, z_host;
    if (is_device_ptr(scales)) {
        s_host.resize(ngroups);
        if (hipMemcpy(s_host.data(), scales, ngroups * 2, hipMemcpyDeviceToHost) != hipSuccess) {
            hip_fail(hipGetLastError(), "copy scales to host");
            return nullptr;
        }
    }
    if (!symmetric && is_device_ptr(zeros)) {
        z_host.resize(ngroups);
        if (hipMemcpy(z_host.data(), zeros, ngroups * 2, hipMemcpyDeviceToHost) != hipSuccess) {
            hip_fail(hipGetLastError(), "copy zero-points to host");
            return nullptr;
        }
    }
    if (check_scales(s_host.empty() ? scales : s_host.data(), ngroups) != QLIN_OK) return nullptr;
    if (!symmetric && check_zeros(z_host.empty() ? zeros : z_host.data(), ngroups) != QLIN_OK) return nullptr;

    qlin_s *h = new qlin_s;
    h->K = K;
    h->N = N;
    h->Kb = (int)(K / kGroup);
    h->Nt = (int)(N / kTileN);
    h->symmetric = symmetric;
    const size_t code_bytes = (size_t)N * K / 2;
    const size_t sz_bytes = ngroups * (symmetric ? 2 : 4);

    void *canon = nullptr, *sc = nullptr, *zc = nullptr;
    hipStream_t st = nullptr;
    hipError_t e = hipSuccess;
    auto bail = [&](const char *what, hipError_t e) -> qlin_t {
        if (e == hipErrorOutOfMemory) fail(QLIN_ERR_OOM, "device allocation failed (%s)", what);
        else hip_fail(e, what);
        if (st) (void)hipStreamSynchronize(st);
        if (canon) (void)hipFree(canon);
        if (sc) (void)hipFree(sc);
        if (zc) (void)hipFree(zc);
        if (st) (void)hipStreamDestroy(st);
        free_handle(h);
        return nullptr;
    };
    if ((e = dev_alloc((void **)&h->codes, code_bytes)) != hipSuccess) return bail("codes", e);
    if ((e = dev_alloc(&h->sz, sz_bytes)) != hipSuccess) return bail("scales", e);
    if ((e = hipGetDevice(&h->device)) != hipSuccess) return bail("hipGetDevice", e);
    if ((e = hipDeviceGetAttribute(&h->num_cu, hipDeviceAttributeMultiprocessorCount, h->device)) != hipSuccess)
        return bail("hipDeviceGetAttribute", e);
    h->cap_rows = capacity_rows(h->Kb);
    h->ws_bytes = handle_ws_bytes(h);
    {
        Target t = target_of(h);
        full_capacity(t);
        set_capacity(t, h->ws_bytes);
        h->auto_plans = new CachedPlan[kMaxSkinnyM];
        for (int M = 1; M <= kMaxSkinnyM; ++M)
            h->auto_plans[M - 1].ok = make_plan(t, kAuto, 0, M, &h->auto_plans[M - 1].p) == QLIN_OK;
        clear_err();
    }
    if (h->ws_bytes && (e = dev_alloc(&h->ws, h->ws_bytes)) != hipSuccess) return bail("workspace", e);
    if ((e = dev_alloc(&canon, code_bytes)) != hipSuccess) return bail("staging", e);
    if ((e = dev_alloc(&sc, ngroups * 2)) != hipSuccess) return bail("staging", e);
    if (!symmetric && (e = dev_alloc(&zc, ngroups * 2)) != hipSuccess) return bail("staging", e);

    static std::once_flag once;
    std::call_once(once, [] { (void)prepare_kernels(); (void)hipGetLastError(); });
    // the copies and the repack run on a stream of the library's own, so the
    // call waits for its own work only; a blocking stream, so that device
    // inputs written by earlier default-stream work (qlin_quantize) are read
    // after it
    if ((e = hipStreamCreate(&st)) != hipSuccess) return bail("stream", e);
    if ((e = hipMemcpyAsync(canon, packed, code_bytes, hipMemcpyDefault, st)) != hipSuccess)
        return bail("copy codes", e);
    if ((e = hipMemcpyAsync(sc, scales, ngroups * 2, hipMemcpyDefault, st)) != hipSuccess)
        return bail("copy scales", e);
    if (!symmetric && (e = hipMemcpyAsync(zc, zeros, ngroups * 2, hipMemcpyDefault, st)) != hipSuccess)
        return bail("copy zeros", e);
    if (h->ws_bytes && (e = hipMemsetAsync(h->ws, 0, h->ws_bytes, st)) != hipSuccess)
        return bail("clear workspace", e);
    // set-up of this device's static scratch (qlin_forward_group_noalloc), once
    if ((e = static_scratch_setup(h->device, st)) != hipSuccess) return bail("static scratch set-up", e);
    if ((e = launch_repack((const uint32_t *)canon, (const uint16_t *)sc, (const uint16_t *)zc, h->codes, h->sz,
                           (int)K, (int)N, symmetric, st)) != hipSuccess)
        return bail("repack launch", e);
    if ((e = hipStreamSynchronize(st)) != hipSuccess) return bail("repack", e);
    (void)hipStreamDestroy(st);
    (void)hipFree(canon);
    (void)hipFree(sc);
    if (zc) (void)hipFree(zc);
    return h;
}

// A forward of one handle with its own workspace.
int run_forward(qlin_s *h, int path, int64_t split_k, int64_t M, const uint16_t *x, uint16_t *y, void *stream) {
    clear_err();
    if (!h) return fail(QLIN_ERR_INVALID, "NULL handle");
    if (path < kAuto || path > kRegs) return fail(QLIN_ERR_INVALID, "unknown path %d", path);
    if (split_k < 0 || split_k > h->Kb) return fail(QLIN_ERR_INVALID, "split_k must be in [0, K/128]");
    Target t = target_of(h);
    full_capacity(t);
    set_capacity(t, h->ws_bytes);
    uint16_t *ys[1] = {y};
    int rc = check_launch(t, M, x, ys, nullptr, 0);
    if (rc != QLIN_OK || M == 0) return rc;
    if (path == kSkinny && M > kMaxSkinnyM) return fail(QLIN_ERR_UNSUPPORTED, "SKINNY path needs M <= 64");
    if (path == kRegs && M > 16) return fail(QLIN_ERR_UNSUPPORTED, "REGS path needs M <= 16");
    if (path == kGemv && M > kMaxGemvM) return fail(QLIN_ERR_UNSUPPORTED, "GEMV path needs M <= %d", kMaxGemvM);
    const hipStream_t st = (hipStream_t)stream;
    const CachedPlan *cp = (path == kAuto && split_k == 0 && M <= kMaxSkinnyM) ? &h->auto_plans[M - 1] : nullptr;
    if (cp && cp->ok && cp->p.rows >= M) {     // the automatic plan, computed at creation: one launch
        const FwdArgs a = fwd_args(t, cp->p, M, x, ys, h->ws, h->ws_bytes, 0);
        const hipError_t e = launch_forward(cp->p.kern, cp->p.mrows, cp->p.tn, t.symmetric, cp->p.grid, cp->p.lds, a, st);
        if (e != hipSuccess) return hip_fail(e, "forward launch");
        rc = QLIN_OK;
    } else {
        rc = launch_all(t, path, split_k, M, x, ys, h->ws, h->ws_bytes, st);
    }
    return rc;
}

// Target of a group call: members checked to share K, format and device.
int group_target(int64_t n, const qlin_t *hs, Target *t) {
    if (n < 1 || n > kMaxMembers) return fail(QLIN_ERR_INVALID, "n must be in [1, %d]", kMaxMembers);
    if (!hs) return fail(QLIN_ERR_INVALID, "NULL handle array");
    for (int64_t i = 0; i < n; ++i) {
        if (!hs[i]) return fail(QLIN_ERR_INVALID, "NULL handle %lld", (long long)i);
        if (hs[i]->K != hs[0]->K) return fail(QLIN_ERR_INVALID, "handles of a group must share K");
        if (hs[i]->symmetric != hs[0]->symmetric)
            return fail(QLIN_ERR_INVALID, "handles of a group must share the format (zero-points or symmetric)");
        if (hs[i]->device != hs[0]->device) return fail(QLIN_ERR_INVALID, "handles of a group must share the device");
    }
    *t = target_of(hs[0]);
    t->nmem = (int)n;
    t->N = 0;
    t->Nt = 0;
    for (int64_t i = 0; i < n; ++i) {
        t->mem[i] = hs[i];
        t->N += hs[i]->N;
        t->Nt += hs[i]->Nt;
    }
    return QLIN_OK;
}

int check_path_rows(int path, int64_t M) {
    if (path < kAuto || path > kRegs) return fail(QLIN_ERR_INVALID, "unknown path %d", path);
    if (path == kGemv && M > kMaxGemvM) return fail(QLIN_ERR_UNSUPPORTED, "GEMV path needs M <= %d", kMaxGemvM);
    if (path == kSkinny && M > kMaxSkinnyM) return fail(QLIN_ERR_UNSUPPORTED, "SKINNY path needs M <= 64");
    if (path == kRegs && M > 16) return fail(QLIN_ERR_UNSUPPORTED, "REGS path needs M <= 16");
    return QLIN_OK;
}

// Target of a group call with the capacity of a workspace of `bytes`
// (< 0: the full capacity).
int group_target_ws(int64_t n, const qlin_t *hs, int64_t bytes, Target *t) {
    if (group_target(n, hs, t) != QLIN_OK) return last_status();
    full_capacity(*t);
    if (bytes >= 0) set_capacity(*t, (size_t)bytes);
    return QLIN_OK;
}

int plan_text(const Target &t, int path, int64_t split_k, int64_t M, char *buf, int64_t buflen) {
    Plan p;
    const int rc = make_plan(t, path, split_k, M, &p);
    if (rc != QLIN_OK) return rc;
    const bool tiled = p.kern == kKernTiled;
    const int64_t launches = (M + p.rows - 1) / p.rows;
    static const char *names[] = {"gemv", "regs", "skinny", "tiled"};
    snprintf(buf, (size_t)buflen, "path=%s kernel=%s grid=%d block=%d split=%d ranges=%d lds=%zu launches=%lld",
             names[p.kern], kernel_name(p.kern, p.mrows, p.tn, t.symmetric), p.grid,
             tiled ? kTiledWaves * 64 * tiled_wsplit(TiledShape{p.mrows / 16, p.tn}) : kThreads, p.S, p.Gn, p.lds,
             (long long)launches);
    return QLIN_OK;
}

}  // namespace

extern "C" {

qlin_t qlin_create(int64_t K, int64_t N, int64_t group, const uint32_t *packed_w, const uint16_t *scales,
                   const uint16_t *zeros) {
    return create_impl(K, N, group, packed_w, scales, zeros, false);
}

qlin_t qlin_create_symmetric(int64_t K, int64_t N, int64_t group, const uint32_t *packed_w,
                             const uint16_t *scales) {
    return create_impl(K, N, group, packed_w, scales, nullptr, true);
}

int qlin_quantize(int64_t K, int64_t N, int64_t group, const uint16_t *w, const uint16_t *scales,
                  const uint16_t *zeros, uint32_t *packed, void *stream) {
    clear_err();
    if (check_shape(K, N, group) != QLIN_OK) return last_status();
    if (!w || !scales || !packed) return fail(QLIN_ERR_INVALID, "NULL pointer");
    if (((uintptr_t)w & 15) || ((uintptr_t)packed & 3) || ((uintptr_t)scales & 1) || ((uintptr_t)zeros & 1))
        return fail(QLIN_ERR_ALIGN, "w must be 16-byte, packed 4-byte and scales/zeros 2-byte aligned");
    if (overlaps((uintptr_t)w, (size_t)(N * K * 2), (uintptr_t)packed, (size_t)(N * K / 2)))
        return fail(QLIN_ERR_INVALID, "packed overlaps w");
    hipError_t e = launch_quantize(w, scales, zeros, packed, (int)K, (int)N, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "quantize launch");
    return QLIN_OK;
}

int qlin_forward(qlin_t h, int64_t M, const uint16_t *x, uint16_t *y, void *stream) {
    return run_forward(h, kAuto, 0, M, x, y, stream);
}

int qlin_forward_path(qlin_t h, int path, int64_t split_k, int64_t M, const uint16_t *x, uint16_t *y,
                      void *stream) {
    return run_forward(h, path, split_k, M, x, y, stream);
}

int qlin_plan(qlin_t h, int path, int64_t split_k, int64_t M, char *buf, int64_t buflen) {
    clear_err();
    if (!h) return fail(QLIN_ERR_INVALID, "NULL handle");
    if (!buf || buflen <= 0) return fail(QLIN_ERR_INVALID, "NULL buffer");
    if (M <= 0 || M > kMaxM) return fail(QLIN_ERR_INVALID, "M must be in [1, 65536]");
    if (check_path_rows(path, M) != QLIN_OK) return last_status();
    Target t = target_of(h);
    full_capacity(t);
    set_capacity(t, h->ws_bytes);
    return plan_text(t, path, split_k, M, buf, buflen);
}

int qlin_forward_group(int64_t n, const qlin_t *hs, int path, int64_t split_k, int64_t M, const uint16_t *x,
                       uint16_t *const *ys, void *workspace, int64_t workspace_bytes, void *stream) {
    clear_err();
    if (workspace_bytes < 0) return fail(QLIN_ERR_INVALID, "workspace_bytes must be >= 0");
    if (!workspace && workspace_bytes) return fail(QLIN_ERR_INVALID, "NULL workspace of non-zero size");
    Target t;
    if (group_target_ws(n, hs, workspace_bytes, &t) != QLIN_OK) return last_status();
    if (!ys) return fail(QLIN_ERR_INVALID, "NULL output array");
    if (split_k < 0 || split_k > t.Kb) return fail(QLIN_ERR_INVALID, "split_k must be in [0, K/128]");
    if (check_path_rows(path, M) != QLIN_OK) return last_status();
    int rc = check_launch(t, M, x, ys, workspace, (size_t)workspace_bytes);
    if (rc != QLIN_OK || M == 0) return rc;
    const hipStream_t st = (hipStream_t)stream;
    return launch_all(t, path, split_k, M, x, ys, workspace, (size_t)workspace_bytes, st);
}

int qlin_forward_group_noalloc(int64_t n, const qlin_t *hs, int path, int64_t split_k, int64_t M,
                               const uint16_t *x, uint16_t *const *ys, void *stream) {
    clear_err();
    Target t;
    if (group_target_ws(n, hs, -1, &t) != QLIN_OK) return last_status();
    if (!ys) return fail(QLIN_ERR_INVALID, "NULL output array");
    if (split_k < 0 || split_k > t.Kb) return fail(QLIN_ERR_INVALID, "split_k must be in [0, K/128]");
    if (check_path_rows(path, M) != QLIN_OK) return last_status();
    void *ws = static_scratch(t.mem[0]->device);
    if (!ws) return fail(QLIN_ERR_INVALID, "no static scratch on device %d", t.mem[0]->device);
    int rc = check_launch(t, M, x, ys, ws, kStaticScratchBytes);
    if (rc != QLIN_OK || M == 0) return rc;
    // the plan qlin_forward_group runs with a workspace of unlimited size,
    // refused when its scratch exceeds the static array
    size_t need = 0;
    if ((rc = workspace_need(t, path, split_k, M, &need)) != QLIN_OK) return rc;
    if (need > kStaticScratchBytes)
        return fail(QLIN_ERR_UNSUPPORTED, "this plan needs %zu bytes of scratch, the static array holds %zu "
                    "(use qlin_forward_group with a workspace)", need, kStaticScratchBytes);
    set_capacity(t, kStaticScratchBytes);
    return launch_all(t, path, split_k, M, x, ys, ws, kStaticScratchBytes, (hipStream_t)stream);
}

int qlin_group_plan(int64_t n, const qlin_t *hs, int path, int64_t split_k, int64_t M, int64_t workspace_bytes,
                    int64_t *workspace_needed, char *buf, int64_t buflen) {
    clear_err();
    Target t;
    if (group_target_ws(n, hs, workspace_bytes, &t) != QLIN_OK) return last_status();
    if (M <= 0 || M > kMaxM) return fail(QLIN_ERR_INVALID, "M must be in [1, 65536]");
    if (split_k < 0 || split_k > t.Kb) return fail(QLIN_ERR_INVALID, "split_k must be in [0, K/128]");
    if (check_path_rows(path, M) != QLIN_OK) return last_status();
    size_t need = 0;
    int rc = workspace_need(t, path, split_k, M, &need);
    if (rc != QLIN_OK) return rc;
    if (workspace_needed) *workspace_needed = (int64_t)need;
    if (buf && buflen > 0) rc = plan_text(t, path, split_k, M, buf, buflen);
    return rc;
}

// The runtime's hipFree waits for the device's outstanding work before it
// releases the memory, so a forward still in flight keeps its buffers until
// it completes.  Recording an event after every forward (to wait for this
// handle's work only) was measured to add about 3 us of device time to each
// eagerly launched forward, for a wait hipFree performs anyway.
void qlin_destroy(qlin_t h) {
    if (!h) return;
    int prev = -1;
    const bool other = hipGetDevice(&prev) == hipSuccess && prev != h->device && hipSetDevice(h->device) == hipSuccess;
    free_handle(h);
    if (other) (void)hipSetDevice(prev);
}

const char *qlin_last_error(void) { return g_err; }

int qlin_last_status(void) { return g_status; }

int qlin_unpack_codes(qlin_t h, uint8_t *q_out, void *stream) {
    clear_err();
    if (!h || !q_out) return fail(QLIN_ERR_INVALID, "NULL argument");
    if ((uintptr_t)q_out & 15) return fail(QLIN_ERR_ALIGN, "q_out must be 16-byte aligned");
    hipError_t e = launch_unpack(h->codes, q_out, (int)h->K, (int)h->N, (hipStream_t)stream);
    return e == hipSuccess ? QLIN_OK : hip_fail(e, "unpack launch");
}

int qlin_dequantize(qlin_t h, int routine, uint16_t *w_out, void *stream) {
    clear_err();
    if (!h || !w_out) return fail(QLIN_ERR_INVALID, "NULL argument");
    if (routine != 0 && routine != 1) return fail(QLIN_ERR_INVALID, "routine must be 0 or 1");
    if ((uintptr_t)w_out & 15) return fail(QLIN_ERR_ALIGN, "w_out must be 16-byte aligned");
    hipError_t e = launch_dequant(routine, h->codes, h->sz, h->symmetric, w_out, (int)h->K, (int)h->N,
                                  (hipStream_t)stream);
    return e == hipSuccess ? QLIN_OK : hip_fail(e, "dequantize launch");
}

int qlin_stream_read(const void *buf, int64_t bytes, int grid, uint32_t *sink, void *stream) {
    clear_err();
    if (!buf || !sink) return fail(QLIN_ERR_INVALID, "NULL argument");
    if (bytes <= 0 || bytes % 16) return fail(QLIN_ERR_INVALID, "bytes must be a positive multiple of 16");
    if ((uintptr_t)buf & 15) return fail(QLIN_ERR_ALIGN, "buf must be 16-byte aligned");
    hipError_t e;
    if (grid <= 0) {
        int dev = 0, cus = 0;
        if ((e = hipGetDevice(&dev)) != hipSuccess) return hip_fail(e, "hipGetDevice");
        if ((e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev)) != hipSuccess)
            return hip_fail(e, "hipDeviceGetAttribute");
        grid = 4 * cus;
    }
    e = launch_stream_read(buf, (size_t)bytes, grid, sink, (hipStream_t)stream);
    return e == hipSuccess ? QLIN_OK : hip_fail(e, "stream-read launch");
}

int qlin_shape(qlin_t h, int64_t *K, int64_t *N) {
    clear_err();
    if (!h) return fail(QLIN_ERR_INVALID, "NULL handle");
    if (K) *K = h->K;
    if (N) *N = h->N;
    return QLIN_OK;
}

int qlin_workspace_bytes(qlin_t h, int64_t *bytes) {
    clear_err();
    if (!h) return fail(QLIN_ERR_INVALID, "NULL handle");
    if (bytes) *bytes = (int64_t)h->ws_bytes;
    return QLIN_OK;
}

}  // extern "C"
