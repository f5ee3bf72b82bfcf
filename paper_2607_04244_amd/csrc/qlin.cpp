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

struct qlin_s {
    int device = -1;
    int num_cu = 0;
    int64_t K = 0, N = 0;
    int Kb = 0, Nt = 0;
    bool symmetric = false;
    uint4 *codes = nullptr;      // Nt * Kb blocks of 1 KiB
    void *sz = nullptr;          // Nt * Kb * 16 entries (u32 s|z<<16, or u16 s)
    float *ws = nullptr;         // split-K partials, ws_floats fp32
    int ws_rows = 0;             // S * M the workspace covers for any column split
    size_t ws_floats = 0;        // allocated fp32 (also covers one 64 x 128 partial block per CU)
    size_t ws_decode = 0;        // 2 * ws_rows * N >= S * Gn * TnMax * M * 16 when S * M <= ws_rows
    uint32_t *counters = nullptr;
    int counters_n = 0;
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

constexpr int kWsRowsMin = 128;        // S * M always allowed by the partial-sum workspace
constexpr int64_t kMaxK = 65536, kMaxN = 1 << 20, kMaxM = 65536;

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

// Scales must be positive normal bf16 numbers in [2^-100, 2^100]: inside that
// range every (128 + q) * s and (q - z) * s is an exact binary32 number, which
// is what makes the matrix-core dequantization exact.
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

void free_handle(qlin_s *h) {
    if (!h) return;
    if (h->codes) (void)hipFree(h->codes);
    if (h->sz) (void)hipFree(h->sz);
    if (h->ws) (void)hipFree(h->ws);
    if (h->counters) (void)hipFree(h->counters);
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
    // rows of partial sums the smallest feasible K split needs, for every M
    // a SKINNY launch can have (the other kernels need no split)
    h->ws_rows = kWsRowsMin;
    for (int M = 1; M <= kMaxSkinnyM; ++M) {
        const int s_min = min_split(M, h->Kb);
        if (s_min > 1) h->ws_rows = std::max(h->ws_rows, s_min * M);
    }

    void *canon = nullptr, *sc = nullptr, *zc = nullptr;
    hipError_t e = hipSuccess;
    auto bail = [&](const char *what, hipError_t e) -> qlin_t {
        if (e == hipErrorOutOfMemory) fail(QLIN_ERR_OOM, "device allocation failed (%s)", what);
        else hip_fail(e, what);
        if (canon) (void)hipFree(canon);
        if (sc) (void)hipFree(sc);
        if (zc) (void)hipFree(zc);
        free_handle(h);
        return nullptr;
    };
    if ((e = dev_alloc((void **)&h->codes, code_bytes)) != hipSuccess) return bail("codes", e);
    if ((e = dev_alloc(&h->sz, sz_bytes)) != hipSuccess) return bail("scales", e);
    if ((e = hipGetDevice(&h->device)) != hipSuccess) return bail("hipGetDevice", e);
    if ((e = hipDeviceGetAttribute(&h->num_cu, hipDeviceAttributeMultiprocessorCount, h->device)) != hipSuccess)
        return bail("hipDeviceGetAttribute", e);
    // arrival counters: one per column range of the decode kernels, or per
    // output block of a K-split tiled launch (at most one per CU)
    h->counters_n = std::max(h->Nt, h->num_cu);
    // partial sums: the decode kernels' smallest feasible split for every M,
    // and one 64 x 128 fp32 partial block per CU for a K-split tiled launch
    h->ws_decode = std::min(2 * (size_t)h->ws_rows * N, (size_t)0xFFFFFFF0u / 4);   // buffer descriptor range
    h->ws_floats = std::max(h->ws_decode, std::min((size_t)h->num_cu * 64 * 128, (size_t)0xFFFFFFF0u / 4));
    if ((e = dev_alloc((void **)&h->ws, h->ws_floats * 4)) != hipSuccess) return bail("workspace", e);
    if ((e = dev_alloc((void **)&h->counters, (size_t)h->counters_n * 4)) != hipSuccess) return bail("counters", e);
    if ((e = dev_alloc(&canon, code_bytes)) != hipSuccess) return bail("staging", e);
    if ((e = dev_alloc(&sc, ngroups * 2)) != hipSuccess) return bail("staging", e);
    if (!symmetric && (e = dev_alloc(&zc, ngroups * 2)) != hipSuccess) return bail("staging", e);

    static std::once_flag once;
    std::call_once(once, [] { (void)prepare_kernels(); (void)hipGetLastError(); });
    if ((e = hipMemcpy(canon, packed, code_bytes, hipMemcpyDefault)) != hipSuccess)
        return bail("copy codes", e);
    if ((e = hipMemcpy(sc, scales, ngroups * 2, hipMemcpyDefault)) != hipSuccess)
        return bail("copy scales", e);
    if (!symmetric && (e = hipMemcpy(zc, zeros, ngroups * 2, hipMemcpyDefault)) != hipSuccess)
        return bail("copy zeros", e);
    if ((e = hipMemset(h->counters, 0, (size_t)h->counters_n * 4)) != hipSuccess)
        return bail("hipMemset", e);
    if ((e = launch_repack((const uint32_t *)canon, (const uint16_t *)sc, (const uint16_t *)zc, h->codes, h->sz,
                           (int)K, (int)N, symmetric, nullptr)) != hipSuccess)
        return bail("repack launch", e);
    if ((e = hipDeviceSynchronize()) != hipSuccess) return bail("repack", e);
    (void)hipFree(canon);
    (void)hipFree(sc);
    if (zc) (void)hipFree(zc);
    return h;
}

// ------------------------------------------------------------------ planning

struct Plan {
    int path = 0;
    int kern = 0;
    int mrows = 0;     // template row count (GEMV: M; MFMA kernels: 16 * m-tiles)
    int S = 1, Gn = 1, grid = 1;
    int tn = 0;        // REGS/GEMV: tile slots (max tiles per range); SKINNY: staged x rows
    size_t lds = 0;
};

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
double plan_cost(const qlin_s *h, int kern, int M, int S, int Gn) {
    const int Kc = (h->Kb + S - 1) / S, Tn = (h->Nt + Gn - 1) / Gn;
    const int rounds = (S * Gn + h->num_cu - 1) / h->num_cu;
    const double blocks = (double)rounds * Tn * Kc;
    double t;
    if (kern == kKernStaged) {
        const double x_kib = (double)M * Kc * 256.0 / 1024.0;
        t = 4200.0 + 60.0 * blocks + 12.0 * rounds * x_kib;
    } else {
        t = 3300.0 + (60.0 + 3.5 * M) * blocks;
    }
    // never faster than streaming the weights at 6 TB/s
    const double blk = 1024.0 + (h->symmetric ? 32.0 : 64.0);
    t = std::max(t, (double)h->Nt * h->Kb * blk / 6.0e3);
    if (S > 1) t += 2500.0 + 100.0 * S;
    return t;
}

// Plans measured on MI355X (256 compute units) for the 4B decoder's linears
// where the cost model below picks a slower one: every kernel family and
// split from 1 to 8 was timed (HIP-graph replays over > 1 GiB of rotating
// weight copies) at M = 1, 2, 4, 8, 12 .. 16, and these won by 4-12%.
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

const TunedPlan *tuned_plan(const qlin_s *h, int M) {
    if (h->num_cu != 256) return nullptr;
    for (const TunedPlan &t : kTunedPlans)
        if (M >= t.m_lo && M <= t.m_hi && h->K == t.K && h->N == t.N) return &t;
    return nullptr;
}

// TILED plan: one launch over all M rows.  The block shape minimises
// (blocks per compute unit, rounded up) x (time of one block), with the
// block times measured on MI355X relative to the 128 x 256 shape (same K):
// 96 x 256 0.95, 64 x 128 0.42.  Ranked this way the three shapes come out
// in the measured order for every decoder linear at M = 512 .. 2048 (or
// within 2%): small blocks for narrow layers at small M, 96 x 256 where 128
// rows would leave part of the chip idle, 128 x 256 otherwise.
int make_tiled_plan(const qlin_s *h, int64_t split_k, int64_t M, Plan *p) {
    if (split_k < 0 || split_k > h->Kb) return fail(QLIN_ERR_INVALID, "split_k must be in [0, K/128]");
    if (M * h->K >= ((int64_t)1 << 31)) return fail(QLIN_ERR_UNSUPPORTED, "TILED path needs M * K < 2^31");
    constexpr int kShapes = (int)(sizeof kTiledShapes / sizeof kTiledShapes[0]);
    static const int forced = [] {                   // tuning knob: QLIN_TILED_SHAPE = index into kTiledShapes
        const char *e = getenv("QLIN_TILED_SHAPE");
        return e ? atoi(e) : -1;
    }();
    auto allowed = [&](int i) { return forced < 0 || forced >= kShapes || i == forced; };
    auto blocks_of = [&](int i) {
        const TiledShape c = kTiledShapes[i];
        return ((M + 16 * c.msw - 1) / (16 * c.msw)) * (int64_t)((h->Nt + 4 * c.nt - 1) / (4 * c.nt));
    };
    // Whole K range: the shape that minimises (blocks per compute unit,
    // rounded up) x (block time relative to 128 x 256).
    constexpr double kBlockTime[] = {1.0, 0.42, 0.95};
    static_assert(sizeof kBlockTime / sizeof kBlockTime[0] == kShapes, "");
    int best_i = -1, best_s = 1;
    double best = 1e300;
    for (int i = 0; i < kShapes; ++i) {
        if (!allowed(i)) continue;
        const double t = (double)((blocks_of(i) + h->num_cu - 1) / h->num_cu) * kBlockTime[i];
        if (t < best) { best = t; best_i = i; }
    }
    // A K split, when that leaves more than half the CUs idle (or when one is
    // asked for).  Time model in us: a pipeline ramp plus a time per 128-wide
    // group of K per block with every CU busy (128 x 256: 2.28, 64 x 128: 0.97,
    // 96 x 256: 2.17), times the rounds of work items over the CUs; a split
    // adds the exchange: ~3 us of latency plus the partial blocks written and
    // read back at ~4 TB/s.
    if (split_k > 1 || (split_k == 0 && blocks_of(best_i) * 2 <= h->num_cu)) {
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
            const int s_hi = split_k > 0 ? (int)split_k : std::min(16, h->Kb);
            for (int S = s_lo; S <= s_hi; ++S) {
                if (S > 1) {   // partial blocks and arrival counters must fit the handle's buffers
                    if (blocks > h->counters_n) continue;
                    if ((double)S * blocks * bm * bn > (double)h->ws_floats) continue;
                }
                const int Kc = (h->Kb + S - 1) / S;
                const double rounds = (double)((blocks * S + h->num_cu - 1) / h->num_cu);
                double t = rounds * (kRamp + kGroupTime[i] * Kc);
                if (S > 1) t += kExchange + 2.0 * S * blocks * bm * bn * 4.0 / kPartialBw;
                if (t < best) { best = t; best_i = i; best_s = S; }
            }
        }
    }
    if (best_i < 0) return fail(QLIN_ERR_UNSUPPORTED, "split_k=%d does not fit (workspace or counters)", (int)split_k);
    const TiledShape sh = kTiledShapes[best_i];
    const int Mt = (int)((M + 16 * sh.msw - 1) / (16 * sh.msw));
    const int Gn = (h->Nt + 4 * sh.nt - 1) / (4 * sh.nt);
    p->path = kTiled;
    p->kern = kKernTiled;
    p->mrows = 16 * sh.msw;
    p->S = best_s;
    p->Gn = Gn;
    p->tn = sh.nt;
    p->grid = 8 * ((Gn * Mt * best_s + 7) / 8);
    p->lds = 0;
    return QLIN_OK;
}

// Does the automatic choice run M rows through the TILED kernel (one
// launch) rather than 64-row slices of the decode kernels?  Above 64 rows,
// always: with its K split the tiled kernel also covers the narrow, deep
// layers at small M (measured on MI355X at M = 128: o projection 14.5 us
// against 35.9 us as two slices, down projection 21.8 us against 74.2 us).
bool auto_tiled(const qlin_s *h, int64_t M) {
    (void)h;
    return M > kMaxSkinnyM;
}

int make_plan(const qlin_s *h, int path, int64_t split_k, int64_t M, Plan *p) {
    const bool auto_pick = path == kAuto;
    if (path == kTiled) return make_tiled_plan(h, split_k, M, p);
    if (path == kAuto) path = (M <= gemv_max_auto()) ? kGemv : kSkinny;
    if (path != kGemv && path != kSkinny && path != kRegs) return fail(QLIN_ERR_INVALID, "unknown path %d", path);
    if (path == kGemv && M > kMaxGemvM) return fail(QLIN_ERR_UNSUPPORTED, "GEMV path needs M <= %d", kMaxGemvM);
    if (path == kRegs && M > 16) return fail(QLIN_ERR_UNSUPPORTED, "REGS path needs M <= 16");
    if (split_k < 0 || split_k > h->Kb) return fail(QLIN_ERR_INVALID, "split_k must be in [0, K/128]");
    const int Mi = (int)std::min<int64_t>(M, kMaxSkinnyM);
    p->path = path;
    // candidate kernel families: the forced one, or for the automatic choice
    // (path SKINNY reached from AUTO) both matrix-core kernels when M <= 16
    int kerns[2], nk = 0;
    if (path == kGemv) kerns[nk++] = kKernGemv;
    else if (path == kRegs) kerns[nk++] = kKernMfma16;
    else if (auto_pick && Mi <= 16) { kerns[nk++] = kKernMfma16; kerns[nk++] = kKernStaged; }
    else kerns[nk++] = kKernStaged;

    auto tn_max_of = [&](int kern) {
        return kern == kKernGemv ? kTnMaxGemv : kern == kKernMfma16 ? kTnMax : h->Nt;
    };
    auto rows_of = [&](int kern) { return kern == kKernGemv ? Mi : 16 * ((Mi + 15) / 16); };
    auto fits = [&](int kern, int S, int Gn) {
        const int Kc = (h->Kb + S - 1) / S, Tn = (h->Nt + Gn - 1) / Gn;
        if (S > 1 && (size_t)S * Gn * Tn * Mi * 16 > h->ws_decode) return false;
        if (Gn > h->counters_n || Tn > tn_max_of(kern)) return false;
        if (kern != kKernStaged) return lds_bytes_regs(rows_of(kern), Tn) <= kLdsMax;
        if (!chunk_fits(Mi, Kc)) return false;
        if ((int64_t)Tn * Kc >= 65536) return false;   // the kernel's block walk divides u < 2^16 by Kc
        if ((int64_t)Tn * h->Kb * 1024 >= ((int64_t)1 << 31)) return false;   // span of its buffer descriptors
        return lds_bytes(Mi, Kc, Tn) <= kLdsMax;
    };
    // column ranges for S chunks: one workgroup per CU (never more: a second
    // round of workgroups would double the time), but no range wider than the
    // kernel's tile limit (and more ranges if LDS demands).  Uneven ranges are
    // fine: splitting the columns over fewer, equal ranges leaves CUs idle,
    // and was measured slower.
    auto gn_for = [&](int kern, int S) {
        const int tm = tn_max_of(kern);
        int Gn = std::max((h->Nt + tm - 1) / tm, std::min(h->Nt, std::max(1, h->num_cu / S)));
        Gn = std::min(Gn, h->Nt);
        while (Gn < h->Nt && !fits(kern, S, Gn)) ++Gn;
        return Gn;
    };

    int bestK = -1, bestS = -1, bestGn = 1;
    // a measured plan for this shape, if it fits; otherwise the cost model
    bool tuned = false;
    if (auto_pick && path == kSkinny && split_k == 0) {
        if (const TunedPlan *t = tuned_plan(h, Mi)) {
            const int Gn = gn_for(t->kern, t->S);
            if (fits(t->kern, t->S, Gn)) { bestK = t->kern; bestS = t->S; bestGn = Gn; tuned = true; }
        }
    }
    double best = 1e300;
    for (int ki = 0; ki < nk && !tuned; ++ki) {
        const int kern = kerns[ki];
        const int s_lo = split_k > 0 ? (int)split_k : 1;
        const int s_hi = split_k > 0 ? (int)split_k : std::min(h->Kb, 64);
        for (int S = s_lo; S <= s_hi; ++S) {
            const int Gn = gn_for(kern, S);
            if (!fits(kern, S, Gn)) continue;
            const double c = plan_cost(h, kern, Mi, S, Gn);
            if (c < best) { best = c; bestK = kern; bestS = S; bestGn = Gn; }
        }
    }
    if (bestS < 0) {
        if (split_k > 0) return fail(QLIN_ERR_UNSUPPORTED, "split_k=%d does not fit (LDS or workspace)", (int)split_k);
        return fail(QLIN_ERR_UNSUPPORTED, "no work split fits this shape");
    }
    p->kern = bestK;
    p->mrows = rows_of(bestK);
    p->S = bestS;
    p->Gn = bestGn;
    p->grid = bestS * bestGn;
    const bool regs = bestK != kKernStaged;
    const int Kc = (h->Kb + bestS - 1) / bestS, Tn = (h->Nt + bestGn - 1) / bestGn;
    p->tn = regs ? Tn : bestK == kKernStaged ? staged_rows(Mi) : 0;
    const size_t need = regs ? lds_bytes_regs(p->mrows, Tn) : lds_bytes(Mi, Kc, Tn);
    // at least 80 KiB + 1 of LDS per workgroup keeps one workgroup per CU, so
    // the grid spreads over all CUs
    p->lds = std::max(need, (size_t)80 * 1024 + 256);
    return QLIN_OK;
}

int check_forward_args(const qlin_s *h, int64_t M, const uint16_t *x, const uint16_t *y) {
    if (!h) return fail(QLIN_ERR_INVALID, "NULL handle");
    if (M < 0) return fail(QLIN_ERR_INVALID, "M must be >= 0");
    if (M == 0) return QLIN_OK;
    if (M > kMaxM) return fail(QLIN_ERR_UNSUPPORTED, "M must be <= 65536");
    if (!x || !y) return fail(QLIN_ERR_INVALID, "NULL x or y");
    if (((uintptr_t)x | (uintptr_t)y) & 15) return fail(QLIN_ERR_ALIGN, "x and y must be 16-byte aligned");
    const uintptr_t xa = (uintptr_t)x, xe = xa + (uintptr_t)(M * h->K * 2);
    const uintptr_t ya = (uintptr_t)y, ye = ya + (uintptr_t)(M * h->N * 2);
    if (xa < ye && ya < xe) return fail(QLIN_ERR_INVALID, "y overlaps x");
    return QLIN_OK;
}

int run_forward(qlin_s *h, int path, int64_t split_k, int64_t M, const uint16_t *x, uint16_t *y, void *stream) {
    clear_err();
    int rc = check_forward_args(h, M, x, y);
    if (rc != QLIN_OK || M == 0) return rc;
    if (path == kSkinny && M > kMaxSkinnyM) return fail(QLIN_ERR_UNSUPPORTED, "SKINNY path needs M <= 64");
    if (path == kRegs && M > 16) return fail(QLIN_ERR_UNSUPPORTED, "REGS path needs M <= 16");
    if (path == kGemv && M > kMaxGemvM) return fail(QLIN_ERR_UNSUPPORTED, "GEMV path needs M <= %d", kMaxGemvM);
    if (path < kAuto || path > kRegs) return fail(QLIN_ERR_INVALID, "unknown path %d", path);
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    if (dev != h->device) return fail(QLIN_ERR_INVALID, "handle belongs to device %d, current is %d", h->device, dev);
    hipStream_t st = (hipStream_t)stream;
    if (path == kTiled || (path == kAuto && auto_tiled(h, M))) {
        Plan p;
        rc = make_tiled_plan(h, split_k, M, &p);
        if (rc != QLIN_OK) return rc;
        TiledArgs a;
        a.codes = h->codes;
        a.sz = h->sz;
        a.x = x;
        a.y = y;
        a.M = (int)M;
        a.K = (int)h->K;
        a.N = (int)h->N;
        a.Kb = h->Kb;
        a.Nt = h->Nt;
        a.Mt = (int)((M + p.mrows - 1) / p.mrows);
        a.Gn = p.Gn;
        a.S = p.S;
        a.Kq = h->Kb / p.S;
        a.Kr = h->Kb % p.S;
        a.ws = h->ws;
        a.counters = h->counters;
        a.ws_bytes = (uint32_t)(h->ws_floats * 4);
        e = launch_tiled(h->symmetric, TiledShape{p.mrows / 16, p.tn}, a, p.grid, st);
        if (e != hipSuccess) return hip_fail(e, "tiled launch");
        return QLIN_OK;
    }
    // GEMV / SKINNY / REGS: rows beyond 64 run as consecutive 64-row slices
    for (int64_t m0 = 0; m0 < M; m0 += kMaxSkinnyM) {
        const int64_t Ms = std::min<int64_t>(kMaxSkinnyM, M - m0);
        Plan p;
        rc = make_plan(h, path, split_k, Ms, &p);
        if (rc != QLIN_OK) return rc;
        FwdArgs a;
        a.codes = h->codes;
        a.sz = h->sz;
        a.x = x + m0 * h->K;
        a.y = y + m0 * h->N;
        a.ws = h->ws;
        a.counters = h->counters;
        a.M = (int)Ms;
        a.K = (int)h->K;
        a.N = (int)h->N;
        a.Kb = h->Kb;
        a.Nt = h->Nt;
        a.S = p.S;
        a.Gn = p.Gn;
        a.Nq = h->Nt / p.Gn;
        a.Nr = h->Nt % p.Gn;
        a.Kq = h->Kb / p.S;
        a.Kr = h->Kb % p.S;
        a.TnMax = a.Nq + (a.Nr > 0 ? 1 : 0);
        a.ws_bytes = (uint32_t)(h->ws_floats * 4);
        e = launch_forward(p.kern, p.mrows, p.tn, h->symmetric, p.grid, p.lds, a, st);
        if (e != hipSuccess) return hip_fail(e, "forward launch");
    }
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
    if (check_shape(K, N, group) != QLIN_OK) return g_status;
    if (!w || !scales || !packed) return fail(QLIN_ERR_INVALID, "NULL pointer");
    if (((uintptr_t)w & 15) || ((uintptr_t)packed & 3) || ((uintptr_t)scales & 1) || ((uintptr_t)zeros & 1))
        return fail(QLIN_ERR_ALIGN, "w must be 16-byte, packed 4-byte and scales/zeros 2-byte aligned");
    const uintptr_t wa = (uintptr_t)w, we = wa + (uintptr_t)(N * K * 2);
    const uintptr_t pa = (uintptr_t)packed, pe = pa + (uintptr_t)(N * K / 2);
    if (wa < pe && pa < we) return fail(QLIN_ERR_INVALID, "packed overlaps w");
    hipError_t e = launch_quantize(w, scales, zeros, packed, (int)K, (int)N, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "quantize launch");
    return QLIN_OK;
}

int qlin_forward(qlin_t h, int64_t M, const uint16_t *x, uint16_t *y, void *stream) {
    return run_forward(h, kAuto, 0, M, x, y, stream);
}

int qlin_forward_path(qlin_t h, int path, int64_t split_k, int64_t M, const uint16_t *x, uint16_t *y,
                      void *stream) {
    if (h && (split_k < 0 || split_k > h->Kb)) {
        clear_err();
        return fail(QLIN_ERR_INVALID, "split_k must be in [0, K/128]");
    }
    return run_forward(h, path, split_k, M, x, y, stream);
}

int qlin_plan(qlin_t h, int path, int64_t split_k, int64_t M, char *buf, int64_t buflen) {
    clear_err();
    if (!h) return fail(QLIN_ERR_INVALID, "NULL handle");
    if (!buf || buflen <= 0) return fail(QLIN_ERR_INVALID, "NULL buffer");
    if (M <= 0 || M > kMaxM) return fail(QLIN_ERR_INVALID, "M must be in [1, 65536]");
    if (path < kAuto || path > kRegs) return fail(QLIN_ERR_INVALID, "unknown path %d", path);
    if (path == kGemv && M > kMaxGemvM) return fail(QLIN_ERR_UNSUPPORTED, "GEMV path needs M <= %d", kMaxGemvM);
    if (path == kSkinny && M > kMaxSkinnyM) return fail(QLIN_ERR_UNSUPPORTED, "SKINNY path needs M <= 64");
    if (path == kRegs && M > 16) return fail(QLIN_ERR_UNSUPPORTED, "REGS path needs M <= 16");
    Plan p;
    const bool tiled = path == kTiled || (path == kAuto && auto_tiled(h, M));
    int rc = tiled ? make_tiled_plan(h, split_k, M, &p) : make_plan(h, path, split_k, std::min<int64_t>(M, kMaxSkinnyM), &p);
    if (rc != QLIN_OK) return rc;
    const int64_t slices = tiled ? 1 : (M + kMaxSkinnyM - 1) / kMaxSkinnyM;
    static const char *names[] = {"gemv", "regs", "skinny", "tiled"};
    snprintf(buf, (size_t)buflen, "path=%s kernel=%s grid=%d block=%d split=%d ranges=%d lds=%zu launches=%lld",
             names[p.kern], kernel_name(p.kern, p.mrows, p.tn, h->symmetric), p.grid,
             tiled ? kTiledWaves * 64 * tiled_wsplit(TiledShape{p.mrows / 16, p.tn}) : kThreads, p.S, p.Gn, p.lds,
             (long long)slices);
    return QLIN_OK;
}

void qlin_destroy(qlin_t h) {
    if (!h) return;
    int prev = -1;
    if (hipGetDevice(&prev) == hipSuccess && prev != h->device && hipSetDevice(h->device) == hipSuccess) {
        (void)hipDeviceSynchronize();
        free_handle(h);
        (void)hipSetDevice(prev);
        return;
    }
    (void)hipDeviceSynchronize();
    free_handle(h);
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

}  // extern "C"
