// C ABI of the drafter block attention (include/qlin_attn.h): argument
// checks, the key-range split planner and the launches.

#include "../../include/qlin_attn.h"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdio>

#include "attn_internal.h"
#include "qlin_internal.h"

using namespace qlin;

namespace {

constexpr int64_t kMaxT = (int64_t)1 << 28;

struct AttnPlan {
    int G = 1, half = -1, lo = 0, hi = 0, ntiles = 0, tps = 1, S = 1;
    int64_t ws_bytes = 0;
};

int check_sizes(int64_t Hq, int64_t Hkv, int64_t D, int64_t nq, int64_t T, int64_t window, int64_t splits) {
    if (Hq <= 0 || Hkv <= 0 || Hq % Hkv) return fail(QLIN_ERR_INVALID, "Hq and Hkv must be positive, Hq a multiple of Hkv");
    if (D != kAttnD) return fail(QLIN_ERR_UNSUPPORTED, "head_dim must be 128 (got %lld)", (long long)D);
    if (Hq / Hkv > kAttnMaxG) return fail(QLIN_ERR_UNSUPPORTED, "at most 8 query heads per key/value head");
    if (Hq > 4096) return fail(QLIN_ERR_UNSUPPORTED, "at most 4096 query heads");
    if (nq < 1 || nq > kAttnQ) return fail(QLIN_ERR_INVALID, "nq must be in [1, 16]");
    if (T < nq || T > kMaxT) return fail(QLIN_ERR_INVALID, "T must be in [nq, 2^28]");
    if (window < 0) return fail(QLIN_ERR_INVALID, "window must be >= 0");
    if (splits < 0) return fail(QLIN_ERR_INVALID, "splits must be >= 0");
    return QLIN_OK;
}

// Key ranges per key/value head.  The automatic choice spreads the tiles
// over about one workgroup per compute unit.
int make_attn_plan(int64_t Hq, int64_t Hkv, int64_t nq, int64_t T, int64_t window, int64_t splits, AttnPlan *p) {
    p->G = (int)(Hq / Hkv);
    const bool full = window == 0 || T <= window;
    p->half = full ? -1 : (int)(window / 2);
    p->hi = (int)T;
    p->lo = full ? 0 : (int)std::max<int64_t>(0, T - nq - window / 2);
    p->ntiles = (p->hi - p->lo + kAttnTile - 1) / kAttnTile;
    int64_t S = splits;
    if (S == 0) {
        int dev = 0, cus = 0;
        hipError_t e = hipGetDevice(&dev);
        if (e == hipSuccess) e = hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev);
        if (e != hipSuccess) return hip_fail(e, "device query");
        S = std::max<int64_t>(1, cus / Hkv);
    }
    S = std::min<int64_t>({S, (int64_t)p->ntiles, (int64_t)kAttnMaxSplits});
    p->tps = (int)((p->ntiles + S - 1) / S);
    p->S = (p->ntiles + p->tps - 1) / p->tps;
    // partials of every (head, split) cover all 16 rows of the query tile
    p->ws_bytes = p->S > 1 ? (int64_t)p->S * Hq * kAttnQ * (kAttnD + 2) * 4 : 0;
    return QLIN_OK;
}

bool overlaps(const void *a, size_t an, const void *b, size_t bn) {
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + bn && b0 < a0 + an;
}

}  // namespace

extern "C" {

int qlin_swa_plan(int64_t Hq, int64_t Hkv, int64_t head_dim, int64_t nq, int64_t T, int64_t window,
                  int64_t splits, int64_t *splits_out, int64_t *workspace_bytes, char *buf, int64_t buflen) {
    clear_err();
    if (check_sizes(Hq, Hkv, head_dim, nq, T, window, splits) != QLIN_OK) return last_status();
    AttnPlan p;
    if (make_attn_plan(Hq, Hkv, nq, T, window, splits, &p) != QLIN_OK) return last_status();
    if (splits_out) *splits_out = p.S;
    if (workspace_bytes) *workspace_bytes = p.ws_bytes;
    if (buf && buflen > 0)
        snprintf(buf, (size_t)buflen, "kernel=%s keys=%d tiles=%d splits=%d grid=%lld combine=%d",
                 attn_kernel_name(p.G), p.hi - p.lo, p.ntiles, p.S, (long long)(Hkv * p.S), p.S > 1 ? 1 : 0);
    return QLIN_OK;
}

int qlin_swa_attention(int64_t Hq, int64_t Hkv, int64_t head_dim, int64_t nq, int64_t T, int64_t kv_stride,
                       int64_t window, int64_t splits, const uint16_t *q, const uint16_t *k, const uint16_t *v,
                       uint16_t *out, void *workspace, int64_t workspace_bytes, void *stream) {
    clear_err();
    if (check_sizes(Hq, Hkv, head_dim, nq, T, window, splits) != QLIN_OK) return last_status();
    if (kv_stride < T || kv_stride > kMaxT) return fail(QLIN_ERR_INVALID, "kv_stride must be in [T, 2^28]");
    if (!q || !k || !v || !out) return fail(QLIN_ERR_INVALID, "NULL q, k, v or out");
    if (workspace_bytes < 0) return fail(QLIN_ERR_INVALID, "workspace_bytes must be >= 0");
    if (((uintptr_t)q | (uintptr_t)k | (uintptr_t)v | (uintptr_t)out | (uintptr_t)workspace) & 15)
        return fail(QLIN_ERR_ALIGN, "q, k, v, out and workspace must be 16-byte aligned");
    AttnPlan p;
    if (make_attn_plan(Hq, Hkv, nq, T, window, splits, &p) != QLIN_OK) return last_status();
    if (p.ws_bytes > 0 && (!workspace || workspace_bytes < p.ws_bytes))
        return fail(QLIN_ERR_INVALID, "workspace of %lld bytes needed (%lld given)", (long long)p.ws_bytes,
                    (long long)(workspace ? workspace_bytes : 0));
    const size_t qo_bytes = (size_t)Hq * nq * kAttnD * 2;
    const size_t kv_bytes = ((size_t)(Hkv - 1) * kv_stride + T) * kAttnD * 2;
    if (overlaps(out, qo_bytes, q, qo_bytes) || overlaps(out, qo_bytes, k, kv_bytes) ||
        overlaps(out, qo_bytes, v, kv_bytes) || (p.ws_bytes && overlaps(out, qo_bytes, workspace, p.ws_bytes)))
        return fail(QLIN_ERR_INVALID, "out overlaps an input or the workspace");

    AttnArgs a;
    a.q = q;
    a.k = k;
    a.v = v;
    a.out = out;
    a.ws_o = (float *)workspace;
    a.ws_ml = p.S > 1 ? (float *)workspace + (size_t)p.S * Hq * kAttnQ * kAttnD : nullptr;
    a.kv_stride = kv_stride * kAttnD;
    a.Hq = (int)Hq;
    a.Hkv = (int)Hkv;
    a.G = p.G;
    a.nq = (int)nq;
    a.T = (int)T;
    a.lo = p.lo;
    a.hi = p.hi;
    a.half = p.half;
    a.ntiles = p.ntiles;
    a.tps = p.tps;
    a.S = p.S;
    a.c = (float)(1.4426950408889634 / std::sqrt((double)kAttnD));
    hipError_t e = launch_attn(a, (hipStream_t)stream);
    if (e != hipSuccess) return hip_fail(e, "attention launch");
    return QLIN_OK;
}

}  // extern "C"
