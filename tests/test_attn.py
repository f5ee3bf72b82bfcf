"""GPU parity of the drafter block attention (qlin_swa_attention) with the
float64 oracle, through the C ABI.

Tolerance (derived, not fitted).  The kernel rounds each softmax weight to
bf16 once (relative error <= 2^-9) and normalises by the sum of the rounded
weights, so the output is a convex combination of the visible value rows
with weights perturbed by a factor (1 + delta_j); then
|out - ref| <= 2 max|delta| max|v| / (1 - max|delta|).  delta also holds the
fp32 score error (at most D 2^-24 sum_d |q_d k_d| / sqrt(D) in exponent
units) and the exp2 error (< 2^-20).  The fp32 accumulation over n keys adds
n 2^-24 max|v|, and the final bf16 rounding 2^-9 |ref|.
"""

import numpy as np
import pytest
import torch

from oracle import attn_ref as ar
from paper_2607_04244_amd import qlin
from synth import gen

pytestmark = pytest.mark.gpu
D = 128


def dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def host_f64(t):
    return ar.bf16_to_f64(t.view(torch.int16).cpu().numpy().view(np.uint16))


def tolerance(q, k, v, T, W, ref):
    qf, kf, vf = ar.bf16_to_f64(q), ar.bf16_to_f64(k[:, :T]), ar.bf16_to_f64(v[:, :T])
    G = q.shape[0] // k.shape[0]
    score_abs = max(float((np.abs(qf[h]) @ np.abs(kf[h // G]).T).max()) for h in range(q.shape[0]))
    delta = 2.0 ** -9 + 2.0 ** -20 + D * 2.0 ** -24 * score_abs / np.sqrt(D)
    maxv = float(np.abs(vf).max())
    return 2.0 * delta / (1 - delta) * maxv + T * 2.0 ** -24 * maxv + 2.0 ** -9 * np.abs(ref) + 1e-30


def case(Hq, Hkv, nq, T, sigma_q=2.0, kv_stride=None, seed=0):
    rng = np.random.default_rng(seed)
    return gen.draw_attention(rng, Hq, Hkv, nq, T, sigma_q, kv_stride=kv_stride)


def run(q, k, v, T, W, splits=0, stream=None):
    qt, kt, vt = dev(q), dev(k), dev(v)
    out = qlin.swa_attention(qt, kt, vt, W, T=T, splits=splits)
    torch.cuda.synchronize()
    return out


def check(q, k, v, T, W, splits=0, what=""):
    out = run(q, k, v, T, W, splits)
    got = host_f64(out)
    ref = ar.swa_attention(q, k[:, :T], v[:, :T], W)
    tol = tolerance(q, k, v, T, W, ref)
    err = np.abs(got - ref)
    assert np.isfinite(got).all(), what
    bad = err > tol
    assert not bad.any(), f"{what}: {bad.sum()} outside tolerance, max err {err.max():.3e} (tol {tol.min():.3e}..)"
    return out


@pytest.mark.parametrize("Hq,Hkv,nq,T,W", [
    (8, 2, 16, 300, 64),        # window inside the cache, one 64-key tile of keys
    (8, 2, 16, 1000, 256),      # window, several tiles, ragged tail
    (8, 2, 16, 200, 256),       # T <= window: full-attention fallback
    (8, 2, 16, 1000, 0),        # no window
    (4, 4, 16, 130, 20),        # G = 1; half window smaller than the block
    (24, 8, 16, 500, 100),      # G = 3: one wave of the workgroup has no head
    (16, 2, 16, 700, 300),      # G = 8: two heads per wave
    (12, 2, 16, 333, 64),       # G = 6: the second head exists for two waves only
    (32, 16, 16, 300, 64),      # 16 key/value heads: two per XCD
    (8, 2, 5, 400, 128),        # ragged block: 5 queries
    (2, 1, 1, 1, 0),            # one token
    (2, 1, 16, 16, 0),          # cache = the block
    (8, 2, 16, 600, 101),       # odd window: half window 50 on each side
    (8, 2, 16, 257, 256),       # cache one token longer than the window
])
def test_matches_oracle(Hq, Hkv, nq, T, W):
    q, k, v = case(Hq, Hkv, nq, T, seed=T + W)
    check(q, k, v, T, W, what=f"{Hq}/{Hkv} nq={nq} T={T} W={W}")


@pytest.mark.parametrize("splits", [1, 2, 3, 7, 16, 256])
def test_forced_splits_match_oracle(splits):
    q, k, v = case(8, 2, 16, 1000, seed=5)
    check(q, k, v, 1000, 0, splits=splits, what=f"splits={splits}")


def test_cache_capacity_beyond_T_is_not_read():
    """kv_stride > T: the tokens after T (set to NaN here) must not matter."""
    T, cap = 250, 384
    q, k, v = case(8, 2, 16, T, kv_stride=cap, seed=7)
    k[:, T:] = 0x7FC0
    v[:, T:] = 0x7FC0
    for W in (0, 64):
        for splits in (1, 3):
            check(q, k, v, T, W, splits=splits, what=f"capacity W={W} splits={splits}")


def test_heads_beyond_two_gib_of_cache():
    """kv_stride = 2^23 tokens: key/value head 1 starts 2 GiB into each cache
    (byte offsets past 2^31); only the first T tokens of a head are filled."""
    T, W, cap = 300, 64, 1 << 23
    q, k, v = case(4, 2, 16, T, seed=11)
    kt = torch.zeros((2, cap, 128), dtype=torch.bfloat16, device="cuda")
    vt = torch.zeros((2, cap, 128), dtype=torch.bfloat16, device="cuda")
    kt[:, :T] = dev(k)
    vt[:, :T] = dev(v)
    for splits in (0, 3):
        out = qlin.swa_attention(dev(q), kt, vt, W, T=T, splits=splits)
        torch.cuda.synchronize()
        got = host_f64(out)
        ref = ar.swa_attention(q, k, v, W)
        bad = np.abs(got - ref) > tolerance(q, k, v, T, W, ref)
        assert not bad.any(), f"splits={splits}: {bad.sum()} outside tolerance"
    del kt, vt
    torch.cuda.empty_cache()


def test_window_of_one_returns_the_own_value_row_exactly():
    """W = 1: half window 0, each query sees only its own key (weight 1)."""
    T, nq = 200, 16
    q, k, v = case(8, 2, nq, T, seed=9)
    out = run(q, k, v, T, 1).view(torch.int16).cpu().numpy().view(np.uint16)
    for hq in range(8):
        assert np.array_equal(out[hq], v[hq // 4, T - nq:T]), hq


@pytest.mark.parametrize("Hq,Hkv,T,W,splits", [
    (8, 2, 600, 7, 0),          # half window 3: both edges inside the cache for most queries
    (8, 2, 600, 8, 1),          # even window, one key range
    (8, 2, 600, 9, 3),          # odd window, key ranges cut inside the window
    (8, 2, 2000, 41, 0),        # half window 20: right edges beyond the cache
    (8, 2, 2000, 40, 5),
    (32, 8, 8192, 1024, 0),     # the benchmarked swa1024 shape and plan
    (32, 8, 8192, 1025, 4),
    (32, 8, 8192, 2048, 0),     # swa2048
    (32, 8, 8192, 2049, 17),
])
def test_window_edge_is_exact(Hq, Hkv, T, W, splits):
    """The window edge, exactly.  With q = 0 every visible key gets weight 1
    (exp of 0, exact in bf16), so out = (sum of visible value rows) / n.
    Value rows are zero except markers: for block query i at position p,
    dimension 4 i + r holds 1 at key p - h - 1, p - h, p + h, p + h + 1
    (r = 0..3, h = W / 2, keys outside the cache skipped).  A key admitted
    or dropped at the edge changes a dimension from 0 to 1/n or back, so
    every dimension whose visible sum is 0 must come out as an exact zero,
    and every other within the rounding of 1/n's multiples."""
    nq = 16
    h = W // 2
    rng = np.random.default_rng(T + W)
    k = gen.draw_attention(rng, 1, Hkv, 1, T, 1.0)[1]
    q = np.zeros((Hq, nq, D), np.uint16)
    v = np.zeros((Hkv, T, D), np.uint16)
    for i in range(nq):
        p = T - nq + i
        for role, j in enumerate((p - h - 1, p - h, p + h, p + h + 1)):
            if 0 <= j < T:
                v[:, j, 4 * i + role] = 0x3F80
    out = host_f64(run(q, k, v, T, W, splits))
    vis = ar.visible(T, W, nq).astype(np.float64)
    vf = ar.bf16_to_f64(v)
    G = Hq // Hkv
    for hq in range(Hq):
        want = (vis @ vf[hq // G]) / vis.sum(axis=1, keepdims=True)      # [nq][D]
        got = out[hq]
        zero = want == 0
        assert np.all(got[zero] == 0), f"head {hq}: {np.argwhere((got != 0) & zero)[:5]} should be 0"
        assert np.all(np.abs(got[~zero] - want[~zero]) <= 2.0 ** -8 * want[~zero]), f"head {hq}"
        # each query's own markers: the two just outside the window are
        # exact zeros, the two on its edge are not
        for i in range(nq):
            p = T - nq + i
            assert got[i, 4 * i] == 0 and got[i, 4 * i + 3] == 0, (hq, i)
            if p - h >= 0:
                assert got[i, 4 * i + 1] > 0, (hq, i)
            if p + h < T:
                assert got[i, 4 * i + 2] > 0, (hq, i)


def test_zero_queries_average_the_visible_values():
    """q = 0: uniform weights, the output is the mean of the visible rows."""
    T, W = 600, 128
    _, k, v = case(8, 2, 16, T, seed=10)
    q = np.zeros((8, 16, D), np.uint16)
    out = host_f64(run(q, k, v, T, W))
    m = ar.visible(T, W)
    vf = ar.bf16_to_f64(v)
    for hq in range(8):
        for i in range(16):
            want = vf[hq // 4][m[i]].mean(axis=0)
            assert np.allclose(out[hq, i], want, rtol=2 ** -8, atol=2 ** -7 * np.abs(vf).max()), (hq, i)


def test_repeat_calls_are_bit_identical_and_splits_agree():
    q, k, v = case(8, 2, 16, 3000, seed=12)
    a = run(q, k, v, 3000, 1024, splits=5).view(torch.int16)
    b = run(q, k, v, 3000, 1024, splits=5).view(torch.int16)
    assert torch.equal(a, b)
    c = host_f64(run(q, k, v, 3000, 1024, splits=1))
    assert np.abs(c - host_f64(a.view(torch.bfloat16))).max() < 2 ** -6


def test_non_default_stream_and_caller_workspace():
    q, k, v = case(8, 2, 16, 900, seed=13)
    S, ws_bytes, _ = qlin.qlin_swa_plan(8, 2, D, 16, 900, 0, 4)
    assert S == 4 and ws_bytes > 0
    ws = torch.empty(ws_bytes, dtype=torch.uint8, device="cuda")
    qt, kt, vt = dev(q), dev(k), dev(v)
    ref = run(q, k, v, 900, 0, splits=4)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        out = qlin.swa_attention(qt, kt, vt, 0, splits=4, workspace=ws)
    s.synchronize()
    assert torch.equal(out.view(torch.int16), ref.view(torch.int16))


@pytest.mark.parametrize("name", ["swa1024", "swa2048", "full", "short"])
def test_drafter_workload_full_size(name):
    """The benchmarked workloads (32 query heads, 8 key/value heads, 16 block
    queries, T = 8192 or 700) in the launch configuration the benchmark
    times, every output element against the oracle."""
    c = gen.attention_case(name)
    check(c["q"], c["k"], c["v"], c["T"], c["window"], what=name)


def test_attention_argument_errors_on_device():
    q, k, v = case(8, 2, 16, 300, seed=14)
    qt, kt, vt = dev(q), dev(k), dev(v)
    with pytest.raises(qlin.QlinError) as e:
        qlin.swa_attention(qt, kt, vt, 0, T=301)          # T beyond the capacity
    assert e.value.code == qlin.QLIN_ERR_INVALID
    with pytest.raises(qlin.QlinError) as e:
        qlin.swa_attention(qt, kt, vt, 0, out=qt)        # out aliases q
    assert e.value.code == qlin.QLIN_ERR_INVALID
