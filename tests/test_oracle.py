"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these tests compares the oracle with a retyped copy of itself: each
uses hand-derived golden values, an exhaustive comparison against torch's own
binary32 multiply and bf16 conversion, integer arithmetic, a correctly rounded
sum (math.fsum), or an invariant of the definition.  CPU only.
"""

import json
import math
import os

import numpy as np
import pytest
import torch

from oracle import qlin_ref as ref
from synth import gen


def _hex(s):
    return int(s, 16)


# ---------------------------------------------------------------- P1 packing

def test_nibble_order_golden(golden_dir):
    fx = json.load(open(os.path.join(golden_dir, "nibble_order.json")))
    for case in fx["cases"]:
        P = np.array([[_hex(case["word"])]], dtype=np.uint32)
        assert ref.unpack_codes(P)[0].tolist() == case["codes"], case["word"]
        assert ref.pack_codes(np.array([case["codes"]]))[0, 0] == _hex(case["word"])


def test_pack_unpack_round_trip():
    rng = np.random.default_rng(11)
    P = rng.integers(0, 2 ** 32, size=(37, 48), dtype=np.uint32)
    assert np.array_equal(ref.pack_codes(ref.unpack_codes(P)), P)
    Q = rng.integers(0, 16, size=(13, 256), dtype=np.uint8)
    assert np.array_equal(ref.unpack_codes(ref.pack_codes(Q)), Q)


def test_unpack_is_a_bijection_on_a_word():
    # every nibble position reaches a distinct code slot
    for i in range(8):
        P = np.array([[np.uint32(0xF) << np.uint32(4 * i)]], dtype=np.uint32)
        q = ref.unpack_codes(P)[0]
        assert q[i] == 15 and q.sum() == 15


# ---------------------------------------------------------------- P2 dequant rounding

def test_dequant_rounding_golden(golden_dir):
    fx = json.load(open(os.path.join(golden_dir, "dequant_rounding.json")))
    for c in fx["cases"]:
        q = np.full((1, 128), c["q"], dtype=np.uint8)
        P = ref.pack_codes(q)
        s = np.array([[_hex(c["s"])]], dtype=np.uint16)
        z = np.array([[_hex(c["z"])]], dtype=np.uint16)
        w = ref.dequant_bf16(P, s, z)
        assert np.all(w == _hex(c["w"])), (c, hex(int(w[0, 0])))


def _all_finite_bf16():
    b = np.arange(1 << 16, dtype=np.uint32).astype(np.uint16)
    exp = (b >> 7) & 0xFF
    return b[exp != 0xFF]          # 65,280 finite patterns (incl. +-0, denormals)


def test_dequant_exhaustive_vs_torch():
    """Every finite bf16 scale x every (q - z) in [-15, 15]: the oracle's
    single RNE of the exact product equals torch's binary32 multiply followed
    by torch's bf16 conversion (binary32 holds every such product exactly
    unless it overflows, in which case both give +-inf)."""
    S = _all_finite_bf16()
    N = S.size
    assert N == 65280
    codes = np.tile(np.arange(16, dtype=np.uint8), 16)          # 256 codes
    q = np.broadcast_to(codes, (N, 256)).copy()
    P = ref.pack_codes(q)
    scales = np.stack([S, S], axis=1)
    zeros = np.empty((N, 2), dtype=np.uint16)
    zeros[:, 0] = 0x0000                                         # z = 0  -> d in [0, 15]
    zeros[:, 1] = 0x4170                                         # z = 15 -> d in [-15, 0]
    with np.errstate(over="ignore"):
        w = ref.dequant_bf16(P, scales, zeros)

    d = torch.from_numpy((codes.astype(np.int32) - np.repeat([0, 15], 128)).astype(np.float32))
    s32 = torch.from_numpy((S.astype(np.uint32) << 16).view(np.float32).copy())
    prod = s32[:, None] * d[None, :]                            # binary32 products
    expect = prod.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    # torch keeps the sign of zero: (+-0 or -s) * 0 may give -0; the oracle's
    # (q - z) * s with q == z gives 0 * s, which is -0 only for negative s.
    same = (w == expect) | ((w & 0x7FFF) == 0) & ((expect & 0x7FFF) == 0)
    assert same.all(), np.argwhere(~same)[:5]
    # and the float64 product is exact in binary32 wherever binary32 is finite
    exact = ref.dequant_exact(P, scales, zeros)
    fin = torch.isfinite(prod).numpy()
    assert np.array_equal(prod.numpy().astype(np.float64)[fin], exact[fin])


def test_power_of_two_scales_are_exact():
    # s = 2**e, |q - z| in {0, 1, 2, 4, 8}: w = (q - z) * s with no rounding
    for e in (-20, -7, 0, 5):
        s_bits = np.uint16(((127 + e) << 7))
        for q, z in ((8, 8), (9, 8), (10, 8), (12, 8), (0, 8), (15, 7)):
            w = ref.dequant_bf16(ref.pack_codes(np.full((1, 128), q, np.uint8)),
                                 np.array([[s_bits]]), np.array([[ref.rne_bf16(float(z))]]))
            assert ref.bf16_to_f64(w[0, 0]) == (q - z) * 2.0 ** e


def test_zero_code_gives_plus_zero():
    for z in range(16):
        q = np.full((1, 128), z, dtype=np.uint8)
        w = ref.dequant_bf16(ref.pack_codes(q), np.array([[0x3C23]], np.uint16),
                             np.array([[ref.rne_bf16(float(z))]], np.uint16))
        assert np.all(w == 0)


def test_group_and_column_indexing_closed_form():
    """s[n, g] = 2**(n - g), every code = z + 1  =>  w[n, k] = 2**(n - k//128)."""
    N, K = 5, 512
    G = K // 128
    z = np.array([[(n + g) % 15 for g in range(G)] for n in range(N)])
    q = np.repeat(z + 1, 128, axis=1).astype(np.uint8)
    s = np.array([[(127 + n - g) << 7 for g in range(G)] for n in range(N)], dtype=np.uint16)
    zb = ref.rne_bf16(z.astype(np.float64))
    w = ref.bf16_to_f64(ref.dequant_bf16(ref.pack_codes(q), s, zb))
    k = np.arange(K)
    for n in range(N):
        assert np.array_equal(w[n], 2.0 ** (n - k // 128))


def test_symmetric_zeros_are_eight():
    z = ref.symmetric_zeros(3, 256)
    assert z.shape == (3, 2) and np.all(ref.bf16_to_f64(z) == 8.0)


def test_rne_bf16_matches_torch_on_random_binary32():
    rng = np.random.default_rng(5)
    u = rng.integers(0, 2 ** 32, size=200_000, dtype=np.uint32)
    f = u.view(np.float32)
    f = f[np.isfinite(f)]
    with np.errstate(over="ignore"):
        mine = ref.rne_bf16(f.astype(np.float64))
    theirs = torch.from_numpy(f.copy()).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(mine, theirs)


def test_rne_bf16_rejects_inexact_binary32():
    with pytest.raises(ValueError):
        ref.rne_bf16(1.0 + 2.0 ** -40)


# ---------------------------------------------------------------- P3 matmul

def test_forward_golden_tiny(golden_dir):
    fx = json.load(open(os.path.join(golden_dir, "tiny_forward.json")))
    K, N, M = fx["K"], fx["N"], fx["M"]
    P = np.stack([np.full(K // 8, _hex(w), dtype=np.uint32) for w in fx["column_words"]])
    s = np.array([[_hex(v) for v in row] for row in fx["scales"]], dtype=np.uint16)
    z = np.array([[_hex(v) for v in row] for row in fx["zeros"]], dtype=np.uint16)
    x = np.empty((M, K), dtype=np.uint16)
    for m, row in enumerate(fx["x_rows"]):
        x[m, :128] = _hex(row["k_lt_128"])
        x[m, 128:] = _hex(row["k_ge_128"])
    y = ref.forward(x, P, s, z)
    assert np.array_equal(y, np.array(fx["y"]))


@pytest.mark.parametrize("K", [128, 256])
@pytest.mark.parametrize("N", [1, 3, 8])
def test_forward_brute_force_fsum(K, N):
    c = gen.random_case(100 + K + N, 1, K, N)
    y = ref.forward(c["x"], c["packed"], c["scales"], c["zeros"])
    w = ref.bf16_to_f64(ref.dequant_bf16(c["packed"], c["scales"], c["zeros"]))
    x = ref.bf16_to_f64(c["x"])[0]
    for n in range(N):
        terms = [float(x[k]) * float(w[n, k]) for k in range(K)]
        exact = math.fsum(terms)                      # correctly rounded sum
        bound = K * 2.0 ** -53 * math.fsum(abs(t) for t in terms)
        assert abs(y[0, n] - exact) <= bound


def test_forward_matches_torch_float64_matmul():
    c = gen.random_case(7, 5, 640, 48)
    y = ref.forward(c["x"], c["packed"], c["scales"], c["zeros"])
    w = torch.from_numpy(ref.bf16_to_f64(ref.dequant_bf16(c["packed"], c["scales"], c["zeros"])))
    x = torch.from_numpy(c["x"].astype(np.int16)).view(torch.bfloat16).to(torch.float64)
    yt = (x @ w.T).numpy()
    assert np.allclose(y, yt, rtol=1e-12, atol=1e-12)


# ---------------------------------------------------------------- P4 linearity

def test_linearity_disjoint_supports_and_power_of_two():
    c = gen.random_case(8, 3, 384, 32)
    x = c["x"]
    x1 = x.copy(); x1[:, 1::2] = 0        # even k only
    x2 = x.copy(); x2[:, 0::2] = 0        # odd k only  (x1 + x2 == x exactly)
    args = (c["packed"], c["scales"], c["zeros"])
    y, y1, y2 = (ref.forward(v, *args) for v in (x, x1, x2))
    scale = np.abs(ref.bf16_to_f64(x)) @ np.abs(ref.bf16_to_f64(ref.dequant_bf16(*args))).T
    assert np.all(np.abs(y - (y1 + y2)) <= 384 * 2.0 ** -52 * scale + 1e-300)
    # multiplying x by 2**j (exponent + j, no overflow here) scales y exactly
    x4 = (x.astype(np.uint32) + np.where((x & 0x7F80) != 0, 2 << 7, 0)).astype(np.uint16)
    nz = (x & 0x7F80) != 0
    assert np.array_equal(ref.bf16_to_f64(x4)[nz], 4.0 * ref.bf16_to_f64(x)[nz])
    xs = np.where(nz, x4, 0).astype(np.uint16)
    xb = np.where(nz, x, 0).astype(np.uint16)
    assert np.array_equal(ref.forward(xs, *args), 4.0 * ref.forward(xb, *args))


# ---------------------------------------------------------------- P5 / P6 / P7

def test_all_codes_equal_zero_point_gives_zero():
    rng = np.random.default_rng(3)
    N, K = 24, 512
    z = rng.integers(0, 16, size=(N, K // 128))
    q = np.repeat(z, 128, axis=1).astype(np.uint8)
    c = gen.random_case(4, 4, K, N)
    y = ref.forward(c["x"], ref.pack_codes(q), c["scales"], ref.rne_bf16(z.astype(np.float64)))
    assert np.all(y == 0.0)


def test_one_hot_rows_select_weights():
    c = gen.random_case(9, 6, 512, 40)
    ks = [0, 1, 127, 128, 300, 511]
    x = np.zeros((6, 512), dtype=np.uint16)
    for m, k in enumerate(ks):
        x[m, k] = 0x3F80                   # 1.0
    y = ref.forward(x, c["packed"], c["scales"], c["zeros"])
    w = ref.bf16_to_f64(ref.dequant_bf16(c["packed"], c["scales"], c["zeros"]))
    for m, k in enumerate(ks):
        assert np.array_equal(y[m], w[:, k])


def test_integer_case_equals_integer_matmul():
    """s = 1, z = 8 (symmetric format), x in {-1, 0, 1}: y = x . (Q - 8)^T in
    integers, computed here with int64 numpy arithmetic."""
    rng = np.random.default_rng(12)
    M, K, N = 7, 1024, 33
    Q = rng.integers(0, 16, size=(N, K), dtype=np.uint8)
    xi = rng.integers(-1, 2, size=(M, K))
    x = np.select([xi == 1, xi == -1], [0x3F80, 0xBF80], 0).astype(np.uint16)
    s = np.full((N, K // 128), 0x3F80, dtype=np.uint16)
    z = ref.symmetric_zeros(N, K)
    y = ref.forward(x, ref.pack_codes(Q), s, z)
    yi = xi.astype(np.int64) @ (Q.astype(np.int64) - 8).T
    assert np.array_equal(y, yi.astype(np.float64))
    # integers below 2**24 round to bf16 exactly as torch rounds them
    yb = ref.round_output(y)
    tb = torch.from_numpy(yi.astype(np.float32)).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    assert np.array_equal(yb, tb)


# ---------------------------------------------------------------- comparison rule

def test_ulp_and_tolerance():
    assert ref.ulp_bf16(1.0) == 2.0 ** -7
    assert ref.ulp_bf16(1.99) == 2.0 ** -7
    assert ref.ulp_bf16(2.0) == 2.0 ** -6
    assert ref.ulp_bf16(-0.75) == 2.0 ** -8
    assert ref.tolerance(0.0) == 1e-3
    assert ref.tolerance(100.0) == 2 * 2.0 ** -1


def test_compare_accepts_two_ulp_and_rejects_more():
    y_ref = np.array([[100.0, -3.0, 0.0]])
    ok = ref.rne_bf16(np.array([[100.0 + 1.0, -3.0 - 2 ** -6, 0.0009765625]]))
    assert ref.compare(ok, y_ref)["ok"]
    bad = ref.rne_bf16(np.array([[100.0 + 1.5, -3.0, 0.0]]))
    r = ref.compare(bad, y_ref)
    assert not r["ok"] and r["nbad"] == 1


def test_rounding_reading_matters():
    """The unrounded-weight reading differs from the bf16-weight reading by more
    than the tolerance on a visible share of outputs, so a kernel cannot mix
    them (this is why the oracle rounds each weight once)."""
    c = gen.random_case(21, 4, 2560, 256)
    args = (c["x"], c["packed"], c["scales"], c["zeros"])
    y_b = ref.forward(*args)
    y_e = ref.forward(*args, mode="exact")
    with np.errstate(over="ignore"):
        r = ref.compare(ref.rne_bf16(y_e.astype(np.float32).astype(np.float64)), y_b)
    assert r["nbad"] > 0.01 * y_b.size


# ---------------------------------------------------------------- P8 generator

def test_generator_distributions():
    c = gen.linear_case(2, M=16)
    q = ref.unpack_codes(c["packed"][:256])
    hist = np.bincount(q.ravel(), minlength=16) / q.size
    assert np.all(np.abs(hist - 1 / 16) < 0.01)
    s = ref.bf16_to_f64(c["scales"])
    assert s.min() >= 0.001 * (1 - 2 ** -8) and s.max() <= 0.01 * (1 + 2 ** -8)
    assert set(np.unique(ref.bf16_to_f64(c["zeros"]))) == {7.0, 8.0, 9.0}
    x = ref.bf16_to_f64(c["x"])
    big = np.abs(x) > 4.0 * 0.5 * 2.5          # beyond ~5 sigma of N(0, 0.5^2)
    assert 0.004 < big.mean() < 0.02            # ~1% outliers x20
    core = x[~big]
    assert abs(core.mean()) < 0.02 and abs(core.std() - 0.5) < 0.03


def test_generator_is_seeded():
    a = gen.linear_case(0)
    b = gen.linear_case(0)
    for k in ("packed", "scales", "zeros", "x"):
        assert np.array_equal(a[k], b[k])
    assert a["x"].shape == (1, 2560) and a["packed"].shape == (2560, 320)


# ---------------------------------------------------------------- fixed-grid RTN quantization

def _rtn_fixture():
    import json
    import os
    with open(os.path.join(os.path.dirname(__file__), "golden", "rtn_rounding.json")) as f:
        return json.load(f)["cases"]


def test_rtn_golden_rounding():
    """Hand-worked ties, zero-points and clamps (golden fixture)."""
    for c in _rtn_fixture():
        w = np.full((1, 128), int(c["w"], 16), np.uint16)
        s = np.array([[int(c["s"], 16)]], np.uint16)
        z = ref.rne_bf16(np.array([[float(c["z"])]]))
        q = ref.quantize_rtn(w, s, z)
        assert np.all(q == c["code"]), c


def test_rtn_inverts_dequantization_exhaustively():
    """quantize(dequant(q)) == q for every code and zero-point over every
    positive normal bf16 scale in [2^-100, 2^100]: the bf16 rounding of
    (q - z) s moves the quotient by at most 15 * 2^-9 < 1/2."""
    sb = np.arange(0x0000, 0x7F80, dtype=np.uint32).astype(np.uint16)   # finite, non-negative
    sv = ref.bf16_to_f64(sb)
    sb = sb[(sv >= 2.0 ** -100) & (sv <= 2.0 ** 100)]
    q = np.arange(16, dtype=np.uint8)
    for z in range(16):
        zz = ref.rne_bf16(np.full((sb.size, 1), float(z)))
        # one row per scale, one group of 128 columns holding every code 8 times
        codes = np.tile(np.repeat(q, 8), (sb.size, 1))
        packed = ref.pack_codes(codes)
        w = ref.dequant_bf16(packed, sb.reshape(-1, 1), zz)
        assert np.array_equal(ref.quantize_rtn(w, sb.reshape(-1, 1), zz), codes), f"z={z}"


def test_rtn_is_monotone_and_clamped():
    """Codes never decrease as w grows (fixed s, z) and stay in [0, 15]."""
    wv = np.linspace(-40.0, 40.0, 4096).astype(np.float32).astype(np.float64)
    wb = ref.rne_bf16(wv).reshape(32, 128)          # rounding keeps the order
    for s_val, z in ((1.0, 8), (0.375, 3), (2.5, 12)):
        s = np.repeat(ref.rne_bf16(np.array([[s_val]])), 32, 0)
        zz = np.repeat(ref.rne_bf16(np.array([[float(z)]])), 32, 0)
        q = ref.quantize_rtn(wb, s, zz).ravel()
        assert np.all(np.diff(q.astype(int)) >= 0) and q.min() == 0 and q.max() == 15


def test_rtn_nan_quotient_gives_zero_point_and_pack_layout():
    w = np.zeros((2, 128), np.uint16)                      # w = 0
    s = np.array([[0x0000], [0x3F80]], np.uint16)          # s = 0 (0/0 = NaN), s = 1
    z = ref.rne_bf16(np.array([[5.0], [9.0]]))
    q = ref.quantize_rtn(w, s, z)
    assert np.all(q[0] == 5) and np.all(q[1] == 9)
    p = ref.quantize_pack(w, s, z)
    assert p.shape == (2, 16) and np.all(p[0] == 0x55555555) and np.all(p[1] == 0x99999999)
