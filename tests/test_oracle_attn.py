"""Pins of the drafter block-attention oracle (CPU only): closed forms, brute
force on tiny inputs, the full-attention fallback and the head mapping."""

import numpy as np

from oracle import attn_ref as ar
from oracle import qlin_ref as ref


def _bf16(a):
    return ref.rne_bf16(np.asarray(a, np.float32).astype(np.float64))


def _rand(rng, *shape, scale=1.0):
    return _bf16(rng.standard_normal(shape) * scale)


def test_visibility_window_edges():
    T, W = 100, 40
    m = ar.visible(T, W)
    for i in range(16):
        p = T - 16 + i
        idx = np.nonzero(m[i])[0]
        assert idx.min() == p - 20 and idx.max() == min(T - 1, p + 20)
    assert ar.visible(40, 40).all() and ar.visible(100, 0).all()     # fallback / no window


def test_uniform_scores_average_the_visible_values():
    """q = 0: every visible key gets the same weight, so the output is the
    plain mean of the visible value rows."""
    rng = np.random.default_rng(1)
    Hq, Hkv, T, D, W = 4, 2, 300, 128, 64
    q = np.zeros((Hq, 16, D), np.uint16)
    k = _rand(rng, Hkv, T, D)
    v = _rand(rng, Hkv, T, D)
    out = ar.swa_attention(q, k, v, W)
    vv = ar.bf16_to_f64(v)
    m = ar.visible(T, W)
    for h in range(Hq):
        for i in range(16):
            assert np.allclose(out[h, i], vv[h // 2][m[i]].mean(axis=0), rtol=1e-12, atol=1e-12)


def test_dominant_key_returns_its_value_row():
    """A key whose score exceeds every other visible score by > 60 gets all
    the weight (to within e^-60)."""
    rng = np.random.default_rng(2)
    Hq, Hkv, T, D, W = 2, 1, 64, 128, 0
    q = np.zeros((Hq, 16, D))
    q[:, :, 0] = 1.0
    k = rng.standard_normal((Hkv, T, D)) * 0.01
    k[0, 37, 0] = 800.0                                # score 800 / sqrt(128) ~ 70.7
    v = rng.standard_normal((Hkv, T, D))
    out = ar.swa_attention(_bf16(q), _bf16(k), _bf16(v), W)
    target = ar.bf16_to_f64(_bf16(v))[0, 37]
    assert np.allclose(out, np.broadcast_to(target, out.shape), atol=1e-12)


def test_matches_brute_force_loops():
    """Vectorized oracle vs explicit loops with math.fsum on tiny inputs,
    windowed, fallback and grouped heads."""
    rng = np.random.default_rng(3)
    for Hq, Hkv, T, D, W in ((2, 1, 40, 8, 10), (4, 2, 30, 16, 64), (3, 3, 24, 8, 4)):
        q = _rand(rng, Hq, 16, D)
        k = _rand(rng, Hkv, T, D)
        v = _rand(rng, Hkv, T, D)
        a = ar.swa_attention(q, k, v, W)
        b = ar.swa_attention_loops(q, k, v, W)
        assert np.allclose(a, b, rtol=1e-12, atol=1e-13), (Hq, Hkv, T, D, W)


def test_fallback_equals_unmasked_attention():
    rng = np.random.default_rng(4)
    q = _rand(rng, 2, 16, 128)
    k = _rand(rng, 1, 200, 128)
    v = _rand(rng, 1, 200, 128)
    assert np.array_equal(ar.swa_attention(q, k, v, 256), ar.swa_attention(q, k, v, 0))
    assert not np.allclose(ar.swa_attention(q, k, v, 64), ar.swa_attention(q, k, v, 0))


def test_grouped_heads_read_their_kv_head():
    """Query head h uses key/value head h // G: permuting the KV heads
    permutes the output groups accordingly."""
    rng = np.random.default_rng(5)
    Hq, Hkv = 8, 4
    q = _rand(rng, Hq, 16, 128)
    k = _rand(rng, Hkv, 120, 128)
    v = _rand(rng, Hkv, 120, 128)
    perm = np.array([2, 0, 3, 1])
    out = ar.swa_attention(q, k, v, 32)
    qp = q.reshape(Hkv, 2, 16, 128)[perm].reshape(Hq, 16, 128)
    outp = ar.swa_attention(qp, k[perm], v[perm], 32)
    assert np.array_equal(outp.reshape(Hkv, 2, 16, 128), out.reshape(Hkv, 2, 16, 128)[perm])


def test_two_keys_closed_form_fixes_the_score_scale():
    """Scores are q.k / sqrt(128): the standard scaled dot-product attention
    the drafter of Sec. 2.3 uses, whose scale the paper does not spell out
    (a reading; head dimension 128).  One query, two keys: q = 7.84375 e0 (exact in bf16),
    k0 = e0, k1 = 0, so the scores are 7.84375 / sqrt(128) = 0.693296 (ln 2 +
    1.5e-4) and 0; with v0 = 1, v1 = 0 every output element is
    e^s / (e^s + 1) = 2/3 + 3.31e-5.  A missing or different scale gives
    0.9996 (none), 0.727 (1/8) or 0.515 (1/128)."""
    D = 128
    q = np.zeros((1, 1, D))
    q[0, 0, 0] = 7.84375
    k = np.zeros((1, 2, D))
    k[0, 0, 0] = 1.0
    v = np.zeros((1, 2, D))
    v[0, 0, :] = 1.0
    out = ar.swa_attention(_bf16(q), _bf16(k), _bf16(v), 0)
    assert np.all(np.abs(out - (2.0 / 3.0 + 3.31e-5)) < 1e-6)
