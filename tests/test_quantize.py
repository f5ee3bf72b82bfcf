"""GPU parity of qlin_quantize (fixed-grid round-to-nearest + packing) with
the CPU oracle, bit-exact on every packed word (needs an MI355X)."""

import numpy as np
import pytest
import torch

from oracle import qlin_ref as ref
from paper_2607_04244_amd import qlin
from synth import gen

pytestmark = pytest.mark.gpu


def dev16(a):
    return torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()


def host_words(t):
    torch.cuda.synchronize()
    return t.cpu().numpy().view(np.uint32)


def _weights_near_grid(rng, N, K, scales, zeros, spread=0.7):
    """bf16 weights around the grid points (q - z) s, with exact ties planted:
    (q - z + 1/2) s is a bf16 value whenever s is a power of two."""
    s = np.repeat(ref.bf16_to_f64(scales), 128, axis=1)
    z = np.repeat(ref.bf16_to_f64(zeros), 128, axis=1)
    q = rng.integers(-2, 18, size=(N, K))                 # a few beyond the clamp
    off = rng.uniform(-spread, spread, size=(N, K))
    tie = rng.random((N, K)) < 0.05
    off[tie] = 0.5 * np.sign(rng.standard_normal(tie.sum()))
    w = ((q - z) + off) * s
    return ref.rne_bf16(w.astype(np.float32).astype(np.float64))


@pytest.mark.parametrize("symmetric", [False, True])
@pytest.mark.parametrize("N,K", [(16, 128), (48, 384), (208, 1152), (1024, 2560)])
def test_quantize_matches_oracle(N, K, symmetric):
    rng = np.random.default_rng(N + K + symmetric)
    e = rng.integers(-8, 3, size=(N, K // 128))
    pow2 = rng.random((N, K // 128)) < 0.5                # power-of-two scales make ties exact
    sv = np.where(pow2, 2.0 ** e, rng.uniform(0.002, 0.05, size=(N, K // 128)))
    scales = ref.rne_bf16(sv.astype(np.float32).astype(np.float64))
    zeros = ref.symmetric_zeros(N, K) if symmetric else ref.rne_bf16(rng.integers(0, 16, size=(N, K // 128)).astype(np.float64))
    w = _weights_near_grid(rng, N, K, scales, zeros)
    got = host_words(qlin.quantize(dev16(w), dev16(scales), None if symmetric else dev16(zeros)))
    assert np.array_equal(got, ref.quantize_pack(w, scales, zeros))


def test_quantize_special_values():
    """Subnormal weights, signed zeros, huge values (clamp) and 0/0 (NaN
    quotient gives the zero-point)."""
    N, K = 16, 256
    w = np.zeros((N, K), np.uint16)
    w[0, :] = 0x8000                                      # -0
    w[1, :] = np.arange(K) % 0x7F + 1                     # subnormals
    w[2, :] = 0x7F00                                      # huge
    w[3, :] = 0xFF00                                      # -huge
    w[4, :] = 0x0001                                      # smallest subnormal
    scales = np.full((N, K // 128), 0x3F80, np.uint16)
    scales[1, :] = 0x0080                                 # 2^-126: subnormal w / s is O(1)
    scales[4, :] = 0x0000                                 # 0 -> w / 0 = inf, and row 5 below 0 / 0 = NaN
    scales[5, :] = 0x0000
    zeros = ref.rne_bf16(np.full((N, K // 128), 6.0))
    got = host_words(qlin.quantize(dev16(w), dev16(scales), dev16(zeros)))
    assert np.array_equal(got, ref.quantize_pack(w, scales, zeros))


# Scales at and just past the bounds of the kernel's reciprocal route
# (2^-60 <= |s| <= 2^60), both signs, plus ordinary and subnormal ones.
_EDGE_SCALES = [2.0 ** -60, 2.0 ** 60, 2.0 ** -61, 2.0 ** 61, 2.0 ** -60 * 1.0078125, 2.0 ** 60 * 0.99609375,
                2.0 ** -62 * 1.9921875, 2.0 ** 60 * 1.0078125, 2.0 ** -127, 0.0, 1.0, 0.0234375, 3.0, 1e-30, 1e30]


@pytest.mark.parametrize("zero_set", ["in_grid", "far"])
def test_quantize_every_weight_pattern_on_route_bounds(zero_set):
    """All 65536 bf16 weight patterns (NaN and infinities included), shuffled
    over groups whose scales sit on either side of the reciprocal route's
    scale bounds, with either sign, and whose zero-points are fractional or
    past the route's |z| <= 64 bound: bit-exact with the oracle's division."""
    N, K = 32, 2048
    rng = np.random.default_rng(11 if zero_set == "in_grid" else 12)
    w = rng.permutation(np.arange(65536, dtype=np.uint32)).astype(np.uint16).reshape(N, K)
    sv = np.array(_EDGE_SCALES * (N * K // 128 // len(_EDGE_SCALES) + 1))[: N * K // 128]
    sv = rng.permutation(sv) * np.where(rng.random(sv.size) < 0.5, -1.0, 1.0)
    scales = ref.rne_bf16(sv.astype(np.float32).astype(np.float64)).astype(np.uint16).reshape(N, K // 128)
    if zero_set == "in_grid":
        zv = rng.choice([0.0, 3.5, 8.0, 15.0, 7.0], size=N * K // 128)
    else:
        # a NaN quotient takes code z, which must then be a code itself
        zv = rng.choice([-64.0, -63.5, 64.0, 66.0, -66.0, 100.0, -1000.0, 40.0], size=N * K // 128)
        wf = ref.bf16_to_f64(w)
        w = np.where(np.isnan(wf), np.uint16(0x7F80), w).astype(np.uint16)
    zeros = ref.rne_bf16(zv).astype(np.uint16).reshape(N, K // 128)
    got = host_words(qlin.quantize(dev16(w), dev16(scales), dev16(zeros)))
    want = ref.quantize_pack(w, scales, zeros)
    assert np.array_equal(got, want), np.argwhere(got != want)[:8]


def test_quantize_inverts_the_handles_dequantization():
    """Round trip on the device: the bf16 weights the handle dequantizes are
    quantized back to the very codes it was built from (config-1 shape)."""
    c = gen.linear_case(1)
    lin = qlin.QLinear(c["packed"], c["scales"], c["zeros"])
    w = lin.dequantize(0)
    got = host_words(qlin.quantize(w, dev16(c["scales"]), dev16(c["zeros"])))
    assert np.array_equal(got, c["packed"])
    lin.close()


def test_handle_from_device_quantized_weights():
    """Quantize on the device, build the handle from the device arrays, and
    run the layer: equals the oracle on the same codes."""
    rng = np.random.default_rng(3)
    N, K, M = 256, 1280, 16
    c = gen.random_case(3, M, K, N)
    w = _weights_near_grid(rng, N, K, c["scales"], c["zeros"])
    s_d, z_d = dev16(c["scales"]), dev16(c["zeros"])
    packed_d = qlin.quantize(dev16(w), s_d, z_d)
    lin = qlin.QLinear(packed_d, s_d, z_d)
    packed = ref.quantize_pack(w, c["scales"], c["zeros"])
    y = lin.forward(dev16(c["x"]))
    torch.cuda.synchronize()
    r = ref.compare(y.view(torch.int16).cpu().numpy().view(np.uint16),
                    ref.forward(c["x"], packed, c["scales"], c["zeros"]))
    assert r["ok"], r
    lin.close()


def test_quantize_argument_errors_on_device():
    w = torch.zeros((32, 256), dtype=torch.bfloat16, device="cuda")
    s = torch.ones((32, 2), dtype=torch.bfloat16, device="cuda")
    out = torch.empty((32, 32), dtype=torch.int32, device="cuda")
    f = qlin.qlin_quantize
    assert f(256, 32, 128, w.data_ptr() + 2, s.data_ptr(), None, out.data_ptr(), None) == qlin.QLIN_ERR_ALIGN
    assert f(256, 32, 128, w.data_ptr(), s.data_ptr(), None, w.data_ptr(), None) == qlin.QLIN_ERR_INVALID
    assert f(256, 32, 128, w.data_ptr(), s.data_ptr(), None, out.data_ptr(), None) == qlin.QLIN_OK
    torch.cuda.synchronize()
    assert torch.all(out.view(torch.int32) == np.int32(np.uint32(0x88888888).view(np.int32)))


@pytest.mark.parametrize("symmetric", [False, True])
def test_quantize_into_output_not_16_byte_aligned(symmetric):
    """Packed output at a 4-byte but not 16-byte aligned address (the word
    stores instead of the 16-byte ones): same words as the oracle, and the
    words around the output untouched."""
    N, K = 48, 640
    rng = np.random.default_rng(21 + symmetric)
    scales = ref.rne_bf16(rng.uniform(0.002, 0.05, size=(N, K // 128)).astype(np.float32).astype(np.float64))
    zeros = ref.symmetric_zeros(N, K) if symmetric else ref.rne_bf16(rng.integers(0, 16, size=(N, K // 128)).astype(np.float64))
    w = _weights_near_grid(rng, N, K, scales, zeros)
    buf = torch.full((N * K // 8 + 8,), -1, dtype=torch.int32, device="cuda")
    wd, sd = dev16(w), dev16(scales)
    zp = None if symmetric else dev16(zeros)
    for off in (1, 2, 3):                                 # words: 4, 8, 12 bytes past a 16-byte boundary
        buf.fill_(-1)
        rc = qlin.qlin_quantize(K, N, 128, wd.data_ptr(), sd.data_ptr(), None if zp is None else zp.data_ptr(),
                                buf.data_ptr() + 4 * off, torch.cuda.current_stream().cuda_stream)
        assert rc == qlin.QLIN_OK
        got = host_words(buf)
        assert np.array_equal(got[off:off + N * K // 8].reshape(N, K // 8), ref.quantize_pack(w, scales, zeros))
        assert np.all(got[:off] == 0xFFFFFFFF) and np.all(got[off + N * K // 8:] == 0xFFFFFFFF)


def test_quantize_every_weight_pattern_under_many_scales():
    """Each of 64 scales across the reciprocal route's range (random sign,
    exponent and mantissa) sees all 65536 bf16 weight patterns."""
    S, N, K = 64, 64 * 32, 2048
    rng = np.random.default_rng(31)
    sv = rng.choice([-1.0, 1.0], S) * 2.0 ** rng.integers(-60, 60, S) * (1 + rng.integers(0, 128, S) / 128)
    scales = np.repeat(ref.rne_bf16(sv), 32 * (K // 128)).astype(np.uint16).reshape(N, K // 128)
    w = np.tile(rng.permutation(np.arange(65536, dtype=np.uint32)).astype(np.uint16).reshape(32, K), (S, 1))
    zeros = ref.rne_bf16(rng.integers(0, 16, size=(N, K // 128)).astype(np.float64)).astype(np.uint16)
    got = host_words(qlin.quantize(dev16(w), dev16(scales), dev16(zeros)))
    want = ref.quantize_pack(w, scales, zeros)
    assert np.array_equal(got, want), np.argwhere(got != want)[:8]
