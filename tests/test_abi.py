"""The C ABI library loads, exports what include/*.h declare, and rejects
bad arguments before any HIP call (CPU only: no compute is launched)."""

import os
import re

import numpy as np
import pytest

from paper_2607_04244_amd import qlin
from synth import gen

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared_functions():
    names = set()
    inc = os.path.join(ROOT, "include")
    for f in sorted(os.listdir(inc)):
        if f.endswith(".h"):
            txt = re.sub(r"/\*.*?\*/", "", open(os.path.join(inc, f)).read(), flags=re.S)
            names |= set(re.findall(r"\b(qlin_[a-z_]+)\s*\(", txt))
    return sorted(names)


def test_header_declares_the_binding_names():
    assert _declared_functions() == sorted(qlin.EXPORTS)


def test_library_exports_every_declared_symbol():
    L = qlin.lib()
    for name in _declared_functions():
        assert hasattr(L, name), name


def test_missing_library_fails_loudly(monkeypatch, tmp_path):
    monkeypatch.setattr(qlin, "_lib", None)
    monkeypatch.setattr(qlin, "LIB_PATH", str(tmp_path / "absent.so"))
    with pytest.raises(RuntimeError, match="missing"):
        qlin.lib()


@pytest.fixture(scope="module")
def case():
    return gen.random_case(1, 1, 256, 32)


def _create_code(K, N, group, packed, scales, zeros, symmetric=False):
    try:
        if symmetric:
            qlin.qlin_create_symmetric(K, N, group, packed, scales)
        else:
            qlin.qlin_create(K, N, group, packed, scales, zeros)
    except qlin.QlinError as e:
        return e.code
    raise AssertionError("create unexpectedly succeeded")


@pytest.mark.parametrize("K,N,group,code", [
    (0, 32, 128, qlin.QLIN_ERR_INVALID),
    (256, 0, 128, qlin.QLIN_ERR_INVALID),
    (256, 32, 0, qlin.QLIN_ERR_INVALID),
    (256, 32, 64, qlin.QLIN_ERR_UNSUPPORTED),
    (200, 32, 128, qlin.QLIN_ERR_INVALID),
    (256, 24, 128, qlin.QLIN_ERR_UNSUPPORTED),
    (65536 + 128, 32, 128, qlin.QLIN_ERR_UNSUPPORTED),
])
def test_create_rejects_bad_shapes(case, K, N, group, code):
    assert _create_code(K, N, group, case["packed"], case["scales"], case["zeros"]) == code


def test_create_rejects_null_pointers(case):
    L = qlin.lib()
    p = case["packed"]
    s = case["scales"]
    assert not L.qlin_create(256, 32, 128, None, s.ctypes.data, s.ctypes.data)
    assert qlin.qlin_last_status() == qlin.QLIN_ERR_INVALID
    assert not L.qlin_create(256, 32, 128, p.ctypes.data, None, s.ctypes.data)
    assert qlin.qlin_last_status() == qlin.QLIN_ERR_INVALID
    assert not L.qlin_create(256, 32, 128, p.ctypes.data, s.ctypes.data, None)
    assert qlin.qlin_last_status() == qlin.QLIN_ERR_INVALID
    assert not L.qlin_create_symmetric(256, 32, 128, p.ctypes.data, None)
    assert qlin.qlin_last_status() == qlin.QLIN_ERR_INVALID


@pytest.mark.parametrize("zbits", [0x40F0, 0x4180, 0xBF80, 0x7FC0, 0x3F00])   # 7.5, 16, -1, nan, 0.5
def test_create_rejects_non_integer_or_out_of_range_zeros(case, zbits):
    z = case["zeros"].copy()
    z[5, 1] = zbits
    assert _create_code(256, 32, 128, case["packed"], case["scales"], z) == qlin.QLIN_ERR_INVALID
    assert "zero-point" in qlin.last_error()


@pytest.mark.parametrize("sbits", [0x0000, 0x8000, 0xBC00, 0x7F80, 0x7FC0, 0x0001, 0x0D00, 0x7300])
def test_create_rejects_scales_outside_the_exact_range(case, sbits):
    # zero, -0, negative, inf, nan, denormal, 2^-101, 2^103
    s = case["scales"].copy()
    s[3, 0] = sbits
    assert _create_code(256, 32, 128, case["packed"], s, case["zeros"]) == qlin.QLIN_ERR_UNSUPPORTED
    assert _create_code(256, 32, 128, case["packed"], s, None, symmetric=True) == qlin.QLIN_ERR_UNSUPPORTED


def test_scale_range_edges_pass_validation(case, monkeypatch):
    # 2^-100 and the largest value below 2^100 are accepted: validation passes
    # and the forced allocation failure is reported instead
    monkeypatch.setenv("QLIN_FAULT", "alloc")
    s = case["scales"].copy()
    s[0, 0] = (127 - 100) << 7
    s[0, 1] = ((127 + 99) << 7) | 0x7F
    assert _create_code(256, 32, 128, case["packed"], s, case["zeros"]) == qlin.QLIN_ERR_OOM


def test_allocation_failure_is_reported_not_aborted(case, monkeypatch):
    monkeypatch.setenv("QLIN_FAULT", "alloc")
    assert _create_code(256, 32, 128, case["packed"], case["scales"], case["zeros"]) == qlin.QLIN_ERR_OOM
    assert "allocation failed" in qlin.last_error()
    assert _create_code(256, 32, 128, case["packed"], case["scales"], None, symmetric=True) == qlin.QLIN_ERR_OOM


def test_calls_on_a_null_handle():
    L = qlin.lib()
    assert L.qlin_forward(None, 1, 16, 32, None) == qlin.QLIN_ERR_INVALID
    assert L.qlin_forward_path(None, 2, 0, 1, 16, 32, None) == qlin.QLIN_ERR_INVALID
    assert L.qlin_unpack_codes(None, 16, None) == qlin.QLIN_ERR_INVALID
    assert L.qlin_dequantize(None, 0, 16, None) == qlin.QLIN_ERR_INVALID
    assert L.qlin_shape(None, None, None) == qlin.QLIN_ERR_INVALID
    buf = qlin.ctypes.create_string_buffer(64)
    assert L.qlin_plan(None, 0, 0, 1, buf, 64) == qlin.QLIN_ERR_INVALID
    L.qlin_destroy(None)                       # NULL-safe
    assert qlin.qlin_last_status() == qlin.QLIN_ERR_INVALID
    assert "NULL" in qlin.last_error()


def test_error_state_is_cleared_by_the_next_call(case, monkeypatch):
    monkeypatch.setenv("QLIN_FAULT", "alloc")
    _create_code(0, 32, 128, case["packed"], case["scales"], case["zeros"])
    assert qlin.qlin_last_status() == qlin.QLIN_ERR_INVALID
    _create_code(256, 32, 128, case["packed"], case["scales"], case["zeros"])
    assert qlin.qlin_last_status() == qlin.QLIN_ERR_OOM


def test_quantize_rejects_bad_arguments():
    """qlin_quantize validates shapes, pointers, alignment and overlap before
    any HIP call (addresses below are never dereferenced)."""
    L = qlin.lib()
    A = 1 << 20                                  # aligned stand-in addresses
    f = L.qlin_quantize
    assert f(0, 32, 128, A, A, A, 2 * A, None) == qlin.QLIN_ERR_INVALID
    assert f(256, 32, 64, A, A, A, 2 * A, None) == qlin.QLIN_ERR_UNSUPPORTED
    assert f(200, 32, 128, A, A, A, 2 * A, None) == qlin.QLIN_ERR_INVALID
    assert f(256, 24, 128, A, A, A, 2 * A, None) == qlin.QLIN_ERR_UNSUPPORTED
    assert f(256, 32, 128, None, A, A, 2 * A, None) == qlin.QLIN_ERR_INVALID
    assert f(256, 32, 128, A, None, A, 2 * A, None) == qlin.QLIN_ERR_INVALID
    assert f(256, 32, 128, A, A, A, None, None) == qlin.QLIN_ERR_INVALID
    assert f(256, 32, 128, A + 8, A, A, 2 * A, None) == qlin.QLIN_ERR_ALIGN
    assert f(256, 32, 128, A, A, A, 2 * A + 2, None) == qlin.QLIN_ERR_ALIGN
    assert f(256, 32, 128, A, A + 1, A, 2 * A, None) == qlin.QLIN_ERR_ALIGN
    assert f(256, 32, 128, A, A, A, A + 256, None) == qlin.QLIN_ERR_INVALID      # packed overlaps w
    assert "overlaps" in qlin.last_error()


# ---------------------------------------------------------------- drafter attention

def test_attention_plan_key_ranges():
    """Explicit splits need no device: the plan is pure arithmetic."""
    # window 1024 at T = 8192: keys [8192 - 16 - 512, 8192) = 528 keys, 9 tiles of 64
    S, ws, txt = qlin.qlin_swa_plan(32, 8, 128, 16, 8192, 1024, 3)
    assert S == 3 and ws == 3 * 32 * 16 * 130 * 4 and "keys=528 tiles=9" in txt and "grid=24" in txt
    # the workspace covers 16 rows per (head, split) whatever nq is
    S, ws, _ = qlin.qlin_swa_plan(32, 8, 128, 5, 8192, 1024, 3)
    assert S == 3 and ws == 3 * 32 * 16 * 130 * 4
    # T <= window: full attention over all T keys
    S, ws, txt = qlin.qlin_swa_plan(32, 8, 128, 16, 700, 1024, 100)
    assert S == 11 and "keys=700 tiles=11" in txt
    # window 0: full attention; one split needs no workspace
    S, ws, txt = qlin.qlin_swa_plan(4, 1, 128, 1, 5, 0, 1)
    assert (S, ws) == (1, 0) and "combine=0" in txt
    # splits that do not divide the tiles: no empty range
    S, _, _ = qlin.qlin_swa_plan(8, 8, 128, 16, 64 * 10, 0, 4)
    assert S == 4          # 3 tiles per range: 3 + 3 + 3 + 1
    S, _, _ = qlin.qlin_swa_plan(8, 8, 128, 16, 64 * 10, 0, 6)
    assert S == 5          # 2 tiles per range
    _, _, txt = qlin.qlin_swa_plan(64, 8, 128, 16, 100, 0, 1)
    assert "k_attn_split<2,3>" in txt


@pytest.mark.parametrize("args,code", [
    ((32, 8, 64, 16, 100, 0, 1), qlin.QLIN_ERR_UNSUPPORTED),     # head_dim
    ((128, 8, 128, 16, 100, 0, 1), qlin.QLIN_ERR_UNSUPPORTED),   # 16 query heads per key/value head
    ((30, 8, 128, 16, 100, 0, 1), qlin.QLIN_ERR_INVALID),        # Hq not a multiple of Hkv
    ((0, 8, 128, 16, 100, 0, 1), qlin.QLIN_ERR_INVALID),
    ((32, 8, 128, 0, 100, 0, 1), qlin.QLIN_ERR_INVALID),         # nq
    ((32, 8, 128, 17, 100, 0, 1), qlin.QLIN_ERR_INVALID),
    ((32, 8, 128, 16, 15, 0, 1), qlin.QLIN_ERR_INVALID),         # T < nq
    ((32, 8, 128, 16, 2 ** 28 + 1, 0, 1), qlin.QLIN_ERR_INVALID),
    ((32, 8, 128, 16, 100, -1, 1), qlin.QLIN_ERR_INVALID),       # window
    ((32, 8, 128, 16, 100, 0, -1), qlin.QLIN_ERR_INVALID),       # splits
])
def test_attention_plan_rejects_bad_sizes(args, code):
    with pytest.raises(qlin.QlinError) as e:
        qlin.qlin_swa_plan(*args)
    assert e.value.code == code


def test_attention_rejects_bad_arguments():
    """Every case fails in the argument checks, before any HIP call."""
    A = 1 << 32                    # fake, 16-byte aligned addresses (never dereferenced)
    q, k, v, o, w = A, A + (1 << 24), A + (2 << 24), A + (3 << 24), A + (4 << 24)
    base = dict(Hq=32, Hkv=8, D=128, nq=16, T=1000, kv_stride=1000, window=0, splits=4,
                q=q, k=k, v=v, o=o, w=w, wb=1 << 24)

    def call(**kw):
        a = dict(base, **kw)
        return qlin.qlin_swa_attention(a["Hq"], a["Hkv"], a["D"], a["nq"], a["T"], a["kv_stride"], a["window"],
                                       a["splits"], a["q"], a["k"], a["v"], a["o"], a["w"], a["wb"], None)

    assert call(kv_stride=999) == qlin.QLIN_ERR_INVALID
    assert call(q=None) == qlin.QLIN_ERR_INVALID
    assert call(o=None) == qlin.QLIN_ERR_INVALID
    assert call(k=k + 8) == qlin.QLIN_ERR_ALIGN
    assert call(w=w + 4) == qlin.QLIN_ERR_ALIGN
    assert call(wb=-1) == qlin.QLIN_ERR_INVALID
    assert call(w=None, wb=0) == qlin.QLIN_ERR_INVALID               # 4 ranges need a workspace
    assert call(wb=4 * 32 * 16 * 130 * 4 - 16) == qlin.QLIN_ERR_INVALID
    assert "workspace" in qlin.last_error()
    assert call(o=q + 1024) == qlin.QLIN_ERR_INVALID                 # out overlaps q
    assert call(o=v + 7 * 1000 * 256) == qlin.QLIN_ERR_INVALID       # out overlaps the last head of v
    assert call(o=w + 4096) == qlin.QLIN_ERR_INVALID                 # out overlaps the workspace
    assert call(D=96) == qlin.QLIN_ERR_UNSUPPORTED
    assert qlin.qlin_last_status() == qlin.QLIN_ERR_UNSUPPORTED


def test_group_calls_reject_bad_arguments_without_a_device():
    """Checks of the grouped launch that need no handle (no HIP call)."""
    L = qlin.lib()
    A = 1 << 32
    assert L.qlin_forward_group(0, None, 0, 0, 16, A, None, None, 0, None) == qlin.QLIN_ERR_INVALID
    assert L.qlin_forward_group(1, None, 0, 0, 16, A, None, None, 0, None) == qlin.QLIN_ERR_INVALID
    assert L.qlin_forward_group(9, None, 0, 0, 16, A, None, None, 0, None) == qlin.QLIN_ERR_INVALID
    hs = (qlin.ctypes.c_void_p * 2)(None, None)
    assert L.qlin_forward_group(2, hs, 0, 0, 16, A, None, None, 0, None) == qlin.QLIN_ERR_INVALID
    assert "NULL handle" in qlin.last_error()
    assert L.qlin_forward_group(1, hs, 0, 0, 16, A, None, A, -5, None) == qlin.QLIN_ERR_INVALID
    assert L.qlin_forward_group(1, hs, 0, 0, 16, A, None, None, 64, None) == qlin.QLIN_ERR_INVALID
    need = qlin.ctypes.c_int64()
    assert L.qlin_group_plan(0, None, 0, 0, 16, -1, qlin.ctypes.byref(need), None, 0) == qlin.QLIN_ERR_INVALID
    assert L.qlin_workspace_bytes(None, qlin.ctypes.byref(need)) == qlin.QLIN_ERR_INVALID
