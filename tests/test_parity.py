"""GPU parity of the HIP path with the CPU oracle (needs an MI355X).

Bit-exact: unpacked codes, dequantized bf16 weights (both device routines),
and outputs whose exact value is representable (one-hot rows, codes equal to
the zero-point, the integer case).  Everything else: within the oracle's
tolerance max(2 bf16 ulp, 1e-3), element by element.
"""

import numpy as np
import pytest
import torch

from oracle import qlin_ref as ref
from paper_2607_04244_amd import qlin
from synth import gen

pytestmark = pytest.mark.gpu

GEMV, SKINNY, TILED, AUTO, REGS = qlin.PATH_GEMV, qlin.PATH_SKINNY, qlin.PATH_TILED, qlin.PATH_AUTO, qlin.PATH_REGS


def dev(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        return torch.from_numpy(a.view(np.int16)).view(torch.bfloat16).cuda()
    return torch.from_numpy(a).cuda()


def host_bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def make(c, symmetric=False):
    if symmetric:
        return qlin.QLinear(c["packed"], c["scales"], None)
    return qlin.QLinear(c["packed"], c["scales"], c["zeros"])


def run(lin, x_bits, path=AUTO, split_k=0):
    """One forward.  A forced path or split runs with a caller workspace of
    the size its unconstrained plan reports (qlin_group_plan); the automatic
    plan runs through qlin_forward_path with the handle's own workspace."""
    x = dev(x_bits)
    if split_k > 0 or path != AUTO:
        need, _ = qlin.group_plan([lin], x.shape[0], path, split_k)
        y = lin.forward(x, path=path, split_k=split_k, workspace=qlin.new_workspace(need))
    else:
        y = lin.forward(x, path=path, split_k=split_k)
    torch.cuda.synchronize()
    return host_bits(y)


def oracle(c, x=None, symmetric=False):
    z = ref.symmetric_zeros(c["N"], c["K"]) if symmetric else c["zeros"]
    return ref.forward(c["x"] if x is None else x, c["packed"], c["scales"], z)


def run_split(lin, x_bits, path, split):
    """run() for a forced split; None when the split does not fit this shape
    (the library refuses it explicitly)."""
    try:
        return run(lin, x_bits, path, split)
    except qlin.QlinError as e:
        assert split > 0 and e.code == qlin.QLIN_ERR_UNSUPPORTED and "does not fit" in str(e), e
        return None


def assert_close(y_bits, y_ref, what=""):
    r = ref.compare(y_bits, y_ref)
    assert r["ok"], f"{what}: {r}"


# ------------------------------------------------------------------ layout hooks

@pytest.mark.parametrize("K,N", [(128, 16), (256, 48), (2560, 2560), (9728, 160)])
def test_unpack_and_dequantize_bit_exact(K, N):
    c = gen.random_case(K + N, 1, K, N)
    lin = make(c)
    q = lin.unpack_codes().cpu().numpy()
    assert np.array_equal(q, ref.unpack_codes(c["packed"]))
    w_ref = ref.dequant_bf16(c["packed"], c["scales"], c["zeros"])
    for routine in (0, 1):
        w = host_bits(lin.dequantize(routine))
        assert np.array_equal(w, w_ref), f"routine {routine}: {np.argwhere(w != w_ref)[:5]}"
    lin.close()


def test_dequantize_rounding_golden_cases():
    # the hand-derived rounding cases, planted in one tile
    s = np.full((16, 1), 0x3F81, np.uint16)
    z = np.full((16, 1), 0x4100, np.uint16)
    q = np.tile(np.array([11, 13, 15, 0, 5, 8, 1, 2], np.uint8), (16, 16))
    c = dict(K=128, N=16, packed=ref.pack_codes(q), scales=s, zeros=z)
    lin = make(c)
    w = host_bits(lin.dequantize(0))
    assert w[0, 0] == 0x4042 and w[0, 1] == 0x40A1 and w[0, 2] == 0x40E2 and w[0, 3] == 0xC101
    for routine in (0, 1):
        assert np.array_equal(host_bits(lin.dequantize(routine)), ref.dequant_bf16(c["packed"], s, z))
    lin.close()


def test_symmetric_handle_dequantizes_with_zero_point_eight():
    c = gen.random_case(5, 1, 512, 64)
    lin = make(c, symmetric=True)
    w_ref = ref.dequant_bf16(c["packed"], c["scales"], ref.symmetric_zeros(64, 512))
    for routine in (0, 1):
        assert np.array_equal(host_bits(lin.dequantize(routine)), w_ref)
    lin.close()


# ------------------------------------------------------------------ exact outputs

def _one_hot(M, K, ks):
    x = np.zeros((M, K), np.uint16)
    for m, k in enumerate(ks):
        x[m, k] = 0x3F80
    return x


@pytest.mark.parametrize("path,M,split", [(GEMV, 1, 0), (GEMV, 4, 3), (SKINNY, 1, 0), (SKINNY, 3, 2),
                                          (SKINNY, 16, 0), (SKINNY, 16, 5), (SKINNY, 37, 2), (SKINNY, 64, 0),
                                          (REGS, 1, 0), (REGS, 7, 3), (REGS, 16, 0), (REGS, 16, 4),
                                          (TILED, 96, 0), (TILED, 96, 3), (TILED, 130, 10)])
def test_one_hot_rows_are_bit_exact(path, M, split):
    K, N = 1280, 320
    c = gen.random_case(31, 1, K, N)
    rng = np.random.default_rng(M)
    ks = rng.integers(0, K, size=M)
    x = _one_hot(M, K, ks)
    lin = make(c)
    y = run(lin, x, path, split)
    w = ref.dequant_bf16(c["packed"], c["scales"], c["zeros"])
    assert np.array_equal(y, w[:, ks].T)
    lin.close()


@pytest.mark.parametrize("path", [GEMV, SKINNY, REGS])
def test_codes_equal_zero_point_give_exact_zero(path):
    K, N, M = 768, 96, 4
    rng = np.random.default_rng(2)
    z = rng.integers(0, 16, size=(N, K // 128))
    c = gen.random_case(3, M, K, N)
    c["packed"] = ref.pack_codes(np.repeat(z, 128, axis=1).astype(np.uint8))
    c["zeros"] = ref.rne_bf16(z.astype(np.float64))
    lin = make(c)
    for split in (0, 2, 6):
        y = run(lin, c["x"], path, split)
        assert np.all((y & 0x7FFF) == 0)
    lin.close()


@pytest.mark.parametrize("path,M", [(GEMV, 2), (GEMV, 3), (SKINNY, 1), (SKINNY, 16), (SKINNY, 50),
                                    (REGS, 1), (REGS, 5), (REGS, 16)])
def test_integer_case_is_bit_exact(path, M):
    """s = 1, z = 8 (symmetric), x in {-1, 0, 1}: every partial sum is an
    integer below 2^24, so fp32 accumulation is exact in any order."""
    K, N = 2048, 160
    rng = np.random.default_rng(M)
    Q = rng.integers(0, 16, size=(N, K), dtype=np.uint8)
    xi = rng.integers(-1, 2, size=(M, K))
    x = np.select([xi == 1, xi == -1], [0x3F80, 0xBF80], 0).astype(np.uint16)
    c = dict(K=K, N=N, packed=ref.pack_codes(Q), scales=np.full((N, K // 128), 0x3F80, np.uint16))
    lin = make(c, symmetric=True)
    y_ref = ref.forward(x, c["packed"], c["scales"], ref.symmetric_zeros(N, K))
    ran_split = False
    for split in (0, 2, 3, 4):
        y = run_split(lin, x, path, split)
        if y is not None:
            ran_split |= split > 1
            assert np.array_equal(y, ref.round_output(y_ref)), f"split {split}"
    assert ran_split
    lin.close()


# ------------------------------------------------------------------ tolerance parity

@pytest.mark.parametrize("K,N", [(128, 16), (384, 48), (1152, 208), (2560, 2560)])
@pytest.mark.parametrize("M", [1, 2, 3, 8, 16, 17, 33, 64])
def test_paths_and_splits_match_oracle(K, N, M):
    c = gen.random_case(K * 7 + N + M, M, K, N, sigma=1.0)
    y_ref = oracle(c)
    lin = make(c)
    Kb = K // 128
    splits = sorted({0, 1, min(2, Kb), Kb, max(1, Kb // 3)})
    paths = [SKINNY, AUTO] + ([GEMV] if M <= 4 else []) + ([REGS] if M <= 16 else [])
    for path in paths:
        for split in splits:
            y = run_split(lin, c["x"], path, split)     # split 0 (the planner's) always runs
            if y is not None:
                assert_close(y, y_ref, f"path={path} split={split}")
    lin.close()


@pytest.mark.parametrize("M", [65, 128, 200])
def test_prefill_rows_match_oracle(M):
    c = gen.random_case(M, M, 1024, 128)
    lin = make(c)
    assert_close(run(lin, c["x"], TILED), oracle(c), "tiled")
    assert_close(run(lin, c["x"], AUTO), oracle(c), "auto")
    lin.close()


@pytest.mark.parametrize("M,K,N", [(1, 256, 16), (128, 1280, 512), (200, 384, 208), (300, 1152, 496),
                                   (129, 2560, 4112)])
def test_tiled_matches_oracle(M, K, N):
    """The prefill kernel: partial row blocks (M % 128), partial column blocks
    (N % 256), several groups, every output compared."""
    c = gen.random_case(M * 3 + K + N, M, K, N, sigma=1.0)
    lin = make(c)
    assert_close(run(lin, c["x"], TILED), oracle(c), f"tiled M={M} K={K} N={N}")
    lin.close()


@pytest.mark.parametrize("M,K,N,shape", [
    (2100, 256, 16384, "k_tiled<8,4>"),     # 128 x 256 blocks: enough of them for every compute unit
    (1500, 256, 8208, "k_tiled<8,4>"),      # 128 x 256 blocks, partial row and column blocks
    (1000, 384, 4112, "k_tiled<6,4>"),      # 96 x 256 blocks, partial row and column blocks
    (1000, 384, 2064, "k_tiled<4,2>"),      # 64 x 128 blocks, partial row and column blocks
    (300, 640, 2576, "k_tiled<4,2>"),       # 64 x 128 blocks for a narrow layer
])
def test_tiled_block_shapes_match_oracle(M, K, N, shape):
    """Each block shape of the prefill kernel, as the planner picks it,
    every output compared."""
    c = gen.random_case(M + K + N, M, K, N, sigma=1.0)
    lin = make(c)
    assert f"kernel={shape}" in qlin.group_plan([lin], M, TILED)[1]
    assert_close(run(lin, c["x"], TILED), oracle(c), f"{shape} M={M} K={K} N={N}")
    lin.close()


@pytest.mark.parametrize("M,K,N,split", [(128, 1152, 496, 4), (200, 2560, 272, 3), (65, 1024, 128, 7),
                                         (300, 640, 2576, 2), (129, 9728, 2560, 6)])
def test_tiled_split_k_matches_oracle(M, K, N, split):
    """The prefill kernel with its K range cut in chunks (partial blocks summed
    by the last workgroup to arrive): uneven chunks, partial row and column
    blocks, every output compared; a second call checks that the arrival
    counters were left at zero."""
    c = gen.random_case(7 * M + K + N + split, M, K, N, sigma=1.0)
    lin = make(c)
    assert f"split={split} " in qlin.group_plan([lin], M, TILED, split)[1]
    y_ref = oracle(c)
    assert_close(run(lin, c["x"], TILED, split), y_ref, f"tiled M={M} K={K} N={N} S={split}")
    assert_close(run(lin, c["x"], TILED, split), y_ref, f"tiled M={M} K={K} N={N} S={split}, second call")
    lin.close()


@pytest.mark.parametrize("K,N", [(9728, 2560), (4096, 2560)])
def test_prefill_narrow_layers_take_the_split_tiled_kernel(K, N):
    """At M = 128 the narrow, deep layers of the decoder (o and down
    projections) run as one K-split tiled launch, not as 64-row slices of the
    decode kernel (measured 2.5-3.4x faster on MI355X); outputs match."""
    import torch
    if torch.cuda.get_device_properties(0).multi_processor_count != 256:
        pytest.skip("plans were measured on a 256-CU device")
    M = 128
    c = gen.random_case(K + 5, M, K, N, sigma=1.0)
    lin = make(c)
    need, plan = qlin.group_plan([lin], M)
    assert "kernel=k_tiled<4,2>" in plan and "split=1 " not in plan and need > 0, plan
    y_ref = oracle(c)
    y = lin.forward(dev(c["x"]), workspace=qlin.new_workspace(need))
    torch.cuda.synchronize()
    assert_close(host_bits(y), y_ref, f"M={M} K={K} N={N} with a caller workspace")
    # the handle's own workspace (sized for M <= 16) runs a plan that fits it
    assert_close(run(lin, c["x"]), y_ref, f"M={M} K={K} N={N} own workspace: {lin.plan(M)}")
    lin.close()


def test_tiled_split_k_integer_case_is_bit_exact():
    """Integer products and sums: with the K range cut in chunks the result
    must still be the exact sum, rounded once."""
    K, N, M = 1280, 272, 130
    rng = np.random.default_rng(6)
    Q = rng.integers(0, 16, size=(N, K), dtype=np.uint8)
    xi = rng.integers(-1, 2, size=(M, K))
    x = np.select([xi == 1, xi == -1], [0x3F80, 0xBF80], 0).astype(np.uint16)
    c = dict(K=K, N=N, packed=ref.pack_codes(Q), scales=np.full((N, K // 128), 0x3F80, np.uint16))
    lin = make(c, symmetric=True)
    y_ref = ref.forward(x, c["packed"], c["scales"], ref.symmetric_zeros(N, K))
    assert np.array_equal(run(lin, x, TILED, 4), ref.round_output(y_ref))
    lin.close()


def test_tiled_integer_case_is_bit_exact():
    K, N, M = 1024, 272, 130
    rng = np.random.default_rng(5)
    Q = rng.integers(0, 16, size=(N, K), dtype=np.uint8)
    xi = rng.integers(-1, 2, size=(M, K))
    x = np.select([xi == 1, xi == -1], [0x3F80, 0xBF80], 0).astype(np.uint16)
    c = dict(K=K, N=N, packed=ref.pack_codes(Q), scales=np.full((N, K // 128), 0x3F80, np.uint16))
    lin = make(c, symmetric=True)
    y_ref = ref.forward(x, c["packed"], c["scales"], ref.symmetric_zeros(N, K))
    assert np.array_equal(run(lin, x, TILED), ref.round_output(y_ref))
    lin.close()


@pytest.mark.parametrize("M", [512])
def test_config4_prefill_down_projection_full_size(M):
    """Chunked-prefill regime at full size (K=9728, N=2560) through the
    automatic plan (the tiled kernel), every output compared."""
    rng_case = gen.random_case(4000 + M, M, 9728, 2560, sigma=1.0)
    lin = make(rng_case)
    assert "path=tiled" in lin.plan(M)
    assert_close(run(lin, rng_case["x"]), oracle(rng_case), f"M={M}")
    lin.close()


def test_symmetric_forward_matches_oracle():
    c = gen.random_case(77, 16, 2560, 1024)
    lin = make(c, symmetric=True)
    y_ref = oracle(c, symmetric=True)
    for path, M in ((GEMV, 1), (GEMV, 2), (SKINNY, 16), (SKINNY, 3), (REGS, 1), (REGS, 16), (TILED, 16)):
        assert_close(run(lin, c["x"][:M], path), y_ref[:M], f"path={path}")
    lin.close()


def test_config0_single_linear():
    c = gen.linear_case(0)
    lin = make(c)
    y_ref = oracle(c)
    for path in (AUTO, GEMV, SKINNY, REGS):
        assert_close(run(lin, c["x"], path), y_ref, f"path={path}")
    lin.close()


def test_config1_draft_block_verify_full_size():
    """The benchmarked workload (M=16, K=2560, N=19456) in the bench's launch
    configuration (automatic plan), compared on every output."""
    c = gen.linear_case(1)
    lin = make(c)
    y_ref = oracle(c)
    assert_close(run(lin, c["x"]), y_ref, "auto")
    assert_close(run(lin, c["x"], SKINNY, 2), y_ref, "skinny split 2")
    assert_close(run(lin, c["x"], REGS), y_ref, "regs")
    lin.close()


@pytest.mark.parametrize("M", [1, 4, 8, 16])
def test_config2_down_projection_with_outliers(M):
    c = gen.linear_case(2, M=M)
    lin = make(c)
    y_ref = oracle(c)
    paths = (AUTO, SKINNY, REGS, GEMV) if M <= 4 else (AUTO, SKINNY, REGS)
    for path in paths:
        assert_close(run(lin, c["x"], path), y_ref, f"M={M} path={path}")
    lin.close()


# ------------------------------------------------------------------ edge cases and API

def test_extreme_shapes():
    for K, N, M in ((65536, 16, 3), (128, 65536, 5)):
        c = gen.random_case(K + N, M, K, N)
        lin = make(c)
        assert_close(run(lin, c["x"]), oracle(c), f"K={K} N={N}")
        lin.close()


def test_maximum_sizes():
    # the largest N and M the boundary accepts: N = 2^20 columns (65536 column
    # tiles, a 64 MiB code array; checked on sampled columns, each of which
    # the oracle computes from its own weights alone), and M = 65536 rows
    # through the tiled kernel
    K, N, M = 128, 1 << 20, 3
    c = gen.random_case(K + N, M, K, N)
    lin = make(c)
    y = run(lin, c["x"])
    lin.close()
    rng = np.random.default_rng(5)
    cols = np.unique(np.concatenate([np.arange(256), np.arange(N - 256, N), rng.integers(0, N, 1024)]))
    y_ref = ref.forward(c["x"], c["packed"][cols], c["scales"][cols], c["zeros"][cols])
    assert_close(np.ascontiguousarray(y[:, cols]), y_ref, f"K={K} N={N} M={M} sampled columns")
    K, N, M = 256, 64, 65536
    c = gen.random_case(K + N + M, M, K, N)
    lin = make(c)
    assert_close(run(lin, c["x"]), oracle(c), f"K={K} N={N} M={M}")
    lin.close()


def test_code_array_beyond_two_gib():
    # K = 65536 (the largest), N = 69632: 2.28 GB of codes, so column tiles
    # past 2 GiB are addressed; checked on sampled columns
    K, N = 65536, 69632
    c = gen.random_case(3, 16, K, N)
    lin = make(c)
    rng = np.random.default_rng(9)
    cols = np.unique(np.concatenate([np.arange(64), np.arange(N - 64, N), rng.integers(0, N, 256)]))
    for M in (1, 16):
        x = c["x"][:M]
        y = run(lin, x)
        y_ref = ref.forward(x, c["packed"][cols], c["scales"][cols], c["zeros"][cols])
        assert_close(np.ascontiguousarray(y[:, cols]), y_ref, f"K={K} N={N} M={M} sampled columns")
    lin.close()


def test_zero_rows_is_a_noop_and_repeat_calls_agree():
    c = gen.random_case(9, 16, 1280, 160)
    lin = make(c)
    x = dev(c["x"])
    y = torch.full((16, 160), 7.0, dtype=torch.bfloat16, device="cuda")
    assert qlin.qlin_forward(lin.h, 0, x.data_ptr(), y.data_ptr(), None) == qlin.QLIN_OK
    torch.cuda.synchronize()
    assert torch.all(y == 7.0)
    # every reduction runs in a fixed order, so repeated calls give identical
    # bits; split-K arrival counters must reset themselves between calls
    y_ref = oracle(c)
    for path, split in ((SKINNY, 4), (SKINNY, 1), (GEMV, 3), (REGS, 5), (REGS, 1)):
        M = 4 if path == GEMV else 16
        first = run(lin, c["x"][:M], path, split)
        assert_close(first, y_ref[:M])
        for _ in range(3):
            assert np.array_equal(run(lin, c["x"][:M], path, split), first)
    lin.close()


def test_non_default_stream():
    c = gen.random_case(10, 4, 1024, 256)
    lin = make(c)
    s = torch.cuda.Stream()
    x = dev(c["x"])
    with torch.cuda.stream(s):
        y = lin.forward(x)
    s.synchronize()
    assert_close(host_bits(y), oracle(c))
    lin.close()


def test_forward_argument_errors():
    c = gen.random_case(11, 4, 256, 32)
    lin = make(c)
    x = torch.zeros((70000, 256), dtype=torch.bfloat16, device="cuda")
    y = torch.zeros((70000, 32), dtype=torch.bfloat16, device="cuda")
    xp, yp = x.data_ptr(), y.data_ptr()
    f = qlin.qlin_forward_path
    assert f(lin.h, AUTO, 0, -1, xp, yp, None) == qlin.QLIN_ERR_INVALID
    assert f(lin.h, AUTO, 0, 4, xp + 2, yp, None) == qlin.QLIN_ERR_ALIGN
    assert f(lin.h, AUTO, 0, 4, xp, yp + 8, None) == qlin.QLIN_ERR_ALIGN
    assert f(lin.h, AUTO, 0, 4, xp, xp + 256, None) == qlin.QLIN_ERR_INVALID      # y overlaps x
    assert f(lin.h, AUTO, 0, 4, None, yp, None) == qlin.QLIN_ERR_INVALID
    assert f(lin.h, AUTO, 0, 65537, xp, yp, None) == qlin.QLIN_ERR_UNSUPPORTED
    assert f(lin.h, GEMV, 0, 5, xp, yp, None) == qlin.QLIN_ERR_UNSUPPORTED
    assert f(lin.h, SKINNY, 0, 65, xp, yp, None) == qlin.QLIN_ERR_UNSUPPORTED
    assert f(lin.h, REGS, 0, 17, xp, yp, None) == qlin.QLIN_ERR_UNSUPPORTED
    assert f(lin.h, 7, 0, 4, xp, yp, None) == qlin.QLIN_ERR_INVALID
    assert f(lin.h, AUTO, 3, 4, xp, yp, None) == qlin.QLIN_ERR_INVALID          # split_k > K/128
    assert f(lin.h, AUTO, -1, 4, xp, yp, None) == qlin.QLIN_ERR_INVALID
    assert qlin.qlin_shape(lin.h) == (256, 32)
    assert "path=" in lin.plan(16)
    torch.cuda.synchronize()
    lin.close()


@pytest.mark.parametrize("M,K,N,kernel,split", [
    (16, 2560, 19456, "k_skinny<1,16>", 1),    # the draft-block verification linear
    (1, 2560, 19456, "k_skinny<1,1>", 1),      # gate|up at one row (measured plan)
    (16, 2560, 6144, "k_skinny<1,16>", 1),     # q|k|v of a layer
    (16, 4096, 2560, "k_skinny<1,16>", 1),     # o projection (measured plan)
    (16, 9728, 2560, "k_skinny<1,16>", 3),     # down projection (measured plan)
    (8, 9728, 2560, "k_mfma16<2>", 3),         # down projection, half a draft block (measured plan)
    (1, 9728, 2560, "k_skinny<1,1>", 1),       # down projection, one row (measured plan)
    (1, 2560, 2560, "k_mfma16<1>", 1),         # single-row layer
])
def test_automatic_plan_for_decoder_shapes(M, K, N, kernel, split):
    """The automatic plan for the decoder's linears on a 256-CU MI355X is the
    one measured fastest (a planner change that silently falls back to a
    slower kernel family fails here)."""
    import torch
    if torch.cuda.get_device_properties(0).multi_processor_count != 256:
        pytest.skip("plans were measured on a 256-CU device")
    c = gen.random_case(3, M, K, N)
    lin = make(c)
    plan = lin.plan(M)
    lin.close()
    assert f"kernel={kernel} " in plan and f"split={split} " in plan, plan


def test_rows_beyond_32_bit_offsets_of_x():
    """M * K = 2^31 (K = 65536, M = 32768: a 4 GiB x) through the automatic
    plan: the tiled kernel addresses x with 32-bit byte offsets, so the rows
    run as two launches (32767 rows, then one).  x is drawn on the device
    (seeded); the rows checked, on both sides of the boundary, are read back
    and compared with the oracle on every column."""
    K, N, M = 65536, 64, 32768
    c = gen.random_case(12, 1, K, N)
    lin = make(c)
    g = torch.Generator(device="cuda").manual_seed(12)
    x = torch.randn((M, K), device="cuda", generator=g).to(torch.bfloat16)
    y = lin.forward(x)
    torch.cuda.synchronize()
    assert "launches=2" in lin.plan(M), lin.plan(M)
    rows = np.array([0, 1, 4095, 32766, 32767])
    xr = host_bits(x[torch.from_numpy(rows).cuda()])
    y_ref = ref.forward(xr, c["packed"], c["scales"], c["zeros"])
    assert_close(np.ascontiguousarray(host_bits(y)[rows]), y_ref, f"K={K} M={M} rows {rows}")
    del x, y
    torch.cuda.empty_cache()
    lin.close()
