"""GPU tests of the grouped launch (qlin_forward_group), caller workspaces
and the drafter's weight pass shapes, through the C ABI (needs an MI355X).

A group is several linears that share their input x: the q, k and v
projections of a decoder layer (the target verifies one 16-token block per
step, Sec. 2.2; the drafter drafts one per step, Sec. 2.3 and 3.2).  Every
member's output is compared with the oracle element by element within
max(2 bf16 ulp, 1e-3); exact cases (integer products and sums) bit for bit.
"""

import numpy as np
import pytest
import torch

from oracle import qlin_ref as ref
from paper_2607_04244_amd import qlin
from synth import gen

pytestmark = pytest.mark.gpu

AUTO, GEMV, SKINNY, TILED, REGS = qlin.PATH_AUTO, qlin.PATH_GEMV, qlin.PATH_SKINNY, qlin.PATH_TILED, qlin.PATH_REGS


def dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def host_bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def make(w, symmetric=False):
    return qlin.QLinear(w["packed"], w["scales"], None if symmetric else w["zeros"])


def zeros_of(w, symmetric=False):
    return ref.symmetric_zeros(w["N"], w["K"]) if symmetric else w["zeros"]


def group_run(lins, x_bits, path=AUTO, split=0, ws_bytes=-1):
    """forward_group with a workspace of the unconstrained plan's size (or
    ws_bytes); returns host bit arrays."""
    x = dev(x_bits)
    need, _ = qlin.group_plan(lins, x.shape[0], path, split)
    nb = need if ws_bytes < 0 else ws_bytes
    ws = qlin.new_workspace(nb) if nb > 0 else None
    ys = qlin.forward_group(lins, x, path=path, split_k=split, workspace=ws)
    torch.cuda.synchronize()
    return [host_bits(y) for y in ys]


def check_members(ys, ws, x, symmetric=False, what=""):
    for i, (y, w) in enumerate(zip(ys, ws)):
        r = ref.compare(y, ref.forward(x, w["packed"], w["scales"], zeros_of(w, symmetric)))
        assert r["ok"], f"{what} member {i} ({w['N']} columns): {r}"


@pytest.fixture(scope="module")
def qkv():
    ws = [gen.model_linear(0, p) for p in range(3)]
    lins = [make(w) for w in ws]
    yield ws, lins
    for l in lins:
        l.close()


@pytest.mark.parametrize("M", [1, 4, 8, 13, 16, 33, 64])
def test_qkv_group_matches_oracle(qkv, M):
    """The q|k|v projections of a decoder layer as one launch, every output of
    every member compared; once with the unconstrained plan's workspace, once
    with none (plans without a K split)."""
    ws, lins = qkv
    x = gen.model_activations(3, M, ws[0]["K"])
    check_members(group_run(lins, x), ws, x, what=f"M={M}")
    check_members(group_run(lins, x, ws_bytes=0), ws, x, what=f"M={M} no workspace")


@pytest.mark.parametrize("M", [65, 128, 300, 2048])
def test_qkv_group_at_prefill_rows(qkv, M):
    """Prefill rows: one tiled launch over the three members (q's 16-tile
    column blocks, then k's, then v's), with and without a workspace for the
    K split; all outputs compared (sampled columns at M = 2048)."""
    ws, lins = qkv
    x = gen.model_activations(4, M, ws[0]["K"])
    need, plan = qlin.group_plan(lins, M)
    assert "path=tiled" in plan and "launches=1" in plan, plan
    for nb in (-1, 0):
        ys = group_run(lins, x, ws_bytes=nb)
        for i, (y, w) in enumerate(zip(ys, ws)):
            cols = np.arange(w["N"]) if M < 2048 else np.unique(np.r_[0:64, w["N"] - 64:w["N"], 200:w["N"]:97])
            y_ref = ref.forward(x, w["packed"][cols], w["scales"][cols], w["zeros"][cols])
            r = ref.compare(np.ascontiguousarray(y[:, cols]), y_ref)
            assert r["ok"], f"M={M} member {i} workspace={nb}: {r}"


def test_qkv_group_is_one_launch(qkv):
    _, lins = qkv
    if torch.cuda.get_device_properties(0).multi_processor_count != 256:
        pytest.skip("plans were measured on a 256-CU device")
    need, plan = qlin.group_plan(lins, 16)
    assert "kernel=k_skinny<1,16> " in plan and "split=1 " in plan and "launches=1" in plan, plan
    assert need == 0


@pytest.mark.parametrize("path,M,split", [(SKINNY, 16, 0), (SKINNY, 16, 3), (SKINNY, 40, 2), (REGS, 7, 0),
                                          (REGS, 16, 4), (GEMV, 3, 0), (GEMV, 4, 5), (AUTO, 1, 0),
                                          (TILED, 130, 0), (TILED, 130, 4)])
def test_mixed_width_group_integer_case_is_bit_exact(path, M, split):
    """Members of unequal width (one tile, three, 64, seventeen), every path
    and forced splits: s = 1, z = 8, x in {-1, 0, 1}, so every sum is an
    integer below 2^24 and each member's output must equal the rounded exact
    product bit for bit."""
    K = 1280
    rng = np.random.default_rng(M * 10 + split)
    xi = rng.integers(-1, 2, size=(M, K))
    x = np.select([xi == 1, xi == -1], [0x3F80, 0xBF80], 0).astype(np.uint16)
    ws, lins = [], []
    for N in (16, 48, 1024, 272):
        Q = rng.integers(0, 16, size=(N, K), dtype=np.uint8)
        w = dict(K=K, N=N, packed=ref.pack_codes(Q), scales=np.full((N, K // 128), 0x3F80, np.uint16))
        ws.append(w)
        lins.append(make(w, symmetric=True))
    ys = group_run(lins, x, path, split)
    for y, w in zip(ys, ws):
        y_ref = ref.forward(x, w["packed"], w["scales"], ref.symmetric_zeros(w["N"], K))
        assert np.array_equal(y, ref.round_output(y_ref)), f"N={w['N']}"
    for l in lins:
        l.close()


def test_eight_member_group_with_split():
    """The largest group (8 members, asymmetric, random values) with the K
    range cut, every output compared."""
    K, M = 2048, 16
    ws = [gen.random_case(50 + i, M, K, 16 * (i + 1)) for i in range(8)]
    lins = [make(w) for w in ws]
    x = ws[0]["x"]
    for path, split in ((AUTO, 0), (SKINNY, 4), (REGS, 2)):
        check_members(group_run(lins, x, path, split), ws, x, what=f"path={path} split={split}")
    for l in lins:
        l.close()


def test_one_workspace_shared_in_stream_order():
    """One zero-filled workspace serves launches of different handles and plans
    (decode splits, a tiled split, slices) issued back to back on one stream
    without synchronisation: each launch leaves its arrival counters at zero
    for the next, whatever plan that one has."""
    cases = [gen.random_case(60, 16, 9728, 2560), gen.random_case(61, 130, 1152, 496),
             gen.random_case(62, 16, 4096, 2560), gen.random_case(63, 48, 2560, 1024)]
    lins = [make(c) for c in cases]
    runs = [(0, SKINNY, 3, 16), (1, TILED, 4, 130), (2, REGS, 5, 16), (3, SKINNY, 2, 48), (0, REGS, 6, 9),
            (1, TILED, 2, 130), (3, AUTO, 0, 48), (2, SKINNY, 8, 16)]
    need = max(qlin.group_plan([lins[i]], M, p, s)[0] for i, p, s, M in runs)
    wsb = qlin.new_workspace(need)
    xs = {i: dev(c["x"]) for i, c in enumerate(cases)}
    outs = []
    for i, p, s, M in runs:
        outs.append(qlin.forward_group([lins[i]], xs[i][:M], path=p, split_k=s, workspace=wsb)[0])
    torch.cuda.synchronize()
    for (i, p, s, M), y in zip(runs, outs):
        c = cases[i]
        r = ref.compare(host_bits(y), ref.forward(c["x"][:M], c["packed"], c["scales"], c["zeros"]))
        assert r["ok"], f"case {i} path={p} split={s} M={M}: {r}"
    for l in lins:
        l.close()


def test_small_workspace_gives_a_plan_that_fits():
    """A workspace smaller than the unconstrained plan's: the planner falls back
    to a plan that fits it (16-row slices or no K split), with the same
    results; a forced split that does not fit is refused."""
    c = gen.random_case(70, 64, 2560, 19456)
    lin = make(c)
    need, plan = qlin.group_plan([lin], 64)
    assert need > 0, plan
    small, plan_small = qlin.group_plan([lin], 64, ws_bytes=need // 2)
    assert small <= need // 2, plan_small
    y_ref = ref.forward(c["x"], c["packed"], c["scales"], c["zeros"])
    for nb in (need, need // 2, 0):
        assert ref.compare(group_run([lin], c["x"], ws_bytes=nb)[0], y_ref)["ok"], nb
    x = dev(c["x"])
    with pytest.raises(qlin.QlinError) as e:
        qlin.forward_group([lin], x, path=SKINNY, split_k=3, workspace=None)
    assert e.value.code == qlin.QLIN_ERR_UNSUPPORTED
    lin.close()


def test_handle_workspace_is_a_small_fraction_of_the_weights():
    """The handles of the 36-layer model own workspaces for their M <= 16
    plans only: at most 5% of the weight bytes together (every layer has the
    same shapes, so one layer's handles stand for all 36)."""
    total_ws, total_w = 0, 0
    for p in range(len(gen.LAYER_SHAPES)):
        w = gen.model_linear(0, p)
        lin = make(w)
        total_ws += lin.workspace_bytes()
        total_w += w["K"] * w["N"] // 2 + 4 * (w["K"] // 128) * w["N"]
        lin.close()
    assert total_ws <= 0.05 * total_w, (total_ws, total_w)


def test_group_argument_errors(qkv):
    ws, lins = qkv
    x = torch.zeros((16, 2560), dtype=torch.bfloat16, device="cuda")
    ys = [torch.empty((16, w["N"]), dtype=torch.bfloat16, device="cuda") for w in ws]
    hs = [l.h for l in lins]
    yp = [y.data_ptr() for y in ys]
    f = qlin.qlin_forward_group
    assert f(hs, AUTO, 0, 16, x.data_ptr(), yp, None, 0, None) == qlin.QLIN_OK
    assert f([], AUTO, 0, 16, x.data_ptr(), [], None, 0, None) == qlin.QLIN_ERR_INVALID
    assert f(hs * 3, AUTO, 0, 16, x.data_ptr(), yp * 3, None, 0, None) == qlin.QLIN_ERR_INVALID   # 9 members
    assert f(hs, AUTO, 0, 16, x.data_ptr(), [yp[0], yp[0], yp[2]], None, 0, None) == qlin.QLIN_ERR_INVALID
    assert f(hs, AUTO, 0, 16, x.data_ptr(), [yp[0], None, yp[2]], None, 0, None) == qlin.QLIN_ERR_INVALID
    assert f(hs, AUTO, 0, 16, x.data_ptr(), [yp[0], yp[1] + 8, yp[2]], None, 0, None) == qlin.QLIN_ERR_ALIGN
    assert f(hs, AUTO, 0, 16, x.data_ptr(), yp, None, -1, None) == qlin.QLIN_ERR_INVALID
    assert f(hs, AUTO, 0, 16, x.data_ptr(), yp, yp[0], 1 << 20, None) == qlin.QLIN_ERR_INVALID     # y in ws
    assert f(hs, AUTO, 21, 16, x.data_ptr(), yp, None, 0, None) == qlin.QLIN_ERR_INVALID           # split > K/128
    o = gen.model_linear(0, 3)                      # K = 4096
    lo = make(o)
    assert f([hs[0], lo.h], AUTO, 0, 16, x.data_ptr(), yp[:2], None, 0, None) == qlin.QLIN_ERR_INVALID
    assert "share K" in qlin.last_error()
    s = make(dict(ws[1], zeros=None), symmetric=True)
    assert f([hs[0], s.h], AUTO, 0, 16, x.data_ptr(), yp[:2], None, 0, None) == qlin.QLIN_ERR_INVALID
    assert "format" in qlin.last_error()
    torch.cuda.synchronize()
    lo.close()
    s.close()


# ------------------------------------------------------------------ the drafter's weight pass

@pytest.mark.parametrize("layer", [0, 4])
def test_drafter_layer_shapes_symmetric(layer):
    """One drafter layer at M = 16 in the paper's symmetric format (Sec. 3.3):
    q|k|v as a group, then o, gate|up and down, every output compared."""
    x25 = gen.model_activations(3, 16, 2560)
    ws = [gen.drafter_linear(layer, p) for p in range(len(gen.LAYER_SHAPES))]
    lins = [make(w, symmetric=True) for w in ws]
    check_members(group_run(lins[:3], x25), ws[:3], x25, symmetric=True, what=f"layer {layer} q|k|v")
    for w, l in zip(ws[3:], lins[3:]):
        x = gen.model_activations(3, 16, w["K"])
        y = host_bits(l.forward(dev(x)))
        torch.cuda.synchronize()
        check_members([y], [w], x, symmetric=True, what=f"layer {layer} {w['name']} ({l.plan(16)})")
    for l in lins:
        l.close()


def test_drafter_context_projection():
    """The drafter's projection of five target layers' hidden states
    (K = 12800 -> N = 2560) at M = 1 and 16, symmetric."""
    w = gen.drafter_linear(0, len(gen.LAYER_SHAPES))
    lin = make(w, symmetric=True)
    for M in (1, 16):
        x = gen.model_activations(3, M, w["K"])
        y = host_bits(lin.forward(dev(x)))
        torch.cuda.synchronize()
        check_members([y], [w], x, symmetric=True, what=f"fc M={M} ({lin.plan(M)})")
    lin.close()
