"""GPU parity of every linear shape of the 4B-shaped decoder at the sizes the
benchmark reports, through the automatic plan (needs an MI355X).

The layer shapes (Sec. 2.1: the target's linears in the W4A16 format; Sec.
2.2 and 3.2: one 16-token block per verification step; chunked prefill over
the same weights): q 2560 -> 4096, k and v 2560 -> 1024, the fused q|k|v
2560 -> 6144, o 4096 -> 2560, gate|up 2560 -> 19456 and down 9728 -> 2560,
with the weights and activations of the whole-model workloads.  Outputs are
compared with the oracle element by element, within max(2 bf16 ulp, 1e-3);
where the oracle's float64 matmul would take minutes (large M x N x K) the
comparison runs on sampled columns (every row of each sampled column), always
including the first and last 128 columns so that the edge tiles are covered.
"""

import numpy as np
import pytest
import torch

from oracle import qlin_ref as ref
from paper_2607_04244_amd import qlin
from synth import gen

pytestmark = pytest.mark.gpu

SHAPES = {name: i for i, (name, _, _) in enumerate(gen.LAYER_SHAPES)}


def dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def host_bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def weights(layer, name):
    if name == "qkv":
        ws = [gen.model_linear(layer, p) for p in range(3)]
        return dict(K=ws[0]["K"], N=sum(w["N"] for w in ws),
                    packed=np.concatenate([w["packed"] for w in ws]),
                    scales=np.concatenate([w["scales"] for w in ws]),
                    zeros=np.concatenate([w["zeros"] for w in ws]))
    return gen.model_linear(layer, SHAPES[name])


def sample_columns(N, seed, n_random=512):
    rng = np.random.default_rng(seed)
    edge = min(128, N)
    cols = np.concatenate([np.arange(edge), np.arange(N - edge, N), rng.integers(0, N, n_random)])
    return np.unique(cols)


def check(y_bits, w, x, M, seed, what):
    """Compare all outputs when the oracle is cheap, else sampled columns."""
    K, N = w["K"], w["N"]
    if M * N * K <= 4e9:
        y_ref = ref.forward(x, w["packed"], w["scales"], w["zeros"])
        r = ref.compare(y_bits, y_ref)
    else:
        cols = sample_columns(N, seed)
        y_ref = ref.forward(x, w["packed"][cols], w["scales"][cols], w["zeros"][cols])
        r = ref.compare(np.ascontiguousarray(y_bits[:, cols]), y_ref)
    assert r["ok"], f"{what}: {r}"


@pytest.mark.parametrize("name", ["q", "k", "v", "qkv", "o", "gate_up", "down"])
def test_decoder_shape_at_verification_block(name):
    """M = 16 (one draft block) through the automatic plan, every output
    compared: the o projection runs the staged kernel with its largest x
    chunk (32 groups of K), k and v the asymmetric format at N = 1024."""
    w = weights(0, name)
    lin = qlin.QLinear(w["packed"], w["scales"], w["zeros"])
    x = gen.model_activations(3, 16, w["K"])
    y = host_bits(lin.forward(dev(x)))
    torch.cuda.synchronize()
    plan = lin.plan(16)
    lin.close()
    check(y, w, x, 16, 1, f"{name} M=16 ({plan})")


@pytest.mark.parametrize("M", [128, 512, 2048])
@pytest.mark.parametrize("name", ["q", "k", "v", "qkv", "o", "gate_up", "down"])
def test_decoder_shape_at_prefill_rows(name, M):
    """Chunked prefill: M rows through every decoder shape in one call of the
    automatic plan (tiled kernel, with a K split where the planner takes
    one)."""
    w = weights(17, name)
    lin = qlin.QLinear(w["packed"], w["scales"], w["zeros"])
    x = gen.model_activations(4, M, w["K"])
    y = host_bits(lin.forward(dev(x)))
    torch.cuda.synchronize()
    plan = lin.plan(M)
    lin.close()
    check(y, w, x, M, M, f"{name} M={M} ({plan})")


@pytest.mark.parametrize("M,name,expect", [
    (512, "down", "kernel=k_tiled<4,2> grid=480 block=256 split=3"),
    (512, "o", "kernel=k_tiled<4,2> grid=480 block=256 split=3"),
    (1024, "down", "kernel=k_tiled<8,4> grid=240 block=512 split=3"),
    (1024, "o", "kernel=k_tiled<6,4> grid=224 block=512 split=2"),
])
def test_measured_tiled_split_with_caller_workspace(M, name, expect):
    """The deep and narrow layers at M = 512 and 1024 take the measured K
    split when the caller's workspace holds it (a handle's own workspace is
    sized for decode and keeps the unsplit plan): the plan is the table's,
    and every sampled output matches the oracle."""
    w = weights(21, name)
    lin = qlin.QLinear(w["packed"], w["scales"], w["zeros"])
    need, plan = qlin.group_plan([lin], M)
    assert expect in plan and need > 0, plan
    x = gen.model_activations(4, M, w["K"])
    y = host_bits(qlin.forward_group([lin], dev(x), workspace=qlin.new_workspace(need))[0])
    torch.cuda.synchronize()
    lin.close()
    check(y, w, x, M, M + 7, f"{name} M={M} ({plan})")


@pytest.mark.parametrize("M,name", [(397, "down"), (639, "o"), (771, "down"), (1279, "o")])
def test_measured_tiled_split_at_ragged_rows(M, name):
    """The measured plans at the edges of their row ranges, where the last
    row block is partial: every sampled output against the oracle."""
    w = weights(22, name)
    lin = qlin.QLinear(w["packed"], w["scales"], w["zeros"])
    need, plan = qlin.group_plan([lin], M)
    assert "split=1 " not in plan and need > 0, plan
    x = gen.model_activations(4, M, w["K"])
    y = host_bits(qlin.forward_group([lin], dev(x), workspace=qlin.new_workspace(need))[0])
    torch.cuda.synchronize()
    lin.close()
    check(y, w, x, M, M + 11, f"{name} M={M} ({plan})")
