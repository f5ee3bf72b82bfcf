"""The entry point that allocates nothing (qlin_forward_group_noalloc),
through the C ABI, against qlin_forward_group with a caller workspace (the
same plan, so the same bits) and the oracle (needs an MI355X).

Two calls in a row on the same static scratch, the second with a smaller
input, for a decode plan that cuts the K range, a tiled plan that cuts it,
and a grouped launch; then the size limit."""

import numpy as np
import pytest
import torch

from oracle import qlin_ref as ref
from paper_2607_04244_amd import qlin
from synth import gen

pytestmark = pytest.mark.gpu

AUTO, SKINNY, TILED, REGS = qlin.PATH_AUTO, qlin.PATH_SKINNY, qlin.PATH_TILED, qlin.PATH_REGS


def dev(bits):
    return torch.from_numpy(np.ascontiguousarray(bits).view(np.int16)).view(torch.bfloat16).cuda()


def host_bits(t):
    return t.view(torch.int16).cpu().numpy().view(np.uint16)


def both(lins, x_bits, path, split):
    """(no-allocation outputs, caller-workspace outputs), each a list of host bit arrays."""
    x = dev(x_bits)
    M = x.shape[0]
    ys_a = [torch.full((M, l.N), 3.0, dtype=torch.bfloat16, device="cuda") for l in lins]
    rc = qlin.qlin_forward_group_noalloc([l.h for l in lins], path, split, M, x.data_ptr(),
                                         [y.data_ptr() for y in ys_a], torch.cuda.current_stream().cuda_stream)
    assert rc == qlin.QLIN_OK, qlin.last_error()
    need, _ = qlin.group_plan(lins, M, path, split)
    ys_b = qlin.forward_group(lins, x, path=path, split_k=split, workspace=qlin.new_workspace(need))
    torch.cuda.synchronize()
    return [host_bits(y) for y in ys_a], [host_bits(y) for y in ys_b]


@pytest.mark.parametrize("K,N,path,split,M1,M2", [
    (9728, 2560, AUTO, 0, 16, 9),        # the down projection: the automatic plan cuts K in 3
    (4096, 2560, REGS, 5, 16, 3),        # a forced 5-way split, register kernel
    (2560, 1024, TILED, 4, 200, 130),    # prefill rows, tiled kernel with a 4-way split
    (4096, 2560, AUTO, 0, 128, 96),      # the automatic tiled plan at prefill rows
])
def test_two_calls_match_the_workspace_entry_point(K, N, path, split, M1, M2):
    c = gen.random_case(K + N + M1, M1, K, N)
    lin = qlin.QLinear(c["packed"], c["scales"], c["zeros"])
    for M in (M1, M2):
        x = c["x"][:M]
        a, b = both([lin], x, path, split)
        assert np.array_equal(a[0], b[0]), f"M={M}: outputs differ from qlin_forward_group's"
        r = ref.compare(a[0], ref.forward(x, c["packed"], c["scales"], c["zeros"]))
        assert r["ok"], f"M={M}: {r}"
    lin.close()


def test_grouped_launch_two_calls():
    ws = [gen.random_case(90 + i, 16, 2560, n) for i, n in enumerate((4096, 1024, 1024))]
    lins = [qlin.QLinear(w["packed"], w["scales"], w["zeros"]) for w in ws]
    for M, split in ((16, 4), (5, 2)):
        x = ws[0]["x"][:M]
        a, b = both(lins, x, SKINNY, split)
        for i, w in enumerate(ws):
            assert np.array_equal(a[i], b[i]), f"member {i} M={M}"
            assert ref.compare(a[i], ref.forward(x, w["packed"], w["scales"], w["zeros"]))["ok"]
    for l in lins:
        l.close()


def test_plans_beyond_the_static_scratch_are_refused():
    """A forced split whose partial sums exceed the 16 MiB array is refused
    before any launch, with the size in the message."""
    K, N, M = 2560, 19456, 64
    c = gen.random_case(5, M, K, N)
    lin = qlin.QLinear(c["packed"], c["scales"], c["zeros"])
    need, _ = qlin.group_plan([lin], M, SKINNY, 4)
    assert need > 16 << 20, need
    x = dev(c["x"])
    y = torch.zeros((M, N), dtype=torch.bfloat16, device="cuda")
    rc = qlin.qlin_forward_group_noalloc([lin.h], SKINNY, 4, M, x.data_ptr(), [y.data_ptr()],
                                         torch.cuda.current_stream().cuda_stream)
    assert rc == qlin.QLIN_ERR_UNSUPPORTED and "static array" in qlin.last_error()
    torch.cuda.synchronize()
    assert torch.all(y == 0)
    lin.close()
