"""Seeded random sweeps of the HIP path against the CPU oracle (needs an MI355X).

The other parity tests enumerate chosen shapes; these draw (M, K, N, format,
path, K split) for single linears, member widths for grouped launches, and
(heads, block size, cache length, window, key ranges) for the drafter
attention from one fixed seed each, so every run checks the same few hundred
planner and kernel combinations, every output element against the oracle:
within max(2 bf16 ulp, 1e-3) for the linears, within the derived attention
bound (tests/test_attn.py) for attention.  A forced split that does not fit
a shape must be refused explicitly (QLIN_ERR_UNSUPPORTED), never run wrong.
"""

import numpy as np
import pytest
import torch

from paper_2607_04244_amd import qlin
from synth import gen

from test_attn import check as attn_check
from test_parity import assert_close, dev, host_bits, make, oracle, run_split

pytestmark = pytest.mark.gpu

GEMV, SKINNY, TILED, AUTO, REGS = qlin.PATH_GEMV, qlin.PATH_SKINNY, qlin.PATH_TILED, qlin.PATH_AUTO, qlin.PATH_REGS


def draw_rows(rng):
    """Decode-sized rows most of the time, some staged-kernel and prefill sizes."""
    u = rng.random()
    if u < 0.5:
        return int(rng.integers(1, 17))
    if u < 0.75:
        return int(rng.integers(17, 65))
    return int(rng.integers(65, 401))


def paths_for(M):
    p = [AUTO, TILED]
    if M <= 4:
        p.append(GEMV)
    if M <= 16:
        p.append(REGS)
    if M <= 64:
        p.append(SKINNY)
    return p


def linear_cases(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        M = draw_rows(rng)
        K = 128 * int(rng.integers(1, 25))
        N = 16 * int(rng.integers(1, 81))
        sym = bool(rng.random() < 0.3)
        path = paths_for(M)[int(rng.integers(0, len(paths_for(M))))]
        Kb = K // 128
        split = 0 if rng.random() < 0.4 else int(rng.integers(1, Kb + 1))
        sigma = float(rng.choice([0.5, 1.0, 4.0]))
        out.append((i, M, K, N, sym, path, split, sigma))
    return out


@pytest.mark.parametrize("i,M,K,N,sym,path,split,sigma", linear_cases(120, 20261202))
def test_random_linear_matches_oracle(i, M, K, N, sym, path, split, sigma):
    c = gen.random_case(9000 + i, M, K, N, sigma=sigma)
    lin = make(c, symmetric=sym)
    y = run_split(lin, c["x"], path, split)
    what = f"case {i}: M={M} K={K} N={N} sym={sym} path={path} split={split}"
    if y is None:
        assert split > 0, what         # only a forced split may be refused
    else:
        assert_close(y, oracle(c, symmetric=sym), what)
    lin.close()


def group_cases(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        nmem = int(rng.integers(2, 9))
        K = 128 * int(rng.integers(1, 21))
        widths = [16 * int(rng.integers(1, 41)) for _ in range(nmem)]
        M = draw_rows(rng)
        sym = bool(rng.random() < 0.3)
        out.append((i, M, K, tuple(widths), sym))
    return out


@pytest.mark.parametrize("i,M,K,widths,sym", group_cases(24, 20261203))
def test_random_group_matches_oracle(i, M, K, widths, sym):
    cases = [gen.random_case(9500 + 10 * i + j, M, K, N) for j, N in enumerate(widths)]
    lins = [make(c, symmetric=sym) for c in cases]
    x = dev(cases[0]["x"])
    need, plan = qlin.group_plan(lins, M)
    ys = qlin.forward_group(lins, x, workspace=qlin.new_workspace(need) if need else None)
    torch.cuda.synchronize()
    for j, (c, y) in enumerate(zip(cases, ys)):
        c = dict(c, x=cases[0]["x"])
        assert_close(host_bits(y), oracle(c, symmetric=sym), f"case {i} member {j} ({plan})")
    for l in lins:
        l.close()


def attention_cases(n, seed):
    rng = np.random.default_rng(seed)
    out = []
    for i in range(n):
        Hkv = int(rng.choice([1, 2, 4, 8]))
        G = int(rng.integers(1, 9))
        nq = int(rng.integers(1, 17))
        T = int(rng.integers(nq, 3001))
        u = rng.random()
        W = 0 if u < 0.25 else int(rng.integers(1, 2 * T + 2))
        cap = T + int(rng.integers(0, 65))
        ntiles_max = (T + 63) // 64
        splits = 0 if rng.random() < 0.5 else int(rng.integers(1, ntiles_max + 1))
        out.append((i, G * Hkv, Hkv, nq, T, W, cap, splits))
    return out


@pytest.mark.parametrize("i,Hq,Hkv,nq,T,W,cap,splits", attention_cases(48, 20261204))
def test_random_attention_matches_oracle(i, Hq, Hkv, nq, T, W, cap, splits):
    rng = np.random.default_rng(9900 + i)
    q, k, v = gen.draw_attention(rng, Hq, Hkv, nq, T, 2.0, kv_stride=cap)
    attn_check(q, k, v, T, W, splits, what=f"case {i}: Hq={Hq} Hkv={Hkv} nq={nq} T={T} W={W} cap={cap} "
                                             f"splits={splits}")
