"""Benchmark of the W4A16 linear layer on one MI355X.

Workload: the draft-block verification linear, M = 16 rows (one 16-token
draft block), K = 2560, N = 19456 (fused gate + up projection of a
4B-shaped decoder), int4 codes with bf16 scales and zero-points in groups of
128 along K.  A step is one qlin_forward of that linear: activation staging,
weight streaming, dequantization, the dot products and the reduction, all in
the HIP kernels.  Weights are re-laid-out once at handle creation (untimed,
like loading a model).

To measure HBM rather than the 256 MB last-level cache, R handles with their
own copies of the weights (over 1 GiB together) are used in turn, and the
steps are replayed from a HIP graph so host launch cost is not measured.

Prints one JSON line.  ``value`` is algorithmic bytes per step / time per step
(GB/s); the algorithmic bytes are the int4 codes, the bf16 scales and zeros,
x and y (K*N/2 + 4*(K/128)*N + 2*M*K + 2*M*N).
"""

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

PEAK_HBM_GBS = 8000.0
METRIC = "W4A16 linear HBM GB/s (% of peak) at M=1/16; µs per 4B-shaped layer"


def algorithmic_bytes(M, K, N, symmetric=False):
    per_group = 2 if symmetric else 4
    return K * N // 2 + per_group * (K // 128) * N + 2 * M * K + 2 * M * N


def file_hash(path):
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()[:16]


def traffic_from_profiles(kernel_src_hash, kernel):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current kernel source; else None."""
    p = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        t = json.load(open(p))
    except (OSError, ValueError):
        return None
    if t.get("kernels_hip_sha256_16") != kernel_src_hash:
        return None
    e = t.get("kernels", {}).get(kernel)
    return None if e is None else e.get("hbm_bytes_per_launch")


def cpu_baseline(case, budget_s=15.0):
    """Time the oracle (as it stands) on the host cores on whole config-1 calls."""
    from oracle import qlin_ref as ref
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
    except Exception:
        threads = 1
    times = []
    t_start = time.perf_counter()
    while True:
        t0 = time.perf_counter()
        ref.forward(case["x"], case["packed"], case["scales"], case["zeros"])
        times.append(time.perf_counter() - t0)
        if time.perf_counter() - t_start > budget_s or len(times) >= 5:
            break
    t = float(np.median(times))
    b = algorithmic_bytes(case["M"], case["K"], case["N"])
    return {"value": round(b / t / 1e9, 4), "unit": "GB/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{len(times)} whole oracle calls of the M=16 K=2560 N=19456 linear "
                      f"(median {t:.2f} s each; numpy unpack/dequant single-threaded, fp64 matmul on "
                      f"{threads} BLAS threads)"}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=4000)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle timing")
    ap.add_argument("--path", type=int, default=0, help="force a kernel path (tuning)")
    ap.add_argument("--split", type=int, default=0, help="force a K split (tuning)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the layer has no multi-GPU path in this build "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)

    import torch

    from paper_2607_04244_amd import qlin
    from synth import gen

    torch.cuda.set_device(0)
    case = gen.linear_case(1)
    M, K, N = case["M"], case["K"], case["N"]
    bytes_step = algorithmic_bytes(M, K, N)
    weight_bytes = K * N // 2 + 4 * (K // 128) * N
    R = max(2, -(-(1 << 30) // weight_bytes))          # > 1 GiB of distinct weights
    lins = [qlin.QLinear(case["packed"], case["scales"], case["zeros"]) for _ in range(R)]
    x = torch.from_numpy(case["x"].view(np.int16)).view(torch.bfloat16).cuda()
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    plan = lins[0].plan(M, args.path, args.split)

    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        for i in range(args.warmup):
            lins[i % R].forward(x, out=y, path=args.path, split_k=args.split)
    stream.synchronize()

    # one graph of R steps (every weight copy once); K steps = whole replays + a tail graph
    def capture(n):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for i in range(n):
                lins[i % R].forward(x, out=y, path=args.path, split_k=args.split)
        return g

    K_steps = args.steps
    g_full = capture(R)
    tail = K_steps % R
    g_tail = capture(tail) if tail else None
    for _ in range(2):
        g_full.replay()
    stream.synchronize()

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        ev0.record(stream)
        for _ in range(K_steps // R):
            g_full.replay()
        if g_tail is not None:
            g_tail.replay()
        ev1.record(stream)
    stream.synchronize()
    torch.cuda.synchronize()
    ms_total = ev0.elapsed_time(ev1)
    ms_step = ms_total / K_steps
    gbs = bytes_step / (ms_step * 1e-3) / 1e9

    # eager launches from Python, for reference (host-launch bound for small kernels)
    ev2 = torch.cuda.Event(enable_timing=True)
    ev3 = torch.cuda.Event(enable_timing=True)
    n_eager = min(K_steps, 2000)
    with torch.cuda.stream(stream):
        ev2.record(stream)
        for i in range(n_eager):
            lins[i % R].forward(x, out=y, path=args.path, split_k=args.split)
        ev3.record(stream)
    stream.synchronize()
    eager_us = ev2.elapsed_time(ev3) * 1e3 / n_eager

    kernel = plan.split("kernel=")[1].split()[0] if "kernel=" in plan else "?"
    src_hash = file_hash(os.path.join(ROOT, "paper_2607_04244_amd", "csrc", "kernels.hip"))
    traffic = traffic_from_profiles(src_hash, kernel)
    out = {
        "metric": METRIC,
        "value": round(gbs, 2),
        "unit": "GB/s",
        "n_gpus": 1,
        "steps": K_steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_step, 6),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "draft-block verification linear: M=16, K=2560, N=19456 (fused gate+up), "
                               "int4 g128 asymmetric, bf16 scales/zeros",
                   "M": M, "K": K, "N": N, "group": 128, "rotating_weight_copies": R,
                   "bytes_per_step": bytes_step, "plan": plan, "timing": "HIP graph replay",
                   "us_per_step": round(ms_step * 1e3, 3), "pct_of_peak_hbm": round(100 * gbs / PEAK_HBM_GBS, 2),
                   "eager_launch_us_per_step": round(eager_us, 3)},
        "roofline": {"bound": "hbm", "kernel": kernel, "achieved": round(gbs, 2), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "traffic": traffic, "bytes_per_launch": bytes_step,
                     "avg_launch_us": round(ms_step * 1e3, 3)},
    }
    for l in lins:
        l.close()
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(case)
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
