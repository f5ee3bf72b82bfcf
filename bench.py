"""Benchmark of the W4A16 linear layer on one MI355X.

Default workload: the draft-block verification linear, M = 16 rows (one
16-token draft block), K = 2560, N = 19456 (fused gate + up projection of a
4B-shaped decoder), int4 codes with bf16 scales and zero-points in groups of
128 along K.  A step is one qlin_forward of that linear: activation staging,
weight streaming, dequantization, the dot products and the reduction, all in
the HIP kernels.  Weights are re-laid-out once at handle creation (untimed,
like loading a model).

To measure HBM rather than the 256 MB last-level cache, R handles with their
own copies of the weights (over 1 GiB together) are used in turn, and the
steps are replayed from a HIP graph so host launch cost is not measured.
The same rotation is timed for a plain 128-bit streaming read of the same
byte count (qlin_stream_read), the achievable ceiling at this size.

Prints one JSON line.  ``value`` is algorithmic bytes per step / time per step
(GB/s); the algorithmic bytes are the int4 codes, the bf16 scales and zeros,
x and y (K*N/2 + 4*(K/128)*N + 2*M*K + 2*M*N).  ``metric_parts`` carries the
rest of the metric, measured in the same run: the M=1 linear (K=N=2560,
GB/s) and the 36-layer 4B-shaped weight pass at M=16 (microseconds per
verification step and per layer: q|k|v as one grouped launch, then o,
gate|up and down, 144 launches in one graph on one stream, so each runs after
the previous one as in a decoder), and the drafter's 5-layer pass, each next
to the same launch structure reduced to plain streaming reads of each
launch's bytes (the ceiling of a pass made of that many dependent launches).

Other modes (not the benchmark line): ``--workload`` c0 | c2m1 | c2m4 |
c2m8 | c2m16 | model (the 36-layer pass at M=16) | drafter (the drafter's
five layers and context projection at M=16, symmetric format) | prefill128
| prefill512 | prefill2048 (the 36-layer linears at M rows, TFLOP/s and
matrix-core utilisation) | quantize (bf16 -> packed int4 codes on a fixed
grid, GB/s) | swa1024 | swa2048 | attn-full | attn-short (the drafter's
block attention: 32 query heads over 8 key/value heads of dimension 128, 16
block queries, a T = 8192 cache with a symmetric window of 1024 or 2048
tokens, full attention, and T = 700 inside the window; GB/s of the visible
key/value span) | gemm128 | gemm512 | gemm2048 (diagnostic only: the
vendor bf16 GEMM on weights already dequantized to bf16, at the same
per-layer shapes and M, summed to a 36-layer pass); ``--separate-qkv`` runs
q, k and v as three launches;
``--calibrate-copy`` runs a plain 256 MiB device copy for the HBM-traffic
counter calibration.
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
PEAK_BF16_TFLOPS = 2500.0          # dense bf16 matrix-core peak of MI355X
METRIC = "W4A16 linear HBM GB/s (% of peak) at M=1/16; µs per 4B-shaped layer"


def algorithmic_bytes(M, K, N, symmetric=False):
    per_group = 2 if symmetric else 4
    return K * N // 2 + per_group * (K // 128) * N + 2 * M * K + 2 * M * N


# device sources each kernel family is built from (the stored counter
# summary of a kernel is valid while these files are unchanged)
KERNEL_SOURCES = {
    "linear": ("kernels.hip", "device_common.h", "qlin_internal.h"),
    "tiled": ("tiled.hip", "device_common.h", "qlin_internal.h"),
    "attention": ("attn.hip", "attn_internal.h", "device_common.h", "qlin_internal.h"),
}


def kernel_family(kernel):
    if kernel.startswith("k_attn"):
        return "attention"
    return "tiled" if kernel.startswith("k_tiled") else "linear"


def code_only(text):
    """C++ source text without its comments, trailing blanks and empty lines
    (the sources hold no string literal with a comment marker in it)."""
    import re
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    text = re.sub(r"//[^\n]*", "", text)
    return "\n".join(l.rstrip() for l in text.splitlines() if l.strip())


def device_sources_hash(family="linear"):
    """sha256 (16 hex digits) of the code of the device sources of one kernel
    family (comments left out), in name order: identifies the kernels a
    stored counter summary was taken on."""
    import hashlib
    d = os.path.join(ROOT, "paper_2607_04244_amd", "csrc")
    h = hashlib.sha256()
    for name in sorted(KERNEL_SOURCES[family]):
        with open(os.path.join(d, name), encoding="utf-8") as f:
            h.update(name.encode() + b"\0" + code_only(f.read()).encode())
    return h.hexdigest()[:16]


def traffic_from_profiles(kernel, key=None):
    """HBM bytes per launch from the committed rocprofv3 counter summary (entry
    `key`, default the kernel's name), if it was taken on the current source
    of the kernel's family; else None."""
    p = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        t = json.load(open(p))
    except (OSError, ValueError):
        return None
    e = t.get("kernels", {}).get(key or kernel)
    if e is None or e.get("sources_sha256_16") != device_sources_hash(kernel_family(kernel)):
        return None
    return e.get("hbm_bytes_per_launch")


class ClockSampler:
    """Samples the GPU's current shader (sclk) and memory (mclk) clocks from
    the driver's sysfs tables (the row marked with '*') in a thread, for the
    timed region; summary: min / median / max MHz over the samples, and the
    table's rows.  Absent tables give an empty summary."""

    def __init__(self, period_s=0.0005):
        import glob
        import threading
        self.period = period_s
        self.paths = {}
        for kind in ("sclk", "mclk"):
            found = sorted(glob.glob(f"/sys/class/drm/card*/device/pp_dpm_{kind}"))
            if found:
                self.paths[kind] = found[0]
        self.samples = {k: [] for k in self.paths}
        self.levels = {k: self._read(k)[1] for k in self.paths}
        self._stop = threading.Event()
        self._thread = threading.Thread(target=self._run, daemon=True)

    def _read(self, kind):
        try:
            lines = open(self.paths[kind]).read().split("\n")
        except OSError:
            return None, []
        cur, levels = None, []
        for line in lines:
            parts = line.replace("Mhz", "").replace("MHz", "").split()
            if len(parts) >= 2 and parts[1].isdigit():
                levels.append(int(parts[1]))
                if line.strip().endswith("*"):
                    cur = int(parts[1])
        return cur, levels

    def _run(self):
        while not self._stop.is_set():
            for k in self.paths:
                cur = self._read(k)[0]
                if cur is not None:
                    self.samples[k].append(cur)
            time.sleep(self.period)

    def __enter__(self):
        if self.paths:
            self._thread.start()
        return self

    def __exit__(self, *exc):
        self._stop.set()
        if self._thread.is_alive():
            self._thread.join()

    def summary(self):
        out = {}
        for k, v in self.samples.items():
            if v:
                v = sorted(v)
                out[f"{k}_mhz"] = {"min": v[0], "median": v[len(v) // 2], "max": v[-1], "samples": len(v)}
                out[f"{k}_levels_mhz"] = self.levels.get(k, [])
        return out


def host_cores():
    """Cores this process may run on (its affinity mask)."""
    try:
        return len(os.sched_getaffinity(0))
    except AttributeError:
        return os.cpu_count() or 1


def cpu_baseline(case, budget_s=12.0, y_gpu=None):
    """Time the oracle (as it stands) on the host cores on whole calls, with
    the BLAS threads set to the cores of the affinity mask; the unpack +
    dequantize step is also timed on its own (the rest is the fp64 matmul).
    With ``y_gpu`` (bf16 bits of the timed kernel's output), every element of
    it is checked against the last timed oracle call, by the tests' rule."""
    from oracle import qlin_ref as ref
    cores = host_cores()
    try:
        from threadpoolctl import threadpool_limits
        limiter = threadpool_limits(limits=cores, user_api="blas")
    except Exception:
        limiter = None
    times, deq = [], []
    t_start = time.perf_counter()
    while time.perf_counter() - t_start < budget_s and len(times) < 50:
        t0 = time.perf_counter()
        y_ref = ref.forward(case["x"], case["packed"], case["scales"], case["zeros"])
        times.append(time.perf_counter() - t0)
        if len(deq) < 3:
            t0 = time.perf_counter()
            ref.dequant_bf16(case["packed"], case["scales"], case["zeros"])
            deq.append(time.perf_counter() - t0)
    if limiter is not None:
        limiter.unregister()
    t, td = float(np.median(times)), float(np.median(deq))
    b = algorithmic_bytes(case["M"], case["K"], case["N"])
    parity = None
    if y_gpu is not None:
        c = ref.compare(y_gpu, y_ref)
        parity = {"outputs": int(y_gpu.size), "ok": c["ok"], "nbad": c["nbad"],
                  "worst_err_over_tol": round(c["worst"], 4), "max_abs_err": c["max_abs"]}
    return {"value": round(b / t / 1e9, 4), "unit": "GB/s", "cores": int(cores), "kind": "oracle",
            "timed_output_vs_oracle": parity,
            "sample": f"{len(times)} whole oracle calls of the M={case['M']} K={case['K']} N={case['N']} "
                      f"linear (median {t:.3f} s each: unpack + dequantize {td:.3f} s in numpy, one thread; "
                      f"fp64 matmul {max(t - td, 0.0):.3f} s on up to {cores} BLAS threads)",
            "unpack_dequant_s": round(td, 4), "matmul_s": round(max(t - td, 0.0), 4)}


def graph_time_us(torch, stream, launches, reps):
    """Capture `launches` (list of callables) in one graph; median us per launch
    over `reps` replays (at least 5) after 3 untimed ones.  The timed replays
    follow one more untimed replay back to back on `stream`, with an event
    between consecutive replays, so each interval is one replay with its work
    already submitted (the GPU never waits for the host inside it).  Every
    replay runs on `stream`: a replay issued outside its context goes to the
    default stream and overlaps the timed ones."""
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, stream=stream):
        for f in launches:
            f()
    with torch.cuda.stream(stream):
        for _ in range(3):
            g.replay()
    torch.cuda.synchronize()
    n = max(reps, 5)
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(n + 1)]
    with torch.cuda.stream(stream):
        g.replay()
        evs[0].record(stream)
        for i in range(n):
            g.replay()
            evs[i + 1].record(stream)
    stream.synchronize()
    times = sorted(evs[i].elapsed_time(evs[i + 1]) * 1e3 / len(launches) for i in range(n))
    return times[len(times) // 2], g


def stream_read_ceiling(torch, qlin, nbytes, stream):
    """Plain streaming read of nbytes per launch over > 1 GiB of rotating buffers."""
    R = max(2, -(-(1 << 30) // nbytes))
    nb = (nbytes + 15) // 16 * 16
    bufs = [torch.empty(nb, dtype=torch.uint8, device="cuda").fill_(i & 0xFF) for i in range(R)]
    sink = torch.zeros(4096, dtype=torch.int32, device="cuda")
    best = None
    for grid in (512, 1024, 2048):
        def mk(b):
            return lambda: qlin.qlin_stream_read(b.data_ptr(), nb, grid, sink.data_ptr(), stream.cuda_stream)
        us, _ = graph_time_us(torch, stream, [mk(b) for b in bufs], reps=max(3, int(4e9 / (nb * R))))
        best = us if best is None else min(best, us)
    del bufs
    return nb / (best * 1e-6) / 1e9, best


def launch_floor_us(torch, qlin, stream, n=200):
    """The per-launch cost of the launch structure itself: n back-to-back
    launches of the streaming-read kernel over 16 bytes (256 workgroups of 512
    threads, the decode kernels' launch shape), replayed from one graph."""
    buf = torch.zeros(16, dtype=torch.uint8, device="cuda")
    sink = torch.zeros(4096, dtype=torch.int32, device="cuda")
    calls = [(lambda: qlin.qlin_stream_read(buf.data_ptr(), 16, 256, sink.data_ptr(), stream.cuda_stream))] * n
    us, g = graph_time_us(torch, stream, calls, reps=10)
    del g
    return us


def make_case(workload):
    from synth import gen
    if workload == "verify":
        return gen.linear_case(1)
    if workload == "c0":
        return gen.linear_case(0)
    if workload.startswith("c2m"):
        return gen.linear_case(2, M=int(workload[3:]))
    raise ValueError(workload)


def calibrate_copy():
    """A plain device-to-device copy of 256 MiB, 20 times (counter calibration:
    each launch reads and writes exactly 268,435,456 bytes)."""
    import torch
    torch.cuda.set_device(0)
    a = torch.ones(1 << 28, dtype=torch.uint8, device="cuda")
    b = torch.empty_like(a)
    for _ in range(20):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"calibration": "device copy", "bytes_read_per_launch": 1 << 28,
                      "bytes_written_per_launch": 1 << 28, "launches": 20}), flush=True)


def structure_ceiling_us(torch, qlin, sizes, stream, reps):
    """The same launch structure with nothing but the weight stream: one plain
    streaming read per launch of that launch's bytes, from distinct regions of
    one buffer, in one graph.  Returns the step time (us)."""
    offs, total = [], 0
    for n in sizes:
        offs.append(total)
        total += (n + 4095) // 4096 * 4096
    buf = torch.empty(total, dtype=torch.uint8, device="cuda").fill_(1)
    sink = torch.zeros(4096, dtype=torch.int32, device="cuda")
    best = None
    for grid in (256, 512, 1024):
        calls = [(lambda o=o, n=n: qlin.qlin_stream_read(buf.data_ptr() + o, (n + 15) // 16 * 16, grid,
                                                          sink.data_ptr(), stream.cuda_stream))
                 for o, n in zip(offs, sizes)]
        us, g = graph_time_us(torch, stream, calls, reps=reps)
        del g
        best = us * len(sizes) if best is None else min(best, us * len(sizes))
    del buf
    torch.cuda.empty_cache()
    return best


def model_pass(M=16, x_seed=3, separate_qkv=False, drafter=False, reps=15, ceiling=False):
    """The linears of a whole decoder step at M rows, one graph on one stream:
    per layer q|k|v (one grouped launch, or three), o, gate|up, down.  The
    target: 36 layers of config-3 weights (asymmetric).  The drafter: its 5
    layers and its context projection (symmetric, Sec. 3.3).  Prefill-sized
    M share one caller workspace sized for the largest plan.  Returns a dict
    of the step time and rates; with ``ceiling``, also the step time of the
    same launches reduced to plain streaming reads of their bytes."""
    import torch

    from paper_2607_04244_amd import qlin
    from synth import gen
    torch.cuda.set_device(0)
    n_layers = gen.DRAFTER_LAYERS if drafter else gen.N_LAYERS
    layers, xs, total, flops = [], {}, 0, 0
    t0 = time.perf_counter()
    for layer in range(n_layers):
        if drafter:
            ws = [gen.drafter_linear(layer, p) for p in range(len(gen.LAYER_SHAPES))]
            lins = [qlin.QLinear(w["packed"], w["scales"], None) for w in ws]
        else:
            ws = [gen.model_linear(layer, p) for p in range(len(gen.LAYER_SHAPES))]
            lins = [qlin.QLinear(w["packed"], w["scales"], w["zeros"]) for w in ws]
        groups = [[l] for l in lins[:3]] if separate_qkv else [lins[:3]]
        groups += [[l] for l in lins[3:]]
        layers.extend(groups)
    if drafter:
        w = gen.drafter_linear(0, len(gen.LAYER_SHAPES))
        layers.insert(0, [qlin.QLinear(w["packed"], w["scales"], None)])
    setup_s = time.perf_counter() - t0
    steps, launch_bytes = [], []
    for grp in layers:
        K = grp[0].K
        if K not in xs:
            xs[K] = torch.from_numpy(gen.model_activations(x_seed, M, K).view(np.int16)).view(torch.bfloat16).cuda()
        ys = [torch.empty((M, l.N), dtype=torch.bfloat16, device="cuda") for l in grp]
        steps.append((grp, ys))
        launch_bytes.append(sum(algorithmic_bytes(M, K, l.N, symmetric=drafter) for l in grp))
        for l in grp:
            total += algorithmic_bytes(M, K, l.N, symmetric=drafter)
            flops += 2 * M * K * l.N
    need = max(qlin.group_plan(grp, M)[0] for grp, _ in steps)
    wsb = qlin.new_workspace(need) if need else None
    stream = torch.cuda.Stream()
    calls = [(lambda grp=grp, ys=ys: qlin.forward_group(grp, xs[grp[0].K], ys, workspace=wsb)) for grp, ys in steps]
    us_per_launch, g = graph_time_us(torch, stream, calls, reps=reps)
    us_step = us_per_launch * len(calls)
    tfs = flops / (us_step * 1e-6) / 1e12
    gbs = total / (us_step * 1e-6) / 1e9
    plans = sorted({qlin.group_plan(grp, M)[1] for grp, _ in steps})
    del g
    for grp, _ in steps:
        for l in grp:
            l.close()
    torch.cuda.empty_cache()
    who = (f"drafter: {n_layers} layers + context projection, symmetric" if drafter
           else f"36-layer 4B decoder weight pass")
    out = {"workload": f"{who}, M={M} ({len(calls)} launches, "
                       f"{'separate' if separate_qkv else 'grouped'} q|k|v, one graph)",
           "us_per_step": round(us_step, 2), "us_per_layer": round(us_step / n_layers, 3),
           "bytes_per_step": total, "GBps": round(gbs, 1), "pct_of_peak_hbm": round(100 * gbs / PEAK_HBM_GBS, 2),
           "TFLOPs": round(tfs, 1), "mfma_util_pct": round(100 * tfs / PEAK_BF16_TFLOPS, 2),
           "workspace_bytes": need, "setup_s": round(setup_s, 1), "plans": plans}
    if ceiling:
        c_us = structure_ceiling_us(torch, qlin, launch_bytes, stream, reps)
        out["stream_read_structure_us"] = round(c_us, 2)
        out["pct_of_stream_read_structure"] = round(100 * c_us / us_step, 1)
    return out


def bench_model(args, M=16, x_seed=3, drafter=False):
    out = model_pass(M, x_seed, separate_qkv=args.separate_qkv, drafter=drafter,
                     reps=max(5, min(50, args.steps // 144)))
    print(json.dumps(out), flush=True)


def bench_gemm_ceiling(args, M):
    """Diagnostic only, never part of the path: the vendor bf16 GEMM
    (torch.matmul -> hipBLASLt) on weights already dequantized to bf16, at
    the decoder's per-layer shapes (q|k|v as one 2560 x 6144 product, o,
    gate|up, down) and M rows.  Reports each shape's time and TFLOP/s and the
    36-layer pass those times add up to, next to which the fused W4A16
    kernel's prefill pass can be read.  Weights rotate over > 600 MB of
    copies; both operands are contiguous row-major (x [M, K] @ w [K, N])."""
    import torch

    from synth import gen
    torch.cuda.set_device(0)
    stream = torch.cuda.Stream()
    shapes = [("q|k|v", 2560, 6144), ("o", 4096, 2560), ("gate|up", 2560, 19456), ("down", 9728, 2560)]
    g = torch.Generator(device="cuda").manual_seed(6)
    out, pass_us, pass_flops = {}, 0.0, 0
    for name, K, N in shapes:
        copies = max(2, -(-600_000_000 // (2 * K * N)))
        ws = [torch.randn((K, N), device="cuda", generator=g).mul_(0.02).to(torch.bfloat16) for _ in range(copies)]
        x = torch.randn((M, K), device="cuda", generator=g).to(torch.bfloat16)
        y = torch.empty((M, N), device="cuda", dtype=torch.bfloat16)
        with torch.cuda.stream(stream):
            for w in ws:
                torch.matmul(x, w, out=y)                 # library set-up outside the capture
        stream.synchronize()
        calls = [(lambda w=w: torch.matmul(x, w, out=y)) for w in ws]
        us, gr = graph_time_us(torch, stream, calls, reps=max(5, min(50, args.steps // len(calls))))
        del gr, ws
        torch.cuda.empty_cache()
        tfs = 2 * M * K * N / (us * 1e-6) / 1e12
        out[name] = {"K": K, "N": N, "us": round(us, 3), "TFLOPs": round(tfs, 1),
                     "pct_of_peak_bf16": round(100 * tfs / PEAK_BF16_TFLOPS, 2)}
        pass_us += us * gen.N_LAYERS
        pass_flops += 2 * M * K * N * gen.N_LAYERS
    tfs = pass_flops / (pass_us * 1e-6) / 1e12
    print(json.dumps({"workload": f"bf16 GEMM on pre-dequantized weights (diagnostic ceiling), M={M}",
                      "shapes": out, "pass_us": round(pass_us, 1), "pass_TFLOPs": round(tfs, 1),
                      "pass_pct_of_peak_bf16": round(100 * tfs / PEAK_BF16_TFLOPS, 2)}), flush=True)


def bench_quantize(args):
    """Fixed-grid RTN quantize + pack of the fused gate+up weight (N = 19456,
    K = 2560) from bf16: HBM-bound, reports GB/s of algorithmic bytes (bf16
    weights in, packed codes out, scales and zeros in)."""
    import torch

    from paper_2607_04244_amd import qlin
    torch.cuda.set_device(0)
    N, K = 19456, 2560
    rng = np.random.default_rng(5)
    g = torch.Generator(device="cuda").manual_seed(5)
    ws = [torch.randn((N, K), device="cuda", generator=g).mul_(0.02).to(torch.bfloat16) for _ in range(12)]
    sc = torch.from_numpy(rng.uniform(0.002, 0.02, size=(N, K // 128)).astype(np.float32)).to(torch.bfloat16).cuda()
    zr = torch.from_numpy(rng.integers(7, 10, size=(N, K // 128)).astype(np.float32)).to(torch.bfloat16).cuda()
    out = torch.empty((N, K // 8), dtype=torch.int32, device="cuda")
    nbytes = N * K * 2 + N * K // 2 + 4 * N * (K // 128)
    stream = torch.cuda.Stream()
    calls = [(lambda w=w: qlin._check(qlin.qlin_quantize(K, N, 128, w.data_ptr(), sc.data_ptr(), zr.data_ptr(),
                                                       out.data_ptr(), torch.cuda.current_stream().cuda_stream)))
             for w in ws]
    us, _ = graph_time_us(torch, stream, calls, reps=max(1, args.steps // len(calls)))
    print(json.dumps({"workload": f"quantize+pack N={N} K={K} bf16 -> int4 g128 (12 rotating weight copies)",
                      "us_per_call": round(us, 3), "bytes_per_call": nbytes,
                      "GBps": round(nbytes / (us * 1e-6) / 1e9, 1),
                      "pct_of_peak_hbm": round(100 * nbytes / (us * 1e-6) / 1e9 / PEAK_HBM_GBS, 2)}), flush=True)


ATTN_WORKLOADS = {"swa1024": "swa1024", "swa2048": "swa2048", "attn-full": "full", "attn-short": "short"}


def attn_span(T, nq, window):
    """Keys [lo, T) some block query can see (the window or the fallback)."""
    if window == 0 or T <= window:
        return 0, T
    return max(0, T - nq - window // 2), T


def bench_attention(args, name):
    """Drafter block attention: one qlin_swa_attention call per step over
    rotating copies of the key/value cache (> 1 GiB together, so the reads
    come from HBM, not the last-level cache), replayed from a HIP graph.
    Algorithmic bytes: the visible key/value span, q and the output."""
    import torch

    from oracle import attn_ref as ar
    from paper_2607_04244_amd import qlin
    from synth import gen
    torch.cuda.set_device(0)
    c = gen.attention_case(ATTN_WORKLOADS[name])
    Hq, Hkv, nq, T, W = c["Hq"], c["Hkv"], c["nq"], c["T"], c["window"]
    lo, hi = attn_span(T, nq, W)
    nbytes = Hkv * (hi - lo) * 128 * 2 * 2 + 2 * Hq * nq * 128 * 2
    dev = lambda a: torch.from_numpy(np.ascontiguousarray(a).view(np.int16)).view(torch.bfloat16).cuda()
    q = dev(c["q"])
    k0, v0 = dev(c["k"]), dev(c["v"])
    cache_bytes = 2 * k0.numel() * 2
    R = max(2, -(-(1 << 30) // cache_bytes))
    kvs = [(k0, v0)] + [(k0.clone(), v0.clone()) for _ in range(R - 1)]
    S, ws_bytes, plan = qlin.qlin_swa_plan(Hq, Hkv, 128, nq, T, W, args.split)
    ws = torch.empty(max(ws_bytes, 16), dtype=torch.uint8, device="cuda")
    out = torch.empty((Hq, nq, 128), dtype=torch.bfloat16, device="cuda")
    stream = torch.cuda.Stream()
    calls = [(lambda k=k, v=v: qlin.swa_attention(q, k, v, W, splits=args.split, out=out, workspace=ws))
             for k, v in kvs]
    with torch.cuda.stream(stream):
        for i in range(args.warmup):
            calls[i % R]()
    stream.synchronize()
    us, _ = graph_time_us(torch, stream, calls, reps=max(2, args.steps // R))
    gbs = nbytes / (us * 1e-6) / 1e9
    kernel = plan.split("kernel=")[1].split()[0]
    res = {"workload": f"drafter block attention {name}: Hq={Hq}, Hkv={Hkv}, d=128, nq={nq}, T={T}, "
                       f"window={W or 'full'} ({hi - lo} visible keys per head, {R} rotating caches)",
           "us_per_call": round(us, 3), "bytes_per_call": nbytes, "GBps": round(gbs, 1),
           "pct_of_peak_hbm": round(100 * gbs / PEAK_HBM_GBS, 2), "plan": plan,
           "roofline": {"bound": "hbm", "kernel": kernel + (" + k_attn_combine" if S > 1 else ""),
                        "achieved": round(gbs, 2), "peak": PEAK_HBM_GBS, "unit": "GB/s",
                        "frac": round(gbs / PEAK_HBM_GBS, 4),
                        "traffic": traffic_from_profiles(kernel, f"call@{name}"),
                        "bytes_per_launch": nbytes, "avg_launch_us": round(us, 3)}}
    if not args.no_cpu:
        times = []
        t_start = time.perf_counter()
        while time.perf_counter() - t_start < 10.0 and len(times) < 20:
            t0 = time.perf_counter()
            o_ref = ar.swa_attention(c["q"], c["k"], c["v"], W)
            times.append(time.perf_counter() - t0)
        t = float(np.median(times))
        threads = host_cores()
        # the last timed call's output against the oracle (every copy of the cache holds the same data)
        o_gpu = ar.bf16_to_f64(out.view(torch.int16).cpu().numpy().view(np.uint16))
        vmax = float(np.abs(ar.bf16_to_f64(c["v"])).max())
        err = float(np.abs(o_gpu - o_ref).max())
        res["cpu_baseline"] = {"value": round(nbytes / t / 1e9, 4), "unit": "GB/s", "cores": int(threads),
                               "kind": "oracle",
                               "timed_output_vs_oracle": {"outputs": int(o_gpu.size), "max_abs_err": err,
                                                          "max_abs_err_over_max_abs_v": round(err / vmax, 6)},
                               "sample": f"{len(times)} whole oracle calls (median {t:.3f} s; float64 numpy, "
                                         f"matmuls on up to {threads} BLAS threads)"}
    print(json.dumps(res), flush=True)


def linear_rate(case, steps, warmup, path=0, split=0):
    """Time `steps` forwards of one linear (HIP-graph replays over R handles
    with their own weight copies, > 1 GiB together, so the weights come from
    HBM), after `warmup` untimed ones; the timed region is bracketed by
    device synchronisations.  Returns a dict of the rates and the plan."""
    import torch

    from paper_2607_04244_amd import qlin
    M, K, N = case["M"], case["K"], case["N"]
    bytes_step = algorithmic_bytes(M, K, N)
    weight_bytes = K * N // 2 + 4 * (K // 128) * N
    R = max(2, -(-(1 << 30) // weight_bytes))          # > 1 GiB of distinct weights
    lins = [qlin.QLinear(case["packed"], case["scales"], case["zeros"]) for _ in range(R)]
    x = torch.from_numpy(case["x"].view(np.int16)).view(torch.bfloat16).cuda()
    y = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    # a forced split or tiled path runs with a caller workspace of its size
    ws = None
    if split or path == qlin.PATH_TILED:
        need, plan = qlin.group_plan([lins[0]], M, path, split)
        ws = qlin.new_workspace(need) if need else None
    else:
        plan = lins[0].plan(M, path, split)

    stream = torch.cuda.Stream()
    with torch.cuda.stream(stream):
        for i in range(warmup):
            lins[i % R].forward(x, out=y, path=path, split_k=split, workspace=ws)
    stream.synchronize()

    # one graph of R steps (every weight copy once); the steps = whole replays + a tail graph
    def capture(n):
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=stream):
            for i in range(n):
                lins[i % R].forward(x, out=y, path=path, split_k=split, workspace=ws)
        return g

    g_full = capture(R)
    tail = steps % R
    with torch.cuda.stream(stream):
        for _ in range(2):
            g_full.replay()
    stream.synchronize()

    ev0 = torch.cuda.Event(enable_timing=True)
    ev1 = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    with ClockSampler() as clocks:
        with torch.cuda.stream(stream):
            # an untimed replay of the rotation just before the timed region:
            # the timed steps start with their work submitted and with the
            # rotation in its steady state (each copy last read R launches
            # ago).  Whole rotations replay the graph; the remaining steps
            # are direct launches (a graph's replay carries a fixed cost of
            # its own, measured at ~1 us per step over a 20-launch graph,
            # that direct launches queued behind busy work do not pay).
            g_full.replay()
            ev0.record(stream)
            for _ in range(steps // R):
                g_full.replay()
            for i in range(tail):
                lins[i].forward(x, out=y, path=path, split_k=split, workspace=ws)
            ev1.record(stream)
        stream.synchronize()
    torch.cuda.synchronize()
    ms_step = ev0.elapsed_time(ev1) / steps
    gbs = bytes_step / (ms_step * 1e-3) / 1e9
    y_bits = y.view(torch.int16).cpu().numpy().view(np.uint16)     # the last timed step's output

    # eager launches from Python, for reference (host-launch bound for small kernels)
    ev2 = torch.cuda.Event(enable_timing=True)
    ev3 = torch.cuda.Event(enable_timing=True)
    n_eager = min(steps, 2000)
    with torch.cuda.stream(stream):
        ev2.record(stream)
        for i in range(n_eager):
            lins[i % R].forward(x, out=y, path=path, split_k=split, workspace=ws)
        ev3.record(stream)
    stream.synchronize()
    eager_us = ev2.elapsed_time(ev3) * 1e3 / n_eager
    del g_full
    for l in lins:
        l.close()
    del lins
    torch.cuda.empty_cache()
    return {"ms_step": ms_step, "GBps": gbs, "plan": plan, "R": R, "bytes": bytes_step, "eager_us": eager_us,
            "stream": stream, "clocks": clocks.summary(), "y_bits": y_bits}


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=4000)
    ap.add_argument("--warmup", type=int, default=200)
    ap.add_argument("--no-cpu", action="store_true", help="skip the oracle timing")
    ap.add_argument("--no-parts", action="store_true", help="skip the M=1, model and drafter passes")
    ap.add_argument("--path", type=int, default=0, help="force a kernel path (tuning)")
    ap.add_argument("--split", type=int, default=0, help="force a K split (tuning)")
    ap.add_argument("--workload", default="verify")
    ap.add_argument("--calibrate-copy", action="store_true")
    ap.add_argument("--separate-qkv", action="store_true", help="model / prefill passes: q, k, v as three launches")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU: the layer has no multi-GPU path in this library "
              "(run with --gpus 1)", file=sys.stderr)
        sys.exit(2)
    if args.calibrate_copy:
        return calibrate_copy()
    if args.workload.startswith("prefill"):
        # chunked-prefill regime: M rows through every linear of the model
        return bench_model(args, M=int(args.workload[len("prefill"):]), x_seed=4)
    if args.workload.startswith("gemm"):
        return bench_gemm_ceiling(args, M=int(args.workload[len("gemm"):]))
    if args.workload == "model":
        return bench_model(args)
    if args.workload == "drafter":
        return bench_model(args, drafter=True)
    if args.workload == "quantize":
        return bench_quantize(args)
    if args.workload in ATTN_WORKLOADS:
        return bench_attention(args, args.workload)

    import torch

    from paper_2607_04244_amd import qlin

    torch.cuda.set_device(0)
    case = make_case(args.workload)
    M, K, N = case["M"], case["K"], case["N"]
    r = linear_rate(case, args.steps, args.warmup, args.path, args.split)
    ms_step, gbs, plan, R, bytes_step, eager_us = r["ms_step"], r["GBps"], r["plan"], r["R"], r["bytes"], r["eager_us"]
    K_steps = args.steps
    ceil_gbs, ceil_us = stream_read_ceiling(torch, qlin, bytes_step, r["stream"])
    floor_us = launch_floor_us(torch, qlin, r["stream"])

    parts = None
    if args.workload == "verify" and not args.no_parts:
        # the rest of the metric: the M=1 linear, and microseconds per layer of
        # the whole 4B-shaped step (and the drafter's) at M=16
        print("measuring the M=1 linear and the model passes", file=sys.stderr, flush=True)
        c0 = linear_rate(make_case("c0"), 2000, 100)
        model = model_pass(16, ceiling=True)
        draft = model_pass(16, drafter=True, ceiling=True)
        parts = {"M1_K2560_N2560": {"us": round(c0["ms_step"] * 1e3, 3), "GBps": round(c0["GBps"], 1),
                                    "pct_of_peak_hbm": round(100 * c0["GBps"] / PEAK_HBM_GBS, 2),
                                    "plan": c0["plan"]},
                 "M16_K2560_N19456": {"us": round(ms_step * 1e3, 3), "GBps": round(gbs, 1),
                                      "pct_of_peak_hbm": round(100 * gbs / PEAK_HBM_GBS, 2)},
                 "model_M16": {k: model[k] for k in ("workload", "us_per_step", "us_per_layer", "GBps",
                                                     "pct_of_peak_hbm", "bytes_per_step", "stream_read_structure_us",
                                                     "pct_of_stream_read_structure")},
                 "drafter_M16": {k: draft[k] for k in ("workload", "us_per_step", "us_per_layer", "GBps",
                                                       "pct_of_peak_hbm", "bytes_per_step", "stream_read_structure_us",
                                                       "pct_of_stream_read_structure")}}
        parts["model_M16"]["us_at_70pct_of_peak"] = round(model["bytes_per_step"] / (0.7 * PEAK_HBM_GBS * 1e3), 1)

    kernel = plan.split("kernel=")[1].split()[0] if "kernel=" in plan else "?"
    traffic = traffic_from_profiles(kernel)
    wl = {"verify": "draft-block verification linear: M=16, K=2560, N=19456 (fused gate+up)"}.get(
        args.workload, f"{args.workload}: M={M}, K={K}, N={N}")
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
        "config": {"workload": wl + ", int4 g128 asymmetric, bf16 scales/zeros",
                   "M": M, "K": K, "N": N, "group": 128, "rotating_weight_copies": R,
                   "bytes_per_step": bytes_step, "plan": plan,
                   "timing": "HIP graph replays of the rotation, remaining steps as direct launches, "
                             "behind one untimed replay",
                   "us_per_step": round(ms_step * 1e3, 3), "pct_of_peak_hbm": round(100 * gbs / PEAK_HBM_GBS, 2),
                   "stream_read_ceiling_GBps": round(ceil_gbs, 1), "stream_read_ceiling_us": round(ceil_us, 3),
                   "pct_of_stream_read_ceiling": round(100 * gbs / ceil_gbs, 1),
                   "launch_floor_us": round(floor_us, 3),
                   "launch_floor_bound_pct_of_peak_hbm": round(
                       100 * bytes_step / ((floor_us + bytes_step / (PEAK_HBM_GBS * 1e3)) * 1e-6) / 1e9 / PEAK_HBM_GBS, 1),
                   "eager_launch_us_per_step": round(eager_us, 3),
                   "clocks_during_timed_region": r["clocks"]},
        "metric_parts": parts,
        "roofline": {"bound": "hbm", "kernel": kernel, "achieved": round(gbs, 2), "peak": PEAK_HBM_GBS,
                     "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
                     "traffic": traffic, "bytes_per_launch": bytes_step,
                     "avg_launch_us": round(ms_step * 1e3, 3)},
    }
    if not args.no_cpu:
        out["cpu_baseline"] = cpu_baseline(case, y_gpu=r["y_bits"])
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
