"""Host logic of bench.py, on the CPU: the one-GPU contract, the algorithmic
byte counts the reported rates divide by, the counter-summary lookup and the
clock sampler's parsing."""

import json
import os
import subprocess
import sys
import threading
import time

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
sys.path.insert(0, ROOT)
import bench  # noqa: E402


def test_more_than_one_gpu_is_refused_before_any_gpu_work():
    r = subprocess.run([sys.executable, os.path.join(ROOT, "bench.py"), "--gpus", "2"], capture_output=True,
                       text=True, timeout=120, cwd=ROOT)
    assert r.returncode == 2 and "one GPU" in r.stderr and r.stdout == ""


def test_algorithmic_bytes():
    # codes K*N/2, 4 bytes of s|z (2 of s) per group and column, x and y in bf16
    assert bench.algorithmic_bytes(16, 2560, 19456) == 24_903_680 + 1_556_480 + 81_920 + 622_592 == 27_164_672
    assert bench.algorithmic_bytes(1, 2560, 2560) == 3_276_800 + 204_800 + 5_120 + 5_120
    assert bench.algorithmic_bytes(16, 2560, 19456, symmetric=True) == 27_164_672 - 778_240


def test_attention_span():
    assert bench.attn_span(8192, 16, 1024) == (8192 - 16 - 512, 8192)
    assert bench.attn_span(700, 16, 1024) == (0, 700)        # inside the window: full attention
    assert bench.attn_span(8192, 16, 0) == (0, 8192)


def test_counter_summary_is_used_only_for_the_sources_it_was_taken_on():
    t = json.load(open(os.path.join(ROOT, "profiles", "traffic.json")))
    e = t["kernels"]["k_skinny<1,16>"]
    got = bench.traffic_from_profiles("k_skinny<1,16>")
    if e["sources_sha256_16"] == bench.device_sources_hash("linear"):
        assert got == e["hbm_bytes_per_launch"]
    else:
        assert got is None
    assert bench.traffic_from_profiles("k_no_such_kernel") is None


def test_clock_sampler_reads_the_marked_row(tmp_path):
    s = tmp_path / "pp_dpm_sclk"
    s.write_text("S: 101Mhz\n0: 500Mhz\n1: 2353Mhz *\n")
    c = bench.ClockSampler(period_s=0.0005)
    c.paths = {"sclk": str(s)}
    c.samples = {"sclk": []}
    c.levels = {"sclk": c._read("sclk")[1]}
    c._thread = threading.Thread(target=c._run, daemon=True)
    with c:
        time.sleep(0.01)
    out = c.summary()
    assert out["sclk_levels_mhz"] == [101, 500, 2353]
    assert out["sclk_mhz"]["min"] == out["sclk_mhz"]["max"] == 2353 and out["sclk_mhz"]["samples"] > 0


def test_clock_sampler_without_tables_is_empty():
    c = bench.ClockSampler()
    c.paths, c.samples = {}, {}
    with c:
        pass
    assert c.summary() == {}


def test_cpu_baseline_checks_the_timed_output():
    """The cpu_baseline leg compares the timed kernel's output with its own
    oracle call: a planted one-element error is reported, a faithful output
    passes."""
    from oracle import qlin_ref as ref
    from synth import gen
    c = gen.random_case(1, 4, 256, 64)
    y = ref.rne_bf16(ref.forward(c["x"], c["packed"], c["scales"], c["zeros"]).astype(np.float32).astype(np.float64))
    good = bench.cpu_baseline(c, budget_s=0.1, y_gpu=y.astype(np.uint16))["timed_output_vs_oracle"]
    assert good["ok"] and good["outputs"] == 4 * 64
    bad = y.astype(np.uint16)
    bad[1, 3] ^= 0x0100
    r = bench.cpu_baseline(c, budget_s=0.1, y_gpu=bad)["timed_output_vs_oracle"]
    assert not r["ok"] and r["nbad"] == 1


def test_source_hash_ignores_comments_only():
    src = "int a; // note\n/* block\n comment */ int b;\n\n"
    assert bench.code_only(src) == bench.code_only("int a;\n int b;")
    assert bench.code_only(src) != bench.code_only("int a; int c;")
