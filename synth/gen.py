"""Seeded synthetic inputs for the W4A16 linear layer.

Shared by the tests, ``bench.py`` and ``__graft_entry__.smoke()``.  This module
only draws random numbers and converts them to storage formats; it holds none
of the layer's arithmetic (no unpacking, dequantization or matmul).

The paper's own data (its model weights, datasets and benchmarks) is not
available, so every workload is synthetic with the shapes of a 4B-parameter
decoder (hidden 2560, intermediate 9728, 36 layers) and these distributions:

* codes: uniform over [0, 15].  Eight uniform 4-bit codes packed per uint32
  are exactly a uniform random uint32, so words are drawn directly.
* scales: uniform U(a, b) drawn in binary32, then rounded to bf16.
* zero-points: uniform over {7, 8, 9}, stored as bf16.
* activations: N(0, sigma^2) drawn in binary32 (sigma is the standard
  deviation), optionally with each entry independently multiplied by 20 with
  probability p (activation outliers), then rounded to bf16.

Draw order inside one generator: packed words, scales, zeros, activations,
outlier mask.  bf16 rounding of drawn values uses torch's conversion.
"""

import numpy as np

GROUP = 128

# (name, K, N) of the linears in one decoder layer of the 4B-shaped model.
LAYER_SHAPES = (
    ("q", 2560, 4096),
    ("k", 2560, 1024),
    ("v", 2560, 1024),
    ("o", 4096, 2560),
    ("gate_up", 2560, 19456),
    ("down", 9728, 2560),
)
N_LAYERS = 36

# Workloads.  "single" workloads name one linear; "model" covers all 216.
CONFIGS = {
    0: dict(name="single-linear M=1 K=2560 N=2560", Ms=(1,), K=2560, N=2560,
            s_range=(0.002, 0.02), sigma=1.0, outlier_p=0.0, seed=0),
    1: dict(name="draft-block verify M=16 K=2560 N=19456 (fused gate+up)", Ms=(16,),
            K=2560, N=19456, s_range=(0.002, 0.02), sigma=1.0, outlier_p=0.0, seed=1),
    2: dict(name="ffn-down M=1/4/8/16 K=9728 N=2560 with outliers", Ms=(1, 4, 8, 16),
            K=9728, N=2560, s_range=(0.001, 0.01), sigma=0.5, outlier_p=0.01, seed=2),
    3: dict(name="36-layer 4B decoder weight pass M=16", Ms=(16,), model=True,
            s_range=(0.002, 0.02), sigma=1.0, outlier_p=0.0, seed=3),
    4: dict(name="chunked prefill M=128/512/2048 over the 36-layer weights",
            Ms=(128, 512, 2048), model=True, s_range=(0.002, 0.02), sigma=1.0,
            outlier_p=0.0, seed=4),
}


def f32_to_bf16_bits(a):
    """binary32 array -> bf16 bit patterns (uint16), via torch's RNE conversion."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16).copy()


def draw_weights(rng, K, N, s_range, z_values=(7, 8, 9), group=GROUP):
    """Packed codes [N][K/8] uint32, scales and zeros [N][K/group] bf16 bits."""
    packed = rng.integers(0, 2 ** 32, size=(N, K // 8), dtype=np.uint32)
    lo, hi = s_range
    scales = f32_to_bf16_bits(rng.uniform(lo, hi, size=(N, K // group)).astype(np.float32))
    zeros = f32_to_bf16_bits(
        np.asarray(z_values, dtype=np.float32)[rng.integers(0, len(z_values), size=(N, K // group))])
    return packed, scales, zeros


def draw_activations(rng, M, K, sigma=1.0, outlier_p=0.0, outlier_mul=20.0):
    """Activations x[M][K] as bf16 bits (outliers scaled before rounding)."""
    x = rng.standard_normal((M, K), dtype=np.float32) * np.float32(sigma)
    if outlier_p > 0.0:
        mask = rng.random((M, K)) < outlier_p
        x = np.where(mask, x * np.float32(outlier_mul), x).astype(np.float32)
    return f32_to_bf16_bits(x)


def linear_case(cfg_id, M=None):
    """One linear of a single-linear workload (configs 0, 1, 2).

    Returns dict(M, K, N, packed, scales, zeros, x).  For config 2 the
    activations are drawn once for the largest M and smaller M take the
    leading rows.
    """
    c = CONFIGS[cfg_id]
    if c.get("model"):
        raise ValueError("use model_linear() for whole-model workloads")
    rng = np.random.default_rng(c["seed"])
    packed, scales, zeros = draw_weights(rng, c["K"], c["N"], c["s_range"])
    Mmax = max(c["Ms"])
    x = draw_activations(rng, Mmax, c["K"], c["sigma"], c["outlier_p"])
    M = Mmax if M is None else M
    if M > Mmax:
        raise ValueError("M larger than the workload's")
    return dict(M=M, K=c["K"], N=c["N"], packed=packed, scales=scales,
                zeros=zeros, x=np.ascontiguousarray(x[:M]))


def model_linear_seed(layer, proj):
    """Seed of linear ``proj`` (index into LAYER_SHAPES) of decoder ``layer``."""
    return 3_000_000 + 10 * layer + proj


def model_linear(layer, proj):
    """Weights of one linear of the 36-layer model (configs 3 and 4)."""
    name, K, N = LAYER_SHAPES[proj]
    rng = np.random.default_rng(model_linear_seed(layer, proj))
    packed, scales, zeros = draw_weights(rng, K, N, CONFIGS[3]["s_range"])
    return dict(name=name, K=K, N=N, packed=packed, scales=scales, zeros=zeros)


# The drafter (Sec. 3.2: five layers, hidden size 2560, block size 16, about
# 537M parameters; Sec. 3.3: group-wise symmetric INT4, group 128).  Its
# layers have the decoder shapes above; the context projection maps the
# hidden states of five target layers (5 x 2560) to 2560, which with the
# five layers (504.6M) accounts for the stated parameter count (537.4M).
DRAFTER_LAYERS = 5
DRAFTER_FC = ("fc", 5 * 2560, 2560)


def drafter_linear_seed(layer, proj):
    """Seed of drafter linear ``proj`` (index into LAYER_SHAPES, or
    len(LAYER_SHAPES) for the context projection, which has no layer)."""
    return 5_000_000 + (100 if proj == len(LAYER_SHAPES) else 10 * layer + proj)


def drafter_linear(layer, proj):
    """Weights of one drafter linear in the symmetric format: packed codes and
    scales only (the zero-point is 8).  Draw order: packed words, scales."""
    name, K, N = DRAFTER_FC if proj == len(LAYER_SHAPES) else LAYER_SHAPES[proj]
    rng = np.random.default_rng(drafter_linear_seed(layer, proj))
    packed = rng.integers(0, 2 ** 32, size=(N, K // GROUP * 16), dtype=np.uint32)
    lo, hi = CONFIGS[3]["s_range"]
    scales = f32_to_bf16_bits(rng.uniform(lo, hi, size=(N, K // GROUP)).astype(np.float32))
    return dict(name=name, K=K, N=N, packed=packed, scales=scales)


def model_activations(cfg_id, M, K):
    """Activations for the whole-model workloads: one x per (M, K)."""
    c = CONFIGS[cfg_id]
    rng = np.random.default_rng([c["seed"], M, K])
    return draw_activations(rng, M, K, c["sigma"], c["outlier_p"])


def random_case(seed, M, K, N, s_range=(0.002, 0.02), z_values=(7, 8, 9),
                sigma=1.0, outlier_p=0.0):
    """A generic seeded case for tests at arbitrary (small) shapes."""
    rng = np.random.default_rng(seed)
    packed, scales, zeros = draw_weights(rng, K, N, s_range, z_values)
    x = draw_activations(rng, M, K, sigma, outlier_p)
    return dict(M=M, K=K, N=N, packed=packed, scales=scales, zeros=zeros, x=x)


# ---------------------------------------------------------------- drafter attention
#
# Block attention of the drafter: 32 query heads over 8 key/value heads of
# dimension 128 (the q/k/v projection widths 4096/1024/1024 of the layer
# shapes above), 16 block queries, a key/value cache of T tokens.  Keys and
# values are N(0, 1); queries are N(0, sigma_q^2), so that the scaled scores
# q.k / sqrt(128) have standard deviation sigma_q (a moderately peaked
# softmax).  All drawn in binary32 and rounded to bf16; draw order q, k, v.
ATTN_HQ, ATTN_HKV, ATTN_D, ATTN_NQ = 32, 8, 128, 16

ATTN_CONFIGS = {
    # long-input decode with the leaderboard window, its wider variant and
    # full attention (the window sweep's end points)
    "swa1024": dict(T=8192, window=1024, sigma_q=2.0, seed=11),
    "swa2048": dict(T=8192, window=2048, sigma_q=2.0, seed=11),
    "full": dict(T=8192, window=0, sigma_q=2.0, seed=11),
    # a short prompt inside the window (full-attention fallback)
    "short": dict(T=700, window=1024, sigma_q=2.0, seed=12),
}


def draw_attention(rng, Hq, Hkv, nq, T, sigma_q=2.0, D=ATTN_D, kv_stride=None):
    """q [Hq][nq][D], k and v [Hkv][kv_stride][D] as bf16 bits (tokens at and
    beyond T up to kv_stride are drawn too: they stand for unused capacity)."""
    kv_stride = T if kv_stride is None else kv_stride
    q = rng.standard_normal((Hq, nq, D), dtype=np.float32) * np.float32(sigma_q)
    k = rng.standard_normal((Hkv, kv_stride, D), dtype=np.float32)
    v = rng.standard_normal((Hkv, kv_stride, D), dtype=np.float32)
    return f32_to_bf16_bits(q), f32_to_bf16_bits(k), f32_to_bf16_bits(v)


def attention_case(name):
    """One drafter attention workload: dict(Hq, Hkv, nq, T, window, q, k, v)."""
    c = ATTN_CONFIGS[name]
    rng = np.random.default_rng(c["seed"])
    q, k, v = draw_attention(rng, ATTN_HQ, ATTN_HKV, ATTN_NQ, c["T"], c["sigma_q"])
    return dict(Hq=ATTN_HQ, Hkv=ATTN_HKV, nq=ATTN_NQ, T=c["T"], window=c["window"], q=q, k=k, v=v)
