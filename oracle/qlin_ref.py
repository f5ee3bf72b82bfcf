"""CPU oracle for the weight-only INT4 (W4A16) group-quantized linear layer.

TEST INFRASTRUCTURE ONLY.  This module is the correctness reference that the
HIP path is checked against.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it.  It shares no code with
``paper_2607_04244_amd`` (the product path) and imports nothing from it.

What it computes (Kim, Lee, Kim, "Quantize the Target, Quantize the Drafter",
arXiv 2607.04244):

* Sec. 2.1 (QAD paragraph): the quantized student keeps INT4 codes W_q with
  frozen per-group scales s; the dequantized weight is W = s (.) W_q, and the
  model is served in the W4A16 format (int4 weights, 16-bit activations).
* Sec. 3.2: the quantized target's weights are dequantized from the INT4 grid
  into floating point (BF16 weights), so the matmul sees bf16 weights.
* Sec. 3.3 (Drafter PTQ): group-wise INT4 with a group size of 128 along K.

Readings taken where the paper is silent:

* Codes are unsigned 4-bit q in [0, 15] with a per-group zero-point z, so the
  signed code of the paper is W_q = q - z.  The paper's symmetric format is the
  special case z = 8.
* Eight codes are packed per uint32 along K; code k = 8j + i lives in bits
  [4i, 4i + 4) of word j (lowest nibble = lowest k).  Tensors are row-major
  ``packed[N][K/8]``, ``scales[N][K/128]``, ``zeros[N][K/128]`` (bf16 bits).
* Each dequantized weight is the exact product (q - z) * s rounded ONCE to
  bf16, round-to-nearest-even; the matmul then multiplies bf16 x by these bf16
  weights exactly and sums in fp64.

Parity status: every function here is pinned by ``tests/test_oracle.py``
(hand-derived golden values, exhaustive comparison against torch's bf16
conversion, closed forms, invariants and brute force); none is "parity
unpinned".

Everything is plain numpy, evaluated in float64 unless stated.
"""

import numpy as np

GROUP = 128          # Sec. 3.3: group size 128 along K
CODES_PER_WORD = 8   # 8 x 4-bit codes per uint32


# --------------------------------------------------------------------------
# bit-level helpers
# --------------------------------------------------------------------------

def bf16_to_f64(bits):
    """bf16 bit patterns (uint16) -> float64 values, exactly.

    A bf16 number is the upper half of an IEEE binary32, so widening the
    pattern by 16 zero bits gives the binary32 with the same value.
    """
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def rne_bf16(values):
    """Round float64 values to bf16 bit patterns, round-to-nearest-even.

    The values must be exactly representable in binary32 (the oracle only
    rounds exact products (q - z) * s and small integers, which are); that is
    asserted, so no double rounding can hide here.  Rounding the binary32
    pattern at bit 16: add 0x7FFF plus the lowest kept bit, then truncate.
    This yields ties-to-even and carries correctly into the exponent.
    NaN inputs are outside the contract.
    """
    v = np.asarray(values, dtype=np.float64)
    f = v.astype(np.float32)
    finite = np.isfinite(f)
    if not np.array_equal(f.astype(np.float64)[finite], v[finite]):
        raise ValueError("rne_bf16: value not exactly representable in binary32")
    u = f.view(np.uint32).astype(np.uint64)
    lsb = (u >> np.uint64(16)) & np.uint64(1)
    r = (u + np.uint64(0x7FFF) + lsb) >> np.uint64(16)
    return r.astype(np.uint16)


# --------------------------------------------------------------------------
# packing (Sec. 2.1: INT4 codes W_q, packed for the W4A16 format)
# --------------------------------------------------------------------------

def unpack_codes(packed):
    """``packed[N][K/8]`` uint32 -> codes ``q[N][K]`` uint8 in [0, 15].

    q[n, 8j + i] = (packed[n, j] >> 4i) & 0xF.
    """
    P = np.asarray(packed, dtype=np.uint32)
    if P.ndim != 2:
        raise ValueError("packed must be 2-D [N][K/8]")
    N, K8 = P.shape
    q = np.empty((N, K8 * CODES_PER_WORD), dtype=np.uint8)
    for i in range(CODES_PER_WORD):
        q[:, i::CODES_PER_WORD] = ((P >> np.uint32(4 * i)) & np.uint32(0xF)).astype(np.uint8)
    return q


def pack_codes(q):
    """Inverse of :func:`unpack_codes`: codes ``q[N][K]`` -> ``packed[N][K/8]``."""
    Q = np.asarray(q)
    if Q.ndim != 2 or Q.shape[1] % CODES_PER_WORD:
        raise ValueError("codes must be [N][K] with K a multiple of 8")
    if Q.min(initial=0) < 0 or Q.max(initial=0) > 15:
        raise ValueError("codes must lie in [0, 15]")
    Q = Q.astype(np.uint32)
    N, K = Q.shape
    P = np.zeros((N, K // CODES_PER_WORD), dtype=np.uint32)
    for i in range(CODES_PER_WORD):
        P |= Q[:, i::CODES_PER_WORD] << np.uint32(4 * i)
    return P


# --------------------------------------------------------------------------
# dequantization (Sec. 2.1: W = s (.) W_q ; Sec. 3.2: BF16 weights)
# --------------------------------------------------------------------------

def dequant_exact(packed, scales, zeros, group=GROUP):
    """Unrounded dequantized weights (q - z) * s in float64, shape [N][K].

    Diagnostic only: the served weights are these values rounded to bf16
    (:func:`dequant_bf16`).  Each product has at most 4 + 8 significant bits,
    so float64 holds it exactly.
    """
    q = unpack_codes(packed).astype(np.float64)
    s = bf16_to_f64(scales)
    z = bf16_to_f64(zeros)
    N, K = q.shape
    if K % group or s.shape != (N, K // group) or z.shape != (N, K // group):
        raise ValueError("scales/zeros must be [N][K/group]")
    s_full = np.repeat(s, group, axis=1)
    z_full = np.repeat(z, group, axis=1)
    return (q - z_full) * s_full


def dequant_bf16(packed, scales, zeros, group=GROUP):
    """Dequantized bf16 weights as uint16 bit patterns, shape [N][K].

    w[n, k] = RNE_bf16((q[n, k] - z[n, g]) * s[n, g]),  g = floor(k / group).
    """
    return rne_bf16(dequant_exact(packed, scales, zeros, group))


def symmetric_zeros(N, K, group=GROUP):
    """Zero-points of the paper's symmetric format (Sec. 2.1, Sec. 3.3).

    A signed code W_q in [-8, 7] stored as the unsigned nibble u = W_q + 8
    dequantizes as (u - 8) * s, i.e. the asymmetric rule with z = 8.
    Returns bf16(8.0) = 0x4100 everywhere.
    """
    return np.full((N, K // group), 0x4100, dtype=np.uint16)


# --------------------------------------------------------------------------
# the linear layer
# --------------------------------------------------------------------------

def quantize_rtn(w_bits, scales, zeros, group=GROUP):
    """Fixed-grid round-to-nearest quantization of bf16 weights.

    Sec. 2.1 (QAD paragraph): at packing time the trained bf16 weights are
    rounded back onto the quantization grid of the frozen scales, giving new
    4-bit codes under the same scales; Sec. 4 (drafter PTQ, Table of drafter
    quantizers): round-to-nearest is the RTN baseline.  With the unsigned
    codes of this library (signed code = q - z):

        code[n][k] = clamp(round(w[n][k] / s[n][g]) + z[n][g], 0, 15),  g = k // group

    Readings (the paper fixes neither): the quotient is formed in binary32
    (IEEE division, correctly rounded) and rounded to the nearest integer with
    ties to even; a NaN quotient (0/0) gives code z.  Returns uint8 [N][K].
    """
    w = bf16_to_f64(w_bits).astype(np.float32)
    s = np.repeat(bf16_to_f64(scales).astype(np.float32), group, axis=1)
    z = np.repeat(bf16_to_f64(zeros), group, axis=1)
    with np.errstate(divide="ignore", invalid="ignore", over="ignore"):
        qf = w / s                                  # binary32 / binary32 -> binary32
        r = np.rint(qf).astype(np.float64)          # nearest integer, ties to even
    code = np.clip(r + z, 0.0, 15.0)
    code = np.where(np.isnan(code), z, code)
    return code.astype(np.uint8)


def quantize_pack(w_bits, scales, zeros, group=GROUP):
    """quantize_rtn() followed by the [N][K/8] packing of pack_codes()."""
    return pack_codes(quantize_rtn(w_bits, scales, zeros, group))


def forward(x_bits, packed, scales, zeros, group=GROUP, mode="bf16"):
    """y[M][N] = x[M][K] . w[N][K]^T in float64.

    ``x_bits`` are bf16 bit patterns.  With ``mode="bf16"`` (the served
    model) w is :func:`dequant_bf16`; ``mode="exact"`` uses the unrounded
    weights and exists only to show how much the rounding matters.  Every
    product of two bf16 numbers is exact in float64; only the float64
    summation rounds (relative error about K * 2**-53).
    """
    if mode == "bf16":
        w = bf16_to_f64(dequant_bf16(packed, scales, zeros, group))
    elif mode == "exact":
        w = dequant_exact(packed, scales, zeros, group)
    else:
        raise ValueError(mode)
    x = bf16_to_f64(x_bits)
    if x.ndim != 2 or x.shape[1] != w.shape[1]:
        raise ValueError("x must be [M][K]")
    return x @ w.T


def round_output(y):
    """bf16 bit pattern of an exactly-binary32-representable float64 result."""
    return rne_bf16(y)


# --------------------------------------------------------------------------
# comparison rule
# --------------------------------------------------------------------------

def ulp_bf16(v):
    """bf16 unit in the last place at |v| (binade of |v|; 2**-133 below 2**-126)."""
    a = np.abs(np.asarray(v, dtype=np.float64))
    _, e = np.frexp(a)                      # a = m * 2**e, m in [0.5, 1)
    ulp = np.ldexp(1.0, e - 1 - 7)          # floor(log2 a) = e - 1
    return np.where(a >= 2.0 ** -126, ulp, 2.0 ** -133)


def tolerance(y_ref):
    """Elementwise acceptance bound: max(2 bf16 ulp of the oracle value, 1e-3)."""
    return np.maximum(2.0 * ulp_bf16(y_ref), 1e-3)


def compare(y_bits, y_ref):
    """Check bf16 results (bit patterns) against float64 oracle values.

    Returns a dict with ``ok`` (every element within :func:`tolerance`),
    ``worst`` (max |err| / tol), ``nbad`` and ``max_abs``.  +0 and -0 compare
    equal because the difference is taken in float64.
    """
    y = bf16_to_f64(y_bits)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    if y.shape != y_ref.shape:
        raise ValueError(f"shape mismatch {y.shape} vs {y_ref.shape}")
    err = np.abs(y - y_ref)
    tol = tolerance(y_ref)
    bad = ~(err <= tol)
    return {
        "ok": not bool(bad.any()),
        "worst": float((err / tol).max(initial=0.0)),
        "nbad": int(bad.sum()),
        "max_abs": float(err.max(initial=0.0)),
    }
