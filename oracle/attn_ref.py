"""CPU oracle for the drafter's block attention with a symmetric sliding window.

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the ``cpu_baseline`` leg of ``bench.py`` may import it.  It shares no code
with ``paper_2607_04244_amd`` (the product path) and imports nothing from it.

What it computes (Kim, Lee, Kim, arXiv 2607.04244):

* Sec. 2.2 / Sec. 3.2: the block-diffusion drafter predicts a block of 16
  tokens at once from mask-token queries, with bidirectional attention among
  them (no causal mask inside the block).
* Sec. 2.3 and Sec. 3.3 (Drafter SWA): the drafter's attention is limited to
  a fixed window of W = 1024 or 2048 tokens that is symmetric around each
  query; it is applied only inside the attention computation while the KV
  cache stays complete; sequences no longer than the window use full
  attention.

Readings taken where the paper is silent:

* The 16 queries of the block sit at the last 16 positions of the cache:
  query i (0 <= i < 16) is at position p_i = T - 16 + i of the T cached keys.
* Key j is visible to the query at position p iff |j - p| <= W / 2; W = 0
  or T <= W means every key is visible (the fallback).
* Grouped-query attention: query head h reads key/value head h // G with
  G = Hq / Hkv; scores are q . k / sqrt(D); softmax over the visible keys;
  output = sum of softmax weights x values.

Parity status: every function here is pinned by ``tests/test_oracle_attn.py``
(closed forms: uniform attention is the mean of the visible values, a
dominant key returns its value row; brute-force loops on tiny inputs; the
fallback equals unmasked attention; the head mapping).

Plain numpy, float64.
"""

import numpy as np

BLOCK = 16            # draft block size (Sec. 3.2)


def bf16_to_f64(bits):
    """bf16 bit patterns (uint16) -> float64 values, exactly."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def visible(T, W, nq=BLOCK):
    """Boolean [nq][T]: key j visible to block query i (positions T - nq + i)."""
    p = np.arange(T - nq, T)[:, None]
    j = np.arange(T)[None, :]
    if W == 0 or T <= W:
        return np.ones((nq, T), dtype=bool)
    return np.abs(j - p) <= W // 2


def swa_attention(q_bits, k_bits, v_bits, W):
    """Block attention of the drafter.

    q_bits: bf16 [Hq][16][D]; k_bits, v_bits: bf16 [Hkv][T][D].
    Returns float64 [Hq][16][D].
    """
    q = bf16_to_f64(q_bits)
    k = bf16_to_f64(k_bits)
    v = bf16_to_f64(v_bits)
    Hq, nq, D = q.shape
    Hkv, T, _ = k.shape
    G = Hq // Hkv
    mask = visible(T, W, nq)
    out = np.empty((Hq, nq, D))
    for h in range(Hq):
        s = q[h] @ k[h // G].T / np.sqrt(D)          # [nq][T]
        s = np.where(mask, s, -np.inf)
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        p /= p.sum(axis=1, keepdims=True)
        out[h] = p @ v[h // G]
    return out


def swa_attention_loops(q_bits, k_bits, v_bits, W):
    """The same definition with explicit loops over heads, queries and keys
    (no masking arithmetic, no vectorization), for tiny inputs."""
    import math
    q = bf16_to_f64(q_bits)
    k = bf16_to_f64(k_bits)
    v = bf16_to_f64(v_bits)
    Hq, nq, D = q.shape
    Hkv, T, _ = k.shape
    G = Hq // Hkv
    out = np.zeros((Hq, nq, D))
    for h in range(Hq):
        kv = h // G
        for i in range(nq):
            p = T - nq + i
            keys = [j for j in range(T) if W == 0 or T <= W or abs(j - p) <= W // 2]
            scores = [math.fsum(q[h, i, d] * k[kv, j, d] for d in range(D)) / math.sqrt(D) for j in keys]
            mx = max(scores)
            e = [math.exp(s - mx) for s in scores]
            tot = math.fsum(e)
            for d in range(D):
                out[h, i, d] = math.fsum(e[t] * v[kv, keys[t], d] for t in range(len(keys))) / tot
    return out
