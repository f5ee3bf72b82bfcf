// Internal interface between the drafter attention's C-ABI host code
// (attn_abi.cpp) and its HIP kernels (attn.hip).  Not installed; the public
// ABI is include/qlin_attn.h.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace qlin {

// Drafter block attention with a symmetric window.
//
// 16 block queries per query head, head dimension 128, grouped heads
// (query head hq reads key/value head hq / G).  The key range [lo, hi) any
// block query can see is cut into 64-key tiles; split s of key/value head h
// (workgroup h * S + s) owns tiles [s * tps, min((s + 1) * tps, ntiles)).
constexpr int kAttnD = 128;        // head dimension
constexpr int kAttnQ = 16;         // block queries (one MFMA tile of rows)
constexpr int kAttnTile = 64;      // keys per pipeline step
constexpr int kAttnWaves = 4;      // one query head per wave (two when G > 4)
constexpr int kAttnMaxG = 8;       // query heads per key/value head
constexpr int kAttnMaxSplits = 256;

struct AttnArgs {
    const uint16_t *q;      // [Hq][nq][128] bf16
    const uint16_t *k, *v;  // [Hkv][kv_stride][128] bf16
    uint16_t *out;          // [Hq][nq][128] bf16
    float *ws_o;            // S > 1: unnormalised partial outputs [Hq][S][8][16 rows][16]
    float *ws_ml;           // S > 1: (running max, sum of weights) [Hq][S][16 rows][2]
    int64_t kv_stride;      // elements between consecutive key/value heads
    int Hq, Hkv, G, nq, T;
    int lo, hi;             // keys [lo, hi) some block query can see
    int half;               // half window: key j visible to the query at p iff |j - p| <= half; < 0: all keys
    int ntiles, tps, S;
    float c;                // log2(e) / sqrt(128): scores to base-2 exponents
};

hipError_t launch_attn(const AttnArgs &a, hipStream_t st);
const char *attn_kernel_name(int G);

}  // namespace qlin
