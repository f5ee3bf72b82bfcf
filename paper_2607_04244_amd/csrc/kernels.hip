// HIP kernels of the W4A16 linear layer for CDNA4 (gfx950).
//
// The layer (Sec. 2.1, 3.2, 3.3 of arXiv 2607.04244): every weight is the
// exact product (q - z) * s of a 4-bit code and its 128-wide group's scale,
// rounded once to bf16; y = x . w^T with fp32 accumulation, rounded once to
// bf16.
//
// Device weight layout ("block layout").  The canonical [N][K/8] words are
// re-laid-out at handle creation into blocks of 16 columns x 128 k (one
// quantization group of one column tile) = 256 words = 1 KiB.  Block (t, kb)
// starts at word (t * Kb + kb) * 256, so a wave that walks the groups of one
// column tile reads consecutive KiB.  Lane l of a wave owns words
// [4l, 4l + 4) of a block (one 128-bit load); word j of lane l covers k in
// [32j, 32j + 32) of the group, and its nibble p holds the code of
//     n = 16 t + 4 * ((l >> 2) & 3) + r,   r  = 2 * (p & 1) + (p >> 2)
//     k = 128 kb + 32 j + 16 h + 4 * (l >> 4) + (l & 3),   h = (p >> 1) & 1.
// That is exactly the operand order of the dequantizing matrix op below, so
// no lane shuffle is needed between HBM and the MFMA.
//
// Dequantization on the matrix cores.  For nibble pairs extracted as bf16
// "128 + q" (bit trick: 0x4300 | q is bf16 128 + q), one
// v_mfma_f32_4x4x4_16b_bf16 computes, for 16 independent 4x4 blocks,
//     D = A . diag(s) + C,  A[k][r] = 128 + q[n_r][k],  C = -(128 + z) s,
// i.e. D[k][n] = (q - z) * s exactly (each product has <= 16 significant
// bits, the sum is exactly representable).  v_cvt_pk_bf16_f32 then rounds
// each value once, to nearest even.  The vector-ALU route does the same with
// v_dot2_f32_bf16 on the same extracted pairs.  Both routes are bit-identical
// to the definition; the unpack/dequantize test hooks check that.

#include "qlin_internal.h"

namespace qlin {

typedef short v4s __attribute__((ext_vector_type(4)));
typedef float v4f __attribute__((ext_vector_type(4)));
typedef float v2f __attribute__((ext_vector_type(2)));
typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
typedef __bf16 v2bf __attribute__((ext_vector_type(2)));
typedef uint32_t v4u __attribute__((ext_vector_type(4)));
typedef uint32_t v2u __attribute__((ext_vector_type(2)));

// ------------------------------------------------------------------ layout

// Column (within the tile) and k (within the group) of nibble p of word j of lane l.
__host__ __device__ inline void block_coord(int l, int j, int p, int &n16, int &k128) {
    const int r = 2 * (p & 1) + (p >> 2);
    const int h = (p >> 1) & 1;
    n16 = 4 * ((l >> 2) & 3) + r;
    k128 = 32 * j + 16 * h + 4 * (l >> 4) + (l & 3);
}

// ------------------------------------------------------------------ small helpers

__device__ inline uint32_t cvt_pk_bf16(float lo, float hi) {
    v2f f = {lo, hi};
    v2bf b = __builtin_convertvector(f, v2bf);   // round to nearest even
    return __builtin_bit_cast(uint32_t, b);
}

__device__ inline uint16_t cvt_bf16(float v) {
    __bf16 b = (__bf16)v;
    return __builtin_bit_cast(uint16_t, b);
}

__device__ inline float bf16_lo_to_f32(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi_to_f32(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// The four "128 + q" bf16 pairs of one packed word: pair i holds nibbles i
// (low half) and i + 4 (high half).
struct Pairs { uint32_t a0, a1, a2, a3; };
__device__ inline Pairs extract_pairs(uint32_t P) {
    constexpr uint32_t kMask = 0x000F000Fu, kMagic = 0x43004300u;   // bf16 128.0 in both halves
    Pairs o;
    o.a0 = (P & kMask) | kMagic;
    o.a1 = ((P >> 4) & kMask) | kMagic;
    o.a2 = ((P >> 8) & kMask) | kMagic;
    o.a3 = ((P >> 12) & kMask) | kMagic;
    return o;
}

// s | z << 16 word of a column (symmetric handles store only s; z = 8).
template <bool SYM>
__device__ inline uint32_t load_sz(const void *sz, size_t idx) {
    if constexpr (SYM) {
        return (uint32_t)((const uint16_t *)sz)[idx] | (0x4100u << 16);
    } else {
        return ((const uint32_t *)sz)[idx];
    }
}

// --- matrix-core dequantization ------------------------------------------

struct MfmaDeq { v4s bdiag; v4f c4; };

// Per-group constants of lane l for column n = 16 t + (l & 15):
// B = diag(s) in the 4x4 block layout (this lane supplies B[r][l & 3],
// non-zero only for r = l & 3) and C = -(128 + z) * s in all four rows.
__device__ inline MfmaDeq mfma_setup(uint32_t sz, uint32_t shift, uint32_t keep_lo) {
    const float s = bf16_lo_to_f32(sz);
    const float z = bf16_hi_to_f32(sz);
    const float c = -((z + 128.0f) * s);
    const uint32_t v = (sz & 0xFFFFu) << shift;     // s in half (l & 1)
    const uint32_t b0 = v & keep_lo, b1 = v & ~keep_lo;
    MfmaDeq d;
    d.bdiag = __builtin_bit_cast(v4s, v2u{b0, b1});
    d.c4 = v4f{c, c, c, c};
    return d;
}

// Dequantize one packed word into the 8 bf16 A-operand values of
// v_mfma_f32_16x16x32_bf16 (row n = l & 15): elements e = 4h + i hold
// w[n][32j + 16h + 4(l >> 4) + i].
__device__ inline v8bf mfma_dequant(uint32_t P, const MfmaDeq &d) {
    const Pairs a = extract_pairs(P);
    const v4s A0 = __builtin_bit_cast(v4s, v2u{a.a0, a.a1});
    const v4s A1 = __builtin_bit_cast(v4s, v2u{a.a2, a.a3});
    const v4f d0 = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(A0, d.bdiag, d.c4, 0, 0, 0);
    const v4f d1 = __builtin_amdgcn_mfma_f32_4x4x4bf16_1k(A1, d.bdiag, d.c4, 0, 0, 0);
    const v4u w = {cvt_pk_bf16(d0[0], d0[1]), cvt_pk_bf16(d0[2], d0[3]),
                   cvt_pk_bf16(d1[0], d1[1]), cvt_pk_bf16(d1[2], d1[3])};
    return __builtin_bit_cast(v8bf, w);
}

// --- vector-ALU dequantization -------------------------------------------

// Constants for the four columns n = 16 t + 4 * ((l >> 2) & 3) + r of lane l.
struct ValuDeq { uint32_t sl[4], sh[4]; float c[4]; };

__device__ inline ValuDeq valu_setup(const uint32_t sz[4]) {
    ValuDeq d;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const float s = bf16_lo_to_f32(sz[r]);
        const float z = bf16_hi_to_f32(sz[r]);
        d.c[r] = -((z + 128.0f) * s);
        d.sl[r] = sz[r] & 0xFFFFu;   // bf16 pair (s, 0)
        d.sh[r] = sz[r] << 16;       // bf16 pair (0, s)
    }
    return d;
}

__device__ inline float dot2(uint32_t a, uint32_t b, float c) {
    return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(v2bf, a), __builtin_bit_cast(v2bf, b), c, false);
}

// Dequantize one packed word: pr[r] = bf16 pair (w[n_r][k0], w[n_r][k0 + 16]) with
// k0 = 32j + 4(l >> 4) + (l & 3).
__device__ inline void valu_dequant(uint32_t P, const ValuDeq &d, uint32_t pr[4]) {
    const Pairs a = extract_pairs(P);
    const float w00 = dot2(a.a0, d.sl[0], d.c[0]), w01 = dot2(a.a0, d.sh[1], d.c[1]);
    const float w02 = dot2(a.a1, d.sl[2], d.c[2]), w03 = dot2(a.a1, d.sh[3], d.c[3]);
    const float w10 = dot2(a.a2, d.sl[0], d.c[0]), w11 = dot2(a.a2, d.sh[1], d.c[1]);
    const float w12 = dot2(a.a3, d.sl[2], d.c[2]), w13 = dot2(a.a3, d.sh[3], d.c[3]);
    pr[0] = cvt_pk_bf16(w00, w10);
    pr[1] = cvt_pk_bf16(w01, w11);
    pr[2] = cvt_pk_bf16(w02, w12);
    pr[3] = cvt_pk_bf16(w03, w13);
}

// ------------------------------------------------------------------ repack

__global__ void k_repack_codes(const uint32_t *__restrict__ canon, uint32_t *__restrict__ out,
                               int K, int N) {
    const int Kb = K / kGroup, K8 = K / 8;
    const size_t total = (size_t)(N / kTileN) * Kb * kBlockU32;
    for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (size_t)gridDim.x * blockDim.x) {
        const size_t b = idx / kBlockU32;
        const int within = (int)(idx % kBlockU32);
        const int l = within >> 2, j = within & 3;
        const int t = (int)(b / Kb), kb = (int)(b % Kb);
        uint32_t word = 0;
        for (int p = 0; p < 8; ++p) {
            int n16, k128;
            block_coord(l, j, p, n16, k128);
            const int n = t * kTileN + n16, k = kb * kGroup + k128;
            const uint32_t src = canon[(size_t)n * K8 + (k >> 3)];
            word |= ((src >> (4 * (k & 7))) & 0xFu) << (4 * p);
        }
        out[idx] = word;
    }
}

__global__ void k_repack_sz(const uint16_t *__restrict__ scales, const uint16_t *__restrict__ zeros,
                            void *__restrict__ out, int K, int N, int symmetric) {
    const int Kb = K / kGroup;
    const size_t total = (size_t)N * Kb;
    for (size_t idx = (size_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total;
         idx += (size_t)gridDim.x * blockDim.x) {
        const int n16 = (int)(idx % kTileN);
        const size_t tb = idx / kTileN;               // t * Kb + kb
        const int kb = (int)(tb % Kb), t = (int)(tb / Kb);
        const size_t n = (size_t)t * kTileN + n16;
        const uint16_t s = scales[n * Kb + kb];
        if (symmetric) {
            ((uint16_t *)out)[idx] = s;
        } else {
            ((uint32_t *)out)[idx] = (uint32_t)s | ((uint32_t)zeros[n * Kb + kb] << 16);
        }
    }
}

// ------------------------------------------------------------------ test hooks

__global__ void k_unpack(const uint4 *__restrict__ codes, uint8_t *__restrict__ q, int K, int N) {
    const int Kb = K / kGroup;
    const size_t nblocks = (size_t)(N / kTileN) * Kb;
    const int l = threadIdx.x & 63;
    for (size_t b = (size_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); b < nblocks;
         b += (size_t)gridDim.x * (blockDim.x >> 6)) {
        const uint4 c = codes[b * 64 + l];
        const uint32_t w[4] = {c.x, c.y, c.z, c.w};
        const int t = (int)(b / Kb), kb = (int)(b % Kb);
        for (int j = 0; j < 4; ++j)
            for (int p = 0; p < 8; ++p) {
                int n16, k128;
                block_coord(l, j, p, n16, k128);
                q[(size_t)(t * kTileN + n16) * K + kb * kGroup + k128] = (uint8_t)((w[j] >> (4 * p)) & 0xFu);
            }
    }
}

template <bool SYM>
__global__ void k_dequant_mfma(const uint4 *__restrict__ codes, const void *__restrict__ sz,
                               uint16_t *__restrict__ w, int K, int N) {
    const int Kb = K / kGroup;
    const size_t nblocks = (size_t)(N / kTileN) * Kb;
    const int l = threadIdx.x & 63;
    const uint32_t shift = (l & 1) * 16, keep_lo = (l & 2) ? 0u : 0xFFFFFFFFu;
    for (size_t b = (size_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); b < nblocks;
         b += (size_t)gridDim.x * (blockDim.x >> 6)) {
        const uint4 c = codes[b * 64 + l];
        const MfmaDeq d = mfma_setup(load_sz<SYM>(sz, b * kTileN + (l & 15)), shift, keep_lo);
        const uint32_t P[4] = {c.x, c.y, c.z, c.w};
        const int t = (int)(b / Kb), kb = (int)(b % Kb);
        const size_t n = (size_t)t * kTileN + (l & 15);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const v4u v = __builtin_bit_cast(v4u, mfma_dequant(P[j], d));
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int k = kb * kGroup + 32 * j + 16 * (e >> 2) + 4 * (l >> 4) + (e & 3);
                w[n * K + k] = (uint16_t)(v[e >> 1] >> (16 * (e & 1)));
            }
        }
    }
}

template <bool SYM>
__global__ void k_dequant_valu(const uint4 *__restrict__ codes, const void *__restrict__ sz,
                               uint16_t *__restrict__ w, int K, int N) {
    const int Kb = K / kGroup;
    const size_t nblocks = (size_t)(N / kTileN) * Kb;
    const int l = threadIdx.x & 63;
    const int b2 = (l >> 2) & 3;
    for (size_t b = (size_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); b < nblocks;
         b += (size_t)gridDim.x * (blockDim.x >> 6)) {
        const uint4 c = codes[b * 64 + l];
        uint32_t s4[4];
        for (int r = 0; r < 4; ++r) s4[r] = load_sz<SYM>(sz, b * kTileN + 4 * b2 + r);
        const ValuDeq d = valu_setup(s4);
        const uint32_t P[4] = {c.x, c.y, c.z, c.w};
        const int t = (int)(b / Kb), kb = (int)(b % Kb);
        for (int j = 0; j < 4; ++j) {
            uint32_t pr[4];
            valu_dequant(P[j], d, pr);
            for (int r = 0; r < 4; ++r) {
                const size_t n = (size_t)t * kTileN + 4 * b2 + r;
                const int k0 = kb * kGroup + 32 * j + 4 * (l >> 4) + (l & 3);
                w[n * K + k0] = (uint16_t)(pr[r] & 0xFFFFu);
                w[n * K + k0 + 16] = (uint16_t)(pr[r] >> 16);
            }
        }
    }
}

// ------------------------------------------------------------------ forward

// Column range and K chunk of workgroup `bid`.
struct WgWork { int c, jn, t0, Tn, g0, Kc; };
__device__ inline WgWork wg_work(const FwdArgs &a, int bid) {
    WgWork w;
    w.c = bid / a.Gn;
    w.jn = bid - w.c * a.Gn;
    w.t0 = (int)(((long long)w.jn * a.Nt) / a.Gn);
    w.Tn = (int)(((long long)(w.jn + 1) * a.Nt) / a.Gn) - w.t0;
    w.g0 = (int)(((long long)w.c * a.Kb) / a.S);
    w.Kc = (int)(((long long)(w.c + 1) * a.Kb) / a.S) - w.g0;
    return w;
}

// Writes the workgroup's accumulated tiles: straight to y as bf16 when the
// whole K range was covered (S == 1); otherwise as fp32 partial sums, and
// the last of the S workgroups of this column range adds the S partials in
// chunk order (a fixed order, so results do not depend on arrival order),
// rounds once and writes y.
__device__ inline void write_out(const FwdArgs &a, const WgWork &w, const float *accs, int rows) {
    const int tid = threadIdx.x;
    const int items = w.Tn * a.M * 2;              // half rows of 8 columns
    const bool direct = (a.S == 1);
    for (int it = tid; it < items; it += blockDim.x) {
        const int tl = it / (a.M * 2);
        const int rem = it - tl * a.M * 2;
        const int m = rem >> 1, hh = rem & 1;
        const float *src = accs + ((size_t)tl * rows + m) * kAccPad + 8 * hh;
        const size_t n = (size_t)(w.t0 + tl) * kTileN + 8 * hh;
        if (direct) {
            uint4 o;
            o.x = cvt_pk_bf16(src[0], src[1]);
            o.y = cvt_pk_bf16(src[2], src[3]);
            o.z = cvt_pk_bf16(src[4], src[5]);
            o.w = cvt_pk_bf16(src[6], src[7]);
            *(uint4 *)(a.y + (size_t)m * a.N + n) = o;
        } else {
            float4 *dst = (float4 *)(a.ws + ((size_t)w.c * a.M + m) * a.N + n);
            dst[0] = make_float4(src[0], src[1], src[2], src[3]);
            dst[1] = make_float4(src[4], src[5], src[6], src[7]);
        }
    }
    if (direct) return;

    __shared__ int s_last;
    __threadfence();
    __syncthreads();
    if (tid == 0) {
        const uint32_t old = __hip_atomic_fetch_add(&a.counters[w.jn], 1u, __ATOMIC_ACQ_REL,
                                                    __HIP_MEMORY_SCOPE_AGENT);
        s_last = (old == (uint32_t)(a.S - 1));
    }
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    for (int it = tid; it < items; it += blockDim.x) {
        const int tl = it / (a.M * 2);
        const int rem = it - tl * a.M * 2;
        const int m = rem >> 1, hh = rem & 1;
        const size_t n = (size_t)(w.t0 + tl) * kTileN + 8 * hh;
        float s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (int cc = 0; cc < a.S; ++cc) {
            const float4 *src = (const float4 *)(a.ws + ((size_t)cc * a.M + m) * a.N + n);
            const float4 v0 = src[0], v1 = src[1];
            s[0] += v0.x; s[1] += v0.y; s[2] += v0.z; s[3] += v0.w;
            s[4] += v1.x; s[5] += v1.y; s[6] += v1.z; s[7] += v1.w;
        }
        uint4 o;
        o.x = cvt_pk_bf16(s[0], s[1]);
        o.y = cvt_pk_bf16(s[2], s[3]);
        o.z = cvt_pk_bf16(s[4], s[5]);
        o.w = cvt_pk_bf16(s[6], s[7]);
        *(uint4 *)(a.y + (size_t)m * a.N + n) = o;
    }
    if (tid == 0) __hip_atomic_store(&a.counters[w.jn], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

constexpr int kDepth = 4;   // 1 KiB blocks in flight per wave

// ---- SKINNY: matrix-core dequantization + v_mfma_f32_16x16x32_bf16 --------
//
// A workgroup owns K chunk c (groups [g0, g0 + Kc)) of column tiles
// [t0, t0 + Tn).  It stages x[:, chunk] in LDS once, in MFMA B-operand order,
// then its 8 waves split the Tn * Kc blocks evenly (tile-major order), each
// streaming its blocks with kDepth 128-bit loads in flight.  A wave adds its
// tile sums into LDS accumulators when it leaves a tile; the workgroup then
// writes y (or partials).
//
// x in LDS: 16-byte fragments F[kbl][g][j][row], row < 16 * MT; fragment
// (kbl, g, j, row) = x[row][k] for k = 128(g0 + kbl) + 32j + 16h + 4g + i,
// element 4h + i.  Lane l of m-tile mt reads fragment (kbl, l >> 4, j, 16 mt + (l & 15)).
template <int MT, bool SYM>
__global__ void __launch_bounds__(kThreads) k_skinny(FwdArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int MR = 16 * MT;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const WgWork w = wg_work(a, blockIdx.x);
    uint4 *xs = (uint4 *)smem;
    float *accs = (float *)(smem + (size_t)w.Kc * MR * 256);

    // stage x chunk (rows >= M are zero)
    {
        const int n8 = w.Kc * 16;
        for (int idx = tid; idx < MR * n8; idx += kThreads) {
            const int m = idx / n8, q8 = idx - m * n8;
            const int kbl = q8 >> 4, r8 = q8 & 15;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (m < a.M) v = *(const uint4 *)(a.x + (size_t)m * a.K + (size_t)(w.g0 + kbl) * kGroup + r8 * 8);
            const int j = r8 >> 2, p0 = (r8 & 3) * 2;
            uint2 *d0 = (uint2 *)&xs[((kbl * 4 + (p0 & 3)) * 4 + j) * MR + m] + (p0 >> 2);
            uint2 *d1 = (uint2 *)&xs[((kbl * 4 + ((p0 + 1) & 3)) * 4 + j) * MR + m] + ((p0 + 1) >> 2);
            *d0 = make_uint2(v.x, v.y);
            *d1 = make_uint2(v.z, v.w);
        }
        for (int idx = tid; idx < w.Tn * MR * kAccPad; idx += kThreads) accs[idx] = 0.0f;
    }
    __syncthreads();

    const int U = w.Tn * w.Kc;
    const int u0 = (int)(((long long)wave * U) / kWaves);
    const int u1 = (int)(((long long)(wave + 1) * U) / kWaves);
    const int lm = lane & 15, lg = lane >> 4;
    const uint32_t shift = (lane & 1) * 16, keep_lo = (lane & 2) ? 0u : 0xFFFFFFFFu;

    if (u0 < u1) {
        auto block_of = [&](int u) -> size_t {
            const int tl = u / w.Kc;
            return (size_t)(w.t0 + tl) * a.Kb + w.g0 + (u - tl * w.Kc);
        };
        uint4 cb[kDepth];
        uint32_t sb[kDepth];
#pragma unroll
        for (int d = 0; d < kDepth; ++d) {
            const size_t b = block_of(min(u0 + d, u1 - 1));
            cb[d] = a.codes[b * 64 + lane];
            sb[d] = load_sz<SYM>(a.sz, b * kTileN + lm);
        }
        v4f acc[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[mt] = v4f{0, 0, 0, 0};

        auto consume = [&](int u, const uint4 &cw, uint32_t szw) {
            const int tl = u / w.Kc, kbl = u - tl * w.Kc;
            v8bf xf[MT][4];
#pragma unroll
            for (int j = 0; j < 4; ++j)
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    xf[mt][j] = __builtin_bit_cast(v8bf, xs[((kbl * 4 + lg) * 4 + j) * MR + 16 * mt + lm]);
            const MfmaDeq d = mfma_setup(szw, shift, keep_lo);
            const uint32_t P[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const v8bf wa = mfma_dequant(P[j], d);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, xf[mt][j], acc[mt], 0, 0, 0);
            }
            if (kbl == w.Kc - 1 || u == u1 - 1) {
                // D of the 16x16 op: lane l holds rows n = 4(l >> 4) + v of column m = l & 15
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
                    for (int v = 0; v < 4; ++v)
                        atomicAdd(&accs[((size_t)tl * MR + 16 * mt + lm) * kAccPad + 4 * lg + v], acc[mt][v]);
                    acc[mt] = v4f{0, 0, 0, 0};
                }
            }
        };

        int u = u0;
        for (; u + kDepth <= u1; u += kDepth) {
#pragma unroll
            for (int d = 0; d < kDepth; ++d) {
                consume(u + d, cb[d], sb[d]);
                const size_t b = block_of(min(u + d + kDepth, u1 - 1));
                cb[d] = a.codes[b * 64 + lane];
                sb[d] = load_sz<SYM>(a.sz, b * kTileN + lm);
            }
        }
#pragma unroll
        for (int d = 0; d < kDepth; ++d)
            if (u + d < u1) consume(u + d, cb[d], sb[d]);
    }
    __syncthreads();
    write_out(a, w, accs, MR);
}

// ---- GEMV: vector-ALU dequantization + v_dot2_f32_bf16 --------------------
//
// Same work split as SKINNY.  x in LDS: for row m, group kbl and
// kk = 4g + i (g = l >> 4, i = l & 3), 16 bytes holding the bf16 pairs
// (x[m][k], x[m][k + 16]) with k = 128(g0 + kbl) + 32j + kk for j = 0..3.
template <int MV, bool SYM>
__global__ void __launch_bounds__(kThreads) k_gemv(FwdArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const WgWork w = wg_work(a, blockIdx.x);
    uint4 *xg = (uint4 *)smem;
    float *accs = (float *)(smem + (size_t)w.Kc * MV * 256);

    {
        uint16_t *xh = (uint16_t *)smem;
        const int n8 = w.Kc * 16;
        for (int idx = tid; idx < MV * n8; idx += kThreads) {
            const int m = idx / n8, q8 = idx - m * n8;
            const int kbl = q8 >> 4, r8 = q8 & 15;
            const uint4 v = *(const uint4 *)(a.x + (size_t)m * a.K + (size_t)(w.g0 + kbl) * kGroup + r8 * 8);
            const uint32_t vv[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int kg = r8 * 8 + e;                 // k within the group
                const int j = kg >> 5, k32 = kg & 31;
                const int hh = k32 >> 4, kk = k32 & 15;
                xh[((((size_t)m * w.Kc + kbl) * 16 + kk) * 4 + j) * 2 + hh] =
                    (uint16_t)(vv[e >> 1] >> (16 * (e & 1)));
            }
        }
        for (int idx = tid; idx < w.Tn * MV * kAccPad; idx += kThreads) accs[idx] = 0.0f;
    }
    __syncthreads();

    const int U = w.Tn * w.Kc;
    const int u0 = (int)(((long long)wave * U) / kWaves);
    const int u1 = (int)(((long long)(wave + 1) * U) / kWaves);
    const int b2 = (lane >> 2) & 3;
    const int kk = 4 * (lane >> 4) + (lane & 3);

    if (u0 < u1) {
        auto block_of = [&](int u) -> size_t {
            const int tl = u / w.Kc;
            return (size_t)(w.t0 + tl) * a.Kb + w.g0 + (u - tl * w.Kc);
        };
        auto load_sz4 = [&](size_t b, uint32_t s4[4]) {
            if constexpr (SYM) {
                const uint2 h = *(const uint2 *)((const uint16_t *)a.sz + b * kTileN + 4 * b2);
                s4[0] = (h.x & 0xFFFFu) | (0x4100u << 16);
                s4[1] = (h.x >> 16) | (0x4100u << 16);
                s4[2] = (h.y & 0xFFFFu) | (0x4100u << 16);
                s4[3] = (h.y >> 16) | (0x4100u << 16);
            } else {
                const uint4 q = *(const uint4 *)((const uint32_t *)a.sz + b * kTileN + 4 * b2);
                s4[0] = q.x; s4[1] = q.y; s4[2] = q.z; s4[3] = q.w;
            }
        };
        uint4 cb[kDepth];
        uint32_t sb[kDepth][4];
#pragma unroll
        for (int d = 0; d < kDepth; ++d) {
            const size_t b = block_of(min(u0 + d, u1 - 1));
            cb[d] = a.codes[b * 64 + lane];
            load_sz4(b, sb[d]);
        }
        float acc[MV][4];
#pragma unroll
        for (int m = 0; m < MV; ++m)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[m][r] = 0.0f;

        auto consume = [&](int u, const uint4 &cw, const uint32_t s4[4]) {
            const int tl = u / w.Kc, kbl = u - tl * w.Kc;
            uint4 xv[MV];
#pragma unroll
            for (int m = 0; m < MV; ++m) xv[m] = xg[((size_t)m * w.Kc + kbl) * 16 + kk];
            const ValuDeq d = valu_setup(s4);
            const uint32_t P[4] = {cw.x, cw.y, cw.z, cw.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                uint32_t pr[4];
                valu_dequant(P[j], d, pr);
#pragma unroll
                for (int m = 0; m < MV; ++m) {
                    const uint32_t xp = (j == 0) ? xv[m].x : (j == 1) ? xv[m].y : (j == 2) ? xv[m].z : xv[m].w;
#pragma unroll
                    for (int r = 0; r < 4; ++r) acc[m][r] = dot2(pr[r], xp, acc[m][r]);
                }
            }
            if (kbl == w.Kc - 1 || u == u1 - 1) {
                // sum over the 16 lanes sharing b2 (lane bits 0, 1, 4, 5)
#pragma unroll
                for (int m = 0; m < MV; ++m)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        float v = acc[m][r];
                        v += __shfl_xor(v, 1);
                        v += __shfl_xor(v, 2);
                        v += __shfl_xor(v, 16);
                        v += __shfl_xor(v, 32);
                        if ((lane & 0x33) == 0)
                            atomicAdd(&accs[((size_t)tl * MV + m) * kAccPad + 4 * b2 + r], v);
                        acc[m][r] = 0.0f;
                    }
            }
        };

        int u = u0;
        for (; u + kDepth <= u1; u += kDepth) {
#pragma unroll
            for (int d = 0; d < kDepth; ++d) {
                consume(u + d, cb[d], sb[d]);
                const size_t b = block_of(min(u + d + kDepth, u1 - 1));
                cb[d] = a.codes[b * 64 + lane];
                load_sz4(b, sb[d]);
            }
        }
#pragma unroll
        for (int d = 0; d < kDepth; ++d)
            if (u + d < u1) consume(u + d, cb[d], sb[d]);
    }
    __syncthreads();
    write_out(a, w, accs, MV);
}

// ------------------------------------------------------------------ host launchers

static inline int grid_for(size_t items, int per_block) {
    size_t g = (items + per_block - 1) / per_block;
    return (int)(g < 65536 ? (g ? g : 1) : 65536);
}

hipError_t launch_repack(const uint32_t *canon, const uint16_t *scales, const uint16_t *zeros,
                         uint4 *codes, void *sz, int K, int N, bool symmetric, hipStream_t st) {
    const size_t words = (size_t)N * K / 8;
    hipLaunchKernelGGL(k_repack_codes, dim3(grid_for(words, 256)), dim3(256), 0, st,
                       canon, (uint32_t *)codes, K, N);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const size_t ent = (size_t)N * (K / kGroup);
    hipLaunchKernelGGL(k_repack_sz, dim3(grid_for(ent, 256)), dim3(256), 0, st,
                       scales, zeros, sz, K, N, symmetric ? 1 : 0);
    return hipGetLastError();
}

hipError_t launch_unpack(const uint4 *codes, uint8_t *q, int K, int N, hipStream_t st) {
    const size_t nblocks = (size_t)(N / kTileN) * (K / kGroup);
    hipLaunchKernelGGL(k_unpack, dim3(grid_for(nblocks, 4)), dim3(256), 0, st, codes, q, K, N);
    return hipGetLastError();
}

hipError_t launch_dequant(int routine, const uint4 *codes, const void *sz, bool symmetric,
                          uint16_t *w, int K, int N, hipStream_t st) {
    const size_t nblocks = (size_t)(N / kTileN) * (K / kGroup);
    const dim3 g(grid_for(nblocks, 4)), b(256);
    if (routine == 0) {
        if (symmetric) hipLaunchKernelGGL(k_dequant_mfma<true>, g, b, 0, st, codes, sz, w, K, N);
        else hipLaunchKernelGGL(k_dequant_mfma<false>, g, b, 0, st, codes, sz, w, K, N);
    } else {
        if (symmetric) hipLaunchKernelGGL(k_dequant_valu<true>, g, b, 0, st, codes, sz, w, K, N);
        else hipLaunchKernelGGL(k_dequant_valu<false>, g, b, 0, st, codes, sz, w, K, N);
    }
    return hipGetLastError();
}

typedef void (*FwdKernel)(FwdArgs);

template <bool SYM>
static FwdKernel pick(int path, int mrows) {
    if (path == kSkinny) {
        switch (mrows) {
            case 16: return k_skinny<1, SYM>;
            case 32: return k_skinny<2, SYM>;
            case 48: return k_skinny<3, SYM>;
            case 64: return k_skinny<4, SYM>;
        }
    } else if (path == kGemv) {
        switch (mrows) {
            case 1: return k_gemv<1, SYM>;
            case 2: return k_gemv<2, SYM>;
            case 3: return k_gemv<3, SYM>;
            case 4: return k_gemv<4, SYM>;
            case 5: return k_gemv<5, SYM>;
            case 6: return k_gemv<6, SYM>;
            case 7: return k_gemv<7, SYM>;
            case 8: return k_gemv<8, SYM>;
        }
    }
    return nullptr;
}

static FwdKernel pick_kernel(int path, int mrows, bool symmetric) {
    return symmetric ? pick<true>(path, mrows) : pick<false>(path, mrows);
}

const char *kernel_name(int path, int mrows, bool symmetric) {
    static const char *sk[2][4] = {{"k_skinny<1>", "k_skinny<2>", "k_skinny<3>", "k_skinny<4>"},
                                   {"k_skinny<1,sym>", "k_skinny<2,sym>", "k_skinny<3,sym>", "k_skinny<4,sym>"}};
    static const char *gv[2][8] = {{"k_gemv<1>", "k_gemv<2>", "k_gemv<3>", "k_gemv<4>", "k_gemv<5>",
                                    "k_gemv<6>", "k_gemv<7>", "k_gemv<8>"},
                                   {"k_gemv<1,sym>", "k_gemv<2,sym>", "k_gemv<3,sym>", "k_gemv<4,sym>",
                                    "k_gemv<5,sym>", "k_gemv<6,sym>", "k_gemv<7,sym>", "k_gemv<8,sym>"}};
    if (path == kSkinny && mrows % 16 == 0 && mrows >= 16 && mrows <= 64) return sk[symmetric][mrows / 16 - 1];
    if (path == kGemv && mrows >= 1 && mrows <= 8) return gv[symmetric][mrows - 1];
    return "?";
}

hipError_t prepare_kernels() {
    for (int sym = 0; sym < 2; ++sym) {
        for (int mr = 16; mr <= 64; mr += 16) {
            hipError_t e = hipFuncSetAttribute((const void *)pick_kernel(kSkinny, mr, sym),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsMax);
            if (e != hipSuccess) return e;
        }
        for (int mv = 1; mv <= 8; ++mv) {
            hipError_t e = hipFuncSetAttribute((const void *)pick_kernel(kGemv, mv, sym),
                                               hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsMax);
            if (e != hipSuccess) return e;
        }
    }
    return hipSuccess;
}

hipError_t launch_forward(int path, int mrows, bool symmetric, int grid, size_t lds,
                          const FwdArgs &a, hipStream_t st) {
    FwdKernel k = pick_kernel(path, mrows, symmetric);
    if (!k) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k, dim3(grid), dim3(kThreads), lds, st, a);
    return hipGetLastError();
}

}  // namespace qlin
