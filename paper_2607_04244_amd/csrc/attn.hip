// Drafter block attention with a symmetric sliding window (Sec. 2.3 and
// Sec. 3.3 of arXiv 2607.04244): the 16 mask-token queries of a draft block
// attend bidirectionally to the key/value cache, each restricted to the keys
// within half a window of its own position; the cache itself stays complete,
// and a cache no longer than the window is attended in full.
//
// Two kernels, flash-decoding style:
//   k_attn_split<HPW>  workgroup (key/value head h, split s): the G query
//       heads of h (one per wave; two per wave when G > 4) against the 64-key
//       tiles of split s.  Q, K and V arrive through direct-to-LDS loads, up
//       to three tiles ahead; K sits in XOR-swizzled 16-byte units (the MFMA
//       A-operand reads are free of bank conflicts) and each V tile is
//       transposed once, LDS to LDS, into key-contiguous rows (the A operand
//       of P.V).  S^T = K Q^T and O^T += V^T P^T run on
//       v_mfma_f32_16x16x32_bf16 with an online softmax in fp32.  With one
//       split the workgroup writes the bf16 output; otherwise it writes its
//       unnormalised partial output and (max, sum) per query row.
//   k_attn_combine     one workgroup per (query head, 16 dimensions):
//       folds the partials of every split in with a running maximum, in a
//       fixed order (deterministic).
//
// MFMA operand layouts (16x16x32 bf16, lane l, g = l >> 4, r = l & 15):
//   A: row r, k = 8 g + e;  B: column r, k = 8 g + e;  D: column r, rows 4 g + i.
// S^T tile kt (keys 16 kt + 4 g + i of the 64-key tile, query r) comes out in
// D layout; two such tiles are exactly the B operand of one P.V step over 32
// keys when the k index e of group g stands for key 4 g + e (e < 4) or
// 16 + 4 g + (e - 4) (e >= 4).  The transposed V rows in LDS store keys in
// that order, so no register shuffle is needed between the two products.
#include "attn_internal.h"
#include "device_common.h"

namespace qlin {

namespace {

constexpr int kTileUnits = kAttnTile * kAttnD / 8;   // 16-byte units of one K or V tile (1024)
constexpr int kQUnits = kAttnQ * kAttnD / 8;         // 16-byte units of one head's block queries (256)
constexpr int kSplitWaves = 2 * kAttnWaves;          // two waves per query head: one per 32-key half
constexpr int kTileLoads = 4;                        // direct-to-LDS loads per wave and tile (2 K + 2 V)
constexpr float kNegInf = -__builtin_huge_valf();

typedef short v4s_t __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4s_t lds_v4s;

// Cross-lane pair reductions without LDS (gfx950 v_permlane{16,32}_swap):
// swapping a register with itself returns, in every lane, the values of the
// lane pair {l, l ^ 16} (resp. {l, l ^ 32}) in the same order for both
// lanes, so both lanes of a pair compute identical results.
__device__ inline float pair16_max(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float pair32_max(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ inline float pair16_sum(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
__device__ inline float pair32_sum(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}
constexpr uint32_t kBf16OnePair = 0x3F803F80u;       // bf16 (1.0, 1.0)

// Transposing LDS read (ds_read_b64_tr_b16): within each group of 16 lanes,
// lane i receives element i & 3 of the 8-byte chunks addressed by lanes
// 4 j + (i >> 2), j = 0..3.
__device__ inline v4s_t lds_read_tr(const void *p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4s *)(const __attribute__((address_space(3))) void *)p);
}

// K and V tiles share one LDS layout: unit c (dimensions 8 c .. 8 c + 7) of
// key kk at 16-byte unit kk * 16 + (c ^ (kk & 15)).  The K reads of S^T
// (key 16 kt + r, unit 4 ks + g) and the transposing V reads of P.V hit
// distinct banks.
__device__ inline int tile_unit(int kk, int c) { return kk * 16 + (c ^ (kk & 15)); }

// Every global read of the split kernel is a direct-to-LDS load (untracked
// by the compiler, waited for explicitly).  The ring holds NS tiles: all NS
// are requested at the start, and each later tile as soon as its slot has
// been consumed, so NS - 1 tiles stream in while one is computed:
//   qs     the block queries of this workgroup's heads, 16 rows x 16 units,
//          unit c of row r at r * 16 + (c ^ r)
//   kring  K tiles, vring V tiles, both in the tile_unit layout
// Wave w takes query head w % 4 (and w % 4 + 4 when G > 4) and keys
// 32 (w / 4) .. + 31 of every tile; the two halves of a head are merged
// through LDS at the end.
template <int HPW, int NS>
__global__ __launch_bounds__(kSplitWaves * 64, 1) void k_attn_split(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) uint4 qs[HPW * kAttnWaves * kQUnits];
    __shared__ __attribute__((aligned(16))) uint4 ring[2][NS][kTileUnits];   // K tiles, V tiles
    uint4 (*kring)[kTileUnits] = ring[0];
    uint4 (*vring)[kTileUnits] = ring[1];

    const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
    const int g = lane >> 4, r = lane & 15;
    const int hw = wave & (kAttnWaves - 1), half = wave >> 2;
    // XCD-aware placement (workgroup b runs on XCD b % 8): with a multiple of
    // 8 key/value heads, every split of head h runs on XCD h % 8, so the
    // head's queries are fetched from HBM once and its partials stay in one L2
    int h, s;
    if ((a.Hkv & 7) == 0) {
        const int q8 = blockIdx.x >> 3, hb = q8 / a.S;
        h = (blockIdx.x & 7) + 8 * hb;
        s = q8 - hb * a.S;
    } else {
        h = blockIdx.x / a.S;
        s = blockIdx.x - h * a.S;
    }
    const int t0 = s * a.tps, t1 = min(t0 + a.tps, a.ntiles);
    const uint16_t *kh = a.k + (size_t)h * a.kv_stride;
    const uint16_t *vh = a.v + (size_t)h * a.kv_stride;

    bool has[HPW];
    int hq[HPW];
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
        const int gl = hw + kAttnWaves * hh;
        has[hh] = gl < a.G;
        hq[hh] = h * a.G + (has[hh] ? gl : 0);
    }

    // block queries (rows >= nq repeat row nq - 1; their results are discarded)
    if (half == 0) {
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) {
            if (!has[hh]) continue;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int u = j * 64 + lane, row = u >> 4, c = (u & 15) ^ row;
                const uint16_t *src = a.q + ((size_t)hq[hh] * a.nq + min(row, a.nq - 1)) * kAttnD + 8 * c;
                load_lds_x16(src, &qs[(hh * kAttnWaves + hw) * kQUnits + j * 64]);
            }
        }
    }

    auto issue = [&](int t) {
        const int st = t % NS;
        const int key0 = a.lo + t * kAttnTile;
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int u = (kSplitWaves * j + wave) * 64 + lane;
            const int kk = u >> 4, c = (u & 15) ^ (kk & 15), key = min(key0 + kk, a.hi - 1);
            load_lds_x16_nt(kh + (size_t)key * kAttnD + 8 * c, &kring[st][(kSplitWaves * j + wave) * 64]);
            load_lds_x16_nt(vh + (size_t)key * kAttnD + 8 * c, &vring[st][(kSplitWaves * j + wave) * 64]);
        }
    };
    for (int t = t0; t < min(t0 + NS, t1); ++t) issue(t);

    float m[HPW], l[HPW];
    v4f o[HPW][8];
    v8bf qf[HPW][4];
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
        m[hh] = kNegInf;
        l[hh] = 0.0f;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) o[hh][dt] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
    }

    // visibility of this lane's row: key j is visible iff j - vis_lo <= vis_span (unsigned)
    const int p = a.T - a.nq + r;
    const int vis_lo = a.half < 0 ? 0 : p - a.half;
    const int vis_hi = a.half < 0 ? a.hi - 1 : min(p + a.half, a.hi - 1);
    const uint32_t vis_span = (uint32_t)(vis_hi - vis_lo);
    // a tile is visible to every block row when it lies inside the smallest row window
    const int all_lo = a.half < 0 ? 0 : a.T - 1 - a.half;
    const int all_hi = a.half < 0 ? a.hi - 1 : min(a.T - a.nq + a.half, a.hi - 1);

    // transposing-read roles: lane (g, 4 j + q) addresses key 4 g + j (+ 16),
    // dimensions 4 q .. 4 q + 3 of a 16-dimension slice
    const int tj = r >> 2, tq = r & 3;

    for (int t = t0; t < t1; ++t) {
        const int st = t % NS;
        // this wave's loads of tile t (and the queries) are complete: the
        // tiles requested after t may still be in flight
        const int after = min(t1 - 1, t + NS - 1) - t;
        if (after >= 3) asm volatile("s_waitcnt vmcnt(%0)" :: "n"(3 * kTileLoads) : "memory");
        else if (after == 2) asm volatile("s_waitcnt vmcnt(%0)" :: "n"(2 * kTileLoads) : "memory");
        else if (after == 1) asm volatile("s_waitcnt vmcnt(%0)" :: "n"(kTileLoads) : "memory");
        else asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        lds_barrier();                 // tile t visible to all waves
        if (t == t0) {
#pragma unroll
            for (int hh = 0; hh < HPW; ++hh)
#pragma unroll
                for (int ks = 0; ks < 4; ++ks)
                    qf[hh][ks] = *(const v8bf *)&qs[(hh * kAttnWaves + hw) * kQUnits + r * 16 + ((4 * ks + g) ^ r)];
        }

        const int key0 = a.lo + t * kAttnTile;
        const int hk0 = key0 + 32 * half;                   // this wave's 32 keys
        const bool masked = hk0 < all_lo || hk0 + 31 > all_hi;
        const uint4 *kb = kring[st];
        const uint4 *vb = vring[st];
#pragma unroll
        for (int hh = 0; hh < HPW; ++hh) {
            if (!has[hh]) continue;                         // wave-uniform
            // S^T = K Q^T over two key tiles of 16
            v4f sc[2];
#pragma unroll
            for (int kt = 0; kt < 2; ++kt) {
                sc[kt] = v4f{0.0f, 0.0f, 0.0f, 0.0f};
                const int kk = 32 * half + 16 * kt + r;
#pragma unroll
                for (int ks = 0; ks < 4; ++ks) {
                    const v8bf kf = *(const v8bf *)&kb[tile_unit(kk, 4 * ks + g)];
                    sc[kt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf, qf[hh][ks], sc[kt], 0, 0, 0);
                }
            }
            if (masked) {
#pragma unroll
                for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                    for (int i = 0; i < 4; ++i) {
                        const int j = hk0 + 16 * kt + 4 * g + i;
                        sc[kt][i] = (uint32_t)(j - vis_lo) <= vis_span ? sc[kt][i] : kNegInf;
                    }
            }
            float mt = fmaxf(fmaxf(fmaxf(sc[0][0], sc[0][1]), fmaxf(sc[0][2], sc[0][3])),
                             fmaxf(fmaxf(sc[1][0], sc[1][1]), fmaxf(sc[1][2], sc[1][3])));
            mt = pair32_max(pair16_max(mt));
            const float mn = fmaxf(m[hh], mt);
            const float muc = (mn == kNegInf ? 0.0f : mn) * a.c;   // exponents are s c - m c
            if (__ballot(mn != m[hh])) {                    // some row maximum moved: rescale
                const float alpha = __builtin_amdgcn_exp2f(__builtin_fmaf(m[hh], a.c, -muc));
                l[hh] *= alpha;
#pragma unroll
                for (int dt = 0; dt < 8; ++dt) o[hh][dt] *= alpha;
                m[hh] = mn;
            }
            // weights in bf16 (the P.V operand); the row sum adds the same rounded values
            uint32_t pw[2][2];
            float ls = 0.0f;
#pragma unroll
            for (int kt = 0; kt < 2; ++kt)
#pragma unroll
                for (int i2 = 0; i2 < 2; ++i2) {
                    const float e0 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[kt][2 * i2], a.c, -muc));
                    const float e1 = __builtin_amdgcn_exp2f(__builtin_fmaf(sc[kt][2 * i2 + 1], a.c, -muc));
                    const uint32_t w = cvt_pk_bf16(e0, e1);
                    pw[kt][i2] = w;
                    ls = dot2(w, kBf16OnePair, ls);         // + both rounded weights
                }
            l[hh] += ls;
            // O^T += V^T P^T over this wave's 32 keys
            const v8bf pb = __builtin_bit_cast(v8bf, v4u{pw[0][0], pw[0][1], pw[1][0], pw[1][1]});
            const int kr0 = 32 * half + 4 * g + tj;           // keys of elements 0..3; +16 for 4..7
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) {
                const int c = 2 * dt + (tq >> 1), off = 8 * (tq & 1);
                const v4s_t lo4 = lds_read_tr((const char *)&vb[tile_unit(kr0, c)] + off);
                const v4s_t hi4 = lds_read_tr((const char *)&vb[tile_unit(kr0 + 16, c)] + off);
                const v8bf vf = __builtin_bit_cast(v8bf, __builtin_shufflevector(lo4, hi4, 0, 1, 2, 3, 4, 5, 6, 7));
                o[hh][dt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pb, o[hh][dt], 0, 0, 0);
            }
        }
        if (t + NS < t1) {
            lds_barrier();             // every wave is done with slot st
            issue(t + NS);
        }
    }

    // merge the two key halves of each head: the second wave hands (m, l, o)
    // to the first through LDS (the rings are free once every wave is past
    // its last tile)
    float *xs = (float *)&ring[0][0][0];
    constexpr int kXch = 64 * (2 + 32);                     // floats per (wave, head)
    static_assert(HPW * kAttnWaves * kXch * 4 <= (int)sizeof(ring), "exchange fits the rings");
    static_assert(NS <= 4, "wait counts cover at most three tiles in flight behind the current one");
    __syncthreads();
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
        if (!has[hh]) continue;
        float *xw = xs + (hh * kAttnWaves + hw) * kXch;
        if (half == 1) {
            xw[lane] = m[hh];
            xw[64 + lane] = l[hh];
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) *(v4f *)(xw + 128 + (dt * 64 + lane) * 4) = o[hh][dt];
        }
    }
    __syncthreads();
    if (half == 1) return;
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
        if (!has[hh]) continue;
        const float *xw = xs + (hh * kAttnWaves + hw) * kXch;
        const float m2 = xw[lane], l2 = xw[64 + lane];
        const float M = fmaxf(m[hh], m2);
        const float mu = M == kNegInf ? 0.0f : M;
        const float a1 = __builtin_amdgcn_exp2f((m[hh] - mu) * a.c), a2 = __builtin_amdgcn_exp2f((m2 - mu) * a.c);
        m[hh] = M;
        l[hh] = l[hh] * a1 + l2 * a2;
#pragma unroll
        for (int dt = 0; dt < 8; ++dt) o[hh][dt] = o[hh][dt] * a1 + *(const v4f *)(xw + 128 + (dt * 64 + lane) * 4) * a2;
    }

    // epilogue: lane holds O^T[d = 16 dt + 4 g + i][query r]
#pragma unroll
    for (int hh = 0; hh < HPW; ++hh) {
        if (!has[hh]) continue;
        const float lt = pair32_sum(pair16_sum(l[hh]));
        if (r >= a.nq) continue;
        const size_t row = (size_t)hq[hh] * a.nq + r;
        if (a.S == 1) {
            uint16_t *op = a.out + row * kAttnD + 4 * g;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) {
                uint2 w;
                w.x = cvt_pk_bf16(o[hh][dt][0] / lt, o[hh][dt][1] / lt);
                w.y = cvt_pk_bf16(o[hh][dt][2] / lt, o[hh][dt][3] / lt);
                *(uint2 *)(op + 16 * dt) = w;
            }
        } else {
            // partials of (head, split): 8 blocks (one per 16 dimensions) of
            // 16 rows x 16 fp32, so each store instruction fills 1 KiB
            const size_t hs = (size_t)hq[hh] * a.S + s;
            float *wp = a.ws_o + hs * 8 * 256 + r * 16 + 4 * g;
#pragma unroll
            for (int dt = 0; dt < 8; ++dt) *(v4f *)(wp + dt * 256) = o[hh][dt];
            if (g == 0) *(float2 *)(a.ws_ml + (hs * 16 + r) * 2) = make_float2(m[hh], lt);
        }
    }
}

// One workgroup of 4 waves per (query head, 16 dimensions).  Thread
// (g, r) of wave sg owns query row r, dimensions 16 dt + 4 g .. + 3, and
// splits s = sg, sg + 4, ...: it requests all of them at once, folds them in
// with a running maximum, and the four waves' results are merged in wave
// order through LDS, so the result does not depend on timing.
constexpr int kCombWaves = 4;
constexpr int kCombBatch = 8;      // splits per thread requested together

struct CombState { float m, l; float4 acc; };

__device__ inline void comb_fold(CombState &st, float m2, float l2, const float4 &v, float c) {
    const float M = fmaxf(st.m, m2);
    const float mu = M == kNegInf ? 0.0f : M;
    const float f1 = __builtin_amdgcn_exp2f((st.m - mu) * c), f2 = __builtin_amdgcn_exp2f((m2 - mu) * c);
    st.m = M;
    st.l = st.l * f1 + l2 * f2;
    st.acc.x = st.acc.x * f1 + v.x * f2;
    st.acc.y = st.acc.y * f1 + v.y * f2;
    st.acc.z = st.acc.z * f1 + v.z * f2;
    st.acc.w = st.acc.w * f1 + v.w * f2;
}

__global__ __launch_bounds__(kCombWaves * 64) void k_attn_combine(AttnArgs a) {
    __shared__ CombState xs[kCombWaves][64];
    // the same XCD placement as the split kernel: the workgroups of query
    // head hq run on the XCD that wrote its partials
    int hq, dt;
    if ((a.Hkv & 7) == 0) {
        const int rest = blockIdx.x >> 3, t2 = rest >> 3, kvl = t2 / a.G;
        dt = rest & 7;
        hq = ((blockIdx.x & 7) + 8 * kvl) * a.G + (t2 - kvl * a.G);
    } else {
        hq = blockIdx.x >> 3;
        dt = blockIdx.x & 7;
    }
    const int lane = threadIdx.x & 63, sg = threadIdx.x >> 6;
    const int r = lane & 15, g = lane >> 4;
    const float2 *ml = (const float2 *)a.ws_ml + (size_t)hq * a.S * 16 + r;          // + 16 s
    const float4 *po = (const float4 *)(a.ws_o + ((size_t)hq * a.S * 8 + dt) * 256 + r * 16 + 4 * g);   // + 512 s
    CombState st{kNegInf, 0.0f, make_float4(0.f, 0.f, 0.f, 0.f)};
    if (r < a.nq) {
        for (int s0 = sg; s0 < a.S; s0 += kCombWaves * kCombBatch) {
            float2 e[kCombBatch];
            float4 v[kCombBatch];
#pragma unroll
            for (int i = 0; i < kCombBatch; ++i) {
                const int si = s0 + kCombWaves * i;
                e[i] = si < a.S ? ml[(size_t)si * 16] : make_float2(kNegInf, 0.0f);
                v[i] = si < a.S ? po[(size_t)si * 512] : make_float4(0.f, 0.f, 0.f, 0.f);
            }
#pragma unroll
            for (int i = 0; i < kCombBatch; ++i) comb_fold(st, e[i].x, e[i].y, v[i], a.c);
        }
    }
    xs[sg][lane] = st;
    __syncthreads();
    if (sg != 0 || r >= a.nq) return;
#pragma unroll
    for (int w = 1; w < kCombWaves; ++w) {
        const CombState o = xs[w][lane];
        comb_fold(st, o.m, o.l, o.acc, a.c);
    }
    uint2 w;
    w.x = cvt_pk_bf16(st.acc.x / st.l, st.acc.y / st.l);
    w.y = cvt_pk_bf16(st.acc.z / st.l, st.acc.w / st.l);
    *(uint2 *)(a.out + ((size_t)hq * a.nq + r) * kAttnD + 16 * dt + 4 * g) = w;
}

}  // namespace

const char *attn_kernel_name(int G) { return G > kAttnWaves ? "k_attn_split<2,3>" : "k_attn_split<1,4>"; }

hipError_t launch_attn(const AttnArgs &a, hipStream_t st) {
    const dim3 block(kSplitWaves * 64);
    const dim3 grid((unsigned)(a.Hkv * a.S));
    // one head per wave: four tiles in flight (144 KiB of LDS); two heads: three (128 KiB)
    if (a.G > kAttnWaves) hipLaunchKernelGGL((k_attn_split<2, 3>), grid, block, 0, st, a);
    else hipLaunchKernelGGL((k_attn_split<1, 4>), grid, block, 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || a.S == 1) return e;
    hipLaunchKernelGGL(k_attn_combine, dim3((unsigned)(a.Hq * 8)), dim3(kCombWaves * 64), 0, st, a);
    return hipGetLastError();
}

}  // namespace qlin
