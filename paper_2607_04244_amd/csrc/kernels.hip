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
// starts at word (t * Kb + kb) * 256 (Kb = K / 128 groups): the K range of a
// column tile is one contiguous run of KiB blocks, so a wave that walks a
// tile's groups reads memory sequentially.  Lane l of a wave owns words
// [4l, 4l + 4) of a block (one 128-bit load); word j of lane l covers k in
// [32j, 32j + 32) of the group, and its nibble p holds the code of
//     n = 16 t + 4 * ((l >> 2) & 3) + r,   r  = 2 * (p & 1) + (p >> 2)
//     k = 128 kb + 32 j + 8 * (l >> 4) + 4 h + (l & 3),   h = (p >> 1) & 1.
// That is exactly the operand order of the dequantizing matrix op below, so
// no lane shuffle is needed between HBM and the MFMA, and each lane ends up
// with 8 consecutive k of one column: its x operand is one contiguous
// 16-byte piece of x.
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

#include "device_common.h"

#include <algorithm>
#include <cstdio>
#include <mutex>

namespace qlin {

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
        const int t = (int)(b / Kb), kb = (int)(b % Kb);     // block b = t * Kb + kb
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
        const size_t tb = idx / kTileN;               // block t * Kb + kb
        const int t = (int)(tb / Kb), kb = (int)(tb % Kb);
        const size_t n = (size_t)t * kTileN + n16;
        const uint16_t s = scales[n * Kb + kb];
        if (symmetric) {
            ((uint16_t *)out)[idx] = s;
        } else {
            // zc = -(128 + z): bf16 sign 1, exponent of 128, mantissa z (z integer in [0, 15])
            const uint32_t z = (uint32_t)__uint_as_float((uint32_t)zeros[n * Kb + kb] << 16);
            ((uint32_t *)out)[idx] = (uint32_t)s | ((0xC300u | z) << 16);
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
    const DiagSel dsel(l);
    const ExtractConsts kx;
    for (size_t b = (size_t)blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6); b < nblocks;
         b += (size_t)gridDim.x * (blockDim.x >> 6)) {
        const uint4 c = codes[b * 64 + l];
        const MfmaDeq d = mfma_setup(load_sz<SYM>(sz, b * kTileN + (l & 15)), dsel);
        const uint32_t P[4] = {c.x, c.y, c.z, c.w};
        const int t = (int)(b / Kb), kb = (int)(b % Kb);
        const size_t n = (size_t)t * kTileN + (l & 15);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const v4u v = __builtin_bit_cast(v4u, mfma_dequant(P[j], d, kx));
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int k = kb * kGroup + 32 * j + 8 * (l >> 4) + e;
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
    const ExtractConsts kx;
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
            valu_dequant(P[j], d, kx, pr);
            for (int r = 0; r < 4; ++r) {
                const size_t n = (size_t)t * kTileN + 4 * b2 + r;
                const int k0 = kb * kGroup + 32 * j + 8 * (l >> 4) + (l & 3);
                w[n * K + k0] = (uint16_t)(pr[r] & 0xFFFFu);
                w[n * K + k0 + 4] = (uint16_t)(pr[r] >> 16);
            }
        }
    }
}

// ------------------------------------------------------------------ forward

// Column range, member and K chunk of workgroup `bid`: chunk c, range jn
// (over all members), the member's tiles [t0, t0 + Tn) and groups
// [g0, g0 + Kc), and the member's weights and output.
struct WgWork {
    int c, jn, t0, Tn, g0, Kc;
    const uint4 *codes;
    const void *sz;
    uint16_t *y;
    int N;
};
// Everything here is wave-uniform scalar work at the start of the kernel:
// the arguments arrive in one batch of scalar loads (the range starts are one
// contiguous array, every index static, and the chunk needs no division),
// then the member's fields in one more.
__device__ inline WgWork wg_work(const FwdArgs &a, int bid) {
    WgWork w;
    // bid / Gn as a multiply-high by ceil(2^32 / Gn): exact because bid * Gn
    // stays below 2^32 (bid < 64 * 4096 workgroups, Gn <= 4096); for Gn = 1
    // the reciprocal is 0 and the chunk is bid itself
    w.c = (int)(__umulhi((uint32_t)bid, a.inv_gn) + (a.Gn == 1 ? (uint32_t)bid : 0u));
    w.jn = bid - w.c * a.Gn;
    int m = 0, g0 = 0;                        // the member owning range jn, its first range
#pragma unroll
    for (int i = 1; i < kMaxMembers; ++i)
        if (w.jn >= a.gn0[i]) {
            m = i;
            g0 = a.gn0[i];
        }
    // one scalar load of the member's fields at a computed offset (reading a
    // member at a fixed index as well would make the compiler copy the
    // whole argument block to scratch memory)
    const FwdMember &f = a.mem[m];
    w.codes = f.codes;
    w.sz = f.sz;
    w.y = f.y;
    w.N = f.N;
    const int j = w.jn - g0;
    w.t0 = j * f.Nq + min(j, f.Nr);
    w.Tn = f.Nq + (j < f.Nr ? 1 : 0);
    w.g0 = w.c * a.Kq + min(w.c, a.Kr);
    w.Kc = a.Kq + (w.c < a.Kr ? 1 : 0);
    return w;
}

// Range [u0, u1) of the U = Tn * Kc blocks (tile-major) that wave i of a
// workgroup handles: U / kWaves blocks each, one more for the first U % kWaves.
__device__ inline void wave_range(int U, int i, int &u0, int &u1) {
    const int q = U / kWaves, r = U % kWaves;    // kWaves is a power of two
    u0 = i * q + min(i, r);
    u1 = u0 + q + (i < r ? 1 : 0);
}

// Split-K partial sums travel between workgroups that may sit on different
// XCDs, whose L2 caches are not coherent with each other for ordinary
// accesses.  They are written and read with agent-scope (sc1) buffer
// accesses, which the hardware performs at the device coherence point; an
// agent-scope release/acquire fence instead would write back and invalidate
// the whole L2 of the XCD on every arrival.  Workgroup (c, jn) owns a
// contiguous region of TnMax * M * 16 fp32 at ((c * Gn + jn) * TnMax * M * 16),
// item it = (tile * M + m) * 2 + half at float offset 8 * it, so the 16-byte
// accesses of a wave are contiguous.

__device__ inline __amdgpu_buffer_rsrc_t ws_rsrc(const FwdArgs &a) {
    return __builtin_amdgcn_make_buffer_rsrc(a.ws, 0, (int)a.ws_bytes, kRsrcFlags);
}
__device__ inline uint32_t ws_region(const FwdArgs &a, int c, int jn) {      // byte offset
    return (uint32_t)((c * a.Gn + jn) * a.TnMax * a.M) * 64u;
}
// The four sums of quarter row `it` of the workgroup's output (row m,
// columns n .. n + 3): bf16 straight to y when the whole K range is covered,
// else fp32 partials to the workspace, quarter it at float offset 4 it of the
// region (half row h = (tile * M + m) * 2 + half is quarters 2h and 2h + 1).
__device__ inline void store_quarter(const FwdArgs &a, const WgWork &w, int it, int m, int n, const float s[4],
                                     bool direct) {
    if (direct) {
        *(uint2 *)(w.y + (size_t)m * w.N + n) = make_uint2(cvt_pk_bf16(s[0], s[1]), cvt_pk_bf16(s[2], s[3]));
    } else {
        const uint32_t off = ws_region(a, w.c, w.jn) + (uint32_t)it * 16u;
        __builtin_amdgcn_raw_buffer_store_b128(
            v4u{__float_as_uint(s[0]), __float_as_uint(s[1]), __float_as_uint(s[2]), __float_as_uint(s[3])},
            ws_rsrc(a), off, 0, kSc1);
    }
}

// The last of the S workgroups of a column range adds the S fp32 partials in
// chunk order (fixed order) and writes y.
__device__ inline void reduce_chunks(const FwdArgs &a, const WgWork &w) {
    const int tid = threadIdx.x;
    const int items = w.Tn * a.M * 2;
    // Every wave waits until its partial-sum stores have completed at the
    // device coherence point before the barrier; one relaxed atomic per
    // workgroup then counts the arrival.  The last arrival reads the other
    // workgroups' partials with agent-scope loads, which do not hit stale
    // cached copies.
    __shared__ int s_last;
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (tid == 0) {
        const uint32_t old = __hip_atomic_fetch_add(&a.counters[w.jn], 1u, __ATOMIC_RELAXED,
                                                    __HIP_MEMORY_SCOPE_AGENT);
        s_last = (old == (uint32_t)(a.S - 1));
    }
    __syncthreads();
    if (!s_last) return;
    const __amdgpu_buffer_rsrc_t r = ws_rsrc(a);
    const uint32_t inv_pt = 0xFFFFFFFFu / (uint32_t)(a.M * 2) + 1u;   // as in write_out()
    for (int it = tid; it < items; it += kThreads) {
        const int tl = (int)__umulhi((uint32_t)it, inv_pt);
        const int rem = it - tl * a.M * 2;
        const int m = rem >> 1, hh = rem & 1;
        const size_t n = (size_t)(w.t0 + tl) * kTileN + 8 * hh;
        // partials of kBatch chunks are loaded together (one memory round
        // trip per batch, not per chunk), then added in chunk order
        constexpr int kBatch = 8;
        float s[8] = {0, 0, 0, 0, 0, 0, 0, 0};
        for (int c0 = 0; c0 < a.S; c0 += kBatch) {
            v4u v[kBatch][2];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int cc = min(c0 + u, a.S - 1);      // unconditional load; extra ones are not added
                const uint32_t off = ws_region(a, cc, w.jn) + (uint32_t)it * 32u;
                v[u][0] = __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kSc1);
                v[u][1] = __builtin_amdgcn_raw_buffer_load_b128(r, off + 16, 0, kSc1);
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u)
                if (c0 + u < a.S)
#pragma unroll
                    for (int i = 0; i < 8; ++i) s[i] += __uint_as_float(v[u][i >> 2][i & 3]);
        }
        uint4 o;
        o.x = cvt_pk_bf16(s[0], s[1]);
        o.y = cvt_pk_bf16(s[2], s[3]);
        o.z = cvt_pk_bf16(s[4], s[5]);
        o.w = cvt_pk_bf16(s[6], s[7]);
        *(uint4 *)(w.y + (size_t)m * w.N + n) = o;
    }
    if (tid == 0) __hip_atomic_store(&a.counters[w.jn], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Writes the workgroup's results.  Each wave left one partial sum per column
// tile it touched in LDS slot (wave, tile), and zeros (from the kernel's start)
// in the slots of the tiles it did not touch; the tile's sum adds the slots of
// all waves in wave order.  With the whole K range covered (S == 1) the sum goes to y as
// bf16; otherwise it goes to the fp32 workspace, and the last of the S
// workgroups of this column range adds the S partials in chunk order and
// writes y.  Every sum runs in a fixed order, so results do not depend on
// timing: repeated calls give identical bits.
//
// The loop strides by the compile-time workgroup size: blockDim.x would be a
// scalar load of the dispatch's hidden arguments here, after the main loop,
// and that load misses the scalar cache and costs a memory round trip on the
// workgroup's critical path.
//
// An item's slot reads do not depend on each other: all kWaves of them are
// issued before the first add.  Adding the zero slots leaves a sum's bits
// unchanged (the sum starts at +0), so the result equals the sum of the
// touched slots alone, without a per-slot test.
__device__ inline void write_out(const FwdArgs &a, const WgWork &w, const float *slots, int rows) {
    const int tid = threadIdx.x;
    const int per_tile = a.M * 4;                  // items (quarter rows of 4 columns) per tile
    const int items = w.Tn * per_tile;
    const bool direct = (a.S == 1);
    // tile of an item: a multiply-high by ceil(2^32 / per_tile), exact since
    // items and per_tile stay below 2^16
    const uint32_t inv_pt = 0xFFFFFFFFu / (uint32_t)per_tile + 1u;
    for (int it = tid; it < items; it += kThreads) {
        const int tl = (int)__umulhi((uint32_t)it, inv_pt);
        const int rem = it - tl * per_tile;
        const int m = rem >> 2, qq = rem & 3;
        float4 v[kWaves];
#pragma unroll
        for (int i = 0; i < kWaves; ++i)
            v[i] = *(const float4 *)(slots + ((size_t)(i * w.Tn + tl) * rows + m) * 16 + 4 * qq);
        float s[4] = {0, 0, 0, 0};
#pragma unroll
        for (int i = 0; i < kWaves; ++i) {
            s[0] += v[i].x;
            s[1] += v[i].y;
            s[2] += v[i].z;
            s[3] += v[i].w;
        }
        store_quarter(a, w, it, m, (w.t0 + tl) * kTileN + 4 * qq, s, direct);
    }
    if (!direct) reduce_chunks(a, w);
}

// ---- SKINNY: matrix-core dequantization + v_mfma_f32_16x16x32_bf16 --------
//
// A workgroup owns K chunk c (groups [g0, g0 + Kc)) of column tiles
// [t0, t0 + Tn).  It stages x[:, chunk] in LDS once, in MFMA B-operand order,
// with direct-to-LDS loads (global_load_lds_dwordx4: no VGPR round trip, no
// LDS write instructions) while its first weight blocks are already in
// flight; its waves then split the Tn * Kc blocks evenly (tile-major order),
// each keeping kDepth 1 KiB blocks in flight.  A wave leaves one partial sum
// per tile it touches in its LDS slot for that tile (slots start at zero);
// write_out() adds the waves' slots in a fixed order.
//
// x in LDS: 16-byte fragments, fragment (row, q8) = x[row][k0 .. k0 + 8)
// with k0 = 128 g0 + 8 q8 (q8 = 16 kbl + c, c = 4j + g < 16), row-major at
// slot row * (n8 + 1) + q8, n8 = 16 Kc: each row is the chunk's 256 Kc
// contiguous bytes plus one 16-byte pad slot.  A direct-to-LDS load fills 64
// consecutive slots = one contiguous KiB of a row of x (coalesced); the pad
// shifts consecutive rows by 4 banks, so the operand reads (16 lanes = 16
// rows of one q8) hit distinct banks; and a lane's four reads of a block are
// one address plus immediate offsets (4 j slots).  XR = staged rows (the
// next power of two >= M for one m-tile, else 16 MT).  Lane l of m-tile mt
// reads row min(16 mt + (l & 15), M - 1); pad slots and rows >= M hold
// copies and are never read.
template <int MT, int XR, bool SYM>
__global__ void __launch_bounds__(kThreads) k_skinny(FwdArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    constexpr int MR = 16 * MT;
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: keeps the walk on the scalar unit
    const ExtractConsts kx;
    const WgWork w = wg_work(a, blockIdx.x);
    uint4 *xs = (uint4 *)smem;
    const int n8 = w.Kc * 16;                         // 16-byte chunks per row of the x chunk
    const int nslots = XR * (n8 + 1);
    const int nload = (nslots + 63) >> 6;             // direct-to-LDS loads of the workgroup
    float *slots = (float *)(smem + (size_t)nload * 1024);   // [kWaves][Tn][MR][16] partial sums

    const int U = w.Tn * w.Kc;
    int u0, u1;
    wave_range(U, wave, u0, u1);
    const int lm = lane & 15, lg = lane >> 4;
    const DiagSel dsel(lane);

    // 1) the x chunk, straight into LDS: load i fills slots [64 i, 64 i + 64)
    //    (the last one may run past the chunk into spare LDS).  The row of a
    //    slot is a quotient by the row pitch d = n8 + 1, taken as the high word
    //    of sl * ceil(2^32 / d): exact because sl and d stay below 2^16 (the
    //    staged chunk fits in LDS), and a generic 32-bit division would cost
    //    a dozen vector instructions per load.
    const uint32_t d = (uint32_t)n8 + 1u;
    const uint32_t inv_d = 0xFFFFFFFFu / d + 1u;
    const uint16_t *xg = a.x + (size_t)w.g0 * kGroup;
    for (int i = wave; i < nload; i += kWaves) {
        const uint32_t sl = (uint32_t)(i * 64 + lane);
        const uint32_t r = __umulhi(sl, inv_d);      // row; q8 == n8 is the pad slot
        const uint32_t q8 = min(sl - r * d, (uint32_t)n8 - 1u);
        const uint32_t row = min(r, (uint32_t)a.M - 1u);
        load_lds_x16(xg + (row * (uint32_t)a.K + q8 * 8u), xs + i * 64);
    }
    // 2) then the first weight blocks (younger than the x loads, so waiting
    //    for x below does not wait for them).  Block u of the workgroup's
    //    work (tile-major, u = tl Kc + kbl) is block base + u + tl (Kb - Kc)
    //    of the device layout, with tl = u / Kc taken as a multiply-high by
    //    ceil(2^32 / Kc) (exact: u and Kc stay below 2^16; Kc = 1, whose
    //    reciprocal needs 33 bits, is taken apart).  All of it is
    //    wave-uniform scalar arithmetic without branches.
    //    The loads go through buffer resources based at the workgroup's first
    //    block (its blocks span at most Tn Kb KiB, well inside the 32-bit
    //    range), so the block offset is a scalar operand of the load.
    //    Prefetches past the wave's last block (the last kDepth of the loop,
    //    or all of them for a wave with an empty range) are clamped to the
    //    wave's last block (block U - 1 of the workgroup for an empty range):
    //    every path issues the same loads, so the wait counts stay static, and
    //    these re-reads are never consumed.
    const bool kc1 = w.Kc == 1;
    const uint32_t inv_kc = kc1 ? 0u : 0xFFFFFFFFu / (uint32_t)w.Kc + 1u;
    const uint32_t kc1_mask = kc1 ? 0xFFFFFFFFu : 0u;       // selects u itself when Kc == 1, without a branch
    auto tile_of = [&](uint32_t u) { return __umulhi(u, inv_kc) + (u & kc1_mask); };
    const size_t base = (size_t)w.t0 * a.Kb + w.g0;
    const uint32_t skip = (uint32_t)(a.Kb - w.Kc);
    const uint32_t ulast = (uint32_t)(u0 < u1 ? u1 - 1 : min(u0, U - 1));
    constexpr int kSzBytes = SYM ? 2 : 4;
    const int span = w.Tn * a.Kb;                      // blocks from base to past the workgroup's last
    const __amdgpu_buffer_rsrc_t rcodes =
        __builtin_amdgcn_make_buffer_rsrc((void *)(w.codes + base * 64), 0, span * 1024, kRsrcFlags);
    const __amdgpu_buffer_rsrc_t rsz = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((const char *)w.sz + base * kTileN * kSzBytes), 0, span * kTileN * kSzBytes, kRsrcFlags);
    uint4 cb[kDepth];
    uint32_t sb[kDepth];
    auto fetch = [&](int d, uint32_t u) {
        u = min(u, ulast);
        const uint32_t rb = u + tile_of(u) * skip;                // block relative to base
        cb[d] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rcodes, lane * 16, rb * 1024, kWeightPolicy));
        if constexpr (SYM) {
            sb[d] = (uint32_t)__builtin_amdgcn_raw_buffer_load_b16(rsz, lm * 2, rb * (kTileN * 2), kWeightPolicy) |
                    (kZcSymmetric << 16);
        } else {
            sb[d] = __builtin_amdgcn_raw_buffer_load_b32(rsz, lm * 4, rb * (kTileN * 4), kWeightPolicy);
        }
    };
#pragma unroll
    for (int d = 0; d < kDepth; ++d) fetch(d, (uint32_t)(u0 + d));
    // the partial-sum slots start at zero (a wave writes only the slots of
    // the tiles it touches); the barrier below orders this before any write
    {
        const int nq = kWaves * w.Tn * MR * 4;     // 16-byte words
        for (int i = tid; i < nq; i += kThreads) ((float4 *)slots)[i] = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    }
    // 3) every wave's x loads have landed in LDS (only the weight prefetch,
    //    2 kDepth loads, may still be in flight)
    asm volatile("s_waitcnt vmcnt(%0)" :: "n"(2 * kDepth) : "memory");
    lds_barrier();

    // per-lane part of the operand read slot: q8 = 16 kbl + 4 j + lg, so the
    // slot is 16 kbl + 4 j + xoff[mt]
    int xoff[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) xoff[mt] = min(16 * mt + lm, a.M - 1) * (n8 + 1) + lg;

    if (u0 < u1) {
        v4f acc[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) acc[mt] = v4f{0, 0, 0, 0};

        auto consume = [&](uint32_t u, const uint4 &cq, uint32_t szw) {
            const uint32_t tl = tile_of(u);
            const uint32_t kbl = u - tl * (uint32_t)w.Kc;
            v8bf xf[MT][4];
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const uint4 *xb = xs + kbl * 16 + xoff[mt];
#pragma unroll
                for (int j = 0; j < 4; ++j) xf[mt][j] = __builtin_bit_cast(v8bf, xb[4 * j]);
            }
            const MfmaDeq d = mfma_setup(szw, dsel);
            const uint32_t P[4] = {cq.x, cq.y, cq.z, cq.w};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const v8bf wa = mfma_dequant(P[j], d, kx);
#pragma unroll
                for (int mt = 0; mt < MT; ++mt)
                    acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa, xf[mt][j], acc[mt], 0, 0, 0);
            }
            // the tile's run in this wave ends here (rare: kept off the
            // straight-line path)
            if (__builtin_expect(kbl == (uint32_t)w.Kc - 1u || u == (uint32_t)u1 - 1u, 0)) {
                // D of the 16x16 op: lane l holds rows n = 4(l >> 4) + v of column m = l & 15
#pragma unroll
                for (int mt = 0; mt < MT; ++mt) {
                    *(v4f *)(slots + ((size_t)(wave * w.Tn + tl) * MR + 16 * mt + lm) * 16 + 4 * lg) = acc[mt];
                    acc[mt] = v4f{0, 0, 0, 0};
                }
            }
        };

        int u = u0;
        for (; u + kDepth <= u1; u += kDepth) {
#pragma unroll
            for (int d = 0; d < kDepth; ++d) {
                consume((uint32_t)(u + d), cb[d], sb[d]);
                fetch(d, (uint32_t)(u + d + kDepth));
            }
        }
#pragma unroll
        for (int d = 0; d < kDepth; ++d)
            if (u + d < u1) consume((uint32_t)(u + d), cb[d], sb[d]);
    }
    lds_barrier();
    write_out(a, w, slots, MR);
}

// ---- register-resident kernels (M <= 16) -------------------------------
//
// A workgroup owns K chunk c (groups [g0, g0 + Kc)) of column tiles
// [t0, t0 + Tn), Tn <= kTnMax.  Its waves split the Tn * Kc blocks evenly in
// group-major order u = kbl * Tn + tl, so a wave covers only ~Kc / kWaves + 2
// groups and loads the x it needs straight into registers: no x staging in
// LDS and no barrier before the main loop.  Per group a wave loads every one
// of its tiles' blocks (contiguous KiB in the device layout) plus that
// group's x, one group ahead of the compute (group_ring with two buffers).
// Each wave keeps one accumulator per tile; at the end it writes them to its
// LDS slots and write_out_waves() adds the waves' slots in wave order.
//
// Out-of-range tiles of a wave's first and last group still load (a valid
// block of the group) so that the loads stay unconditional and the compiler
// can count them; they are not computed.

// Sum over the waves' slots (fixed order) and write y, or fp32 partials plus
// the last-arrival reduction when the K range is cut (S > 1).  Slot (wave, tl)
// holds rows x 16 fp32 (row-major, 16 columns).
template <int TN>
__device__ inline void write_out_waves(const FwdArgs &a, const WgWork &w, const float *slots, int rows) {
    const int tid = threadIdx.x;
    const int per_tile = a.M * 4;                  // items (quarter rows of 4 columns) per tile
    const int items = w.Tn * per_tile;
    const bool direct = (a.S == 1);
    const uint32_t inv_pt = 0xFFFFFFFFu / (uint32_t)per_tile + 1u;   // as in write_out()
    for (int it = tid; it < items; it += kThreads) {
        const int tl = (int)__umulhi((uint32_t)it, inv_pt);
        const int rem = it - tl * per_tile;
        const int m = rem >> 2, qq = rem & 3;
        float4 v[kWaves];
#pragma unroll
        for (int i = 0; i < kWaves; ++i)
            v[i] = *(const float4 *)(slots + (((size_t)i * TN + tl) * rows + m) * 16 + 4 * qq);
        float s[4] = {0, 0, 0, 0};
#pragma unroll
        for (int i = 0; i < kWaves; ++i) {
            s[0] += v[i].x;
            s[1] += v[i].y;
            s[2] += v[i].z;
            s[3] += v[i].w;
        }
        store_quarter(a, w, it, m, (w.t0 + tl) * kTileN + 4 * qq, s, direct);
    }
    if (!direct) reduce_chunks(a, w);
}

// Group buffers in flight per wave.  Deeper rings were measured slower for
// narrow column ranges: every group also reloads its x fragments (4 KiB per
// wave), so the vector-memory return path of the CU, not HBM latency, is
// what a deeper ring fills.
template <int TN>
constexpr int ring_groups() { return 2; }

// Runs groups [kg0, kg1] through a ring of NG group buffers.  Each buffer is
// refilled NG groups ahead right after its group is consumed.  The loads are
// unconditional (a group index past the end is clamped to the last group):
// a load on only some paths would leave the compiler unsure how many loads
// are younger than the one it waits for, and it would then drain every load
// in flight.  The clamped reloads of the last round are not computed.
template <int NG, typename Buf, typename Load, typename Compute>
__device__ inline void group_ring(int kg0, int kg1, Buf (&buf)[NG], Load load, Compute compute) {
#pragma unroll
    for (int i = 0; i < NG; ++i) load(buf[i], min(kg0 + i, kg1));
    int kb = kg0;
    for (; kb + NG <= kg1; kb += NG) {
#pragma unroll
        for (int i = 0; i < NG; ++i) {
            compute(buf[i], kb + i);
            load(buf[i], min(kb + i + NG, kg1));
        }
    }
#pragma unroll
    for (int i = 0; i < NG; ++i)
        if (kb + i <= kg1) compute(buf[i], kb + i);
}

// The wave's groups [kg0, kg1] and, in the first and last of them, the tile
// range [ta0, Tn) and [0, tb1).
struct WaveGroups {
    int kg0, kg1, ta0, tb1;
    __device__ inline void init(int u0, int u1, int Tn) {
        kg0 = u0 / Tn;                // scalar, once per wave
        kg1 = (u1 - 1) / Tn;
        ta0 = u0 - kg0 * Tn;
        tb1 = u1 - kg1 * Tn;
    }
    __device__ inline int ta(int kbl) const { return kbl == kg0 ? ta0 : 0; }
    __device__ inline int tb(int kbl, int Tn) const { return kbl == kg1 ? tb1 : Tn; }
};

template <int TN>
struct MfmaGroup {
    uint4 c[TN];
    uint32_t s[TN];
    v8bf x[4];
};

// x fragment of lane l for step j of group kb: row l & 15, k = 128 kb + 32 j + 8 (l >> 4).
// Lanes of rows >= M read row M - 1: in the 16x16 product those lanes only
// feed output columns >= M, which are never written.
__device__ inline v8bf load_xfrag(const FwdArgs &a, int kb, int j, int lane) {
    const int m = min(lane & 15, a.M - 1);
    return __builtin_bit_cast(v8bf, *(const uint4 *)(a.x + (size_t)m * a.K + (size_t)kb * kGroup + 32 * j +
                                                      8 * (lane >> 4)));
}

template <int TN, bool SYM>
__global__ void __launch_bounds__(kThreads) k_mfma16(FwdArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    float *slots = (float *)smem;                  // [kWaves][TN][16][16]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const ExtractConsts kx;
    const WgWork w = wg_work(a, blockIdx.x);
    const int Tn = w.Tn;
    int u0, u1;
    wave_range(Tn * w.Kc, wave, u0, u1);
    const int lm = lane & 15, lg = lane >> 4;
    const DiagSel dsel(lane);

    v4f acc[TN];
#pragma unroll
    for (int t = 0; t < TN; ++t) acc[t] = v4f{0, 0, 0, 0};

    if (u0 < u1) {
        WaveGroups wg;
        wg.init(u0, u1, Tn);
        auto load_group = [&](MfmaGroup<TN> &B, int kbl) {
            const int ta = wg.ta(kbl), tb = wg.tb(kbl, Tn);
            const size_t base = (size_t)w.t0 * a.Kb + w.g0 + kbl;
#pragma unroll
            for (int t = 0; t < TN; ++t) {
                const size_t b = base + (size_t)min(max(t, ta), tb - 1) * a.Kb;
                B.c[t] = load_block_nt(w.codes, b * 64 + lane);
                B.s[t] = load_sz_nt<SYM>(w.sz, b * kTileN + lm);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) B.x[j] = load_xfrag(a, w.g0 + kbl, j, lane);
        };
        auto compute_group = [&](const MfmaGroup<TN> &B, int kbl) {
            const int ta = wg.ta(kbl), tb = wg.tb(kbl, Tn);
#pragma unroll
            for (int t = 0; t < TN; ++t) {
                if (t >= ta && t < tb) {
                    const MfmaDeq d = mfma_setup(B.s[t], dsel);
                    const uint32_t P[4] = {B.c[t].x, B.c[t].y, B.c[t].z, B.c[t].w};
#pragma unroll
                    for (int j = 0; j < 4; ++j)
                        acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(mfma_dequant(P[j], d, kx), B.x[j], acc[t], 0,
                                                                         0, 0);
                }
            }
        };
        MfmaGroup<TN> ring[ring_groups<TN>()];
        group_ring(wg.kg0, wg.kg1, ring, load_group, compute_group);
    }
    // D of the 16x16 op: lane l holds rows n = 4(l >> 4) + v of column m = l & 15
#pragma unroll
    for (int t = 0; t < TN; ++t)
        if (t < Tn) *(v4f *)(slots + (((size_t)wave * TN + t) * 16 + lm) * 16 + 4 * lg) = acc[t];
    lds_barrier();
    write_out_waves<TN>(a, w, slots, 16);
}

// ---- GEMV: vector-ALU dequantization + v_dot2_f32_bf16 (M <= 4) ---------
//
// Same walk as k_mfma16.  Lane l (b2 = (l >> 2) & 3, g = l >> 4, i = l & 3)
// holds, for every row m and step j, the bf16 pair (x[m][k], x[m][k + 4]) with
// k = 128 kb + 32 j + 8 g + i, matching valu_dequant()'s weight pairs.
template <int MV, int TN>
struct GemvGroup {
    uint4 c[TN];
    uint4 s[TN];
    uint32_t x[MV][4];
};

template <int MV, int TN, bool SYM>
__global__ void __launch_bounds__(kThreads) k_gemv4(FwdArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    float *slots = (float *)smem;                  // [kWaves][TN][MV][16]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const ExtractConsts kx;
    const WgWork w = wg_work(a, blockIdx.x);
    const int Tn = w.Tn;
    int u0, u1;
    wave_range(Tn * w.Kc, wave, u0, u1);
    const int b2 = (lane >> 2) & 3, li = lane & 3, lg = lane >> 4;
    const uint32_t xsel = (li & 1) ? 0x07060302u : 0x05040100u;   // high or low halves

    float acc[TN][MV][4];
#pragma unroll
    for (int t = 0; t < TN; ++t)
#pragma unroll
        for (int m = 0; m < MV; ++m)
#pragma unroll
            for (int r = 0; r < 4; ++r) acc[t][m][r] = 0.0f;

    if (u0 < u1) {
        WaveGroups wg;
        wg.init(u0, u1, Tn);
        auto load_group = [&](GemvGroup<MV, TN> &B, int kbl) {
            const int ta = wg.ta(kbl), tb = wg.tb(kbl, Tn);
            const size_t base = (size_t)w.t0 * a.Kb + w.g0 + kbl;
#pragma unroll
            for (int t = 0; t < TN; ++t) {
                const size_t b = base + (size_t)min(max(t, ta), tb - 1) * a.Kb;
                B.c[t] = load_block_nt(w.codes, b * 64 + lane);
                if constexpr (SYM) {
                    const uint2 h = __builtin_bit_cast(uint2, __builtin_nontemporal_load((const v2u *)((const uint16_t *)w.sz + b * kTileN + 4 * b2)));
                    B.s[t] = make_uint4((h.x & 0xFFFFu) | (kZcSymmetric << 16), (h.x >> 16) | (kZcSymmetric << 16),
                                        (h.y & 0xFFFFu) | (kZcSymmetric << 16), (h.y >> 16) | (kZcSymmetric << 16));
                } else {
                    B.s[t] = __builtin_bit_cast(uint4, __builtin_nontemporal_load((const v4u *)((const uint32_t *)w.sz + b * kTileN + 4 * b2)));
                }
            }
#pragma unroll
            for (int m = 0; m < MV; ++m)
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const uint4 q = *(const uint4 *)(a.x + (size_t)m * a.K + (size_t)(w.g0 + kbl) * kGroup + 32 * j +
                                                     8 * lg);
                    const uint32_t lo = (li < 2) ? q.x : q.y, hi = (li < 2) ? q.z : q.w;
                    B.x[m][j] = __builtin_amdgcn_perm(hi, lo, xsel);
                }
        };
        auto compute_group = [&](const GemvGroup<MV, TN> &B, int kbl) {
            const int ta = wg.ta(kbl), tb = wg.tb(kbl, Tn);
#pragma unroll
            for (int t = 0; t < TN; ++t) {
                if (t >= ta && t < tb) {
                    const uint32_t s4[4] = {B.s[t].x, B.s[t].y, B.s[t].z, B.s[t].w};
                    const ValuDeq d = valu_setup(s4);
                    const uint32_t P[4] = {B.c[t].x, B.c[t].y, B.c[t].z, B.c[t].w};
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        uint32_t pr[4];
                        valu_dequant(P[j], d, kx, pr);
#pragma unroll
                        for (int m = 0; m < MV; ++m)
#pragma unroll
                            for (int r = 0; r < 4; ++r) acc[t][m][r] = dot2(pr[r], B.x[m][j], acc[t][m][r]);
                    }
                }
            }
        };
        GemvGroup<MV, TN> ring[ring_groups<TN>()];
        group_ring(wg.kg0, wg.kg1, ring, load_group, compute_group);
    }
    // sum over the 16 lanes sharing b2 (lane bits 0, 1, 4, 5), then one lane per b2 writes
#pragma unroll
    for (int t = 0; t < TN; ++t) {
        if (t < Tn) {
#pragma unroll
            for (int m = 0; m < MV; ++m) {
                float t4[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    float v = acc[t][m][r];
                    v += __shfl_xor(v, 1);
                    v += __shfl_xor(v, 2);
                    v += __shfl_xor(v, 16);
                    v += __shfl_xor(v, 32);
                    t4[r] = v;
                }
                if ((lane & 0x33) == 0)
                    *(float4 *)(slots + (((size_t)wave * TN + t) * MV + m) * 16 + 4 * b2) =
                        make_float4(t4[0], t4[1], t4[2], t4[3]);
            }
        }
    }
    lds_barrier();
    write_out_waves<TN>(a, w, slots, MV);
}

// ------------------------------------------------------------------ quantize + pack

// Fixed-grid round-to-nearest quantization of bf16 weights and packing into
// the canonical [N][K/8] words (Sec. 2.1: at packing time the trained bf16
// weights are rounded back onto the grid of the frozen scales; Sec. 4: the
// RTN quantizer):  code = clamp(rint(w / s) + z, 0, 15), quotient in binary32
// with a correctly rounded division, nearest integer with ties to even, a
// NaN quotient gives z; code k = 8j + i goes to bits [4i, 4i + 4) of word j.
//
// Exact route, any operands: the correctly rounded division per weight.
__device__ __forceinline__ uint32_t rtn_code_div(float b, float s, float z) {
    const float qf = __fdiv_rn(b, s);
    const float c = __builtin_rintf(qf) + z;
    return (uint32_t)(qf != qf ? z : fminf(fmaxf(c, 0.0f), 15.0f));
}

// Reciprocal route, for 2^-60 <= |s| <= 2^60 and |z| <= 64 (NaN z excluded),
// giving the same integer code as the exact route for every bf16 weight.
// With bf16 operands the exact quotient e = w / s is either a half-integer
// or at least 1/1020 away from every half-integer (w = mw 2^p, s = ms 2^t,
// mw and ms in [128, 255]: e - (k + 1/2) has numerator an integer, or a
// half-integer below 1/2, over 2 ms or 4 ms).  q = w * rcp(s) is within
// 2 ulp of e, the fma residual w - q s is then formed with one rounding,
// and q + residual * rcp(s) is within 2^-19 ulp of e before the fma's one
// rounding: q' is e itself when e is a half-integer (representable), and
// within an ulp of e, on the same side of every half-integer, otherwise;
// for |e| < 128 an ulp is below 2^-17, so rint(q') = rint(RN(e)).  For
// |e| >= 128 both roundings exceed 64 + 16 in magnitude with the sign of e,
// and the code clamps to the same end.  Clamping q to +-2^30 before the
// residual keeps an overflowed product (or an infinite weight) from turning
// into inf - inf; a NaN weight stays NaN through the residual.  The range
// keeps every product and residual that decides a code normal.
__device__ __forceinline__ uint32_t rtn_code_rcp(float b, float s, float r, float z) {
    const float q = fminf(fmaxf(b * r, -0x1p30f), 0x1p30f);
    const float qf = __builtin_fmaf(__builtin_fmaf(-q, s, b), r, q);
    const float c = __builtin_rintf(qf) + z;
    return (uint32_t)(qf != qf ? z : fminf(fmaxf(c, 0.0f), 15.0f));
}

// Four consecutive packed words per thread: four 16-byte weight loads (64
// contiguous bytes) and, when the output is 16-byte aligned, one 16-byte
// store.  Word j of row n is word n K/8 + j of the flat output, and since
// K/8 is a multiple of 16 the four words 4t .. 4t + 3 lie in one group,
// group t / 4 of the flat [N][K/128] scales: one scale, zero-point and
// reciprocal per thread.
template <bool SYM, bool V16>
__global__ __launch_bounds__(256) void k_quantize_pack(const uint4 *__restrict__ w,
                                                       const uint16_t *__restrict__ scales,
                                                       const uint16_t *__restrict__ zeros,
                                                       uint32_t *__restrict__ packed, size_t quads) {
    for (size_t t = (size_t)blockIdx.x * 256 + threadIdx.x; t < quads; t += (size_t)gridDim.x * 256) {
        uint4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) v[u] = w[4 * t + u];
        const float s = __uint_as_float((uint32_t)scales[t >> 2] << 16);
        const float z = SYM ? 8.0f : __uint_as_float((uint32_t)zeros[t >> 2] << 16);
        uint32_t word[4] = {0, 0, 0, 0};
        const float as = fabsf(s);
        if (as >= 0x1p-60f && as <= 0x1p60f && fabsf(z) <= 64.0f) {
            const float r = __builtin_amdgcn_rcpf(s);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const uint32_t half[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const uint32_t b = (i & 1) ? (half[i >> 1] & 0xFFFF0000u) : (half[i >> 1] << 16);
                    word[u] |= rtn_code_rcp(__uint_as_float(b), s, r, z) << (4 * i);
                }
            }
        } else {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const uint32_t half[4] = {v[u].x, v[u].y, v[u].z, v[u].w};
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    const uint32_t b = (i & 1) ? (half[i >> 1] & 0xFFFF0000u) : (half[i >> 1] << 16);
                    word[u] |= rtn_code_div(__uint_as_float(b), s, z) << (4 * i);
                }
            }
        }
        if (V16) {
            *(uint4 *)(packed + 4 * t) = make_uint4(word[0], word[1], word[2], word[3]);
        } else {
#pragma unroll
            for (int u = 0; u < 4; ++u) packed[4 * t + u] = word[u];
        }
    }
}

hipError_t launch_quantize(const uint16_t *w, const uint16_t *scales, const uint16_t *zeros, uint32_t *packed,
                           int K, int N, hipStream_t st) {
    const size_t quads = (size_t)N * (K / 32);
    const int grid = (int)std::min<size_t>((quads + 255) / 256, 65536);
    const bool v16 = ((uintptr_t)packed & 15) == 0;
    auto kern = zeros ? (v16 ? k_quantize_pack<false, true> : k_quantize_pack<false, false>)
                      : (v16 ? k_quantize_pack<true, true> : k_quantize_pack<true, false>);
    hipLaunchKernelGGL(kern, dim3(grid), dim3(256), 0, st, (const uint4 *)w, scales, zeros, packed, quads);
    return hipGetLastError();
}

// ------------------------------------------------------------------ measurement

// Stream-read ceiling: 8 independent 128-bit loads in flight per thread,
// XOR-folded; writes only if the fold hits an (in practice) impossible value.
__global__ void __launch_bounds__(512) k_stream_read(const uint4 *__restrict__ p, size_t n16,
                                                     uint32_t *__restrict__ sink) {
    constexpr int U = 8;
    const size_t stride = (size_t)gridDim.x * blockDim.x;
    size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t acc = 0;
    for (; i + (U - 1) * stride < n16; i += U * stride) {
        uint4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = p[i + u * stride];
#pragma unroll
        for (int u = 0; u < U; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
    }
    for (; i < n16; i += stride) {
        const uint4 v = p[i];
        acc ^= v.x ^ v.y ^ v.z ^ v.w;
    }
    if (acc == 0x12345678u) sink[blockIdx.x] = acc;
}

hipError_t launch_stream_read(const void *buf, size_t bytes, int grid, uint32_t *sink, hipStream_t st) {
    hipLaunchKernelGGL(k_stream_read, dim3(grid), dim3(512), 0, st, (const uint4 *)buf, bytes / 16, sink);
    return hipGetLastError();
}

// ------------------------------------------------------------------ static scratch

// The split-K scratch of qlin_forward_group_noalloc: arrival counters and
// partial sums in the layout of any workspace, in a file-scope device array
// that each device holds from the library's load until the process ends.
// Host code never passes `scratch` itself to a kernel (in host code the name
// stands for a host-side shadow, not a device address): it uses the address
// hipGetSymbolAddress returns for the current device.
static __device__ __align__(256) unsigned char scratch[kStaticScratchBytes];

namespace {
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};
}  // namespace

hipError_t static_scratch_setup(int device, hipStream_t st) {
    if (device < 0 || device >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_ptr[device]) return hipSuccess;
    void *ptr = nullptr;
    hipError_t e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
    if (e != hipSuccess) return e;
    // the arrival counters must start at zero (every launch leaves them so)
    if ((e = hipMemsetAsync(ptr, 0, kScratchCounterBytes, st)) != hipSuccess) return e;
    if ((e = hipStreamSynchronize(st)) != hipSuccess) return e;
    g_scratch_ptr[device] = ptr;
    return hipSuccess;
}

void *static_scratch(int device) {
    if (device < 0 || device >= kMaxDevices) return nullptr;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    return g_scratch_ptr[device];
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

template <int TN, bool SYM>
static FwdKernel pick_regs(int kern, int mrows) {
    if (kern == kKernMfma16) return k_mfma16<TN, SYM>;
    if constexpr (TN <= kTnMaxGemv) {
        switch (mrows) {
            case 1: return k_gemv4<1, TN, SYM>;
            case 2: return k_gemv4<2, TN, SYM>;
            case 3: return k_gemv4<3, TN, SYM>;
            case 4: return k_gemv4<4, TN, SYM>;
        }
    }
    return nullptr;
}

template <bool SYM>
static FwdKernel pick(int kern, int mrows, int tn) {
    if (kern == kKernStaged) {        // tn = staged rows XR
        switch (tn) {
            case 1: return k_skinny<1, 1, SYM>;
            case 2: return k_skinny<1, 2, SYM>;
            case 4: return k_skinny<1, 4, SYM>;
            case 8: return k_skinny<1, 8, SYM>;
            case 16: return k_skinny<1, 16, SYM>;
            case 32: return k_skinny<2, 32, SYM>;
            case 48: return k_skinny<3, 48, SYM>;
            case 64: return k_skinny<4, 64, SYM>;
        }
        return nullptr;
    }
    switch (tn) {
        case 1: return pick_regs<1, SYM>(kern, mrows);
        case 2: return pick_regs<2, SYM>(kern, mrows);
        case 3: return pick_regs<3, SYM>(kern, mrows);
        case 4: return pick_regs<4, SYM>(kern, mrows);
        case 5: return pick_regs<5, SYM>(kern, mrows);
        case 6: return pick_regs<6, SYM>(kern, mrows);
        case 7: return pick_regs<7, SYM>(kern, mrows);
        case 8: return pick_regs<8, SYM>(kern, mrows);
    }
    return nullptr;
}

static FwdKernel pick_kernel(int kern, int mrows, int tn, bool symmetric) {
    return symmetric ? pick<true>(kern, mrows, tn) : pick<false>(kern, mrows, tn);
}

const char *kernel_name(int kern, int mrows, int tn, bool symmetric) {
    static thread_local char buf[64];
    if (kern == kKernTiled) snprintf(buf, sizeof buf, "k_tiled<%d,%d%s>", mrows / 16, tn, symmetric ? ",sym" : "");
    else if (kern == kKernMfma16) snprintf(buf, sizeof buf, "k_mfma16<%d%s>", tn, symmetric ? ",sym" : "");
    else if (kern == kKernGemv) snprintf(buf, sizeof buf, "k_gemv4<%d,%d%s>", mrows, tn, symmetric ? ",sym" : "");
    else snprintf(buf, sizeof buf, "k_skinny<%d,%d%s>", mrows / 16, tn, symmetric ? ",sym" : "");
    return buf;
}

hipError_t prepare_kernels() {
    for (int sym = 0; sym < 2; ++sym) {
        for (int tn = 1; tn <= kTnMax; ++tn) {
            (void)hipFuncSetAttribute((const void *)pick_kernel(kKernMfma16, 16, tn, sym),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsMax);
            for (int mv = 1; tn <= kTnMaxGemv && mv <= kMaxGemvM; ++mv)
                (void)hipFuncSetAttribute((const void *)pick_kernel(kKernGemv, mv, tn, sym),
                                          hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsMax);
        }
        for (int xr : {1, 2, 4, 8, 16, 32, 48, 64})
            (void)hipFuncSetAttribute((const void *)pick_kernel(kKernStaged, 0, xr, sym),
                                      hipFuncAttributeMaxDynamicSharedMemorySize, (int)kLdsMax);
    }
    return hipSuccess;
}

hipError_t launch_forward(int kern, int mrows, int tn, bool symmetric, int grid, size_t lds,
                          const FwdArgs &a, hipStream_t st) {
    FwdKernel k = pick_kernel(kern, mrows, tn, symmetric);
    if (!k) return hipErrorInvalidValue;
    hipLaunchKernelGGL(k, dim3(grid), dim3(kThreads), lds, st, a);
    return hipGetLastError();
}

}  // namespace qlin
