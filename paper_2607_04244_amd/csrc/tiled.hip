// Prefill-sized M: the tiled W4A16 GEMM kernel for CDNA4 (gfx950).
//
// Same layer as the decode kernels (Sec. 2.1, 3.2, 3.3 of arXiv 2607.04244):
// each weight is the exact (q - z) * s rounded once to bf16, y = x . w^T in
// fp32, rounded once to bf16.  This file is compiled on its own with
// matrix-core results kept in ordinary VGPRs (see build.py): the
// dequantizing 4x4x4 products feed vector instructions, and with results in
// accumulation registers every value would need a copy back.

#include "device_common.h"


namespace qlin {

// ---- TILED: prefill-sized M (GEMM), matrix-core dequantization ----------
//
// A workgroup of 4 WS waves computes a BM x BN = 16 MSW x 64 NT block of y:
// rows [BM im, BM im + BM), column tiles [4 NT j, 4 NT j + 4 NT) of one
// member of the launch (column block jn of all members is block j of the
// member that owns it).  Wave w
// owns all BM rows (MSW m-subtiles of 16) of the NW = NT / WS tiles NW w + t:
// each tile is dequantized once per workgroup and every dequantized operand
// feeds MSW matrix products.  With WS = 2 two waves share each SIMD, so the
// stalls of one (LDS reads, matrix-result latency, barriers) are covered by
// the other; each x fragment is then read from LDS by two waves.  Per group
// kb the workgroup stages the BM x 128 x-tile and its 4 NT weight blocks
// (plus their scales) in LDS with direct-to-LDS loads, kTiledStages groups
// deep, the loads spread over all its waves.  Dequantization (the
// matrix-core route) produces the A operand of v_mfma_f32_16x16x32_bf16
// directly.
//
// x tile in LDS: 16-byte chunk (row r, c) = x[row][128 kb + 8c .. + 8],
// c < 16, at slot 16 r + (c ^ (r & 15)): a wave's direct-to-LDS load fills 64
// consecutive slots (4 rows, each a permutation of one row's 256 bytes, so
// the global reads stay coalesced), and the operand reads (16 lanes = 16
// rows of one c) hit 16 distinct bank groups.
//
// Each XCD (block index mod 8) gets an equal share of the work items, a
// contiguous run in column-block-major order taken in dispatch order: the
// row blocks of a column block run on one XCD (two where a run boundary
// splits it), so the block's weights are fetched into that XCD's L2 once and
// reused, and no XCD gets a second round while others idle.  Rows >= M and
// tiles >= Nt load a clamped valid row or tile and are not written.
//
// With few output blocks (small M over a narrow layer) the K range is cut in
// S chunks: work item (block, chunk c) covers groups [g0, g0 + Kc) of its
// block and stores its fp32 partial block with agent-scope stores; the last
// of the S workgroups of a block to arrive (one relaxed atomic per workgroup,
// after its stores have completed) reads the S partials back and adds them
// in chunk order (a fixed order: repeated calls give identical bits), and
// writes y.  Partial block (block, c) sits at float
// offset (block S + c) BM BN, element (ms, tile, lane) at 4 ((ms 4 NT + tile)
// 64 + lane): one 16-byte access per lane and product.

template <bool SYM, int MSW, int NT, int WS, bool SPLIT>
__global__ void __launch_bounds__(kTiledWaves * WS * 64, MSW * NT <= 8 ? 2 : 1) k_tiled(TiledArgs a) {
    constexpr int kWavesWg = kTiledWaves * WS;
    constexpr int BM = 16 * MSW;
    constexpr int NW = NT / WS;                           // column tiles per wave
    constexpr int kTiles = kTiledWaves * NT;              // column tiles per workgroup
    constexpr int kXLoads = BM * 16 / (kWavesWg * 64);    // direct-to-LDS x loads per wave and group
    constexpr int kRowsPerWave = BM / kWavesWg;
    static_assert(kXLoads * kWavesWg * 64 == BM * 16 && NW * WS == NT, "tile shape does not split over the waves");
    __shared__ __align__(16) uint4 xs[kTiledStages][BM * 16];
    // the workgroup's weight blocks (1 KiB each) and their s|z words (64 per
    // tile: lane l of a load writes the word of column l & 15, the other 48
    // are copies), one buffer per pipeline stage
    __shared__ __align__(16) uint4 ws_codes[kTiledStages][kTiles * 64];
    __shared__ __align__(16) uint32_t ws_sz[kTiledStages][kTiles * 64];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const ExtractConsts kx;
    // block index -> (column block jn, row block im, K chunk c): XCD x (=
    // block index mod 8) takes an equal contiguous slice of the Gn Mt S work
    // items in column-block-major order, in dispatch order
    const int xcd = blockIdx.x & 7, q = blockIdx.x >> 3;
    const int nitem = a.Gn * a.Mt * (SPLIT ? a.S : 1), per = nitem >> 3, rem = nitem & 7;
    if (q >= per + (xcd < rem ? 1 : 0)) return;      // uniform: padding of the grid
    const int s0 = xcd * per + min(xcd, rem);        // the XCD's run of items
    int blk, c = 0, jn, im;
    if constexpr (SPLIT) {
        const int item = s0 + q;
        blk = item / a.S;                             // once per workgroup
        c = item - blk * a.S;
        jn = blk / a.Mt;                              // column block over all members
        im = blk - jn * a.Mt;
    } else {
        // the run's blocks (column blocks ja .. jb: rows r0 .. of ja, all of
        // the ones between, rows .. r1 of jb) are taken row block by row
        // block, so the workgroups running together on the XCD share their x
        // rows in its L2 as well as their weights
        const int last = s0 + per + (xcd < rem ? 1 : 0) - 1;
        const int ja = s0 / a.Mt, jb = last / a.Mt;
        const int r0 = s0 - ja * a.Mt, r1 = last - jb * a.Mt;
        if (ja == jb) {
            jn = ja;
            im = r0 + q;
        } else {
            const int mid = jb - ja - 1;
            auto before = [&](int i) { return i * mid + max(0, i - r0) + min(i, r1 + 1); };   // items in rows < i
            int lo = 0, hi = a.Mt - 1;                // the row holding the q-th item
            while (lo < hi) {
                const int md = (lo + hi + 1) >> 1;
                if (before(md) <= q) lo = md;
                else hi = md - 1;
            }
            im = lo;
            jn = (im >= r0 ? ja : ja + 1) + (q - before(im));
        }
        blk = jn * a.Mt + im;
    }
    // the member owning column block jn (every index of the argument arrays
    // static but one, see wg_work in kernels.hip) and its tiles [t0, t0 + 4 NT)
    int m = 0, gb = 0;
#pragma unroll
    for (int i = 1; i < kMaxMembers; ++i)
        if (jn >= a.gb0[i]) {
            m = i;
            gb = a.gb0[i];
        }
    const TiledMember &f = a.mem[m];
    const int Nt = f.Nt;
    const int g0 = SPLIT ? c * a.Kq + min(c, a.Kr) : 0;   // the chunk's groups [g0, g1]
    const int g1 = SPLIT ? g0 + a.Kq + (c < a.Kr ? 1 : 0) - 1 : a.Kb - 1;
    const int lm = lane & 15, lg = lane >> 4;
    const DiagSel dsel(lane);

    // All global reads are direct-to-LDS buffer loads issued through inline
    // assembly (load_lds_buf16 / load_lds_buf4): the compiler does not track
    // them, so the only waits are the explicit vmcnt below and the pipeline
    // keeps kTiledStages - 1 groups in flight across the barriers.  Each
    // load's per-lane offset is fixed for the whole K walk and the group
    // enters as a scalar offset, so issuing a load costs no vector
    // instruction; the LDS destinations are scalars too.
    //
    // x: load i of wave w fills rows kRowsPerWave w + 4 i + (lane >> 4), slot
    // position lane & 15, which holds chunk (lane & 15) ^ (row & 15) of that
    // row.  Byte offsets from x at group 0; the planner keeps M * K below
    // 2^31, so x spans less than 4 GiB.
    const __amdgpu_buffer_rsrc_t rx =
        __builtin_amdgcn_make_buffer_rsrc((void *)a.x, 0, (int)((uint32_t)a.M * (uint32_t)a.K * 2u), kRsrcFlags);
    uint32_t xv[kXLoads];
#pragma unroll
    for (int i = 0; i < kXLoads; ++i) {
        const int r = wave * kRowsPerWave + 4 * i + lg;
        const int row = min(im * BM + r, a.M - 1);
        xv[i] = ((uint32_t)row * (uint32_t)a.K + (uint32_t)(((lane & 15) ^ (r & 15)) * 8)) * 2u;
    }
    constexpr uint32_t kXStage = BM * 16 * 16, kXLoad = 4 * 16 * 16;   // LDS bytes per stage, per load
    const uint32_t lds_x = lds_addr(&xs[0][wave * kRowsPerWave * 16]);
    auto load_x = [&](int kb, int buf) {
#pragma unroll
        for (int i = 0; i < kXLoads; ++i)
            load_lds_buf16(rx, xv[i], (uint32_t)kb * (kGroup * 2), lds_x + (uint32_t)buf * kXStage + i * kXLoad);
    };
    // weights: wave w loads its own tiles NW w + u (clamped to the last
    // tile), through resources based at the workgroup's first tile (its
    // blocks span at most 16 Kb KiB); wv / sv = byte offsets of this lane's
    // part of block (tile, 0)
    const int t0 = (jn - gb) * kTiles, ntw = min(kTiles, Nt - t0);
    constexpr uint32_t kSzBlk = SYM ? kTileN * 2 : kTileN * 4;          // s|z bytes per block
    const __amdgpu_buffer_rsrc_t rc = __builtin_amdgcn_make_buffer_rsrc(
        (void *)(f.codes + (size_t)t0 * a.Kb * 64), 0, ntw * a.Kb * 1024, kRsrcFlags);
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void *)((const char *)f.sz + (size_t)t0 * a.Kb * kSzBlk), 0, ntw * a.Kb * (int)kSzBlk, kRsrcFlags);
    uint32_t wv[NW], sv[NW];
#pragma unroll
    for (int u = 0; u < NW; ++u) {
        const uint32_t tr = (uint32_t)(min(t0 + wave * NW + u, Nt - 1) - t0) * (uint32_t)a.Kb;   // block (tile, 0)
        wv[u] = tr * 1024u + lane * 16u;
        // 2-byte scales: one dword per lane covers columns 2i, 2i + 1 (read_w picks the half)
        sv[u] = tr * kSzBlk + (SYM ? (lane & 7) : lm) * 4u;
    }
    constexpr uint32_t kWStage = kTiles * 64 * 16, kSStage = kTiles * 64 * 4;
    const uint32_t lds_w = lds_addr(&ws_codes[0][wave * NW * 64]), lds_s = lds_addr(&ws_sz[0][wave * NW * 64]);
    auto load_w = [&](int kb, int buf) {
#pragma unroll
        for (int u = 0; u < NW; ++u) {
            load_lds_buf16(rc, wv[u], (uint32_t)kb * 1024u, lds_w + (uint32_t)buf * kWStage + u * 1024u);
            load_lds_buf4(rs, sv[u], (uint32_t)kb * kSzBlk, lds_s + (uint32_t)buf * kSStage + u * 256u);
        }
    };
    // this lane's code words and s|z word of the wave's tile t from LDS
    auto read_w = [&](int buf, uint4 (&cw)[NW], uint32_t (&sw)[NW]) {
#pragma unroll
        for (int t = 0; t < NW; ++t) {
            const int slot = (wave * NW + t) * 64;
            cw[t] = ws_codes[buf][slot + lane];
            if constexpr (SYM) {
                const uint32_t pair = ws_sz[buf][slot + (lm >> 1)];
                sw[t] = ((lm & 1) ? (pair >> 16) : (pair & 0xFFFFu)) | (kZcSymmetric << 16);
            } else {
                sw[t] = ws_sz[buf][slot + lm];
            }
        }
    };

    v4f acc[MSW][NW];
#pragma unroll
    for (int ms = 0; ms < MSW; ++ms)
#pragma unroll
        for (int t = 0; t < NW; ++t) acc[ms][t] = v4f{0, 0, 0, 0};

    // LDS slot of this lane's operand read: row 16 ms + lm, chunk 4 j + lg
    auto xslot = [&](int ms, int j) { return ms * 256 + lm * 16 + ((4 * j + lg) ^ lm); };

    auto compute = [&](int buf, const uint4 (&cw)[NW], const uint32_t (&sw)[NW]) {
        MfmaDeq d[NW];
#pragma unroll
        for (int t = 0; t < NW; ++t) d[t] = mfma_setup(sw[t], dsel);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            v8bf wa[NW];
#pragma unroll
            for (int t = 0; t < NW; ++t) {
                const uint32_t P = j == 0 ? cw[t].x : j == 1 ? cw[t].y : j == 2 ? cw[t].z : cw[t].w;
                wa[t] = mfma_dequant(P, d[t], kx);
            }
#pragma unroll
            for (int ms = 0; ms < MSW; ++ms) {
                const v8bf xf = __builtin_bit_cast(v8bf, xs[buf][xslot(ms, j)]);
#pragma unroll
                for (int t = 0; t < NW; ++t)
                    acc[ms][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa[t], xf, acc[ms][t], 0, 0, 0);
            }
        }
    };

    // Pipeline of kTiledStages LDS buffers: groups kb + 1 .. kb + S - 1 are
    // in flight (straight into LDS) while group kb is computed.  Each step
    // waits for group kb's loads (kIssued memory instructions per wave), then
    // one barrier both publishes group kb and shows that every wave is done
    // with the previous step's buffer, which the step refills with group
    // kb + S - 1 (past the last group the loads reload it into a buffer
    // nobody reads) before computing group kb.  A wave's weight blocks and
    // s|z words are its own loads, in LDS once its own wait is over: it reads
    // them before the barrier, which only the x tile (loaded by all the
    // waves) needs, so that LDS round trip overlaps the wait for the others.
    // For the two taller block shapes the wave also sends its next weight
    // loads before the barrier (measured faster for them, slower for 64 x
    // 128 blocks).
    constexpr int kIssued = kXLoads + 2 * NW;
    constexpr int S = kTiledStages;
    static_assert(S >= 2, "the pipeline needs two stages");
#pragma unroll
    for (int i = 0; i < S - 1; ++i) {
        load_x(min(g0 + i, g1), i);
        load_w(min(g0 + i, g1), i);
    }
    int buf = 0;
    for (int kb = g0; kb <= g1; ++kb) {
        asm volatile("s_waitcnt vmcnt(%0)" :: "n"((S - 2) * kIssued) : "memory");
        uint4 cw[NW];
        uint32_t sw[NW];
        read_w(buf, cw, sw);
        const int nb = buf == 0 ? S - 1 : buf - 1;             // (kb - g0 + S - 1) % S
        if constexpr (MSW >= 6) {
            // the wave's own blocks in nb were read (and waited for) in the
            // previous step: their refill can go out before the barrier
            load_w(min(kb + S - 1, g1), nb);
            lds_barrier();                    // group kb is in LDS for every wave; buffer nb is free
            load_x(min(kb + S - 1, g1), nb);
        } else {
            lds_barrier();
            load_x(min(kb + S - 1, g1), nb);
            load_w(min(kb + S - 1, g1), nb);
        }
        compute(buf, cw, sw);
        buf = buf == S - 1 ? 0 : buf + 1;
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");   // the reloads past the end

    if constexpr (SPLIT) {
        // partial block to the workspace, then the arrival count; the last
        // arrival of the block sums the S partials in chunk order
        constexpr int kBlkFloats = BM * 64 * NT;
        const __amdgpu_buffer_rsrc_t r = __builtin_amdgcn_make_buffer_rsrc(a.ws, 0, (int)a.ws_bytes, kRsrcFlags);
        auto part_off = [&](int cc, int ms, int t) {   // byte offset of this lane's 16 bytes
            return (uint32_t)(((size_t)blk * a.S + cc) * kBlkFloats * 4) +
                   (uint32_t)(((ms * kTiles + wave * NW + t) * 64 + lane) * 16);
        };
#pragma unroll
        for (int ms = 0; ms < MSW; ++ms)
#pragma unroll
            for (int t = 0; t < NW; ++t)
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, acc[ms][t]), r, part_off(c, ms, t), 0,
                                                       kSc1);
        __shared__ int s_last;
        asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
        __syncthreads();
        if (tid == 0) {
            const uint32_t old = __hip_atomic_fetch_add(&a.counters[blk], 1u, __ATOMIC_RELAXED,
                                                        __HIP_MEMORY_SCOPE_AGENT);
            s_last = (old == (uint32_t)(a.S - 1));
        }
        __syncthreads();
        if (!s_last) return;
        // kBatch chunks of all the lane's MSW NW products are loaded together
        // (one memory round trip per batch), then added in chunk order
        constexpr int kBatch = MSW * NW >= 32 ? 1 : 32 / (MSW * NW);
        v4f sum[MSW][NW];
#pragma unroll
        for (int ms = 0; ms < MSW; ++ms)
#pragma unroll
            for (int t = 0; t < NW; ++t) sum[ms][t] = v4f{0, 0, 0, 0};
        for (int c0 = 0; c0 < a.S; c0 += kBatch) {
            v4f v[kBatch][MSW][NW];
#pragma unroll
            for (int u = 0; u < kBatch; ++u) {
                const int cc = min(c0 + u, a.S - 1);      // unconditional load; extra ones are not added
#pragma unroll
                for (int ms = 0; ms < MSW; ++ms)
#pragma unroll
                    for (int t = 0; t < NW; ++t)
                        v[u][ms][t] = __builtin_bit_cast(
                            v4f, __builtin_amdgcn_raw_buffer_load_b128(r, part_off(cc, ms, t), 0, kSc1));
            }
#pragma unroll
            for (int u = 0; u < kBatch; ++u)
                if (c0 + u < a.S)
#pragma unroll
                    for (int ms = 0; ms < MSW; ++ms)
#pragma unroll
                        for (int t = 0; t < NW; ++t) sum[ms][t] += v[u][ms][t];
        }
#pragma unroll
        for (int ms = 0; ms < MSW; ++ms)
#pragma unroll
            for (int t = 0; t < NW; ++t) acc[ms][t] = sum[ms][t];
        if (tid == 0) __hip_atomic_store(&a.counters[blk], 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }

    // D of the 16x16 op: lane l holds rows n = 4 (l >> 4) + v of column m = l & 15
#pragma unroll
    for (int ms = 0; ms < MSW; ++ms) {
        const int row = im * BM + ms * 16 + lm;
        if (row >= a.M) continue;
#pragma unroll
        for (int t = 0; t < NW; ++t) {
            const int tt = t0 + wave * NW + t;
            if (tt >= Nt) continue;
            const v4f v = acc[ms][t];
            const uint2 o = make_uint2(cvt_pk_bf16(v[0], v[1]), cvt_pk_bf16(v[2], v[3]));
            *(uint2 *)(f.y + (size_t)row * f.N + (size_t)tt * kTileN + 4 * lg) = o;
        }
    }
}

template <bool SYM, bool SPLIT>
hipError_t launch_tiled_kernel(TiledShape sh, const TiledArgs &a, int grid, hipStream_t st) {
    const dim3 g(grid);
    const dim3 b(kTiledWaves * 64 * tiled_wsplit(sh));
    if (sh.msw == 8 && sh.nt == 4) hipLaunchKernelGGL((k_tiled<SYM, 8, 4, tiled_wsplit({8, 4}), SPLIT>), g, b, 0, st, a);
    else if (sh.msw == 4 && sh.nt == 2) hipLaunchKernelGGL((k_tiled<SYM, 4, 2, tiled_wsplit({4, 2}), SPLIT>), g, b, 0, st, a);
    else if (sh.msw == 6 && sh.nt == 4) hipLaunchKernelGGL((k_tiled<SYM, 6, 4, tiled_wsplit({6, 4}), SPLIT>), g, b, 0, st, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

// The whole-K kernel is a separate instantiation from the K-split one, so
// that the split's epilogue does not weigh on its register allocation.
template <bool SYM>
hipError_t launch_tiled_sym(TiledShape sh, const TiledArgs &a, int grid, hipStream_t st) {
    return a.S > 1 ? launch_tiled_kernel<SYM, true>(sh, a, grid, st) : launch_tiled_kernel<SYM, false>(sh, a, grid, st);
}

hipError_t launch_tiled(bool symmetric, TiledShape shape, const TiledArgs &a, int grid, hipStream_t st) {
    return symmetric ? launch_tiled_sym<true>(shape, a, grid, st) : launch_tiled_sym<false>(shape, a, grid, st);
}

}  // namespace qlin
