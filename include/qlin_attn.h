/*
 * qlin_attn.h -- C ABI of the drafter's block attention with a symmetric
 * sliding window, on MI355X (gfx950).  Part of libqlin.so; status codes,
 * qlin_last_error() and qlin_last_status() are those of qlin.h.
 *
 * The operation (Kim, Lee, Kim, arXiv 2607.04244):
 *   Sec. 2.2, 3.2  the block-diffusion drafter predicts a block of 16 tokens
 *                  from mask-token queries that attend bidirectionally;
 *   Sec. 2.3, 3.3  its attention is limited to a fixed window (1024 or 2048
 *                  tokens) that is symmetric around each query, applied only
 *                  inside the attention computation: the key/value cache
 *                  stays complete (no eviction), and a sequence no longer
 *                  than the window is attended in full.
 *
 * Computed here, with the nq block queries at the last nq cache positions
 * (query i at position p_i = T - nq + i), for every query head hq, query i
 * and dimension d < 128:
 *   kv       = hq / (Hq / Hkv)                        (grouped heads)
 *   visible  = { j < T : window == 0 or T <= window or |j - p_i| <= window / 2 }
 *   s_j      = q[hq][i] . k[kv][j] / sqrt(128)         (fp32)
 *   out[hq][i][d] = RNE_bf16( sum_{j visible} softmax_j(s) v[kv][j][d] )
 * The softmax is evaluated in fp32 with the weights rounded to bf16 once (the
 * operand of the matrix-core product) and normalised by the sum of those
 * rounded weights.
 *
 * Layouts (row-major, bf16 as uint16_t bit patterns, all DEVICE memory of the
 * current device, 16-byte aligned):
 *   q    [Hq][nq][128]
 *   k, v [Hkv][kv_stride][128]: token j of head kv at (kv * kv_stride + j) * 128;
 *        only tokens j < T are read (kv_stride >= T is the cache capacity)
 *   out  [Hq][nq][128], must not overlap q, k, v or the workspace
 */
#ifndef QLIN_ATTN_H
#define QLIN_ATTN_H

#include <stdint.h>

#include "qlin.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * qlin_swa_plan -- the work split qlin_swa_attention would use, without
 * launching anything.
 *
 *   Hq, Hkv    query and key/value heads: Hkv > 0, Hq a multiple of Hkv,
 *              Hq / Hkv <= 8
 *   head_dim   must be 128
 *   nq         block queries, 1 <= nq <= 16
 *   T          cached tokens including the block, nq <= T <= 2^28
 *   window     W >= 0; 0 = full attention (no window)
 *   splits     0 = the planner's choice, else the number of key ranges per
 *              key/value head (clamped to the number of 64-key tiles, at
 *              most 256)
 * Outputs (each may be NULL): *splits_out = the key ranges per key/value
 * head; *workspace_bytes = the device workspace qlin_swa_attention needs
 * (0 when one range suffices); buf = NUL-terminated text such as
 * "kernel=k_attn_split<1,4> keys=528 tiles=9 splits=9 grid=72 combine=1"
 * (at most buflen bytes; buf may be NULL).
 * Errors: INVALID (sizes out of range), UNSUPPORTED (head_dim != 128,
 * Hq / Hkv > 8), HIP (device query).
 */
int qlin_swa_plan(int64_t Hq, int64_t Hkv, int64_t head_dim, int64_t nq, int64_t T, int64_t window,
                  int64_t splits, int64_t *splits_out, int64_t *workspace_bytes, char *buf, int64_t buflen);

/*
 * qlin_swa_attention -- the block attention defined above (asynchronous).
 *
 *   kv_stride        tokens between consecutive key/value heads (>= T)
 *   workspace        DEVICE fp32 scratch of at least the workspace_bytes
 *                    qlin_swa_plan reports for the same sizes and splits
 *                    (may be NULL when that is 0), 16-byte aligned; its
 *                    contents need no initialisation and are overwritten
 *   stream           hipStream_t; NULL = the default stream
 * Other arguments as qlin_swa_plan and the layouts above.  The call is
 * deterministic: the same inputs give the same bits for a fixed split.
 * Calls sharing one workspace must be ordered on one stream.
 * Errors: INVALID (sizes, NULL, overlap, workspace too small),
 * UNSUPPORTED (as qlin_swa_plan), ALIGN, HIP.
 */
int qlin_swa_attention(int64_t Hq, int64_t Hkv, int64_t head_dim, int64_t nq, int64_t T, int64_t kv_stride,
                       int64_t window, int64_t splits, const uint16_t *q, const uint16_t *k, const uint16_t *v,
                       uint16_t *out, void *workspace, int64_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* QLIN_ATTN_H */
