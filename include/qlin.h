/*
 * qlin.h -- C ABI of the MI355X (gfx950) weight-only INT4 linear layer (W4A16).
 *
 * The operation (Kim, Lee, Kim, "Quantize the Target, Quantize the Drafter",
 * arXiv 2607.04244):
 *   Sec. 2.1  the served model keeps INT4 codes W_q with frozen per-group
 *             scales s; the dequantized weight is W = s (.) W_q and the model
 *             runs in the W4A16 format (4-bit weights, 16-bit activations).
 *   Sec. 3.2  the INT4 grid is dequantized into floating point: the matmul
 *             sees bf16 weights.
 *   Sec. 3.3  groups of 128 consecutive input features share one scale.
 *   Sec. 2.2, 3.2, 3.3  the target verifies, and the drafter proposes, one
 *             16-token block per speculative step, so the layer runs at small
 *             row counts M (16 per block, 1 for plain decode).
 *
 * Computed here, for every m < M, n < N:
 *   w[n][k]  = RNE_bf16( (q[n][k] - z[n][k/128]) * s[n][k/128] )
 *   y[m][n]  = RNE_bf16( sum_k x[m][k] * w[n][k] )      (fp32 accumulation)
 * with unsigned codes q in [0, 15] and zero-points z; the paper's symmetric
 * format is z = 8 (see qlin_create_symmetric).
 *
 * Conventions: all tensors are row-major and contiguous; bf16 values travel
 * as uint16_t bit patterns; every call returns a QLIN_* status except
 * qlin_create* (NULL on failure) and qlin_destroy.  Argument checks run
 * before any HIP call.  The library never aborts and never prints.  After a
 * failure, qlin_last_error() returns a message for the calling thread.
 */
#ifndef QLIN_H
#define QLIN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct qlin_s *qlin_t;   /* opaque; immutable after creation */

enum {
    QLIN_OK = 0,
    QLIN_ERR_INVALID = -1,      /* bad argument (size, NULL, aliasing, zero-point value) */
    QLIN_ERR_UNSUPPORTED = -2,  /* valid but outside this library (group != 128, N % 16, scale range, M) */
    QLIN_ERR_ALIGN = -3,        /* x or y not 16-byte aligned */
    QLIN_ERR_OOM = -4,          /* device allocation failed */
    QLIN_ERR_HIP = -5           /* a HIP runtime call or kernel launch failed */
};

/* Kernel paths for qlin_forward_path (qlin_forward picks one itself). */
enum {
    QLIN_PATH_AUTO = 0,
    QLIN_PATH_GEMV = 1,    /* vector-ALU dequantize + v_dot2 dot product, M <= 4 */
    QLIN_PATH_SKINNY = 2,  /* matrix-core dequantize + MFMA 16x16x32, x chunk staged in LDS, M <= 64 */
    QLIN_PATH_TILED = 3,   /* LDS-tiled MFMA GEMM for prefill-sized M */
    QLIN_PATH_REGS = 4     /* matrix-core dequantize + MFMA 16x16x32, x fragments in registers, M <= 16 */
};

/*
 * qlin_create -- build a handle for one linear layer (K inputs, N outputs).
 *
 *   packed_w  uint32 [N][K/8]; code of (n, k = 8j + i) is
 *             (packed_w[n*K/8 + j] >> 4i) & 0xF (lowest nibble = lowest k)
 *   scales    bf16 [N][K/group]; positive normal numbers in [2^-100, 2^100]
 *   zeros     bf16 [N][K/group]; integer values in [0, 15]
 *   group     must be 128 (Sec. 3.3)
 * Each of the three may be host memory or device memory of the current
 * device (such as qlin_quantize's output, written on the default stream or
 * complete); device scales and zero-points are copied to the host for the
 * checks.
 *
 * Constraints: K > 0, N > 0, K % 128 == 0, N % 16 == 0, K <= 65536,
 * N <= 1048576.  The call copies and re-lays-out the weights into device
 * memory owned by the handle on the current device and returns after that
 * work has finished, so the caller may free its buffers at once.
 * Errors: NULL with qlin_last_error() set (INVALID / UNSUPPORTED / OOM / HIP).
 * Not thread-safe with respect to other HIP work on the default stream.
 */
qlin_t qlin_create(int64_t K, int64_t N, int64_t group,
                   const uint32_t *packed_w, const uint16_t *scales,
                   const uint16_t *zeros);

/*
 * qlin_create_symmetric -- the paper's symmetric format (Sec. 2.1 "symmetric
 * per-group scales", Sec. 3.3 "group-wise symmetric INT4"): no zero-point
 * tensor; the signed code W_q in [-8, 7] is stored as the nibble W_q + 8, so
 * w = RNE_bf16((q - 8) * s).  Same arguments and rules as qlin_create.
 */
qlin_t qlin_create_symmetric(int64_t K, int64_t N, int64_t group,
                             const uint32_t *packed_w, const uint16_t *scales);

/*
 * qlin_quantize -- round bf16 weights onto a fixed quantization grid and pack
 * the codes (Sec. 2.1: at packing time the trained bf16 weights are rounded
 * back onto the grid of the frozen scales; Sec. 4: the round-to-nearest
 * quantizer of the drafter comparison):
 *   code[n][k] = clamp(rint(w[n][k] / s[n][k/128]) + z[n][k/128], 0, 15)
 * The quotient is a correctly rounded binary32 division, rint rounds to the
 * nearest integer with ties to even, and a NaN quotient gives z.
 *
 *   w       DEVICE bf16 [N][K], 16-byte aligned
 *   scales  DEVICE bf16 [N][K/group]; positive for a meaningful grid
 *   zeros   DEVICE bf16 [N][K/group] integers in [0, 15], or NULL for the
 *           symmetric format (z = 8)
 *   packed  DEVICE uint32 [N][K/8] output in qlin_create's layout, 4-byte
 *           aligned (16-byte aligned is written with 16-byte stores, faster),
 *           must not overlap w
 *   stream  hipStream_t; NULL = the default stream
 *
 * Shape rules as qlin_create.  Asynchronous.  Errors: INVALID (shape, NULL,
 * overlap), UNSUPPORTED (group, N % 16, limits), ALIGN, HIP.
 */
int qlin_quantize(int64_t K, int64_t N, int64_t group, const uint16_t *w, const uint16_t *scales,
                  const uint16_t *zeros, uint32_t *packed, void *stream);

/*
 * qlin_forward -- y[M][N] = x[M][K] . w^T as defined above (asynchronous).
 *
 *   x       DEVICE bf16 [M][K], 16-byte aligned, read-only
 *   y       DEVICE bf16 [M][N], 16-byte aligned, must not overlap x
 *   stream  hipStream_t to launch on; NULL = the default stream
 *
 * M = 0 is a no-op returning QLIN_OK.  0 < M <= 65536.  x and y must stay
 * valid until the stream's work completes.  The handle owns a workspace
 * sized for the plans of M <= 16 (the decode regime: one draft block), so one
 * handle must not run on two streams at the same time (different handles
 * are independent).  Larger M run with plans that fit that workspace; the
 * fastest plans for prefill-sized M take a caller workspace through
 * qlin_forward_group.  The device current at call time must be the handle's
 * device.
 * Errors: INVALID (NULL, M < 0, overlap, wrong device), UNSUPPORTED (M too
 * large), ALIGN, HIP.
 */
int qlin_forward(qlin_t h, int64_t M, const uint16_t *x, uint16_t *y, void *stream);

/*
 * qlin_forward_path -- qlin_forward with the kernel path and the number of
 * K-chunks (split_k; 0 = the planner's choice) forced, for tests and tuning.
 * Errors as qlin_forward, plus INVALID for an unknown path, split_k < 0 or
 * split_k > K/128, and UNSUPPORTED when the path cannot run this M
 * (GEMV: M <= 4; REGS: M <= 16; SKINNY: M <= 64) or the forced split does
 * not fit LDS or the handle's workspace.  The TILED path takes any M: rows
 * beyond M * K < 2^31 run as further launches.
 */
int qlin_forward_path(qlin_t h, int path, int64_t split_k, int64_t M,
                      const uint16_t *x, uint16_t *y, void *stream);

/*
 * qlin_plan -- describe, without launching, what qlin_forward_path would run
 * for (path, split_k, M): writes a NUL-terminated text such as
 * "path=skinny kernel=k_skinny<1,16> grid=256 block=512 split=1 ranges=256
 * lds=123904 launches=1" into buf (at most buflen bytes).  Returns QLIN_OK or an error as
 * qlin_forward_path.
 */
int qlin_plan(qlin_t h, int path, int64_t split_k, int64_t M, char *buf, int64_t buflen);

/*
 * qlin_forward_group -- y_i[M][N_i] = x[M][K] . w_i^T for the n handles hs[i]
 * that share the input x: one launch of the decode kernels covers all of
 * them (M <= 64), e.g. the q, k and v projections of a decoder layer, which
 * the target runs on every verification step (Sec. 2.2) and the drafter on
 * every drafting step (Sec. 2.3).  For M > 64 (or path TILED) one tiled
 * launch covers all members as well.  n = 1 is a forward of one handle with
 * a caller workspace.
 *
 *   n          1 <= n <= 8 handles, all with the same K, the same format
 *              (zero-points or symmetric) and on the current device
 *   path, split_k   as qlin_forward_path (QLIN_PATH_AUTO, 0: the planner's)
 *   x          DEVICE bf16 [M][K], 16-byte aligned
 *   ys         HOST array of n DEVICE pointers, ys[i] bf16 [M][N_i],
 *              16-byte aligned; no output may overlap x, another output or
 *              the workspace
 *   workspace  DEVICE memory of workspace_bytes (16-byte aligned), or NULL
 *              with 0 bytes.  It must be zero-filled before its first use;
 *              every call leaves it in a state the next call can use, so
 *              one workspace can serve any handles and plans in stream
 *              order (calls sharing one must not overlap in time).  The
 *              planner picks the fastest plan whose K split fits it;
 *              qlin_group_plan reports the size the unconstrained plan uses.
 *   stream     hipStream_t; NULL = the default stream
 * Asynchronous.  M = 0 is a no-op.
 * Errors: INVALID (n, NULL, overlaps, K / format / device mismatch, sizes),
 * UNSUPPORTED (as qlin_forward_path), ALIGN, HIP.
 */
int qlin_forward_group(int64_t n, const qlin_t *hs, int path, int64_t split_k, int64_t M, const uint16_t *x,
                       uint16_t *const *ys, void *workspace, int64_t workspace_bytes, void *stream);

/*
 * qlin_group_plan -- without launching: the plan qlin_forward_group would run
 * for (n, hs, path, split_k, M) with a workspace of workspace_bytes bytes
 * (< 0: no limit), as text in buf (see qlin_plan; buf may be NULL), and in
 * *workspace_needed (may be NULL) the workspace bytes that plan uses (0 when
 * it does not cut the K range).  With workspace_bytes < 0 that is the size
 * to allocate for the fastest plans.
 * Errors as qlin_forward_group's argument checks.
 */
int qlin_group_plan(int64_t n, const qlin_t *hs, int path, int64_t split_k, int64_t M, int64_t workspace_bytes,
                    int64_t *workspace_needed, char *buf, int64_t buflen);

/*
 * qlin_forward_group_noalloc -- qlin_forward_group without a workspace
 * argument and without any allocation, for callers that cannot allocate
 * device memory (code under HIP-graph capture, tight serving loops, hosts
 * that forbid allocation).  The K-split scratch comes from a static array of
 * the library on each device (16 MiB, held from the first handle created on
 * the device until the process ends); its arrival counters are cleared once
 * when that first handle is created, and every call leaves them at zero.
 *
 * Arguments and plan as qlin_forward_group with an unlimited workspace.  All
 * calls on one device share the array: calls that overlap in time on one
 * device (different streams, or threads) race and must not be issued.
 * Errors as qlin_forward_group, plus UNSUPPORTED when that plan needs more
 * scratch than the array holds (qlin_group_plan reports the need).
 */
int qlin_forward_group_noalloc(int64_t n, const qlin_t *hs, int path, int64_t split_k, int64_t M,
                               const uint16_t *x, uint16_t *const *ys, void *stream);

/* qlin_workspace_bytes -- device bytes of the handle's own workspace (0 when
 * its plans for M <= 16 never cut the K range). */
int qlin_workspace_bytes(qlin_t h, int64_t *bytes);

/* qlin_destroy -- free the handle and its device memory.  The runtime's free
 * waits for the device's outstanding work first, so a forward still in
 * flight completes; captured graphs that use the handle must not be replayed
 * afterwards.  NULL-safe. */
void qlin_destroy(qlin_t h);

/* qlin_last_error -- message of the calling thread's last failure ("" if none). */
const char *qlin_last_error(void);

/* qlin_last_status -- QLIN_* code of the calling thread's last call (QLIN_OK if it
 * succeeded); the way to learn why qlin_create* returned NULL. */
int qlin_last_status(void);

/*
 * Test hooks.  Both read the handle's device layout with the same device
 * routines the forward kernels use, so comparing them with the oracle
 * checks the layout and the dequantization bit by bit.
 *
 * qlin_unpack_codes: q_out DEVICE uint8 [N][K], codes in [0, 15].
 * qlin_dequantize:   w_out DEVICE bf16 [N][K]; routine 0 = the matrix-core
 *                    routine (SKINNY/TILED/REGS paths), 1 = the vector-ALU
 *                    routine (GEMV path).  Both must give identical bits.
 *                    The routine argument exists because the library has two
 *                    dequantization routes and each must be checked bit by
 *                    bit against the definition.
 * Outputs must be 16-byte aligned.  Asynchronous on stream.
 */
int qlin_unpack_codes(qlin_t h, uint8_t *q_out, void *stream);
int qlin_dequantize(qlin_t h, int routine, uint16_t *w_out, void *stream);

/* qlin_shape -- K and N of a handle (either pointer may be NULL). */
int qlin_shape(qlin_t h, int64_t *K, int64_t *N);

/*
 * qlin_stream_read -- measurement utility: the HBM read ceiling the layer is
 * compared with.  Reads `bytes` bytes at `buf` (DEVICE, 16-byte aligned,
 * bytes a multiple of 16) with 128-bit loads over `grid` workgroups of 512
 * threads (grid <= 0: 4 per CU), 8 loads in flight per thread, and XOR-folds
 * them; one uint32 per workgroup is written to `sink` (DEVICE, grid entries)
 * only in the practically impossible case that the fold equals 0x12345678, so
 * the traffic is reads only.  Asynchronous on stream.
 * Errors: INVALID (NULL, bytes <= 0 or not a multiple of 16), ALIGN, HIP.
 */
int qlin_stream_read(const void *buf, int64_t bytes, int grid, uint32_t *sink, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* QLIN_H */
