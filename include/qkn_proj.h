/*
 * qkn_proj.h -- C ABI of libqkn, part 2: the column-parallel Q/K projection
 * with Phase A in its epilogue (AMD MI355X, gfx950).
 *
 * Under tensor parallelism the first projection of attention is split along
 * its output dimension (Sec. II-B of SwiftQK, arXiv 2608.09160): rank r holds
 * rows [r*d_local, (r+1)*d_local) of each weight W (a linear layer's
 * out x in layout) and computes its slice of the projected activations from
 * the full layer input x. Layerwise QK-Norm then needs, per token, the sum of
 * squares of that slice (Phase A, Sec. III-A, Alg. 1). This entry point forms
 * both in one pass over the projection's output tiles: the statistic is taken
 * while the tile is still on chip, so Phase B (the exchange and the factor)
 * and Phase C need no separate Phase A read (`qkn_apply` consumes them).
 *
 *   y[t, j]     = bf16( sum_k x[t, k] * W[j, k] )      fp32 accumulation,
 *                                                     one rounding to nearest even
 *   partials[t] = sum_j y[t, j]^2                      fp32, of the stored bf16 values
 *
 * Conventions are those of qkn.h (device pointers owned by the caller, bf16 as
 * uint16_t bits, asynchronous on `stream`, validation before any HIP call,
 * negative status codes, T == 0 a no-op).
 *
 * Summation tree of partials[t] (fixed; depends only on d_local): the columns
 * are taken in tiles of 128; within a tile, two fused-multiply-add chains in
 * ascending column order over columns [0, 64) and [64, 128) of the tile, added
 * (first + second); the tile sums are then added in ascending tile order.
 * Results are deterministic and independent of the launch shape; they are
 * not bit-identical to qkn_partial_sumsq of y, whose tree differs (both are
 * fp32 sums of the same squares).
 *
 * Decode-sized launches (T <= 1024, hidden >= 256) split k into 2^s contiguous
 * slices of ceil(hidden / 2^s) rounded up to a multiple of 8 (the last one
 * shorter), with 2^s the largest power of two <= 16 / ceil(T / 128) that
 * keeps slices at least 128 deep, computed by separate workgroups. Each slice's fp32 sum is
 * stored; a reduction adds the slices in ascending order, rounds once to bf16
 * and takes the statistic with the same tree as above. The slice count
 * depends only on T and hidden, so results are deterministic and Q and K in
 * one launch equal Q and K in two; y's last bit can differ from an unsplit
 * accumulation (fp32 sums in another order).
 */
#ifndef QKN_PROJ_H
#define QKN_PROJ_H

#include <stdint.h>

#include "qkn.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * One projection output (Q or K) of one rank.
 *   w        bf16 [d_local, ldw], the rank's rows of the weight; columns
 *            [0, hidden) are used; ldw >= hidden.
 *   y        bf16 [T, ldy] output, columns [0, d_local); ldy >= d_local.
 *   partials fp32 [T] output: the Phase A statistic of y's rows.
 *   d_local  rows of w = columns of y (>= 1).
 */
typedef struct qkn_proj_seg {
  const uint16_t* w;
  int64_t ldw;
  uint16_t* y;
  int64_t ldy;
  float* partials;
  int64_t d_local;
} qkn_proj_seg;

/*
 * Bytes of device workspace qkn_proj_partial needs for these segments, T
 * tokens and `hidden` input columns: the per-chunk statistics before they are
 * added in chunk order (4 * T * sum over segments of ceil(d_local / 128)),
 * or, on the split-k path, the per-slice fp32 sums (4 * splits * T * sum of
 * d_local). Returns a negative status for invalid arguments (segs NULL,
 * nseg not 1 or 2, T < 0, hidden < 1,
 * d_local < 1).
 */
int64_t qkn_proj_workspace_bytes(int64_t T, int64_t hidden, const qkn_proj_seg* segs, int nseg);

/*
 * Projection of the layer input x (bf16 [T, ldx], columns [0, hidden)) onto
 * 1 or 2 weight slices (Q and K of the same tokens) in one launch, each
 * output tile's Phase A statistic taken in the epilogue, then the tile
 * statistics added in a second, small launch (split-k: the slice sums, then
 * one reduction launch that also adds the statistics).
 *   workspace  device memory of at least qkn_proj_workspace_bytes(...) bytes,
 *              16-byte aligned; its contents on entry do not matter.
 * Requirements of the MFMA path (else QKN_ENOTSUP): x, every w and y 16-byte
 * aligned; hidden, ldx, ldw, ldy and d_local multiples of 8; T * ldx * 2 and
 * d_local * ldw * 2 below 2^31 bytes.
 * QKN_EINVAL: x NULL with T > 0, T < 0, hidden < 1, ldx < hidden, segs NULL,
 * nseg not 1 or 2, a segment with NULL w/y/partials, d_local < 1,
 * ldw < hidden, ldy < d_local, workspace NULL or smaller than required.
 * QKN_EOVERLAP: an output (y, partials, workspace) overlapping an input or
 * another output.
 */
int qkn_proj_partial(const uint16_t* x, int64_t ldx, int64_t T, int64_t hidden,
                     const qkn_proj_seg* segs, int nseg, void* workspace,
                     int64_t workspace_bytes, void* stream);

/*
 * Size of the fixed device workspace of qkn_proj_partial_noalloc: 32 MiB,
 * held on each GPU the entry point runs on from its first call there until
 * the process ends. It covers every decode-sized (split-k) launch of up to
 * 4096 output columns over Q and K together (the split workspace is at most
 * 4 * 2048 * columns bytes) and the chunk statistics of prefill launches up to
 * T * sum of ceil(d_local / 128) = 8 M.
 */
#define QKN_PROJ_SCRATCH_BYTES (INT64_C(32) << 20)

/*
 * For callers that cannot allocate device memory -- code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc: the same
 * computation, kernels and results (bit for bit) as qkn_proj_partial, with the
 * workspace taken from a fixed per-device array of QKN_PROJ_SCRATCH_BYTES
 * instead of an argument. It calls no allocator (no hipMalloc, no hipFree);
 * its first call on a device looks the array's address up once (a runtime
 * query, no allocation; code that captures a HIP graph makes that first call
 * before capturing). Every call on one GPU shares that GPU's array, which
 * keeps the last call's contents (no call needs it cleared: every workspace
 * byte a call's kernels read was written earlier by the same call's kernels,
 * in stream order); calls that overlap in time on
 * one GPU -- on different streams, or from different threads -- race on it
 * and must be ordered by the caller.
 * Status codes as qkn_proj_partial, and QKN_ENOTSUP when the launch needs more
 * than QKN_PROJ_SCRATCH_BYTES (qkn_proj_workspace_bytes tells how much).
 */
int qkn_proj_partial_noalloc(const uint16_t* x, int64_t ldx, int64_t T, int64_t hidden,
                             const qkn_proj_seg* segs, int nseg, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* QKN_PROJ_H */
