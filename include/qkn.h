/*
 * qkn.h -- C ABI of libqkn: sharded layerwise QK-Norm on AMD MI355X (gfx950).
 *
 * Layerwise QK-Norm applies RMSNorm (Eq. 1, Sec. II-A of SwiftQK,
 * arXiv 2608.09160) to each token's full projected Q vector and, separately,
 * to its full projected K vector:
 *
 *     y = x / sqrt( (1/H) * sum_j x_j^2 + eps ) * gamma,     H = full width.
 *
 * Under tensor parallelism (Sec. II-B) rank r of tp holds a contiguous slice of
 * the hidden dimension. The method (Sec. III, Alg. 1) splits the norm into
 *   Phase A  the rank's partial sum of squares of its slice, in fp32;
 *   Phase B  the sum of all ranks' partials in ascending rank order, the factor
 *            1/sqrt(S/H_total + eps), and -- independent of it -- x * gamma;
 *   Phase C  the scaled shard, the only output written.
 * This library computes one rank's share on one GPU. The other ranks' partials
 * are inputs: device memory that the caller filled (in a real deployment they
 * would arrive over the interconnect).
 *
 * Conventions for every entry point
 *   - bf16 tensors are passed as uint16_t bit patterns, FP8-E4M3 tensors (the
 *     *_fp8 entry points) as uint8_t bit patterns; fp32 as float.
 *   - Every pointer is DEVICE memory, owned by the caller. The library never
 *     allocates or frees device memory and keeps no pointer after returning.
 *   - A row-major tensor [T, ld] uses columns [0, d_local) of each row;
 *     ld is in elements and must be >= d_local.
 *   - `stream` is a hipStream_t passed as void*; NULL is the null stream.
 *     Calls are asynchronous on that stream and never synchronise the host.
 *   - Arguments are validated before any HIP call, so an invalid call fails
 *     without touching the GPU. T == 0 is a valid no-op (nothing launched).
 *   - Errors are returned as negative status codes; nothing aborts and no C++
 *     exception crosses the ABI. Faults during kernel execution surface, as
 *     usual for HIP, at the caller's next synchronisation.
 *   - Arithmetic: inputs are widened exactly, all sums and products are fp32
 *     (Sec. IV-C: fp32 accumulation for bf16 and FP8-E4M3 activations), and
 *     the output is rounded once to the input's format (nearest, ties to
 *     even). The factor 1/sqrt(S/d_full + eps) is evaluated as the hardware
 *     reciprocal square root (within 1 ulp) of fma(S, 1/d_full, eps), with
 *     1/d_full rounded to fp32 once: within a few fp32 ulps of the exact
 *     factor. NaN and infinities propagate by IEEE rules (eps = 0 with an
 *     all-zero row gives NaN).
 *   - Determinism: a row's partial sum depends only on d_local and the row's
 *     values (one fixed fp32 summation tree), never on the launch shape or the
 *     entry point, so every rank combines bit-identical statistics.
 *   - Fast paths: 128-bit accesses when x, y and w are 16-byte aligned and ld
 *     and d_local are multiples of 8 (bf16) or 16 (fp8), with tp <= 64: rows
 *     held in registers up to d_local = 4096, wider rows with gamma in LDS up
 *     to 16384 columns over both tensors together; otherwise a general path
 *     gives the same bits, more slowly. Alignment is never an error.
 */
#ifndef QKN_H
#define QKN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define QKN_OK 0
#define QKN_EINVAL (-1)   /* bad argument: NULL required pointer, bad size, tp/rank, eps */
#define QKN_EOVERLAP (-2) /* an output overlaps an input or another output in part */
#define QKN_EHIP (-3)     /* the HIP runtime refused a query or a launch */
#define QKN_ENOTSUP (-4)  /* shape/alignment outside what this entry point supports */
#define QKN_EDRYRUN (-5)  /* "validate_only" is set on the calling thread: the arguments
                             were accepted and a kernel chosen, but nothing was launched */

/*
 * One tensor (Q or K) of one rank.
 *   x        bf16 [T, ldx], the rank's slice; columns [0, d_local) are used.
 *   w        fp32 [d_local], the rank's slice of gamma.
 *   partials fp32 [tp * T], rank-major: element k*T + t is rank k's partial
 *            sum of squares of token t (the per-rank statistic exchanged in
 *            Sec. III-A; a buffer slot per rank and token as in Alg. 1).
 *            The fused call writes slot `rank` and reads every other slot.
 *   y        bf16 [T, ldy] output; y == x with ldy == ldx runs in place
 *            (Alg. 1 overwrites the local input); any other overlap with an
 *            input is QKN_EOVERLAP.
 *   inv_rms  optional fp32 [T]: receives 1/sqrt(S/d_full + eps). NULL skips.
 *   d_local  width of the slice (>= 1).
 *   d_full   width of the full vector, H_total of Alg. 1: the divisor of the
 *            mean (>= d_local).
 */
typedef struct qkn_seg {
  const uint16_t* x;
  int64_t ldx;
  const float* w;
  float* partials;
  uint16_t* y;
  int64_t ldy;
  float* inv_rms;
  int64_t d_local;
  int64_t d_full;
} qkn_seg;

/*
 * Phase A alone (Sec. III-A; Alg. 1, Phase A):
 *   partial_out[t] = sum_{j < d_local} x[t, j]^2   (fp32, fixed tree).
 * x bf16 [T, ldx]; partial_out fp32 [T]. The result is bit-identical to the
 * statistic the fused call computes for the same slice, so it serves as a
 * peer rank's contribution. QKN_EINVAL: x or partial_out NULL with T > 0,
 * T < 0, d_local < 1, ldx < d_local. QKN_EOVERLAP: partial_out overlaps x.
 */
int qkn_partial_sumsq(const uint16_t* x, int64_t ldx, int64_t T, int64_t d_local,
                      float* partial_out, void* stream);

/*
 * Phases B and C from precomputed statistics (the unfused second step of a
 * scalar-aggregation norm, Sec. IV-A):
 *   S[t] = sum_{k=0}^{tp-1} partials[k*T + t]   (ascending k, fp32),
 *   y[t, j] = bf16( (x[t, j] * w[j]) * (1 / sqrt(S[t]/d_full + eps)) ).
 * partials fp32 [tp * T] holds every rank's slot, this rank's included.
 * inv_rms may be NULL. QKN_EINVAL: NULL x/w/partials/y with T > 0, T < 0,
 * tp < 1, d_local < 1, d_full < d_local, ldx or ldy < d_local, eps < 0 or not
 * finite. QKN_EOVERLAP: y overlaps x in part, or a float output overlaps a
 * bf16 tensor or the other float arrays.
 */
int qkn_apply(const uint16_t* x, int64_t ldx, const float* w, const float* partials,
              int tp, int64_t T, int64_t d_local, int64_t d_full, float eps,
              uint16_t* y, int64_t ldy, float* inv_rms, void* stream);

/*
 * The fused sharded QK-Norm of one rank (Sec. III, Alg. 1), Phases A+B+C in
 * one persistent launch for 1 or 2 tensors (Q and K of the same tokens):
 * each resident wavefront loops over tokens; per token and tensor it computes
 * the slice's partial sum of squares, writes it to partials[rank*T + t] (if
 * partials is not NULL), combines it with the other ranks' slots in ascending
 * rank order, forms x * w while those slots are in flight, and writes the
 * scaled slice. With tp == 1 no slot is read and partials may be NULL.
 * QKN_EINVAL: segs NULL, nseg not 1 or 2, tp < 1, rank not in [0, tp), T < 0,
 * eps < 0 or not finite, or a segment with a NULL x/w/y, partials NULL while
 * tp > 1, d_local < 1, d_full < d_local, ldx or ldy < d_local.
 * QKN_EOVERLAP: as for qkn_apply, across both segments.
 */
int qkn_fused_shard(const qkn_seg* segs, int nseg, int tp, int rank, int64_t T, float eps,
                    void* stream);

/*
 * Full-vector QK-Norm at TP = 1 (Eq. 1 on whole rows), the compute half of
 * the all-gather baseline (Sec. II-C, Sec. IV-A). Same as qkn_fused_shard
 * with tp = 1, rank = 0; each segment must have d_local == d_full; partials
 * may be NULL (else it receives the full sum of squares per token).
 */
int qkn_full(const qkn_seg* segs, int nseg, int64_t T, float eps, void* stream);

/*
 * FP8-E4M3 activations (Sec. IV-C evaluates SwiftQK on them): the OCP
 * e4m3fn format -- 1 sign, 4 exponent (bias 7), 3 mantissa bits; largest
 * finite value 448; no infinities; NaN is S.1111.111. x and y are uint8_t bit
 * patterns; gamma, statistics and factors are fp32 as above, and every sum
 * and product is fp32. Inputs decode exactly. The output is
 * e4m3fn( (x * w) * factor ), rounded to nearest even; a result whose
 * magnitude rounds above 448 is NaN (the format has no infinity), as in the
 * usual non-saturating cast. The partial sums of a slice are bit-identical
 * across these entry points (one fixed tree, as for bf16), so
 * qkn_partial_sumsq_fp8 serves as a peer rank's contribution to
 * qkn_fused_shard_fp8. Arguments, errors and overlap rules are those of the
 * bf16 entry point of the same name, with sizes and strides in elements
 * (bytes).
 */
typedef struct qkn_seg8 {
  const uint8_t* x;
  int64_t ldx;
  const float* w;
  float* partials;
  uint8_t* y;
  int64_t ldy;
  float* inv_rms;
  int64_t d_local;
  int64_t d_full;
} qkn_seg8;

int qkn_partial_sumsq_fp8(const uint8_t* x, int64_t ldx, int64_t T, int64_t d_local,
                          float* partial_out, void* stream);
int qkn_apply_fp8(const uint8_t* x, int64_t ldx, const float* w, const float* partials,
                  int tp, int64_t T, int64_t d_local, int64_t d_full, float eps,
                  uint8_t* y, int64_t ldy, float* inv_rms, void* stream);
int qkn_fused_shard_fp8(const qkn_seg8* segs, int nseg, int tp, int rank, int64_t T,
                        float eps, void* stream);
int qkn_full_fp8(const qkn_seg8* segs, int nseg, int64_t T, float eps, void* stream);

/*
 * Published statistics, for ranks that run concurrently (Sec. III-B; Alg. 1
 * Phase B, where each GPU signals its peers and spins on a local flag).
 * A slot is one 8-byte word: the fp32 statistic's bits in the low half and the
 * round's epoch in the high half, written by one aligned 64-bit store, so a
 * reader that sees the epoch also sees the value. Slot arrays are uint64
 * [tp * T], rank-major (slot k*T + t), one per tensor; they need no reset
 * between rounds: each round uses a new nonzero epoch. The epoch is an
 * argument of the launch, so a HIP graph that captured a waiting launch keeps
 * its epoch: replaying it would accept the slots that an earlier replay
 * published. Such a graph needs its slot arrays cleared to zero (epoch 0 is
 * never a round's) at the start of every replay, e.g. by a fill kernel
 * captured before the producers' launches, or one graph per round.
 */

/*
 * Phase A of one rank's slice, published: slots_out[t] = {sum_j x[t, j]^2,
 * epoch} (the same fp32 value as qkn_partial_sumsq). slots_out is uint64 [T]
 * (point it at rank k's part, slots + k*T, of a slot array), 8-byte aligned.
 * Register path only: QKN_ENOTSUP unless x is 16-byte aligned, ldx and
 * d_local are multiples of 8 and d_local <= 4096. QKN_EINVAL: NULL pointers
 * with T > 0, epoch 0, misaligned slots_out, T < 0, d_local < 1,
 * ldx < d_local. QKN_EOVERLAP: slots_out overlaps x.
 */
int qkn_publish_partials(const uint16_t* x, int64_t ldx, int64_t T, int64_t d_local,
                         uint64_t* slots_out, uint32_t epoch, void* stream);

/*
 * Largest spin_limit: about 4 million polls of one slot, each a round trip to
 * memory after a short sleep, i.e. seconds at most before a wavefront whose
 * peer never publishes gives up -- so a wait stays bounded whatever the
 * caller asks for.
 */
#define QKN_MAX_SPIN_LIMIT (INT64_C(1) << 22)

typedef struct qkn_wait {
  uint64_t* slots[2];  /* per segment: slot array [tp * T] (see above) */
  uint32_t epoch;      /* nonzero: the slots of this round carry it */
  int64_t spin_limit;  /* polls of one slot before giving up, 1..QKN_MAX_SPIN_LIMIT */
  int co_resident;     /* kernels on this GPU that wait on each other (>= 1): the
                          grid is sized so that all of their wavefronts are
                          resident together (Sec. III-D's bound) */
  int32_t* status;     /* device int, set to 1 if any wait gave up; the caller
                          clears it. Outputs of tokens that gave up are NaN. */
} qkn_wait;

/*
 * qkn_fused_shard for ranks that run concurrently: per token and tensor the
 * kernel publishes its own statistic to slots[i][rank*T + t], forms x * w,
 * and then waits (lanes 0..tp-1, one peer each) until every other rank's slot
 * of that token carries `epoch`, before combining them in ascending rank order
 * (Alg. 1). Results are bit-identical to qkn_fused_shard given the same
 * statistics. A wait that exceeds spin_limit polls sets *status = 1 and the
 * wavefront stops waiting for its later tokens; every kernel exits normally.
 * segs[i].partials must be NULL (statistics travel in the slots).
 * QKN_EINVAL: as qkn_fused_shard, and wait NULL, epoch 0, spin_limit < 1 or
 * > QKN_MAX_SPIN_LIMIT, co_resident < 1, a NULL or misaligned slot array or
 * status, partials set.
 * QKN_ENOTSUP: a segment outside the register path (see qkn_publish_partials),
 * or tp * T * 8 >= 2^31 (the kernel addresses a token's slots by 32-bit byte
 * offsets from rank 0's).
 * QKN_EOVERLAP: slot arrays or status overlapping anything else.
 */
int qkn_fused_shard_wait(const qkn_seg* segs, int nseg, int tp, int rank, int64_t T, float eps,
                         const qkn_wait* wait, void* stream);

/*
 * Every rank of a tp group in one launch (ranks that share one GPU, or a
 * single-GPU rehearsal of the exchange): segs describe the FULL tensors --
 * x, y bf16 [T, ld >= d_full], w fp32 [d_full] -- with d_local the slice width
 * and d_full == tp * d_local; rank r's slice is columns [r*d_local,
 * (r+1)*d_local). Wavefront w computes rank w mod tp: it publishes that rank's
 * statistic to slots[i][r*T + t] and waits for the other ranks' as in
 * qkn_fused_shard_wait. Because all ranks are in one launch whose grid fits
 * on the GPU at once, every wavefront a wait depends on is resident (the
 * bound of Sec. III-D), which separate kernels on separate streams do not
 * guarantee on one GPU. inv_rms, if not NULL, is fp32 [tp * T] (rank-major;
 * every rank's factors are equal). The output y is the unsharded QK-Norm.
 * QKN_EINVAL/QKN_ENOTSUP/QKN_EOVERLAP as qkn_fused_shard_wait, and
 * d_full != tp * d_local or ld < d_full.
 */
int qkn_fused_group_wait(const qkn_seg* segs, int nseg, int tp, int64_t T, float eps,
                         const qkn_wait* wait, void* stream);

/*
 * The three entry points above for FP8-E4M3 activations (qkn_seg8, uint8
 * codes; conventions of the FP8 entry points): the published statistic of a
 * slice equals qkn_partial_sumsq_fp8's, and the waiting kernels' results are
 * bit-identical to qkn_fused_shard_fp8 given the same statistics. Register
 * path: x 16-byte aligned, ldx and d_local multiples of 16, d_local <= 4096.
 */
int qkn_publish_partials_fp8(const uint8_t* x, int64_t ldx, int64_t T, int64_t d_local,
                             uint64_t* slots_out, uint32_t epoch, void* stream);
int qkn_fused_shard_wait_fp8(const qkn_seg8* segs, int nseg, int tp, int rank, int64_t T,
                             float eps, const qkn_wait* wait, void* stream);
int qkn_fused_group_wait_fp8(const qkn_seg8* segs, int nseg, int tp, int64_t T, float eps,
                             const qkn_wait* wait, void* stream);

/* Static text for a status code (never NULL). */
const char* qkn_strerror(int status);

/*
 * Launch description of the calling thread's most recent successful launch (or
 * validate_only call, with grid 0),
 * for tests and benchmarks. kernel is a static string naming the variant
 * ("rows<4,1>/fused", "wide<16,2>/fused", "generic/apply", "rows_fp8<2,1>/fused",
 * ...; the numbers are 16-byte chunks per lane); grid is in workgroups, block in
 * threads, waves = grid * block / 64, lds_bytes is the dynamic LDS per
 * workgroup.
 */
typedef struct qkn_launch_info {
  const char* kernel;
  int64_t grid;
  int64_t block;
  int64_t waves;
  int64_t lds_bytes;
} qkn_launch_info;
int qkn_last_launch(qkn_launch_info* info);

/*
 * Tuning knobs for benchmarks and tests. Each setting applies only to launches
 * made later from the calling thread (options are thread-local: a setting in
 * one thread never changes another thread's launches); a new thread starts
 * with the defaults. Keys:
 *   "waves_per_cu"   wavefronts per CU used to size the grid (0 = the
 *                    default: enough to keep ~24 KB (bf16) or ~28 KB (fp8)
 *                    of rows requested per CU, at least 6, at most the
 *                    occupancy limit; larger values oversubscribe, which is
 *                    correct but not persistent);
 *   "prefetch"       1 = pipelined kernels that request the next token
 *                    before writing the current one (bf16 register path,
 *                    modes without a wait), 0 = not (default);
 *   "wait_schedule"  the waiting kernels' order of work per wavefront:
 *                    0 = token by token (publish, x * gamma, wait, store),
 *                    1 = the same with the next token's rows and first poll
 *                    requested early, 2 = publish ahead: a token's
 *                    statistics are published one token before it waits for
 *                    the other ranks', 3 = two tokens before, 4 = three
 *                    tokens before (default; bf16 Q and K rows that are both
 *                    wider than 2048 per rank take 1 instead); same results;
 *   "balance"        1 = shrink the grid so every wavefront takes the same
 *                    number of tokens, 0 = use the full grid (default);
 *   "token_blocks"   1 = each wavefront takes a contiguous range of tokens,
 *                    0 = tokens strided by the wavefront count (default);
 *   "waves_per_block" 1..4, 0 = automatic (register path: 1 for bf16,
 *                    4 for fp8; wide path: always 4);
 *   "force_generic"  1 = always take the general path (same results);
 *   "proj_tile"      qkn_proj_partial's kernel: 0 = automatic (split k for
 *                    decode-sized launches, else kernel 1), 1 = direct-to-
 *                    LDS two-stage kernel on 16 x 16 x 32 MFMAs, never split,
 *                    2 = register-staged kernel, never split, 3 = direct-to-
 *                    LDS kernel on 32 x 32 x 16 MFMAs, never split (2 and 3
 *                    give the same results as 1);
 *   "validate_only"  1 = entry points validate their arguments and choose a
 *                    kernel (reported by qkn_last_launch, grid 0) but make no
 *                    HIP call, launch nothing and return QKN_EDRYRUN (never
 *                    QKN_OK, so a caller that checks the status cannot take
 *                    a call that launched nothing for one that ran; calls
 *                    with T == 0 still return QKN_OK).
 * Returns QKN_OK or QKN_EINVAL for an unknown key or a bad value.
 */
int qkn_set_option(const char* key, int64_t value);

#ifdef __cplusplus
}
#endif

#endif /* QKN_H */
