/*
 * qkn_calib.h -- C ABI of libqkn, part 3: measurement references (AMD MI355X,
 * gfx950). Not part of the QK-Norm method: two kernels the benchmark times in
 * the same run as the QK-Norm kernels, so that their achieved bandwidth and
 * latency can be read against what the part delivers to any kernel.
 *
 * Conventions are those of qkn.h (device pointers owned by the caller,
 * asynchronous on `stream`, validation before any HIP call, negative status
 * codes; the "validate_only" option applies).
 */
#ifndef QKN_CALIB_H
#define QKN_CALIB_H

#include <stdint.h>

#include "qkn.h"

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Streaming copy y[0, bytes) = x[0, bytes): `blocks` workgroups of 256
 * threads, grid-stride over 16-byte vectors with non-temporal loads and
 * stores -- the practical ceiling of a kernel that reads its input once and
 * writes its output once.
 * QKN_EINVAL: bytes < 0 or not a multiple of 16, blocks outside [1, 65536],
 * x or y NULL or not 16-byte aligned (bytes > 0). QKN_EOVERLAP: the regions
 * overlap. bytes == 0 is a no-op.
 */
int qkn_calib_copy(const void* x, void* y, int64_t bytes, int64_t blocks, void* stream);

/* One workgroup of one wavefront that does nothing: the launch floor. */
int qkn_calib_empty(void* stream);

#ifdef __cplusplus
}
#endif

#endif /* QKN_CALIB_H */
