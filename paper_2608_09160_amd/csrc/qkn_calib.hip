// Measurement references for libqkn (AMD MI355X, gfx950): a streaming copy,
// the practical ceiling of any kernel that reads its input once and writes its
// output once, and an empty kernel, the launch floor. The benchmark reports
// both next to the QK-Norm kernels, measured in the same run.

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "qkn_calib.h"
#include "qkn_host.h"

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

// Grid-stride copy of n16 16-byte vectors with non-temporal loads and stores
// (the data is streamed once; keeping it in the caches helps nothing).
__global__ __launch_bounds__(256) void qkn_calib_copy_kernel(const u32x4* __restrict__ x,
                                                             u32x4* __restrict__ y, int64_t n16) {
  const int64_t stride = static_cast<int64_t>(gridDim.x) * blockDim.x;
  for (int64_t i = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x; i < n16;
       i += stride)
    __builtin_nontemporal_store(__builtin_nontemporal_load(x + i), y + i);
}

__global__ void qkn_calib_empty_kernel() {}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

}  // namespace

extern "C" {

int qkn_calib_copy(const void* x, void* y, int64_t bytes, int64_t blocks, void* stream) {
  if (bytes < 0 || bytes % 16 || blocks < 1 || blocks > 65536) return QKN_EINVAL;
  if (bytes == 0) return QKN_OK;
  if (!x || !y || !aligned16(x) || !aligned16(y)) return QKN_EINVAL;
  const qkn_host::Span a{reinterpret_cast<uintptr_t>(x), 1, bytes, bytes, 1};
  const qkn_host::Span b{reinterpret_cast<uintptr_t>(y), 1, bytes, bytes, 1};
  if (qkn_host::spans_overlap(a, b)) return QKN_EOVERLAP;
  const qkn_launch_info info{"calib_copy", blocks, 256, blocks * 4, 0};
  if (qkn_host::validate_only()) {
    qkn_host::record_launch(qkn_launch_info{info.kernel, 0, 0, 0, 0});
    return QKN_EDRYRUN;
  }
  hipLaunchKernelGGL(qkn_calib_copy_kernel, dim3(static_cast<unsigned>(blocks)), dim3(256), 0,
                     static_cast<hipStream_t>(stream), static_cast<const u32x4*>(x),
                     static_cast<u32x4*>(y), bytes / 16);
  if (hipGetLastError() != hipSuccess) return QKN_EHIP;
  qkn_host::record_launch(info);
  return QKN_OK;
}

int qkn_calib_empty(void* stream) {
  const qkn_launch_info info{"calib_empty", 1, 64, 1, 0};
  if (qkn_host::validate_only()) {
    qkn_host::record_launch(qkn_launch_info{info.kernel, 0, 0, 0, 0});
    return QKN_EDRYRUN;
  }
  hipLaunchKernelGGL(qkn_calib_empty_kernel, dim3(1), dim3(64), 0,
                     static_cast<hipStream_t>(stream));
  if (hipGetLastError() != hipSuccess) return QKN_EHIP;
  qkn_host::record_launch(info);
  return QKN_OK;
}

}  // extern "C"
