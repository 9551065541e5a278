// Host-side pieces shared by the entry points of libqkn: the overlap test of
// strided byte regions (argument validation) and the process-wide options and
// launch record that qkn_set_option / qkn_last_launch expose. No device code.
#ifndef QKN_HOST_H
#define QKN_HOST_H

#include <stdint.h>

#include "qkn.h"

namespace qkn_host {

// The "validate_only" option: entry points validate, choose a kernel and
// record it, but launch nothing. Defined in qkn.hip.
__attribute__((visibility("hidden"))) bool validate_only();

// The projection's tile-shape choice ("proj_tile" option). Defined in qkn_proj.hip.
__attribute__((visibility("hidden"))) int set_proj_tile(int64_t choice);

// Records the calling thread's latest launch for qkn_last_launch.
__attribute__((visibility("hidden"))) void record_launch(const qkn_launch_info& info);

// A strided byte region: `rows` rows of `width` elements every `ld` elements.
struct Span {
  uintptr_t base;
  int64_t rows, ld, width, esz;
};

inline int64_t floor_div(int64_t a, int64_t b) {  // b > 0
  int64_t q = a / b;
  if ((a % b != 0) && ((a < 0) != (b < 0))) --q;
  return q;
}

inline bool spans_overlap(const Span& a, const Span& b) {
  if (a.rows <= 0 || b.rows <= 0 || a.width <= 0 || b.width <= 0) return false;
  const __int128 a_lo = a.base, b_lo = b.base;
  const __int128 a_hi = a_lo + ((__int128)(a.rows - 1) * a.ld + a.width) * a.esz;
  const __int128 b_hi = b_lo + ((__int128)(b.rows - 1) * b.ld + b.width) * b.esz;
  if (a_hi <= b_lo || b_hi <= a_lo) return false;  // disjoint extents
  // Same element size and stride: exact test on element offsets.
  if (a.esz == b.esz && a.ld == b.ld && a.ld > 0) {
    const __int128 off_bytes = b_lo - a_lo;
    if (off_bytes % a.esz == 0) {
      const int64_t o = static_cast<int64_t>(off_bytes / a.esz);
      const int64_t ld = a.ld;
      // rows r of a and s of b overlap iff o - wa < (r - s) * ld < o + wb
      const int64_t dmin = -(b.rows - 1), dmax = a.rows - 1;
      int64_t d = floor_div(o - a.width, ld) + 1;
      if (d < dmin) d = dmin;
      return d <= dmax && (__int128)d * ld < (__int128)o + b.width;
    }
  }
  return true;  // conservative
}

}  // namespace qkn_host

#endif  // QKN_HOST_H
