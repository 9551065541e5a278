// libqkn: host side of the sharded layerwise QK-Norm for AMD MI355X (gfx950):
// argument validation, the choice of kernel and launch shape, the C ABI of
// include/qkn.h. The kernels and their design are in qkn_kernels.h.

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdio.h>
#include <stdint.h>
#include <string.h>

#include <mutex>

#include "qkn.h"
#include "qkn_host.h"
#include "qkn_kernels.h"

namespace {

using namespace qkn_dev;
using qkn_host::Span;
using qkn_host::spans_overlap;

// ------------------------------------------------------------------ host side

enum Format { kBf16 = 0, kFp8 = 1 };

// Per-format limits of the specialised kernels. The register path keeps, per
// chunk and lane, the packed row, its fp32 products with gamma and gamma
// itself: 8 bf16 chunks (d_local <= 4096) or 4 fp8 chunks (d_local <= 4096)
// per tensor take the same registers. The wide path keeps only the packed rows
// (slot 0 up to 32 bf16 / 16 fp8 chunks per lane, slot 1 as the register path).
//
// Register-path grid (measured on MI355X, prefill shards of 8192 and 32768
// tokens): bf16 peaks with about 24 KB of rows requested per CU in one-wave
// workgroups; fp8 rows are half as long and need more of them in flight,
// about 28 KB per CU (12 wavefronts for both shards' row lengths; 16, which
// 32 KB gave the 32768-token shard, ran 5 % slower), best spread in four-wave
// workgroups.
struct FormatInfo {
  int esz;                 // bytes per element
  int per;                 // elements per 16-byte chunk
  int reg_max;             // register path: chunks per lane
  int wide_n0[2];          // wide path: chunks per lane of the kernels for slot 0
  const char* suffix;      // kernel-family suffix in launch names
  int64_t inflight_bytes;  // register path: row bytes to keep requested per CU
  int waves_per_block;     // register path: default workgroup size in wavefronts
};
constexpr FormatInfo kFormat[2] = {{2, 8, 8, {16, 32}, "", 24 * 1024, 1},
                                   {1, 16, 4, {8, 16}, "_fp8", 28 * 1024, 4}};

constexpr int kMaxWideLdsBytes = 64 * 1024;  // gamma of both tensors staged by the wide path

// Chunks per lane are rounded up to 1, 2, 4 or 8; unused chunks are masked.
constexpr int kNIdx[9] = {-1, 0, 1, 2, 2, 3, 3, 3, 3};  // chunks/lane -> table index
constexpr int kNVal[4] = {1, 2, 4, 8};

const char* const kModeName[5] = {"fused", "apply", "partial", "fused_wait", "publish"};

// Static names "rows<N0,N1>/mode" ("rows_pf<...>" when pipelined, "rows_fp8<...>" for fp8).
const char* rows_name(int fmt, int mode, int sched, int i0, int i1) {
  static char names[2][5][5][4][5][40];
  static std::once_flag once;
  std::call_once(once, [] {
    const char* const prefix[2][5] = {
        {"rows", "rows_pf", "rows_pa", "rows_pa2", "rows_pa3"},
        {"rows_fp8", "rows_pf_fp8", "rows_pa_fp8", "rows_pa2_fp8", "rows_pa3_fp8"}};
    for (int fm = 0; fm < 2; ++fm)
      for (int m = 0; m < 5; ++m)
        for (int f = 0; f < 5; ++f)
          for (int a = 0; a < 4; ++a)
            for (int b = 0; b < 5; ++b)
              snprintf(names[fm][m][f][a][b], sizeof(names[fm][m][f][a][b]), "%s<%d,%d>/%s",
                       prefix[fm][f], kNVal[a], b == 0 ? 0 : kNVal[b - 1], kModeName[m]);
  });
  return names[fmt][mode][sched][i0][i1];
}
const char* const kGenericName[2][3] = {{"generic/fused", "generic/apply", "generic/partial"},
                                        {"generic_fp8/fused", "generic_fp8/apply",
                                         "generic_fp8/partial"}};

// Static names "wide<N0,N1>/mode" ("wide_fp8<...>" for fp8).
const char* wide_name(int fmt, int mode, int i0, int i1) {
  static char names[2][3][2][5][40];
  static std::once_flag once;
  std::call_once(once, [] {
    for (int fm = 0; fm < 2; ++fm)
      for (int m = 0; m < 3; ++m)
        for (int a = 0; a < 2; ++a)
          for (int b = 0; b < 5; ++b)
            snprintf(names[fm][m][a][b], sizeof(names[fm][m][a][b]), "wide%s<%d,%d>/%s",
                     kFormat[fm].suffix, kFormat[fm].wide_n0[a], b == 0 ? 0 : kNVal[b - 1],
                     kModeName[m]);
  });
  return names[fmt][mode][i0][i1];
}

// Options (qkn_set_option): per calling thread, so that a setting made by
// one thread (a test, a tuning sweep) never changes another thread's launches.
thread_local int64_t g_opt_waves_per_cu = 0;
thread_local int64_t g_opt_wait_schedule = 4;  // publish three tokens ahead
thread_local int64_t g_opt_waves_per_block = 0;
thread_local int64_t g_opt_force_generic = 0;
thread_local int64_t g_opt_validate_only = 0;
thread_local int64_t g_opt_prefetch = 0;
thread_local int64_t g_opt_token_blocks = 0;
thread_local int64_t g_opt_balance = 0;

thread_local qkn_launch_info t_last = {nullptr, 0, 0, 0, 0};

// Per-device CU count and per-kernel occupancy, filled on first use.
constexpr int kMaxDevices = 64;
struct OccEntry {
  const void* fn;
  int block;
  int lds;
  int blocks_per_cu;
};
struct DeviceCache {
  int cu_count = 0;
  OccEntry occ[256];
  int nocc = 0;
};
std::mutex g_mu;
DeviceCache g_dev[kMaxDevices];

int query_device(int* dev, int* cu_count) {
  if (hipGetDevice(dev) != hipSuccess || *dev < 0 || *dev >= kMaxDevices) return QKN_EHIP;
  std::lock_guard<std::mutex> lock(g_mu);
  DeviceCache& dc = g_dev[*dev];
  if (dc.cu_count == 0) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, *dev) != hipSuccess ||
        n <= 0)
      return QKN_EHIP;
    dc.cu_count = n;
  }
  *cu_count = dc.cu_count;
  return QKN_OK;
}

int blocks_per_cu(int dev, const void* fn, int block, int lds, int* out) {
  std::lock_guard<std::mutex> lock(g_mu);
  DeviceCache& dc = g_dev[dev];
  for (int i = 0; i < dc.nocc; ++i) {
    if (dc.occ[i].fn == fn && dc.occ[i].block == block && dc.occ[i].lds == lds) {
      *out = dc.occ[i].blocks_per_cu;
      return QKN_OK;
    }
  }
  int n = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&n, fn, block, lds) != hipSuccess || n <= 0)
    return QKN_EHIP;
  if (dc.nocc < 256) dc.occ[dc.nocc++] = OccEntry{fn, block, lds, n};
  *out = n;
  return QKN_OK;
}

// ---------------------------------------------------------------- validation

// Host view of a segment of either format (qkn_seg or qkn_seg8).
struct HSeg {
  const void* x;
  int64_t ldx;
  const float* w;
  float* partials;
  void* y;
  int64_t ldy;
  float* inv_rms;
  int64_t d_local;
  int64_t d_full;
};

template <class S>
HSeg to_hseg(const S& s) {
  return HSeg{s.x, s.ldx, s.w, s.partials, s.y, s.ldy, s.inv_rms, s.d_local, s.d_full};
}

bool bad_eps(float eps) { return !(eps >= 0.0f) || !isfinite(eps); }

Span elem_span(const void* p, int64_t rows, int64_t ld, int64_t width, int esz) {
  return Span{reinterpret_cast<uintptr_t>(p), rows, ld, width, esz};
}
Span f32_span(const void* p, int64_t n) {
  return Span{reinterpret_cast<uintptr_t>(p), 1, n, n, 4};
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int64_t kMaxWidth = (int64_t{1} << 30);  // d_local and strides fit in int32 chunk math

int check_seg_shape(const HSeg& s, int mode) {
  if (!s.x) return QKN_EINVAL;
  if (s.d_local < 1 || s.d_local > kMaxWidth || s.ldx < s.d_local) return QKN_EINVAL;
  if (mode != kPartial && mode != kPublish) {
    if (!s.w || !s.y) return QKN_EINVAL;
    if (s.d_full < s.d_local || s.ldy < s.d_local) return QKN_EINVAL;
  }
  return QKN_OK;
}

// Overlap rules: outputs (y, own statistic slots, inv_rms) may not overlap any
// input or another output, except y == x with equal strides (in place) and a
// segment's own slots inside its own partials array.
int check_overlaps(const HSeg* segs, int nseg, int tp, int rank, int64_t T, int mode, int esz,
                   const Span* extra = nullptr, int nextra = 0) {
  struct Item {
    Span s;
    bool out;
    int seg;
    int kind;  // 0 x, 1 w, 2 partials (read), 3 y, 4 own slots, 5 inv, 6 extra output
  };
  Item items[16];
  int n = 0;
  for (int i = 0; i < nextra; ++i) items[n++] = Item{extra[i], true, 100 + i, 6};
  for (int i = 0; i < nseg; ++i) {
    const HSeg& s = segs[i];
    items[n++] = Item{elem_span(s.x, T, s.ldx, s.d_local, esz), false, i, 0};
    if (mode == kPartial) {
      items[n++] = Item{f32_span(s.partials, T), true, i, 4};
      continue;
    }
    if (mode == kPublish) continue;
    items[n++] = Item{f32_span(s.w, s.d_local), false, i, 1};
    if (s.partials) {
      if (mode == kApply || tp > 1) items[n++] = Item{f32_span(s.partials, tp * T), false, i, 2};
      if (mode == kFused) items[n++] = Item{f32_span(s.partials + (int64_t)rank * T, T), true, i, 4};
    }
    items[n++] = Item{elem_span(s.y, T, s.ldy, s.d_local, esz), true, i, 3};
    if (s.inv_rms) items[n++] = Item{f32_span(s.inv_rms, T), true, i, 5};
  }
  for (int a = 0; a < n; ++a) {
    for (int b = a + 1; b < n; ++b) {
      const Item& A = items[a];
      const Item& B = items[b];
      if (!A.out && !B.out) continue;
      if (A.seg == B.seg) {
        const int lo = A.kind < B.kind ? A.kind : B.kind;
        const int hi = A.kind < B.kind ? B.kind : A.kind;
        if (lo == 2 && hi == 4) continue;  // own slots live inside the partials array
        if (lo == 0 && hi == 3 && A.s.base == B.s.base && A.s.ld == B.s.ld) continue;  // in place
      }
      if (spans_overlap(A.s, B.s)) return QKN_EOVERLAP;
    }
  }
  return QKN_OK;
}

bool seg_vec_ok(const HSeg& s, int mode, int per) {
  if (!aligned16(s.x) || (s.ldx % per) || (s.d_local % per)) return false;
  if (mode != kPartial && mode != kPublish) {
    if (!aligned16(s.y) || !aligned16(s.w) || (s.ldy % per)) return false;
  }
  return true;
}

DevSeg to_dev(const HSeg& s, int mode, const FormatInfo& fi) {
  DevSeg d;
  d.x = s.x;
  d.w = s.w;
  d.partials = s.partials;
  d.y = s.y;
  d.inv_rms = s.inv_rms;
  d.ldx = s.ldx;
  d.ldy = (mode == kPartial || mode == kPublish) ? 0 : s.ldy;
  d.d = static_cast<int32_t>(s.d_local);
  d.nchunks = static_cast<int32_t>((s.d_local + fi.per - 1) / fi.per);
  d.rcp_d_full = static_cast<float>(
      1.0 / static_cast<double>((mode == kPartial || mode == kPublish) ? s.d_local : s.d_full));
  d.vec = seg_vec_ok(s, mode, fi.per) ? 1 : 0;
  return d;
}

// Arguments of the waiting and publishing modes.
struct WaitArgs {
  uint64_t* slots[2];
  int32_t* status;
  int64_t spin_limit;
  uint32_t epoch;
  int co_resident;  // kernels sharing the GPU that wait on each other
  int group;        // > 1: every rank of the group in this launch
};

int launch(const HSeg* segs, int nseg, int tp, int rank, int64_t T, float eps, int mode, int fmt,
           void* stream, const WaitArgs* wa = nullptr) {
  const FormatInfo& fi = kFormat[fmt];
  KParams kp;
  memset(&kp, 0, sizeof(kp));
  kp.T = T;
  kp.nseg = nseg;
  kp.tp = tp;
  kp.rank = rank;
  kp.eps = eps;
  const bool waits = (mode == kFusedWait || mode == kPublish);
  if (waits) {
    kp.slots[0] = wa->slots[0];
    kp.slots[1] = wa->slots[1];
    kp.status = wa->status;
    kp.spin_limit = wa->spin_limit;
    kp.epoch = wa->epoch;
    kp.group = wa->group;
  }
  const int group = (waits && wa->group > 1) ? wa->group : 1;
  // the register path addresses a token's statistic slots by 32-bit byte
  // offsets from rank 0's: 4-byte statistics, or 8-byte flagged slots
  const int slot_bytes = waits ? 8 : 4;
  const bool buffer_ok = (g_opt_force_generic == 0) && tp <= kMaxFastTp &&
                         static_cast<__int128>(tp) * T * slot_bytes <
                             (static_cast<__int128>(1) << 31);
  bool fast = buffer_ok;
  bool wide = buffer_ok && !waits;
  int idx[2] = {0, 0};
  int max_chunks = 0;
  int64_t gamma_floats = 0;
  for (int i = 0; i < nseg; ++i) {
    kp.seg[i] = to_dev(segs[i], mode, fi);
    const int per_lane = (kp.seg[i].nchunks + kWave - 1) / kWave;
    if (!kp.seg[i].vec || per_lane > fi.reg_max) fast = false;
    else idx[i] = kNIdx[per_lane];
    if (!kp.seg[i].vec || per_lane > fi.wide_n0[1]) wide = false;
    if (kp.seg[i].nchunks > max_chunks) max_chunks = kp.seg[i].nchunks;
    gamma_floats += kp.seg[i].d;
  }
  if (fast) wide = false;
  if (mode != kPartial && gamma_floats * 4 > kMaxWideLdsBytes) wide = false;
  int wide_i0 = 0, wide_i1 = 0;
  if (wide) {
    // the wider tensor goes first (slot 0 takes the wide row, slot 1 a register-path one)
    if (nseg == 2 && kp.seg[1].nchunks > kp.seg[0].nchunks) {
      const DevSeg tmp = kp.seg[0];
      kp.seg[0] = kp.seg[1];
      kp.seg[1] = tmp;
    }
    const int pl0 = (kp.seg[0].nchunks + kWave - 1) / kWave;
    wide_i0 = pl0 <= fi.wide_n0[0] ? 0 : 1;
    if (nseg == 2) {
      const int pl1 = (kp.seg[1].nchunks + kWave - 1) / kWave;
      if (pl1 > fi.reg_max) wide = false;  // both tensors wide: general path
      else wide_i1 = kNIdx[pl1] + 1;
    }
  }

  if (waits && !fast) return QKN_ENOTSUP;  // the flagged-slot modes exist on the register path only
  const void* fn;
  const char* name;
  int lds = 0;
  int32_t stage_elems = 0;
  const int i1 = nseg == 2 ? idx[1] + 1 : 0;
  if (wide) {
    fn = reinterpret_cast<const void*>(kWideTable[fmt][wide_i0][mode][wide_i1]);
    name = wide_name(fmt, mode, wide_i0, wide_i1);
    lds = (mode == kPartial) ? 0 : static_cast<int>(gamma_floats * 4);
  } else if (waits) {
    int sched = (mode == kFusedWait) ? static_cast<int>(g_opt_wait_schedule) : 0;
    // Q and K rows both of 8 bf16 chunks per lane: the publish-ahead
    // schedules' extra token registers do not fit (they spilled to scratch),
    // so those launches take the pipelined token-by-token schedule
    if (fmt == kBf16 && idx[0] == 3 && i1 == 4 && sched > 1) sched = 1;
    if (mode == kFusedWait)
      fn = reinterpret_cast<const void*>(fmt == kBf16 ? kFusedWaitTable[sched][idx[0]][i1]
                                                      : kFusedWaitTable8[sched][idx[0]][i1]);
    else
      fn = reinterpret_cast<const void*>(fmt == kBf16 ? kPublishTable[idx[0]]
                                                      : kPublishTable8[idx[0]]);
    name = rows_name(fmt, mode, sched, idx[0], i1);
    if (!fn) return QKN_ENOTSUP;
  } else if (fast) {
    const int sched = (fmt == kBf16 && g_opt_prefetch) ? 1 : 0;  // pipelining: bf16 kernels only
    if (fmt == kBf16) {
      if (mode == kFused) fn = reinterpret_cast<const void*>(kFusedTable[sched][idx[0]][i1]);
      else if (mode == kApply) fn = reinterpret_cast<const void*>(kApplyTable[sched][idx[0]]);
      else fn = reinterpret_cast<const void*>(kPartialTable[sched][idx[0]]);
    } else {
      if (mode == kFused) fn = reinterpret_cast<const void*>(kFusedTable8[idx[0]][i1]);
      else if (mode == kApply) fn = reinterpret_cast<const void*>(kApplyTable8[idx[0]]);
      else fn = reinterpret_cast<const void*>(kPartialTable8[idx[0]]);
    }
    name = rows_name(fmt, mode, sched, idx[0], i1);
  } else {
    fn = reinterpret_cast<const void*>(kGenericTable[fmt][mode]);
    name = kGenericName[fmt][mode];
    if (mode == kFused && static_cast<int64_t>(max_chunks) * 16 <= kMaxStageBytes) {
      stage_elems = max_chunks * fi.per;
      lds = max_chunks * 16;
    }
  }
  if (!fn) return QKN_ENOTSUP;  // not reached: every selectable entry is instantiated
  if (g_opt_validate_only) {  // arguments accepted and a kernel chosen; no HIP call
    t_last = qkn_launch_info{name, 0, 0, 0, lds};
    return QKN_EDRYRUN;
  }

  int dev = 0, cus = 0;
  int rc = query_device(&dev, &cus);
  if (rc != QKN_OK) return rc;
  int wpb = 1;
  if (fast && !waits) {
    // multi-wave workgroups only when the tokens fill every CU several times
    // over; short launches (decode) spread one-wave workgroups over more CUs
    if (g_opt_waves_per_block > 0) wpb = static_cast<int>(g_opt_waves_per_block);
    else if (T >= static_cast<int64_t>(cus) * fi.waves_per_block * kMinWavesPerCu)
      wpb = fi.waves_per_block;
  }
  if (wide) wpb = 4;  // four wavefronts share the gamma staged in LDS
  const int block = wpb * kWave;
  int bpc = 0;
  rc = blocks_per_cu(dev, fn, block, lds, &bpc);
  if (rc != QKN_OK) return rc;
  // Persistent grid: enough wavefronts per CU to keep about fi.inflight_bytes
  // of rows requested per CU, at least kMinWavesPerCu, at most what fits.
  int64_t waves_per_cu = static_cast<int64_t>(bpc) * wpb;
  if (fast || wide) {  // waiting launches too: fewer waves only loosen the co-residency bound below
    int64_t token_bytes = 0;
    for (int i = 0; i < nseg; ++i) token_bytes += fi.esz * static_cast<int64_t>(kp.seg[i].d);
    int64_t want = (fi.inflight_bytes + token_bytes - 1) / token_bytes;
    if (want < kMinWavesPerCu) want = kMinWavesPerCu;
    // whole workgroups per CU: the dispatcher deals workgroups out evenly over
    // the XCDs and their CUs, so a grid that is not a multiple of the CU count
    // leaves some CUs with one workgroup more than others (measured: 13 waves
    // per CU in 4-wave workgroups runs 15 % slower than 12)
    want = (want + wpb / 2) / wpb * wpb;
    if (want < wpb) want = wpb;
    if (want < waves_per_cu) waves_per_cu = want;
  }
  if (g_opt_waves_per_cu > 0) waves_per_cu = g_opt_waves_per_cu;
  if (mode == kFusedWait) {
    // every wavefront of every co-resident waiting kernel must be resident at
    // once, or a spinning one could hold the place of the one it waits for
    const int64_t fit = static_cast<int64_t>(bpc) * wpb / wa->co_resident;
    if (waves_per_cu > fit) waves_per_cu = fit;
  }
  if (waves_per_cu < 1) waves_per_cu = 1;
  int64_t waves = waves_per_cu * cus;
  if (group > 1) {
    // all ranks of the group share the resident wavefronts equally
    int64_t per_rank = waves / group;
    if (per_rank > T) per_rank = T;
    if (per_rank < 1) return QKN_ENOTSUP;  // the group does not fit on the GPU at once
    waves = per_rank * group;
  } else if (waves > T) {
    waves = T;
  } else if (fast && g_opt_balance) {
    // equal shares: k tokens per wavefront for every wavefront (but the last),
    // so that none runs an extra token while the others are done
    const int64_t k = (T + waves - 1) / waves;
    waves = (T + k - 1) / k;
  }
  int64_t grid = (waves + wpb - 1) / wpb;
  if (grid > 0x7fffffff) grid = 0x7fffffff;
  if (fast && g_opt_token_blocks) kp.tok_chunk = (T + grid * wpb - 1) / (grid * wpb);

  hipError_t err;
  if (fast || wide) {
    void* args[] = {&kp};
    err = hipLaunchKernel(fn, dim3(static_cast<unsigned>(grid)), dim3(block), args, lds,
                          static_cast<hipStream_t>(stream));
  } else {
    void* args[] = {&kp, &stage_elems};
    err = hipLaunchKernel(fn, dim3(static_cast<unsigned>(grid)), dim3(block), args, lds,
                          static_cast<hipStream_t>(stream));
  }
  if (err != hipSuccess) return QKN_EHIP;
  t_last = qkn_launch_info{name, grid, block, grid * wpb, lds};
  return QKN_OK;
}

int validate_common(int64_t T, float eps, int tp, int rank) {
  if (T < 0 || tp < 1 || rank < 0 || rank >= tp || bad_eps(eps)) return QKN_EINVAL;
  if (T > 0 && static_cast<__int128>(T) * tp > INT64_MAX / 8) return QKN_EINVAL;
  return QKN_OK;
}

bool seg_dims_bad(const HSeg& s) {
  return s.d_local < 1 || s.d_local > kMaxWidth || s.ldx < s.d_local || s.d_full < s.d_local ||
         s.ldy < s.d_local;
}

int partial_impl(const void* x, int64_t ldx, int64_t T, int64_t d_local, float* partial_out,
                 int fmt, void* stream) {
  if (T < 0 || d_local < 1 || d_local > kMaxWidth || ldx < d_local) return QKN_EINVAL;
  if (T == 0) return QKN_OK;
  if (!x || !partial_out) return QKN_EINVAL;
  HSeg s;
  memset(&s, 0, sizeof(s));
  s.x = x;
  s.ldx = ldx;
  s.partials = partial_out;
  s.d_local = d_local;
  s.d_full = d_local;
  int rc = check_seg_shape(s, kPartial);
  if (rc != QKN_OK) return rc;
  rc = check_overlaps(&s, 1, 1, 0, T, kPartial, kFormat[fmt].esz);
  if (rc != QKN_OK) return rc;
  return launch(&s, 1, 1, 0, T, 0.0f, kPartial, fmt, stream);
}

int apply_impl(const HSeg& s, int tp, int64_t T, float eps, int fmt, void* stream) {
  int rc = validate_common(T, eps, tp, 0);
  if (rc != QKN_OK) return rc;
  if (seg_dims_bad(s)) return QKN_EINVAL;
  if (T == 0) return QKN_OK;
  rc = check_seg_shape(s, kApply);
  if (rc != QKN_OK) return rc;
  if (!s.partials) return QKN_EINVAL;
  rc = check_overlaps(&s, 1, tp, 0, T, kApply, kFormat[fmt].esz);
  if (rc != QKN_OK) return rc;
  return launch(&s, 1, tp, 0, T, eps, kApply, fmt, stream);
}

int fused_impl(const HSeg* segs, int nseg, int tp, int rank, int64_t T, float eps, int fmt,
               void* stream) {
  int rc = validate_common(T, eps, tp, rank);
  if (rc != QKN_OK) return rc;
  for (int i = 0; i < nseg; ++i)
    if (seg_dims_bad(segs[i])) return QKN_EINVAL;
  if (T == 0) return QKN_OK;
  for (int i = 0; i < nseg; ++i) {
    rc = check_seg_shape(segs[i], kFused);
    if (rc != QKN_OK) return rc;
    if (tp > 1 && !segs[i].partials) return QKN_EINVAL;
  }
  rc = check_overlaps(segs, nseg, tp, rank, T, kFused, kFormat[fmt].esz);
  if (rc != QKN_OK) return rc;
  return launch(segs, nseg, tp, rank, T, eps, kFused, fmt, stream);
}

template <class S>
int fused_entry(const S* segs, int nseg, int tp, int rank, int64_t T, float eps, int fmt,
                void* stream) {
  if (!segs || nseg < 1 || nseg > 2) return QKN_EINVAL;
  HSeg h[2];
  for (int i = 0; i < nseg; ++i) h[i] = to_hseg(segs[i]);
  return fused_impl(h, nseg, tp, rank, T, eps, fmt, stream);
}

template <class S>
int full_entry(const S* segs, int nseg, int64_t T, float eps, int fmt, void* stream) {
  if (!segs || nseg < 1 || nseg > 2) return QKN_EINVAL;
  for (int i = 0; i < nseg; ++i)
    if (segs[i].d_full != segs[i].d_local) return QKN_EINVAL;
  return fused_entry(segs, nseg, 1, 0, T, eps, fmt, stream);
}

int publish_impl(const void* x, int64_t ldx, int64_t T, int64_t d_local, uint64_t* slots_out,
                 uint32_t epoch, int fmt, void* stream) {
  if (T < 0 || d_local < 1 || d_local > kMaxWidth || ldx < d_local) return QKN_EINVAL;
  if (T == 0) return QKN_OK;
  if (!x || !slots_out || epoch == 0 || (reinterpret_cast<uintptr_t>(slots_out) & 7u))
    return QKN_EINVAL;
  HSeg s;
  memset(&s, 0, sizeof(s));
  s.x = x;
  s.ldx = ldx;
  s.d_local = d_local;
  s.d_full = d_local;
  const Span out{reinterpret_cast<uintptr_t>(slots_out), 1, T, T, 8};
  int rc = check_overlaps(&s, 1, 1, 0, T, kPublish, kFormat[fmt].esz, &out, 1);
  if (rc != QKN_OK) return rc;
  WaitArgs wa;
  memset(&wa, 0, sizeof(wa));
  wa.slots[0] = slots_out;
  wa.epoch = epoch;
  wa.spin_limit = 1;
  wa.co_resident = 1;
  wa.group = 1;
  return launch(&s, 1, 1, 0, T, 0.0f, kPublish, fmt, stream, &wa);
}

template <class S>
int wait_impl(const S* segs_in, int nseg, int tp, int rank, int64_t T, float eps,
              const qkn_wait* wait, int fmt, void* stream) {
  if (!segs_in || nseg < 1 || nseg > 2 || !wait) return QKN_EINVAL;
  int rc = validate_common(T, eps, tp, rank);
  if (rc != QKN_OK) return rc;
  if (wait->epoch == 0 || wait->spin_limit < 1 || wait->spin_limit > QKN_MAX_SPIN_LIMIT ||
      wait->co_resident < 1)
    return QKN_EINVAL;
  HSeg segs[2];
  for (int i = 0; i < nseg; ++i) {
    segs[i] = to_hseg(segs_in[i]);
    if (seg_dims_bad(segs[i])) return QKN_EINVAL;
  }
  if (T == 0) return QKN_OK;
  if (!wait->status || (reinterpret_cast<uintptr_t>(wait->status) & 3u)) return QKN_EINVAL;
  Span extra[3];
  int nextra = 0;
  for (int i = 0; i < nseg; ++i) {
    rc = check_seg_shape(segs[i], kFusedWait);
    if (rc != QKN_OK) return rc;
    if (segs[i].partials) return QKN_EINVAL;  // statistics travel in wait->slots
    uint64_t* sl = wait->slots[i];
    if (!sl || (reinterpret_cast<uintptr_t>(sl) & 7u)) return QKN_EINVAL;
    extra[nextra++] = Span{reinterpret_cast<uintptr_t>(sl), 1, tp * T, tp * T, 8};
  }
  extra[nextra++] = Span{reinterpret_cast<uintptr_t>(wait->status), 1, 1, 1, 4};
  rc = check_overlaps(segs, nseg, tp, rank, T, kFusedWait, kFormat[fmt].esz, extra, nextra);
  if (rc != QKN_OK) return rc;
  WaitArgs wa;
  wa.slots[0] = wait->slots[0];
  wa.slots[1] = nseg == 2 ? wait->slots[1] : nullptr;
  wa.status = wait->status;
  wa.spin_limit = wait->spin_limit;
  wa.epoch = wait->epoch;
  wa.co_resident = wait->co_resident;
  wa.group = 1;
  return launch(segs, nseg, tp, rank, T, eps, kFusedWait, fmt, stream, &wa);
}

template <class S>
int group_impl(const S* segs_in, int nseg, int tp, int64_t T, float eps, const qkn_wait* wait,
               int fmt, void* stream) {
  if (!segs_in || nseg < 1 || nseg > 2 || !wait) return QKN_EINVAL;
  int rc = validate_common(T, eps, tp, 0);
  if (rc != QKN_OK) return rc;
  if (wait->epoch == 0 || wait->spin_limit < 1 || wait->spin_limit > QKN_MAX_SPIN_LIMIT ||
      wait->co_resident < 1)
    return QKN_EINVAL;
  HSeg segs[2];
  HSeg view[2];  // the full tensors, for shape and overlap checks
  for (int i = 0; i < nseg; ++i) {
    const HSeg s = to_hseg(segs_in[i]);
    if (s.d_local < 1 || s.d_local > kMaxWidth || s.d_full != s.d_local * tp ||
        s.ldx < s.d_full || s.ldy < s.d_full)
      return QKN_EINVAL;
    segs[i] = s;
    view[i] = s;
    view[i].d_local = s.d_full;
    view[i].inv_rms = nullptr;
  }
  if (T == 0) return QKN_OK;
  if (!wait->status || (reinterpret_cast<uintptr_t>(wait->status) & 3u)) return QKN_EINVAL;
  Span extra[5];
  int nextra = 0;
  for (int i = 0; i < nseg; ++i) {
    rc = check_seg_shape(view[i], kFusedWait);
    if (rc != QKN_OK) return rc;
    if (segs[i].partials) return QKN_EINVAL;
    uint64_t* sl = wait->slots[i];
    if (!sl || (reinterpret_cast<uintptr_t>(sl) & 7u)) return QKN_EINVAL;
    extra[nextra++] = Span{reinterpret_cast<uintptr_t>(sl), 1, tp * T, tp * T, 8};
    if (segs[i].inv_rms)
      extra[nextra++] = Span{reinterpret_cast<uintptr_t>(segs[i].inv_rms), 1, tp * T, tp * T, 4};
  }
  extra[nextra++] = Span{reinterpret_cast<uintptr_t>(wait->status), 1, 1, 1, 4};
  rc = check_overlaps(view, nseg, tp, 0, T, kFusedWait, kFormat[fmt].esz, extra, nextra);
  if (rc != QKN_OK) return rc;
  WaitArgs wa;
  wa.slots[0] = wait->slots[0];
  wa.slots[1] = nseg == 2 ? wait->slots[1] : nullptr;
  wa.status = wait->status;
  wa.spin_limit = wait->spin_limit;
  wa.epoch = wait->epoch;
  wa.co_resident = wait->co_resident;
  wa.group = tp;
  return launch(segs, nseg, tp, 0, T, eps, kFusedWait, fmt, stream, &wa);
}

}  // namespace

namespace qkn_host {
bool validate_only() { return g_opt_validate_only != 0; }
void record_launch(const qkn_launch_info& info) { t_last = info; }
}  // namespace qkn_host

extern "C" {

int qkn_partial_sumsq(const uint16_t* x, int64_t ldx, int64_t T, int64_t d_local,
                      float* partial_out, void* stream) {
  return partial_impl(x, ldx, T, d_local, partial_out, kBf16, stream);
}

int qkn_partial_sumsq_fp8(const uint8_t* x, int64_t ldx, int64_t T, int64_t d_local,
                          float* partial_out, void* stream) {
  return partial_impl(x, ldx, T, d_local, partial_out, kFp8, stream);
}

int qkn_apply(const uint16_t* x, int64_t ldx, const float* w, const float* partials, int tp,
              int64_t T, int64_t d_local, int64_t d_full, float eps, uint16_t* y, int64_t ldy,
              float* inv_rms, void* stream) {
  const HSeg s{x, ldx, w, const_cast<float*>(partials), y, ldy, inv_rms, d_local, d_full};
  return apply_impl(s, tp, T, eps, kBf16, stream);
}

int qkn_apply_fp8(const uint8_t* x, int64_t ldx, const float* w, const float* partials, int tp,
                  int64_t T, int64_t d_local, int64_t d_full, float eps, uint8_t* y, int64_t ldy,
                  float* inv_rms, void* stream) {
  const HSeg s{x, ldx, w, const_cast<float*>(partials), y, ldy, inv_rms, d_local, d_full};
  return apply_impl(s, tp, T, eps, kFp8, stream);
}

int qkn_fused_shard(const qkn_seg* segs, int nseg, int tp, int rank, int64_t T, float eps,
                    void* stream) {
  return fused_entry(segs, nseg, tp, rank, T, eps, kBf16, stream);
}

int qkn_fused_shard_fp8(const qkn_seg8* segs, int nseg, int tp, int rank, int64_t T, float eps,
                        void* stream) {
  return fused_entry(segs, nseg, tp, rank, T, eps, kFp8, stream);
}

int qkn_full(const qkn_seg* segs, int nseg, int64_t T, float eps, void* stream) {
  return full_entry(segs, nseg, T, eps, kBf16, stream);
}

int qkn_full_fp8(const qkn_seg8* segs, int nseg, int64_t T, float eps, void* stream) {
  return full_entry(segs, nseg, T, eps, kFp8, stream);
}

int qkn_publish_partials(const uint16_t* x, int64_t ldx, int64_t T, int64_t d_local,
                         uint64_t* slots_out, uint32_t epoch, void* stream) {
  return publish_impl(x, ldx, T, d_local, slots_out, epoch, kBf16, stream);
}

int qkn_publish_partials_fp8(const uint8_t* x, int64_t ldx, int64_t T, int64_t d_local,
                             uint64_t* slots_out, uint32_t epoch, void* stream) {
  return publish_impl(x, ldx, T, d_local, slots_out, epoch, kFp8, stream);
}

int qkn_fused_shard_wait(const qkn_seg* segs, int nseg, int tp, int rank, int64_t T, float eps,
                         const qkn_wait* wait, void* stream) {
  return wait_impl(segs, nseg, tp, rank, T, eps, wait, kBf16, stream);
}

int qkn_fused_shard_wait_fp8(const qkn_seg8* segs, int nseg, int tp, int rank, int64_t T,
                             float eps, const qkn_wait* wait, void* stream) {
  return wait_impl(segs, nseg, tp, rank, T, eps, wait, kFp8, stream);
}

int qkn_fused_group_wait(const qkn_seg* segs, int nseg, int tp, int64_t T, float eps,
                         const qkn_wait* wait, void* stream) {
  return group_impl(segs, nseg, tp, T, eps, wait, kBf16, stream);
}

int qkn_fused_group_wait_fp8(const qkn_seg8* segs, int nseg, int tp, int64_t T, float eps,
                             const qkn_wait* wait, void* stream) {
  return group_impl(segs, nseg, tp, T, eps, wait, kFp8, stream);
}

const char* qkn_strerror(int status) {
  switch (status) {
    case QKN_OK: return "ok";
    case QKN_EINVAL: return "invalid argument";
    case QKN_EOVERLAP: return "output overlaps an input or another output";
    case QKN_EHIP: return "HIP runtime error";
    case QKN_ENOTSUP: return "shape or alignment not supported by this entry point";
    case QKN_EDRYRUN: return "validated only: validate_only is set on this thread, nothing launched";
    default: return "unknown status";
  }
}

int qkn_last_launch(qkn_launch_info* info) {
  if (!info) return QKN_EINVAL;
  *info = t_last;
  return QKN_OK;
}

int qkn_set_option(const char* key, int64_t value) {
  if (!key) return QKN_EINVAL;
  if (strcmp(key, "waves_per_cu") == 0) {
    if (value < 0 || value > 64) return QKN_EINVAL;
    g_opt_waves_per_cu = value;
  } else if (strcmp(key, "waves_per_block") == 0) {
    if (value < 0 || value > 4) return QKN_EINVAL;
    g_opt_waves_per_block = value;
  } else if (strcmp(key, "force_generic") == 0) {
    if (value != 0 && value != 1) return QKN_EINVAL;
    g_opt_force_generic = value;
  } else if (strcmp(key, "prefetch") == 0) {
    if (value != 0 && value != 1) return QKN_EINVAL;
    g_opt_prefetch = value;
  } else if (strcmp(key, "wait_schedule") == 0) {
    if (value < 0 || value > 4) return QKN_EINVAL;
    g_opt_wait_schedule = value;
  } else if (strcmp(key, "balance") == 0) {
    if (value != 0 && value != 1) return QKN_EINVAL;
    g_opt_balance = value;
  } else if (strcmp(key, "token_blocks") == 0) {
    if (value != 0 && value != 1) return QKN_EINVAL;
    g_opt_token_blocks = value;
  } else if (strcmp(key, "proj_tile") == 0) {
    return qkn_host::set_proj_tile(value);
  } else if (strcmp(key, "validate_only") == 0) {
    if (value != 0 && value != 1) return QKN_EINVAL;
    g_opt_validate_only = value;
  } else {
    return QKN_EINVAL;
  }
  return QKN_OK;
}

}  // extern "C"
