// libqkn, part 2: column-parallel Q/K projection with Phase A in the epilogue
// (AMD MI355X, gfx950, CDNA4).
//
// y = bf16(x . W^T) for the rank's rows of the projection weight (Sec. II-B),
// and per token the fp32 sum of squares of the stored y row (Phase A,
// Sec. III-A / Alg. 1), taken from the output tile while it is on chip.
//
// Kernel design (gfx950):
//   * The contraction runs on the matrix cores: v_mfma_f32_32x32x16_bf16,
//     fp32 accumulation. Both operands are k-contiguous (x is [T, hidden],
//     W is [d_local, hidden]), so one 16-byte vector of 8 k-values is exactly
//     one lane's A or B operand: lane l holds row (l mod 32), k-values
//     8*(l/32) .. 8*(l/32)+7 of a 32 x 16 slab; the 32x32 result block leaves
//     column (l mod 32), rows 8*(r/4) + 4*(l/32) + (r mod 4) in accumulator r.
//   * A 256-thread workgroup owns a 128 x 128 output tile (four wavefronts in
//     2 x 2, 64 x 64 each = 2 x 2 MFMA blocks); k advances 64 at a time
//     through two LDS stages: the next stage's global loads are issued before
//     the current stage's MFMAs and written to the other LDS buffer after
//     them, one barrier per stage. LDS rows are padded to 144 bytes, which
//     spreads a 16-lane group's 16-byte reads over all 64 banks.
//   * Global loads are raw buffer loads whose descriptors end at the last
//     valid row, so rows past T or d_local read zeros; the k tail (hidden not
//     a multiple of 64) is masked by moving the offset out of range.
//   * Tiles are numbered so that each XCD (workgroup id mod 8 on MI355X) takes
//     a contiguous run of them, in groups of 8 row tiles sweeping the column
//     tiles: concurrently running tiles of one XCD share x rows and W rows in
//     its L2.
//   * Epilogue: the fp32 tile is rounded to bf16 once, staged in LDS, written
//     to y with coalesced 16-byte stores, and each row's statistic over the
//     tile's 128 columns is summed from the staged bf16 values (two ascending
//     FMA chains of 64 columns, added). A second launch adds the per-tile
//     statistics of each token in ascending tile order.

#include <hip/hip_runtime.h>

#include <stdint.h>
#include <string.h>

#include "qkn_proj.h"
#include "qkn_host.h"

namespace {

using qkn_host::Span;
using qkn_host::spans_overlap;

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __amdgpu_buffer_rsrc_t Rsrc;

constexpr int kBM = 128;                  // output rows (tokens) per tile
constexpr int kBN = 128;                  // output columns per tile
constexpr int kBK = 64;                   // k per LDS stage
constexpr int kThreads = 256;             // four wavefronts, 2 x 2 over the tile
constexpr int kLdsRow = kBK + 8;          // bf16 per staged row (144 bytes)
constexpr int kStage = kBM * kLdsRow;     // bf16 per staged operand tile
constexpr int kOutRow = kBN + 8;          // bf16 per staged output row (272 bytes)
constexpr int kGroupM = 8;                // row tiles per tile group
constexpr int kXcds = 8;                  // MI355X: workgroup id mod 8 selects the XCD
constexpr int kRsrcWord3 = 0x00020000;    // raw (untyped) buffer

static_assert(kBM * kOutRow <= 4 * kStage, "the output tile reuses the operand stages");

struct ProjSegDev {
  const uint16_t* w;
  uint16_t* y;
  float* tile_partials;  // [ntiles, T]
  float* partials;       // [T]
  int64_t ldw, ldy;
  int32_t d;
  int32_t tile0;         // first column tile of this segment in the launch
  int32_t ntiles;
};

struct ProjParams {
  const uint16_t* x;
  int64_t ldx;
  int64_t T;
  int32_t hidden;
  int32_t m_tiles;
  int32_t n_tiles;       // column tiles of all segments
  int32_t nseg;
  ProjSegDev seg[2];
};

__device__ __forceinline__ Rsrc make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                           static_cast<int>(bytes), kRsrcWord3);
}

__device__ __forceinline__ u32x4 ld16(Rsrc r, uint32_t off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

__device__ __forceinline__ void st16(u32x4 v, Rsrc r, uint32_t off) {
  __builtin_amdgcn_raw_buffer_store_b128(
      __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(r, 0, 0, 0)), v), r, off,
      0, 0);
}

__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(f32x2{lo, hi}, bf16x2));
}

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __builtin_bit_cast(float, u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) {
  return __builtin_bit_cast(float, u & 0xffff0000u);
}

// Tile number -> (row tile, column tile): XCD-contiguous runs, then groups of
// kGroupM row tiles sweeping all column tiles.
__device__ __forceinline__ bool tile_of(int bid, int grid, const ProjParams& p, int& mt, int& nt) {
  const int per_xcd = grid / kXcds;  // the grid is a multiple of kXcds
  const int logical = (bid % kXcds) * per_xcd + bid / kXcds;
  if (logical >= p.m_tiles * p.n_tiles) return false;
  const int group_size = kGroupM * p.n_tiles;
  const int group = logical / group_size;
  const int first_m = group * kGroupM;
  const int gm = (p.m_tiles - first_m < kGroupM) ? p.m_tiles - first_m : kGroupM;
  const int in_group = logical - group * group_size;
  mt = first_m + in_group % gm;
  nt = in_group / gm;
  return true;
}

__global__ __launch_bounds__(kThreads) void qkn_proj_gemm(const ProjParams p) {
  __shared__ __align__(16) uint16_t lds[4 * kStage];  // [stage][A, B][row][k]
  int mt, nt;
  if (!tile_of(static_cast<int>(blockIdx.x), static_cast<int>(gridDim.x), p, mt, nt)) return;
  const int si = (p.nseg == 2 && nt >= p.seg[1].tile0) ? 1 : 0;
  const ProjSegDev& s = p.seg[si];
  const int64_t m0 = static_cast<int64_t>(mt) * kBM;
  const int n0 = (nt - s.tile0) * kBN;
  const int rows_a = static_cast<int>((p.T - m0 < kBM) ? p.T - m0 : kBM);
  const int rows_b = (s.d - n0 < kBN) ? s.d - n0 : kBN;

  const int tid = static_cast<int>(threadIdx.x);
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // descriptors end at the last valid row: rows past it read zeros
  const uint32_t a_bytes = static_cast<uint32_t>(rows_a * p.ldx * 2);
  const uint32_t b_bytes = static_cast<uint32_t>(rows_b * s.ldw * 2);
  const Rsrc ra = make_rsrc(p.x + m0 * p.ldx, a_bytes);
  const Rsrc rb = make_rsrc(s.w + static_cast<int64_t>(n0) * s.ldw, b_bytes);

  // this thread's four 16-byte vectors of each operand tile per stage
  uint32_t a_row_off[4], b_row_off[4];
  int lds_off[4];
  int kv8[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int v = tid + kThreads * i;
    const int row = v >> 3, kv = v & 7;
    a_row_off[i] = static_cast<uint32_t>(row * p.ldx * 2);
    b_row_off[i] = static_cast<uint32_t>(row * s.ldw * 2);
    lds_off[i] = row * kLdsRow + kv * 8;
    kv8[i] = kv * 8;
  }
  u32x4 ga[4], gb[4];
  auto load_stage = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const bool in_k = k0 + kv8[i] < p.hidden;
      const uint32_t ko = static_cast<uint32_t>((k0 + kv8[i]) * 2);
      ga[i] = ld16(ra, in_k ? a_row_off[i] + ko : a_bytes);
      gb[i] = ld16(rb, in_k ? b_row_off[i] + ko : b_bytes);
    }
  };
  auto store_stage = [&](int buf) {
    uint16_t* a = lds + buf * 2 * kStage;
    uint16_t* b = a + kStage;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<u32x4*>(a + lds_off[i]) = ga[i];
      *reinterpret_cast<u32x4*>(b + lds_off[i]) = gb[i];
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = (p.hidden + kBK - 1) / kBK;
  load_stage(0);
  store_stage(0);
  __syncthreads();
  const int frag_row = lane & 31;
  const int frag_k = (lane >> 5) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) load_stage((kt + 1) * kBK);
    const uint16_t* a = lds + cur * 2 * kStage;
    const uint16_t* b = a + kStage;
#pragma unroll
    for (int kk = 0; kk < kBK; kk += 16) {
      bf16x8 af[2], bfr[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        af[i] = *reinterpret_cast<const bf16x8*>(
            a + (wm * 64 + i * 32 + frag_row) * kLdsRow + kk + frag_k);
        bfr[i] = *reinterpret_cast<const bf16x8*>(
            b + (wn * 64 + i * 32 + frag_row) * kLdsRow + kk + frag_k);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (more) store_stage(cur ^ 1);
    __syncthreads();
  }

  // ---- epilogue: round once to bf16, stage the tile in LDS
  uint16_t* out = lds;  // [kBM][kOutRow]
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = wn * 64 + j * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        const int row = wm * 64 + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const uint32_t pk = pack_bf16x2(acc[i][j][r], acc[i][j][r + 1]);
        out[row * kOutRow + col] = static_cast<uint16_t>(pk & 0xffffu);
        out[(row + 1) * kOutRow + col] = static_cast<uint16_t>(pk >> 16);
      }
    }
  __syncthreads();

  // coalesced 16-byte stores of the tile rows (columns past d_local skipped)
  const uint32_t y_bytes = static_cast<uint32_t>(rows_a * s.ldy * 2);
  const Rsrc ry = make_rsrc(s.y + m0 * s.ldy + n0, y_bytes);
#pragma unroll
  for (int i = 0; i < (kBM * kBN / 8) / kThreads; ++i) {
    const int v = tid + kThreads * i;
    const int row = v >> 4, cv = (v & 15) * 8;
    const u32x4 val = *reinterpret_cast<const u32x4*>(out + row * kOutRow + cv);
    const bool ok = cv < rows_b;  // rows_b = valid columns of this tile
    st16(val, ry, ok ? static_cast<uint32_t>((row * s.ldy + cv) * 2) : y_bytes);
  }

  // Phase A over the tile's columns: thread pair (2r, 2r+1) takes row r,
  // columns [0, 64) and [64, 128) in ascending order; the pair then adds.
  {
    const int row = tid >> 1, half = tid & 1;
    const uint16_t* src = out + row * kOutRow + half * 64;
    float acc_s = 0.0f;
#pragma unroll
    for (int c = 0; c < 64; c += 8) {
      const u32x4 v = *reinterpret_cast<const u32x4*>(src + c);
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const float lo = bf16_lo(v[e]), hi = bf16_hi(v[e]);
        acc_s = __builtin_fmaf(lo, lo, acc_s);
        acc_s = __builtin_fmaf(hi, hi, acc_s);
      }
    }
    // the partner lane's sum (quad_perm [1,0,3,2]: lanes 2r and 2r+1 swap)
    const float other = __builtin_bit_cast(
        float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, acc_s), 0xB1, 0xF, 0xF, false));
    const float first = half ? other : acc_s;
    const float second = half ? acc_s : other;
    const float tile_sum = first + second;
    if (half == 0 && row < rows_a)
      s.tile_partials[static_cast<int64_t>(nt - s.tile0) * p.T + m0 + row] = tile_sum;
  }
}

// partials[t] = tile statistics of token t added in ascending tile order.
__global__ __launch_bounds__(256) void qkn_proj_finish(const ProjParams p) {
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int si = static_cast<int>(blockIdx.y);
  if (t >= p.T || si >= p.nseg) return;
  const ProjSegDev& s = p.seg[si];
  float S = s.tile_partials[t];
  for (int n = 1; n < s.ntiles; ++n) S = S + s.tile_partials[static_cast<int64_t>(n) * p.T + t];
  s.partials[t] = S;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int64_t tiles_of(int64_t d) { return (d + kBN - 1) / kBN; }

}  // namespace

extern "C" {

int64_t qkn_proj_workspace_bytes(int64_t T, const qkn_proj_seg* segs, int nseg) {
  if (!segs || nseg < 1 || nseg > 2 || T < 0) return QKN_EINVAL;
  int64_t tiles = 0;
  for (int i = 0; i < nseg; ++i) {
    if (segs[i].d_local < 1) return QKN_EINVAL;
    tiles += tiles_of(segs[i].d_local);
  }
  return 4 * T * tiles;
}

int qkn_proj_partial(const uint16_t* x, int64_t ldx, int64_t T, int64_t hidden,
                     const qkn_proj_seg* segs, int nseg, void* workspace,
                     int64_t workspace_bytes, void* stream) {
  if (!segs || nseg < 1 || nseg > 2 || T < 0 || hidden < 1 || ldx < hidden) return QKN_EINVAL;
  for (int i = 0; i < nseg; ++i) {
    const qkn_proj_seg& s = segs[i];
    if (s.d_local < 1 || s.ldw < hidden || s.ldy < s.d_local) return QKN_EINVAL;
  }
  if (T == 0) return QKN_OK;
  if (!x) return QKN_EINVAL;
  for (int i = 0; i < nseg; ++i)
    if (!segs[i].w || !segs[i].y || !segs[i].partials) return QKN_EINVAL;
  const int64_t need = qkn_proj_workspace_bytes(T, segs, nseg);
  if (!workspace || workspace_bytes < need) return QKN_EINVAL;

  // the MFMA path's shape and alignment requirements
  const int64_t lim = int64_t{1} << 31;
  if (!aligned16(x) || !aligned16(workspace) || hidden % 8 || ldx % 8 || T * ldx * 2 >= lim ||
      hidden > (int64_t{1} << 30))
    return QKN_ENOTSUP;
  for (int i = 0; i < nseg; ++i) {
    const qkn_proj_seg& s = segs[i];
    if (!aligned16(s.w) || !aligned16(s.y) || s.ldw % 8 || s.ldy % 8 || s.d_local % 8 ||
        s.d_local * s.ldw * 2 >= lim || int64_t{kBM} * s.ldy * 2 >= lim)
      return QKN_ENOTSUP;
  }

  // overlap: outputs (y, partials, workspace) against inputs and each other
  Span items[8];
  bool out[8];
  int n = 0;
  items[n] = Span{reinterpret_cast<uintptr_t>(x), T, ldx, hidden, 2};
  out[n++] = false;
  items[n] = Span{reinterpret_cast<uintptr_t>(workspace), 1, need, need, 1};
  out[n++] = true;
  for (int i = 0; i < nseg; ++i) {
    const qkn_proj_seg& s = segs[i];
    items[n] = Span{reinterpret_cast<uintptr_t>(s.w), s.d_local, s.ldw, hidden, 2};
    out[n++] = false;
    items[n] = Span{reinterpret_cast<uintptr_t>(s.y), T, s.ldy, s.d_local, 2};
    out[n++] = true;
    items[n] = Span{reinterpret_cast<uintptr_t>(s.partials), 1, T, T, 4};
    out[n++] = true;
  }
  for (int a = 0; a < n; ++a)
    for (int b = a + 1; b < n; ++b)
      if ((out[a] || out[b]) && spans_overlap(items[a], items[b])) return QKN_EOVERLAP;

  ProjParams p;
  memset(&p, 0, sizeof(p));
  p.x = x;
  p.ldx = ldx;
  p.T = T;
  p.hidden = static_cast<int32_t>(hidden);
  p.m_tiles = static_cast<int32_t>((T + kBM - 1) / kBM);
  p.nseg = nseg;
  float* ws = static_cast<float*>(workspace);
  int32_t tile0 = 0;
  for (int i = 0; i < nseg; ++i) {
    const qkn_proj_seg& s = segs[i];
    ProjSegDev& d = p.seg[i];
    d.w = s.w;
    d.y = s.y;
    d.partials = s.partials;
    d.ldw = s.ldw;
    d.ldy = s.ldy;
    d.d = static_cast<int32_t>(s.d_local);
    d.tile0 = tile0;
    d.ntiles = static_cast<int32_t>(tiles_of(s.d_local));
    d.tile_partials = ws;
    ws += static_cast<int64_t>(d.ntiles) * T;
    tile0 += d.ntiles;
  }
  p.n_tiles = tile0;
  const int64_t tiles = static_cast<int64_t>(p.m_tiles) * p.n_tiles;
  if (tiles > 0x7fffffff - kXcds) return QKN_ENOTSUP;
  const int64_t grid = (tiles + kXcds - 1) / kXcds * kXcds;
  const qkn_launch_info info{"proj<128,128>/gemm+phase_a", grid, kThreads, grid * (kThreads / 64),
                             static_cast<int64_t>(4 * kStage * sizeof(uint16_t))};
  if (qkn_host::validate_only()) {
    qkn_host::record_launch(qkn_launch_info{info.kernel, 0, 0, 0, info.lds_bytes});
    return QKN_OK;
  }
  hipStream_t st = static_cast<hipStream_t>(stream);
  void* args[] = {&p};
  if (hipLaunchKernel(reinterpret_cast<const void*>(qkn_proj_gemm), dim3(static_cast<unsigned>(grid)),
                      dim3(kThreads), args, 0, st) != hipSuccess)
    return QKN_EHIP;
  const dim3 fgrid(static_cast<unsigned>((T + 255) / 256), static_cast<unsigned>(nseg));
  if (hipLaunchKernel(reinterpret_cast<const void*>(qkn_proj_finish), fgrid, dim3(256), args, 0, st) !=
      hipSuccess)
    return QKN_EHIP;
  qkn_host::record_launch(info);
  return QKN_OK;
}

}  // extern "C"
