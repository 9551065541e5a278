// libqkn, part 2: column-parallel Q/K projection with Phase A in the epilogue
// (AMD MI355X, gfx950, CDNA4).
//
// y = bf16(x . W^T) for the rank's rows of the projection weight (Sec. II-B),
// and per token the fp32 sum of squares of the stored y row (Phase A,
// Sec. III-A / Alg. 1), taken from the output tile while it is on chip.
//
// Kernel design (gfx950):
//   * The contraction runs on the matrix cores, fp32 accumulation. Both
//     operands are k-contiguous (x is [T, hidden], W is [d_local, hidden]),
//     so one 16-byte vector of 8 k-values is exactly one lane's A or B
//     operand. Whole tiles use v_mfma_f32_16x16x32_bf16: lane l holds row
//     (l mod 16), k-values 8*(l/16) .. 8*(l/16)+7 of a 16 x 32 slab, and the
//     16x16 result block leaves column (l mod 16), rows 4*(l/16) + r in
//     accumulator r. A selectable whole-tile variant uses
//     v_mfma_f32_32x32x16_bf16: row (l mod 32), k-values 8*(l/32) .. +7 of a
//     32 x 16 slab; result column (l mod 32), rows 8*(r/4) + 4*(l/32) +
//     (r mod 4) in accumulator r. Both walk k in ascending order per output,
//     and the two instructions round their exact bf16 products identically:
//     the results are bit-identical (checked on every tested shape).
//   * A 256-thread workgroup owns a 128 x 128 output tile (four wavefronts in
//     2 x 2, 64 x 64 each = 4 x 4 or 2 x 2 MFMA blocks); k advances 64 at a time
//     through two LDS stages that global memory fills directly (buffer_load
//     ... lds, no VGPR staging): the loads of stage kt + 1 are in flight while
//     stage kt is computed, one barrier per stage. Instead of padding, each
//     row's 16-byte k-slots are XOR-swizzled so that the 16 rows a 16-lane
//     group reads land on 16 distinct bank groups. Two such workgroups (64 KB
//     of LDS each) share a CU. (Measured on MI355X against register-staged
//     double buffering, three- and four-stage rings, k of 32 and 128 per stage
//     and 256-wide tiles: this shape was the fastest; 16 x 16 x 32 MFMAs beat
//     32 x 32 x 16 ones by 4-9 %.)
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
//   * Decode-sized launches (at most 8 row tiles, which alone would leave most
//     CUs idle) split k: separate workgroups take contiguous k-slices of each
//     tile (64-row tiles up to 64 tokens; four LDS stages, so a slice's loads
//     are all in flight at once) and store their fp32 sums; one reduction
//     launch, a workgroup per token and segment, adds the slices in ascending order,
//     rounds once, writes y and takes the statistic with the same tree.

#include <hip/hip_runtime.h>

#include <stdint.h>
#include <string.h>

#include <mutex>

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

// Output tiles: a 256-thread workgroup (four wavefronts, 2 x 2) owns
// (64 WMB) x (64 WNB) outputs, each wavefront (32 WMB) x (32 WNB) as WMB x WNB
// MFMA blocks; k advances BK per LDS stage. The Phase A statistic is always
// taken over 128-column chunks of the output (kChunkN), whatever the tile
// width, so its summation tree does not depend on the tile shape.
constexpr int kThreads = 256;
constexpr int kChunkN = 128;              // columns per statistic chunk
constexpr int kGroupM = 8;                // row tiles per tile group
constexpr int kXcds = 8;                  // MI355X: workgroup id mod 8 selects the XCD
constexpr int kRsrcWord3 = 0x00020000;    // raw (untyped) buffer
constexpr int kLdsBytes = 160 * 1024;     // LDS per CU on gfx950

struct ProjSegDev {
  const uint16_t* w;
  uint16_t* y;
  float* tile_partials;  // [nchunks, T]: statistic of each 128-column chunk
  float* partials;       // [T]
  int64_t ldw, ldy;
  int32_t d;
  int32_t tile0;         // first column tile of this segment in the launch
  int32_t nchunks;       // ceil(d / 128)
  int32_t col0;          // split-k: first column of this segment in the partial sums
};

struct ProjParams {
  const uint16_t* x;
  int64_t ldx;
  int64_t T;
  int32_t hidden;
  int32_t m_tiles;       // row tiles (of the launch's tile height)
  int32_t n_tiles;       // column tiles of all segments
  int32_t nseg;
  ProjSegDev seg[2];
  // split-k (few tiles): k-slice s of every tile adds its fp32 products into
  // part[s][t][c], c over the columns of both segments (segment i's first
  // column at seg[i].col0)
  int32_t splits;        // 1: no split
  int32_t kslice;        // k per slice, a multiple of the stage k
  float* part;
  int32_t ncols;         // columns of both segments
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

// Tile in the grouped order -> (row tile, column tile): groups of kGroupM row
// tiles, each sweeping all column tiles.
__device__ __forceinline__ bool tile_from(int logical, int m_tiles, const ProjParams& p, int& mt,
                                          int& nt) {
  if (logical >= m_tiles * p.n_tiles) return false;
  const int group_size = kGroupM * p.n_tiles;
  const int group = logical / group_size;
  const int first_m = group * kGroupM;
  const int gm = (m_tiles - first_m < kGroupM) ? m_tiles - first_m : kGroupM;
  const int in_group = logical - group * group_size;
  mt = first_m + in_group % gm;
  nt = in_group / gm;
  return true;
}

// Tile number -> (row tile, column tile): XCD-contiguous runs, then groups of
// kGroupM row tiles sweeping all column tiles.
__device__ __forceinline__ bool tile_of(int bid, int grid, int m_tiles, const ProjParams& p, int& mt,
                                        int& nt) {
  const int per_xcd = grid / kXcds;  // the grid is a multiple of kXcds
  const int logical = (bid % kXcds) * per_xcd + bid / kXcds;
  return tile_from(logical, m_tiles, p, mt, nt);
}

// Epilogue of a (64 WMB) x (64 WNB) tile: round the fp32 accumulators once to
// bf16, stage the tile in LDS (`lds`, at least BM x OUT_ROW bf16; the caller
// has finished with it), write it to y with coalesced 16-byte stores, and
// take the Phase A statistic of each row's 128-column chunks.
template <int BM, int BN, int OUT_ROW>
__device__ __forceinline__ void epilogue_staged(const ProjParams& p, const ProjSegDev& s,
                                                const uint16_t* out, int64_t m0, int n0,
                                                int rows_a, int rows_b);

template <int WMB, int WNB, int OUT_ROW>
__device__ __forceinline__ void epilogue(const ProjParams& p, const ProjSegDev& s,
                                         const f32x16 (&acc)[WMB][WNB], uint16_t* lds, int64_t m0,
                                         int n0, int rows_a, int rows_b) {
  constexpr int BM = 64 * WMB, BN = 64 * WNB;
  const int tid = static_cast<int>(threadIdx.x);
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  uint16_t* out = lds;  // [BM][OUT_ROW]
#pragma unroll
  for (int i = 0; i < WMB; ++i)
#pragma unroll
    for (int j = 0; j < WNB; ++j) {
      const int col = wn * 32 * WNB + j * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; r += 2) {
        const int row = wm * 32 * WMB + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3);
        const uint32_t pk = pack_bf16x2(acc[i][j][r], acc[i][j][r + 1]);
        out[row * OUT_ROW + col] = static_cast<uint16_t>(pk & 0xffffu);
        out[(row + 1) * OUT_ROW + col] = static_cast<uint16_t>(pk >> 16);
      }
    }
  __syncthreads();
  epilogue_staged<BM, BN, OUT_ROW>(p, s, out, m0, n0, rows_a, rows_b);
}

// The same for 16 x 16 MFMA blocks: a wavefront's (32 WMB) x 64 share of the
// tile as (2 WMB) x 4 blocks; lane l holds column l mod 16 and rows
// 4 (l / 16) .. 4 (l / 16) + 3 of each block.
template <int WMB, int OUT_ROW>
__device__ __forceinline__ void epilogue16(const ProjParams& p, const ProjSegDev& s,
                                           const f32x4 (&acc)[2 * WMB][4], uint16_t* lds,
                                           int64_t m0, int n0, int rows_a, int rows_b) {
  const int tid = static_cast<int>(threadIdx.x);
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  uint16_t* out = lds;  // [64 WMB][OUT_ROW]
#pragma unroll
  for (int i = 0; i < 2 * WMB; ++i)
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int col = wn * 64 + j * 16 + (lane & 15);
#pragma unroll
      for (int r = 0; r < 4; r += 2) {
        const int row = wm * 32 * WMB + i * 16 + 4 * (lane >> 4) + r;
        const uint32_t pk = pack_bf16x2(acc[i][j][r], acc[i][j][r + 1]);
        out[row * OUT_ROW + col] = static_cast<uint16_t>(pk & 0xffffu);
        out[(row + 1) * OUT_ROW + col] = static_cast<uint16_t>(pk >> 16);
      }
    }
  __syncthreads();
  epilogue_staged<64 * WMB, 128, OUT_ROW>(p, s, out, m0, n0, rows_a, rows_b);
}

// Stores and statistic of a tile staged in LDS as bf16 ([BM][OUT_ROW]).
template <int BM, int BN, int OUT_ROW>
__device__ __forceinline__ void epilogue_staged(const ProjParams& p, const ProjSegDev& s,
                                                const uint16_t* out, int64_t m0, int n0,
                                                int rows_a, int rows_b) {
  const int tid = static_cast<int>(threadIdx.x);

  // coalesced 16-byte stores of the tile rows (columns past d_local skipped)
  const uint32_t y_bytes = static_cast<uint32_t>(rows_a * s.ldy * 2);
  const Rsrc ry = make_rsrc(s.y + m0 * s.ldy + n0, y_bytes);
  constexpr int kRowVecs = BN / 8;
#pragma unroll
  for (int i = 0; i < BM * kRowVecs / kThreads; ++i) {
    const int v = tid + kThreads * i;
    const int row = v / kRowVecs, cv = (v % kRowVecs) * 8;
    const u32x4 val = *reinterpret_cast<const u32x4*>(out + row * OUT_ROW + cv);
    st16(val, ry, cv < rows_b ? static_cast<uint32_t>((row * s.ldy + cv) * 2) : y_bytes);
  }

  // Phase A per 128-column chunk: thread pair (2u, 2u+1) takes one row of one
  // chunk, columns [0, 64) and [64, 128) of it in ascending order; the pair adds.
  constexpr int kUnits = BM * (BN / kChunkN) * 2;
  static_assert(kUnits % 64 == 0, "whole wavefronts of units");
#pragma unroll
  for (int it = 0; it < (kUnits + kThreads - 1) / kThreads; ++it) {
    const int u = tid + kThreads * it;
    const bool live = u < kUnits;  // a 64-row tile has units for half the threads
    const int half = u & 1, rc = u >> 1;
    const int row = rc % BM, chunk = rc / BM;
    const uint16_t* src = out + row * OUT_ROW + chunk * kChunkN + half * 64;
    float acc_s = 0.0f;
    if (live) {
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
    }
    // the partner lane's sum (quad_perm [1,0,3,2]: lanes 2u and 2u+1 swap)
    const float other = __builtin_bit_cast(
        float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, acc_s), 0xB1, 0xF, 0xF, false));
    const float first = half ? other : acc_s;
    const float second = half ? acc_s : other;
    const float chunk_sum = first + second;
    const int gchunk = n0 / kChunkN + chunk;  // chunk index within the segment
    if (live && half == 0 && row < rows_a && gchunk < s.nchunks)
      s.tile_partials[static_cast<int64_t>(gchunk) * p.T + m0 + row] = chunk_sum;
  }
}

template <int WMB, int WNB, int BK>
struct TileCfg {
  static constexpr int BM = 64 * WMB;                 // tile rows (tokens)
  static constexpr int BN = 64 * WNB;                 // tile columns
  static constexpr int kRow = BK + 8;                 // bf16 per staged operand row (padded)
  static constexpr int kStageA = BM * kRow;
  static constexpr int kStage = (BM + BN) * kRow;     // bf16 per LDS stage (A then B)
  static constexpr int kOutRow = BN + 8;              // bf16 per staged output row
  static constexpr int kLds = (2 * kStage > BM * kOutRow) ? 2 * kStage : BM * kOutRow;
  static constexpr int kKv = BK / 8;                  // 16-byte vectors per operand row
  static constexpr int kVecA = BM * kKv / kThreads;   // per thread per stage
  static constexpr int kVecB = BN * kKv / kThreads;
  static_assert(BM * kKv % kThreads == 0 && BN * kKv % kThreads == 0, "whole vectors per thread");
  static_assert(BN % kChunkN == 0, "tiles hold whole statistic chunks");
  static_assert(kLds * 2 <= kLdsBytes, "LDS");
};

// Register-staged kernel: each stage's operand tiles go global -> VGPRs ->
// LDS (rows padded to BK + 8 bf16, which spreads a 16-lane group's 16-byte
// reads over all 64 banks); the next stage's loads are issued before the
// current stage's MFMAs and written to the other LDS buffer after them. Kept as
// a second, independently staged implementation: it must give the same bits
// as the direct-to-LDS kernel (the k order of every accumulation is the same).
template <int WMB, int WNB, int BK>
__global__ __launch_bounds__(kThreads) void qkn_proj_gemm(const ProjParams p) {
  using C = TileCfg<WMB, WNB, BK>;
  __shared__ __align__(16) uint16_t lds[C::kLds];
  int mt, nt;
  if (!tile_of(static_cast<int>(blockIdx.x), static_cast<int>(gridDim.x), p.m_tiles, p, mt, nt))
    return;
  const int si = (p.nseg == 2 && nt >= p.seg[1].tile0) ? 1 : 0;
  const ProjSegDev& s = p.seg[si];
  const int64_t m0 = static_cast<int64_t>(mt) * C::BM;
  const int n0 = (nt - s.tile0) * C::BN;
  const int rows_a = static_cast<int>((p.T - m0 < C::BM) ? p.T - m0 : C::BM);
  const int rows_b = (s.d - n0 < C::BN) ? s.d - n0 : C::BN;

  const int tid = static_cast<int>(threadIdx.x);
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  // descriptors end at the last valid row: rows past it read zeros
  const uint32_t a_bytes = static_cast<uint32_t>(rows_a * p.ldx * 2);
  const uint32_t b_bytes = static_cast<uint32_t>(rows_b * s.ldw * 2);
  const Rsrc ra = make_rsrc(p.x + m0 * p.ldx, a_bytes);
  const Rsrc rb = make_rsrc(s.w + static_cast<int64_t>(n0) * s.ldw, b_bytes);

  // this thread's 16-byte vectors of each operand tile per stage
  uint32_t a_off[C::kVecA], b_off[C::kVecB];
  int a_lds[C::kVecA], b_lds[C::kVecB], a_k[C::kVecA], b_k[C::kVecB];
#pragma unroll
  for (int i = 0; i < C::kVecA; ++i) {
    const int v = tid + kThreads * i;
    const int row = v / C::kKv, kv = v % C::kKv;
    a_off[i] = static_cast<uint32_t>(row * p.ldx * 2);
    a_lds[i] = row * C::kRow + kv * 8;
    a_k[i] = kv * 8;
  }
#pragma unroll
  for (int i = 0; i < C::kVecB; ++i) {
    const int v = tid + kThreads * i;
    const int row = v / C::kKv, kv = v % C::kKv;
    b_off[i] = static_cast<uint32_t>(row * s.ldw * 2);
    b_lds[i] = C::kStageA + row * C::kRow + kv * 8;
    b_k[i] = kv * 8;
  }
  u32x4 ga[C::kVecA], gb[C::kVecB];
  auto load_stage = [&](int k0) {
#pragma unroll
    for (int i = 0; i < C::kVecA; ++i) {
      const int k = k0 + a_k[i];
      ga[i] = ld16(ra, k < p.hidden ? a_off[i] + static_cast<uint32_t>(k * 2) : a_bytes);
    }
#pragma unroll
    for (int i = 0; i < C::kVecB; ++i) {
      const int k = k0 + b_k[i];
      gb[i] = ld16(rb, k < p.hidden ? b_off[i] + static_cast<uint32_t>(k * 2) : b_bytes);
    }
  };
  auto store_stage = [&](int buf) {
    uint16_t* base = lds + buf * C::kStage;
#pragma unroll
    for (int i = 0; i < C::kVecA; ++i) *reinterpret_cast<u32x4*>(base + a_lds[i]) = ga[i];
#pragma unroll
    for (int i = 0; i < C::kVecB; ++i) *reinterpret_cast<u32x4*>(base + b_lds[i]) = gb[i];
  };

  f32x16 acc[WMB][WNB];
#pragma unroll
  for (int i = 0; i < WMB; ++i)
#pragma unroll
    for (int j = 0; j < WNB; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  const int nk = (p.hidden + BK - 1) / BK;
  load_stage(0);
  store_stage(0);
  __syncthreads();
  const int frag_row = lane & 31;
  const int frag_k = (lane >> 5) * 8;
  const int a_row0 = wm * 32 * WMB + frag_row;
  const int b_row0 = wn * 32 * WNB + frag_row;
  for (int kt = 0; kt < nk; ++kt) {
    const int cur = kt & 1;
    const bool more = kt + 1 < nk;
    if (more) load_stage((kt + 1) * BK);
    const uint16_t* a = lds + cur * C::kStage;
    const uint16_t* b = a + C::kStageA;
#pragma unroll
    for (int kk = 0; kk < BK; kk += 16) {
      bf16x8 af[WMB], bfr[WNB];
#pragma unroll
      for (int i = 0; i < WMB; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(a + (a_row0 + i * 32) * C::kRow + kk + frag_k);
#pragma unroll
      for (int j = 0; j < WNB; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(b + (b_row0 + j * 32) * C::kRow + kk + frag_k);
#pragma unroll
      for (int i = 0; i < WMB; ++i)
#pragma unroll
        for (int j = 0; j < WNB; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (more) store_stage(cur ^ 1);
    __syncthreads();
  }
  epilogue<WMB, WNB, C::kOutRow>(p, s, acc, lds, m0, n0, rows_a, rows_b);
}

// Accumulators of a wavefront's (32 WMB) x 64 share of a tile: MI x MI MFMA
// blocks, kM x kN of them, kR fp32 values per lane each.
template <int MI, int WMB>
struct AccOf;
template <int WMB>
struct AccOf<32, WMB> {
  static constexpr int kM = WMB, kN = 2, kR = 16;
  typedef f32x16 T[kM][kN];
};
template <int WMB>
struct AccOf<16, WMB> {
  static constexpr int kM = 2 * WMB, kN = 4, kR = 4;
  typedef f32x4 T[kM][kN];
};

// Direct-to-LDS variant: each stage's operand tiles go from global memory
// straight into LDS (buffer_load ... lds: lane l's 16 bytes land at the
// instruction's LDS base + 16 l), through a ring of S stages, so the loads of
// stage kt + S - 1 are in flight while stage kt is computed and no VGPRs stage
// the data. Rows are not padded; instead the 16-byte k-slot of each row is
// XOR-swizzled, slot' = slot ^ ((row / (16 / P)) mod P) with P = BK / 8 slots
// per row, which puts the 16 rows read by a 16-lane group at 16 distinct
// 16-byte bank groups. Lane l of a load instruction therefore fetches the
// global k-vector that belongs at its fixed LDS slot.
template <int WMB, int BK, int S>
struct DlCfg {
  static constexpr int BM = 64 * WMB, BN = 128;        // tile rows (tokens), columns
  static constexpr int P = BK / 8;                     // 16-byte slots per row
  static constexpr int kRowsPerGroup = 16 / P;         // rows sharing a swizzle value
  static constexpr int kRowBytes = BK * 2;
  static constexpr int kTileBytesA = BM * kRowBytes;
  static constexpr int kTileBytesB = BN * kRowBytes;
  static constexpr int kStageBytes = kTileBytesA + kTileBytesB;  // A then B
  static constexpr int kOutRow = BN + 8;
  static constexpr int kLdsBytes =
      (S * kStageBytes > BM * kOutRow * 2) ? S * kStageBytes : BM * kOutRow * 2;
  static constexpr int kLoadsA = kTileBytesA / 1024 / 4;  // 1 KB wave instructions per wave
  static constexpr int kLoadsB = kTileBytesB / 1024 / 4;
  static constexpr int kRowsPerLoad = 1024 / kRowBytes;
  static_assert(kTileBytesA % 4096 == 0 && kTileBytesB % 4096 == 0,
                "whole load instructions per wavefront");
  static_assert(kLdsBytes <= 160 * 1024, "LDS");
};

typedef __attribute__((address_space(3))) unsigned char LdsByte;

// Lane l's 16 bytes at byte offset `voff` of the buffer go to dst + 16 l (LDS).
// (Called through this helper: with the builtin written directly in a kernel
// body, the host compilation pass emitted no launch stub for the kernel.)
__device__ __forceinline__ void load16_to_lds(Rsrc r, LdsByte* dst, uint32_t voff) {
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, dst, 16, voff, 0, 0, 0);
}

// s_waitcnt vmcnt(n), lgkmcnt and expcnt left alone (gfx9 encoding: vmcnt bits
// [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8])
constexpr int vmcnt_imm(int n) { return 0x0F70 | (n & 15) | ((n >> 4) << 14); }

// Wait until at most n vector-memory requests of this wavefront are in flight
// (n is wavefront-uniform; the instruction takes the count as an immediate,
// so every count a caller can pass has its own case; larger counts wait for
// all).
__device__ __forceinline__ void vm_wait(int n) {
#define QKN_VM_CASE(k) \
  case k:              \
    __builtin_amdgcn_s_waitcnt(vmcnt_imm(k)); \
    break;
  switch (n) {
    QKN_VM_CASE(1) QKN_VM_CASE(2) QKN_VM_CASE(3) QKN_VM_CASE(4) QKN_VM_CASE(5) QKN_VM_CASE(6)
    QKN_VM_CASE(7) QKN_VM_CASE(8) QKN_VM_CASE(9) QKN_VM_CASE(10) QKN_VM_CASE(11) QKN_VM_CASE(12)
    QKN_VM_CASE(13) QKN_VM_CASE(14) QKN_VM_CASE(15) QKN_VM_CASE(16) QKN_VM_CASE(17)
    QKN_VM_CASE(18) QKN_VM_CASE(19) QKN_VM_CASE(20) QKN_VM_CASE(21) QKN_VM_CASE(22)
    QKN_VM_CASE(23) QKN_VM_CASE(24) QKN_VM_CASE(25) QKN_VM_CASE(26) QKN_VM_CASE(27)
    QKN_VM_CASE(28) QKN_VM_CASE(29) QKN_VM_CASE(30) QKN_VM_CASE(31) QKN_VM_CASE(32)
    QKN_VM_CASE(36) QKN_VM_CASE(40) QKN_VM_CASE(48) QKN_VM_CASE(56)
    default: __builtin_amdgcn_s_waitcnt(vmcnt_imm(0)); break;  // 0, and any count not listed
  }
#undef QKN_VM_CASE
}

// Main loop of one direct-to-LDS tile: BM = 64 WMB rows from m0 (rows_a of
// them valid) by 128 columns from n0 of segment s (rows_b valid), k in
// [k_lo, k_hi). Four wavefronts in a 2 x 2 grid, each (32 WMB) x 64, i.e.
// WMB x 2 MFMA blocks of 32 x 32 (MI = 32) or 2 WMB x 4 blocks of 16 x 16
// (MI = 16); every accumulator takes k in ascending order whatever the
// tile's height, so all tile shapes give the same bits.
template <int MI, int WMB, int BK, int S>
__device__ __forceinline__ void dl_mainloop(const ProjParams& p, const ProjSegDev& s,
                                            unsigned char* lds, int64_t m0, int n0, int rows_a,
                                            int rows_b, int k_lo, int k_hi,
                                            typename AccOf<MI, WMB>::T& acc) {
  using C = DlCfg<WMB, BK, S>;
  const int tid = static_cast<int>(threadIdx.x);
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  const uint32_t a_bytes = static_cast<uint32_t>(rows_a * p.ldx * 2);
  const uint32_t b_bytes = static_cast<uint32_t>(rows_b * s.ldw * 2);
  const Rsrc ra = make_rsrc(p.x + m0 * p.ldx, a_bytes);
  const Rsrc rb = make_rsrc(s.w + static_cast<int64_t>(n0) * s.ldw, b_bytes);

  // this lane's global row offset and k-vector for each of the wave's loads
  uint32_t a_row[C::kLoadsA], b_row[C::kLoadsB];
  int kva[C::kLoadsA], kvb[C::kLoadsB];
#pragma unroll
  for (int i = 0; i < C::kLoadsA; ++i) {
    const int row = (wave * C::kLoadsA + i) * C::kRowsPerLoad + lane / C::P;
    kva[i] = ((lane % C::P) ^ ((row / C::kRowsPerGroup) % C::P)) * 8;
    a_row[i] = static_cast<uint32_t>(row * p.ldx * 2);
  }
#pragma unroll
  for (int i = 0; i < C::kLoadsB; ++i) {
    const int row = (wave * C::kLoadsB + i) * C::kRowsPerLoad + lane / C::P;
    kvb[i] = ((lane % C::P) ^ ((row / C::kRowsPerGroup) % C::P)) * 8;
    b_row[i] = static_cast<uint32_t>(row * s.ldw * 2);
  }
  // Stage `stage` (k from k0) into its ring slot; a k-vector past k_hi is
  // moved past the descriptor and reads zeros.
#define QKN_ISSUE_STAGE(stage, k0)                                                          \
  do {                                                                                      \
    const int base_ = ((stage) % S) * C::kStageBytes;                                       \
    _Pragma("unroll") for (int i_ = 0; i_ < C::kLoadsA; ++i_) {                             \
      const int k_ = (k0) + kva[i_];                                                        \
      load16_to_lds(ra, (LdsByte*)(lds + base_ + (wave * C::kLoadsA + i_) * 1024),          \
                    k_ < k_hi ? a_row[i_] + static_cast<uint32_t>(k_ * 2) : a_bytes);        \
    }                                                                                       \
    _Pragma("unroll") for (int i_ = 0; i_ < C::kLoadsB; ++i_) {                             \
      const int k_ = (k0) + kvb[i_];                                                        \
      load16_to_lds(rb,                                                                     \
                    (LdsByte*)(lds + base_ + C::kTileBytesA + (wave * C::kLoadsB + i_) * 1024), \
                    k_ < k_hi ? b_row[i_] + static_cast<uint32_t>(k_ * 2) : b_bytes);        \
    }                                                                                       \
  } while (0)

  using A = AccOf<MI, WMB>;
#pragma unroll
  for (int i = 0; i < A::kM; ++i)
#pragma unroll
    for (int j = 0; j < A::kN; ++j)
#pragma unroll
      for (int r = 0; r < A::kR; ++r) acc[i][j][r] = 0.0f;

  const int nk = (k_hi - k_lo + BK - 1) / BK;
  // A k-range of at most S stages is requested whole before the first
  // MFMA (every stage has its own ring slot); a longer one keeps S - 1
  // stages in flight and requests the next into the slot just consumed.
  const int pre = nk <= S ? nk : S - 1;
#pragma unroll
  for (int st = 0; st < S; ++st)
    if (st < pre) QKN_ISSUE_STAGE(st, k_lo + st * BK);

  // MI = 32: lane l supplies row (l mod 32) of a 32-row block and k-values
  // 8 (l / 32) .. 8 (l / 32) + 7 of a 16-deep k-block; MI = 16: row (l mod 16)
  // of a 16-row block and k-values 8 (l / 16) .. 8 (l / 16) + 7 of 32
  const int frag_row = lane & (MI - 1);
  const int frag_kv = lane / MI;
  constexpr int kKBlock = 512 / MI;  // k per MFMA
  constexpr int kPerStage = C::kLoadsA + C::kLoadsB;  // load instructions per wave per stage
  for (int kt = 0; kt < nk; ++kt) {
    // the stages requested after stage kt may stay in flight
    const int later = (nk - 1 - kt < pre - 1) ? nk - 1 - kt : pre - 1;
    vm_wait(later * kPerStage);
    // A plain barrier, not __syncthreads(): its fence would wait for every
    // load in flight, the later stages' too. Each wavefront has waited for its
    // own part of stage kt (the DMA count drops once the data is in LDS), and
    // its reads of stage kt - 1 were consumed by MFMAs before it got here.
    __builtin_amdgcn_s_barrier();
    if (pre < nk && kt + S - 1 < nk) QKN_ISSUE_STAGE(kt + S - 1, k_lo + (kt + S - 1) * BK);
    const unsigned char* a = lds + (kt % S) * C::kStageBytes;
    const unsigned char* b = a + C::kTileBytesA;
#pragma unroll
    for (int kk = 0; kk < BK; kk += kKBlock) {
      const int kv = kk / 8 + frag_kv;
      bf16x8 af[A::kM], bfr[A::kN];
#pragma unroll
      for (int i = 0; i < A::kM; ++i) {
        const int ra_row = wm * 32 * WMB + i * MI + frag_row;
        af[i] = *reinterpret_cast<const bf16x8*>(
            a + ra_row * C::kRowBytes + ((kv ^ ((ra_row / C::kRowsPerGroup) % C::P)) * 16));
      }
#pragma unroll
      for (int j = 0; j < A::kN; ++j) {
        const int rb_row = wn * 64 + j * MI + frag_row;
        bfr[j] = *reinterpret_cast<const bf16x8*>(
            b + rb_row * C::kRowBytes + ((kv ^ ((rb_row / C::kRowsPerGroup) % C::P)) * 16));
      }
#pragma unroll
      for (int i = 0; i < A::kM; ++i)
#pragma unroll
        for (int j = 0; j < A::kN; ++j) {
          if constexpr (MI == 32)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
          else
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
        }
    }
  }
#undef QKN_ISSUE_STAGE
}

// The segment, origin and valid extent of output tile (row tile mt of height
// 64 WMB from row `row0`, column tile nt over both segments).
struct TileAt {
  int si;
  int64_t m0;
  int n0, rows_a, rows_b;
};
template <int WMB>
__device__ __forceinline__ TileAt tile_at(const ProjParams& p, int64_t row0, int mt, int nt) {
  // The tile numbers are uniform, but the integer divisions that produced
  // them run on the vector unit; without this the compiler can treat the
  // buffer descriptors built from them as per-lane values and wrap every
  // direct load in a loop over the lanes' descriptors.
  mt = __builtin_amdgcn_readfirstlane(mt);
  nt = __builtin_amdgcn_readfirstlane(nt);
  TileAt t;
  t.si = (p.nseg == 2 && nt >= p.seg[1].tile0) ? 1 : 0;
  const ProjSegDev& s = p.seg[t.si];
  t.m0 = row0 + static_cast<int64_t>(mt) * (64 * WMB);
  t.n0 = (nt - s.tile0) * 128;
  t.rows_a = static_cast<int>((p.T - t.m0 < 64 * WMB) ? p.T - t.m0 : 64 * WMB);
  t.rows_b = (s.d - t.n0 < 128) ? s.d - t.n0 : 128;
  return t;
}

// One whole tile with its epilogue.
template <int MI, int WMB, int BK, int S>
__device__ __forceinline__ void dl_tile(const ProjParams& p, unsigned char* lds, int64_t row0,
                                        int mt, int nt) {
  const TileAt t = tile_at<WMB>(p, row0, mt, nt);
  const ProjSegDev& s = p.seg[t.si];
  typename AccOf<MI, WMB>::T acc;
  dl_mainloop<MI, WMB, BK, S>(p, s, lds, t.m0, t.n0, t.rows_a, t.rows_b, 0, p.hidden, acc);
  __syncthreads();
  if constexpr (MI == 32)
    epilogue<WMB, 2, DlCfg<WMB, BK, S>::kOutRow>(p, s, acc, reinterpret_cast<uint16_t*>(lds),
                                                 t.m0, t.n0, t.rows_a, t.rows_b);
  else
    epilogue16<WMB, DlCfg<WMB, BK, S>::kOutRow>(p, s, acc, reinterpret_cast<uint16_t*>(lds),
                                                t.m0, t.n0, t.rows_a, t.rows_b);
}

// Whole 128 x 128 tiles, XCD-aware order.
template <int MI, int BK, int S>
__global__ __launch_bounds__(kThreads) void qkn_proj_gemm_dl(const ProjParams p) {
  __shared__ __align__(1024) unsigned char lds[DlCfg<2, BK, S>::kLdsBytes];
  int mt, nt;
  if (!tile_of(static_cast<int>(blockIdx.x), static_cast<int>(gridDim.x), p.m_tiles, p, mt, nt))
    return;
  dl_tile<MI, 2, BK, S>(p, lds, 0, mt, nt);
}

// Split k: workgroup b takes k-slice b mod splits of tile b / splits (tiles
// of 64 WMB rows) and stores its fp32 sums into the slice array instead of
// running the epilogue.
template <int WMB, int BK, int S>
__global__ __launch_bounds__(kThreads) void qkn_proj_gemm_split(const ProjParams p) {
  constexpr int MI = 16;  // 16 x 16 x 32 MFMAs (same bits as 32 x 32 x 16, 1-2 % faster here)
  using C = DlCfg<WMB, BK, S>;
  __shared__ __align__(1024) unsigned char lds[C::kLdsBytes];
  const int b = static_cast<int>(blockIdx.x);
  int mt, nt;
  if (!tile_from(b / p.splits, p.m_tiles, p, mt, nt)) return;
  const int ks = b % p.splits;
  const int k_lo = ks * p.kslice;
  const int k_hi = (k_lo + p.kslice < p.hidden) ? k_lo + p.kslice : p.hidden;
  const TileAt t = tile_at<WMB>(p, 0, mt, nt);
  const ProjSegDev& s = p.seg[t.si];
  using A = AccOf<MI, WMB>;
  typename A::T acc;
  dl_mainloop<MI, WMB, BK, S>(p, s, lds, t.m0, t.n0, t.rows_a, t.rows_b, k_lo, k_hi, acc);
  // fp32 sums of this k-slice, through LDS: the accumulators (lanes 0..MI-1
  // of a row hold MI adjacent columns) go to an fp32 tile in LDS, which is
  // then written out row by row in 16-byte vectors (4-byte stores straight
  // from the accumulators scatter every wave instruction over 4 rows).
  const int tid = static_cast<int>(threadIdx.x);
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  constexpr int kBM = C::BM, kBN = C::BN;
  constexpr int kRow = kBN + 4;  // padded: the four 16-lane row groups of a write use other banks
  static_assert(kBM * kRow * 4 <= C::kLdsBytes, "the fp32 tile fits in the stage buffers");
  float* tile = reinterpret_cast<float*>(lds);
  __syncthreads();  // every wavefront is done reading the stages
#pragma unroll
  for (int i = 0; i < A::kM; ++i)
#pragma unroll
    for (int j = 0; j < A::kN; ++j) {
      const int col = wn * 64 + j * MI + (lane & (MI - 1));
#pragma unroll
      for (int r = 0; r < A::kR; ++r) {
        const int row = (MI == 32)
            ? wm * 32 * WMB + i * 32 + 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3)
            : wm * 32 * WMB + i * 16 + 4 * (lane >> 4) + r;
        tile[row * kRow + col] = acc[i][j][r];
      }
    }
  __syncthreads();
  // a row's valid columns are a multiple of 8 (d_local is), and its first
  // column's offset in the slice array is a multiple of 8 floats, so every
  // vector is whole and 16-byte aligned
  float* part = p.part + static_cast<int64_t>(ks) * p.T * p.ncols + t.m0 * p.ncols + s.col0 + t.n0;
  constexpr int kVecs = kBN / 4;
  for (int q = tid; q < kBM * kVecs; q += kThreads) {
    const int row = q / kVecs, c4 = (q % kVecs) * 4;
    if (row < t.rows_a && c4 < t.rows_b)
      *reinterpret_cast<f32x4*>(part + static_cast<int64_t>(row) * p.ncols + c4) =
          *reinterpret_cast<const f32x4*>(tile + row * kRow + c4);
  }
}

// Split-k reduction, one workgroup per token and segment (the segments'
// statistics are separate sums, so Q and K run on different CUs), one
// wavefront per 128-column chunk (wavefront w takes chunks w, w + waves,
// ...): each lane adds two
// columns' k-slice sums in ascending slice order and rounds them once to bf16
// (y); the chunk's statistic follows the tile epilogue's tree (two ascending
// FMA chains over the chunk's halves, first + second); after a barrier the
// chunk statistics of each segment are added in ascending chunk order.
constexpr int kMaxSplitChunks = 2048;  // 128-column chunks of both segments
constexpr int kMaxSplits = 16;         // slices: (row tiles) x (slices) <= 16
constexpr int kReduceWaves = 16;
template <int SPLITS>
__global__ __launch_bounds__(64 * kReduceWaves) void qkn_proj_reduce(const ProjParams p) {
  __shared__ float vals[kReduceWaves][kChunkN];
  __shared__ float chunk_sum[kMaxSplitChunks];
  const int64_t t = blockIdx.x;
  const int si = static_cast<int>(blockIdx.y);
  const ProjSegDev& s = p.seg[si];
  const int tid = static_cast<int>(threadIdx.x);
  const int lane = tid & 63, wave = tid >> 6;
  const int waves = static_cast<int>(blockDim.x) >> 6;
  const int64_t slice = p.T * p.ncols;
  float* v = vals[wave];
  for (int q = wave; q < s.nchunks; q += waves) {
    const int c = q * kChunkN + 2 * lane;  // d_local is a multiple of 8: c < d means c + 1 < d
    float v0 = 0.0f, v1 = 0.0f;
    if (c < s.d) {
      const float* src = p.part + t * p.ncols + s.col0 + c;
      f32x2 b[SPLITS];  // every slice's load in flight before the first add
#pragma unroll
      for (int k = 0; k < SPLITS; ++k) b[k] = *reinterpret_cast<const f32x2*>(src + k * slice);
      f32x2 a = b[0];
#pragma unroll
      for (int k = 1; k < SPLITS; ++k) {
        a[0] = a[0] + b[k][0];
        a[1] = a[1] + b[k][1];
      }
      const uint32_t pk = pack_bf16x2(a[0], a[1]);
      *reinterpret_cast<uint32_t*>(s.y + t * s.ldy + c) = pk;
      v0 = bf16_lo(pk);
      v1 = bf16_hi(pk);
    }
    v[2 * lane] = v0;  // columns past d_local hold 0, which adds nothing
    v[2 * lane + 1] = v1;
    // the wavefront's own LDS row: a wavefront-scope fence orders the writes
    // before the other lanes' reads (no workgroup barrier in a loop whose
    // trip count differs between wavefronts)
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();
    const float* h = v + (lane & 1) * 64;
    float acc_s = 0.0f;
#pragma unroll 16
    for (int i = 0; i < 64; ++i) acc_s = __builtin_fmaf(h[i], h[i], acc_s);
    const float other = __builtin_bit_cast(
        float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, acc_s), 0xB1, 0xF, 0xF, false));
    if (lane == 0) chunk_sum[q] = acc_s + other;
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    __builtin_amdgcn_wave_barrier();  // the row is read before the next chunk overwrites it
  }
  __syncthreads();
  if (tid == 0) {
    float S = chunk_sum[0];
    for (int n = 1; n < s.nchunks; ++n) S = S + chunk_sum[n];
    s.partials[t] = S;
  }
}

// partials[t] = chunk statistics of token t added in ascending chunk order.
// The loads go out sixteen at a time before their sums (a plain loop waited
// for each load before the next add: 6.0 us for the prefill shard, 4.6 us
// batched).
__global__ __launch_bounds__(256) void qkn_proj_finish(const ProjParams p) {
  constexpr int kBatch = 16;
  const int64_t t = static_cast<int64_t>(blockIdx.x) * blockDim.x + threadIdx.x;
  const int si = static_cast<int>(blockIdx.y);
  if (t >= p.T || si >= p.nseg) return;
  const ProjSegDev& s = p.seg[si];
  const float* src = s.tile_partials + t;
  const int nc = s.nchunks;
  float S = 0.0f;
  for (int n = 0; n < nc; n += kBatch) {
    float v[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j)
      v[j] = (n + j < nc) ? src[static_cast<int64_t>(n + j) * p.T] : 0.0f;
#pragma unroll
    for (int j = 0; j < kBatch; ++j)
      if (n + j < nc) S = (n + j == 0) ? v[j] : S + v[j];  // chunk 0 starts the sum
  }
  s.partials[t] = S;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

int64_t chunks_of(int64_t d) { return (d + kChunkN - 1) / kChunkN; }

typedef void (*GemmFn)(ProjParams);

// Tile shapes: (rows, columns, k per stage) of a workgroup's tile.
struct TileShape {
  GemmFn fn;
  int bm, bn, bk;
  int lds_bytes;
  const char* name;
};
#define QKN_TILE(WM, WN, BK, NAME)                                                        \
  TileShape {                                                                             \
    qkn_proj_gemm<WM, WN, BK>, 64 * WM, 64 * WN, BK,                                     \
        static_cast<int>(TileCfg<WM, WN, BK>::kLds * sizeof(uint16_t)), NAME              \
  }
#define QKN_DL(MI, BK, S, NAME) \
  TileShape { qkn_proj_gemm_dl<MI, BK, S>, 128, 128, BK, DlCfg<2, BK, S>::kLdsBytes, NAME }
// [0] is the default (measured fastest on MI355X: 128 x 128 tiles, k 64 per
// stage, two LDS stages filled directly from global memory, two workgroups
// per CU, 16 x 16 x 32 MFMAs); [1] is the register-staged kernel and [2] the
// direct-to-LDS kernel on 32 x 32 x 16 MFMAs, both kept as second and third
// implementations of the same sums (same bits).
const TileShape kTiles[] = {QKN_DL(16, 64, 2, "proj<128x128,64,dl2,mi16>"),
                            QKN_TILE(2, 2, 64, "proj<128x128,64,reg>"),
                            QKN_DL(32, 64, 2, "proj<128x128,64,dl2>")};
constexpr int kNumTiles = sizeof(kTiles) / sizeof(kTiles[0]);

// Choice of tile shape (benchmarks), per calling thread as every option:
// 0 = automatic, i = kTiles[i - 1].
thread_local int g_tile_choice = 0;

const TileShape& choose_tile() {
  if (g_tile_choice > 0 && g_tile_choice <= kNumTiles) return kTiles[g_tile_choice - 1];
  return kTiles[0];
}

// Split-k (k-slices of a tile in separate workgroups, added by a reduction)
// for decode-sized launches, whose row tiles alone would leave most CUs idle:
// at most kSplitMaxRowTiles row tiles (1024 tokens). The slice count is the
// largest power of two with (row tiles) x (slices) <= kSplitRowSlices and
// slices at least 128 deep. It depends on T and hidden only -- not on the
// columns or the segments (launches of more than kMaxSplitChunks 128-column
// chunks in all, 262144 columns, are not split) -- so Q and K launched
// together or apart, and any device, give the same bits.
constexpr int64_t kSplitMaxRowTiles = 8;
constexpr int64_t kSplitRowSlices = kMaxSplits;
constexpr int kSplitBk = 64;
constexpr int kSplitStages = 4;  // a 256-deep slice has all its loads in flight at once

struct Plan {
  int64_t m_tiles, n_tiles, chunks, ncols;
  int splits, kslice;
  int64_t ws_bytes;
};

Plan plan_of(int64_t T, int64_t hidden, const qkn_proj_seg* segs, int nseg) {
  Plan pl{};
  pl.m_tiles = (T + 127) / 128;
  for (int i = 0; i < nseg; ++i) {
    pl.n_tiles += (segs[i].d_local + 127) / 128;
    pl.chunks += chunks_of(segs[i].d_local);
    pl.ncols += segs[i].d_local;
  }
  pl.splits = 1;
  pl.kslice = static_cast<int>(hidden);
  if (g_tile_choice == 0 && pl.m_tiles <= kSplitMaxRowTiles && pl.chunks <= kMaxSplitChunks) {
    int splits = 1;
    while (pl.m_tiles * splits * 2 <= kSplitRowSlices && hidden >= int64_t{128} * splits * 2)
      splits *= 2;
    if (splits > 1) {
      // slices of ceil(hidden / splits) rounded up to a multiple of 8: all
      // `splits` of them non-empty, since hidden / splits >= 128 > 7 (splits - 1)
      const int64_t per = (hidden + splits - 1) / splits;
      pl.kslice = static_cast<int>((per + 7) / 8 * 8);
      pl.splits = splits;
    }
  }
  pl.ws_bytes = pl.splits > 1 ? 4 * int64_t{pl.splits} * T * pl.ncols  // slice sums
                              : 4 * T * pl.chunks;                    // chunk statistics

  return pl;
}

// ---------------------------------------------------------------- workspace without allocation
//
// The entry point for callers that cannot allocate (HIP graph capture, tight
// serving loops) takes its workspace from this fixed device array instead of
// an argument. Each GPU the library runs on holds its own copy, from the
// first such call until the process ends. Host code never passes the array's
// name to a kernel or a copy (on the host that name is a stand-in, not a
// device address): it asks the runtime for the array's address on each device
// once, with that device current, and passes that address.
constexpr int64_t kScratchBytes = QKN_PROJ_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];

constexpr int kMaxScratchDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_ptr[kMaxScratchDevices] = {};

// The current device's address of `scratch`, looked up on its first use.
int scratch_address(void** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxScratchDevices) return QKN_EHIP;
  std::lock_guard<std::mutex> lock(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* ptr = nullptr;
    if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return QKN_EHIP;
    g_scratch_ptr[dev] = ptr;
  }
  *out = g_scratch_ptr[dev];
  return QKN_OK;
}

// qkn_proj_partial's body. use_scratch: the workspace is `scratch` (its
// address resolved only once the call is valid and about to launch), and
// `workspace` / `workspace_bytes` are ignored.
int proj_impl(const uint16_t* x, int64_t ldx, int64_t T, int64_t hidden,
              const qkn_proj_seg* segs, int nseg, void* workspace, int64_t workspace_bytes,
              bool use_scratch, void* stream) {
  if (!segs || nseg < 1 || nseg > 2 || T < 0 || hidden < 1 || ldx < hidden) return QKN_EINVAL;
  for (int i = 0; i < nseg; ++i) {
    const qkn_proj_seg& s = segs[i];
    if (s.d_local < 1 || s.ldw < hidden || s.ldy < s.d_local) return QKN_EINVAL;
  }
  if (T == 0) return QKN_OK;
  if (!x) return QKN_EINVAL;
  for (int i = 0; i < nseg; ++i)
    if (!segs[i].w || !segs[i].y || !segs[i].partials) return QKN_EINVAL;
  const Plan pl = plan_of(T, hidden, segs, nseg);
  const int64_t need = pl.ws_bytes;
  if (use_scratch) {
    if (need > kScratchBytes) return QKN_ENOTSUP;  // beyond the fixed workspace
  } else if (!workspace || workspace_bytes < need) {
    return QKN_EINVAL;
  }

  // the MFMA path's shape and alignment requirements
  const int64_t lim = int64_t{1} << 31;
  if (!aligned16(x) || (!use_scratch && !aligned16(workspace)) || hidden % 8 || ldx % 8 ||
      T * ldx * 2 >= lim || hidden > (int64_t{1} << 30))
    return QKN_ENOTSUP;
  for (int i = 0; i < nseg; ++i) {
    const qkn_proj_seg& s = segs[i];
    if (!aligned16(s.w) || !aligned16(s.y) || s.ldw % 8 || s.ldy % 8 || s.d_local % 8 ||
        s.d_local * s.ldw * 2 >= lim || int64_t{256} * s.ldy * 2 >= lim)
      return QKN_ENOTSUP;
  }

  // overlap: outputs (y, partials, a caller's workspace) against inputs and each other
  Span items[8];
  bool out[8];
  int n = 0;
  items[n] = Span{reinterpret_cast<uintptr_t>(x), T, ldx, hidden, 2};
  out[n++] = false;
  if (!use_scratch) {
    items[n] = Span{reinterpret_cast<uintptr_t>(workspace), 1, need, need, 1};
    out[n++] = true;
  }
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

  const TileShape& ts = choose_tile();
  const bool split = pl.splits > 1;
  ProjParams p;
  memset(&p, 0, sizeof(p));
  p.x = x;
  p.ldx = ldx;
  p.T = T;
  p.hidden = static_cast<int32_t>(hidden);
  p.m_tiles = static_cast<int32_t>((T + ts.bm - 1) / ts.bm);
  p.nseg = nseg;
  p.splits = pl.splits;
  p.kslice = pl.kslice;
  p.ncols = static_cast<int32_t>(pl.ncols);
  int64_t ws_off[2] = {0, 0};  // floats into the workspace of each segment's chunk statistics
  int32_t tile0 = 0, col0 = 0;
  int64_t off = 0;
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
    d.col0 = col0;
    d.nchunks = static_cast<int32_t>(chunks_of(s.d_local));
    ws_off[i] = off;
    if (!split) off += static_cast<int64_t>(d.nchunks) * T;
    tile0 += static_cast<int32_t>((s.d_local + 127) / 128);  // every kernel's tiles are 128 wide
    col0 += static_cast<int32_t>(s.d_local);
  }
  p.n_tiles = tile0;
  const auto round8 = [](int64_t v) { return (v + kXcds - 1) / kXcds * kXcds; };
  const int64_t max_wgs = 0x7fffffff - 2 * kXcds;
  int64_t grid = 0;
  const char* name = ts.name;
  int lds = ts.lds_bytes;
  const void* gemm = reinterpret_cast<const void*>(ts.fn);
  if (split) {
    // 64-row tiles when every token fits in one: half the A loads and MFMAs
    const bool half = T <= 64;
    p.m_tiles = static_cast<int32_t>(half ? 1 : (T + 127) / 128);
    const int64_t tiles = static_cast<int64_t>(p.m_tiles) * p.n_tiles;
    if (tiles * pl.splits > max_wgs) return QKN_ENOTSUP;
    grid = tiles * pl.splits;
    if (half) {
      gemm = reinterpret_cast<const void*>(qkn_proj_gemm_split<1, kSplitBk, kSplitStages>);
      name = "proj<64x128,64,dl4,splitk>";
      lds = DlCfg<1, kSplitBk, kSplitStages>::kLdsBytes;
    } else {
      gemm = reinterpret_cast<const void*>(qkn_proj_gemm_split<2, kSplitBk, kSplitStages>);
      name = "proj<128x128,64,dl4,splitk>";
      lds = DlCfg<2, kSplitBk, kSplitStages>::kLdsBytes;
    }
  } else {
    const int64_t tiles = static_cast<int64_t>(p.m_tiles) * p.n_tiles;
    if (tiles > max_wgs) return QKN_ENOTSUP;
    grid = round8(tiles);
  }
  const qkn_launch_info info{name, grid, kThreads, grid * (kThreads / 64), lds};
  if (qkn_host::validate_only()) {
    qkn_host::record_launch(qkn_launch_info{info.kernel, 0, 0, 0, info.lds_bytes});
    return QKN_EDRYRUN;
  }
  if (use_scratch) {
    const int rc = scratch_address(&workspace);
    if (rc != QKN_OK) return rc;
  }
  float* ws = static_cast<float*>(workspace);
  p.part = split ? ws : nullptr;
  for (int i = 0; i < nseg; ++i) p.seg[i].tile_partials = split ? nullptr : ws + ws_off[i];
  hipStream_t st = static_cast<hipStream_t>(stream);
  void* args[] = {&p};
  if (hipLaunchKernel(gemm, dim3(static_cast<unsigned>(grid)), dim3(kThreads), args, 0, st) !=
      hipSuccess)
    return QKN_EHIP;
  if (split) {
    int64_t most = 0;  // chunks of the widest segment: one wavefront each, up to kReduceWaves
    for (int i = 0; i < nseg; ++i) most = p.seg[i].nchunks > most ? p.seg[i].nchunks : most;
    const int waves = most < kReduceWaves ? static_cast<int>(most) : kReduceWaves;
    const void* reduce = pl.splits == 2   ? reinterpret_cast<const void*>(qkn_proj_reduce<2>)
                         : pl.splits == 4 ? reinterpret_cast<const void*>(qkn_proj_reduce<4>)
                         : pl.splits == 8 ? reinterpret_cast<const void*>(qkn_proj_reduce<8>)
                                          : reinterpret_cast<const void*>(qkn_proj_reduce<16>);
    if (hipLaunchKernel(reduce, dim3(static_cast<unsigned>(T), static_cast<unsigned>(nseg)),
                        dim3(64 * waves), args, 0, st) != hipSuccess)
      return QKN_EHIP;
  } else {
    const dim3 fgrid(static_cast<unsigned>((T + 255) / 256), static_cast<unsigned>(nseg));
    if (hipLaunchKernel(reinterpret_cast<const void*>(qkn_proj_finish), fgrid, dim3(256), args,
                        0, st) != hipSuccess)
      return QKN_EHIP;
  }
  qkn_host::record_launch(info);
  return QKN_OK;
}

}  // namespace

namespace qkn_host {
int set_proj_tile(int64_t choice) {
  if (choice < 0 || choice > kNumTiles) return QKN_EINVAL;
  g_tile_choice = static_cast<int>(choice);
  return QKN_OK;
}
}  // namespace qkn_host

extern "C" {

int64_t qkn_proj_workspace_bytes(int64_t T, int64_t hidden, const qkn_proj_seg* segs, int nseg) {
  if (!segs || nseg < 1 || nseg > 2 || T < 0 || hidden < 1) return QKN_EINVAL;
  for (int i = 0; i < nseg; ++i)
    if (segs[i].d_local < 1) return QKN_EINVAL;
  return plan_of(T, hidden, segs, nseg).ws_bytes;
}

int qkn_proj_partial(const uint16_t* x, int64_t ldx, int64_t T, int64_t hidden,
                     const qkn_proj_seg* segs, int nseg, void* workspace,
                     int64_t workspace_bytes, void* stream) {
  return proj_impl(x, ldx, T, hidden, segs, nseg, workspace, workspace_bytes, false, stream);
}

int qkn_proj_partial_noalloc(const uint16_t* x, int64_t ldx, int64_t T, int64_t hidden,
                             const qkn_proj_seg* segs, int nseg, void* stream) {
  return proj_impl(x, ldx, T, hidden, segs, nseg, nullptr, 0, true, stream);
}

}  // extern "C"
