// libqkn: sharded layerwise QK-Norm for AMD MI355X (gfx950, CDNA4, wave64).
//
// What is computed (SwiftQK, arXiv 2608.09160): RMSNorm of Eq. 1 (Sec. II-A)
// applied to each token's full projected Q and, separately, K vector, when the
// hidden dimension is split over tensor-parallel ranks (Sec. II-B). One rank's
// share follows the three phases of Sec. III / Alg. 1:
//   Phase A  partial sum of squares of the rank's slice, fp32;
//   Phase B  ascending-rank sum of all ranks' partials and the factor
//            1/sqrt(S/H_total + eps); independently of it, x * gamma;
//   Phase C  the scaled slice, rounded once to bf16 and written.
//
// Design for gfx950 (the paper's warp/block layout is prior art, not reused):
//   * One wavefront owns one token at a time: its Q row and K row are spread
//     over the 64 lanes in 16-byte chunks (8 bf16), chunk c on lane c % 64, so
//     the row reduction needs no LDS and no barrier: four DPP row steps and
//     four readlanes.
//   * The rows stay in registers between Phase A and Phase C (one HBM read of
//     x, one write of y); gamma is loaded into registers once per wavefront and
//     reused for every token of the persistent loop.
//   * The other ranks' statistics are fetched by lanes 0..tp-1 together with
//     the row, so their latency overlaps Phase A and the x * gamma products.
//   * The grid is persistent: at most (resident waves per CU) x (CU count)
//     wavefronts, each striding over tokens (Sec. III-D bounds the grid the
//     same way, there for deadlock safety across GPUs).
//   * x and y are streamed with non-temporal 128-bit accesses.
//   * A general kernel covers any width, stride and alignment with the same
//     summation tree (so the same bits), staging the row in LDS.
//
// Summation tree of a row (fixed, depends only on d_local): lane l
// accumulates, with fused multiply-adds in ascending column order, the
// elements of chunks l, l+64, l+128, ...; the 16 lanes of each DPP row are then
// combined by symmetric butterflies (every lane of a row ends with the same
// bits) and the four row sums r0..r3 are added as (r0 + r1) + (r2 + r3).

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdio.h>
#include <stdint.h>
#include <string.h>

#include <mutex>

#include "qkn.h"

namespace {

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kChunk = 8;           // bf16 elements per 128-bit access
constexpr int kMaxRegChunks = 8;    // chunks per lane held in registers (d_local <= 4096)
constexpr int kMaxFastTp = kWave;   // one statistic slot per lane
constexpr int kMaxStageBytes = 64 * 1024;
// Grid sizing of the register path (measured on MI355X: HBM throughput peaks
// with few, long-lived wavefronts per CU rather than full occupancy).
constexpr int64_t kInFlightBytes = 24 * 1024;
constexpr int64_t kMinWavesPerCu = 6;

// kFusedWait: fused, with the other ranks' statistics published concurrently
// as flagged slots that the kernel waits for; kPublish: Phase A into flagged slots.
enum Mode { kFused = 0, kApply = 1, kPartial = 2, kFusedWait = 3, kPublish = 4 };

struct DevSeg {
  const uint16_t* x;
  const float* w;
  float* partials;  // [tp * T], rank-major
  uint16_t* y;
  float* inv_rms;   // optional [T]
  int64_t ldx;
  int64_t ldy;
  int32_t d;        // d_local
  int32_t nchunks;  // ceil(d_local / 8)
  float d_full;     // divisor of the mean (H_total)
  int32_t vec;      // 128-bit accesses allowed
};

struct KParams {
  DevSeg seg[2];
  uint64_t* slots[2];  // flagged slots [tp * T] per segment (wait/publish modes)
  int32_t* status;     // wait mode: set to 1 when a wait gives up
  int64_t spin_limit;  // wait mode: polls per slot
  uint32_t epoch;      // wait/publish modes: the flag of this round
  int32_t group;       // wait mode: > 1 = every rank of the group in this launch
  int64_t T;
  int64_t tok_chunk;  // 0: wave w takes tokens w, w + W, ...; else [w*chunk, (w+1)*chunk)
  int32_t nseg;
  int32_t tp;
  int32_t rank;
  float eps;
};

// ------------------------------------------------------------------ device helpers

__device__ __forceinline__ float bf16_lo(uint32_t u) { return __builtin_bit_cast(float, u << 16); }
__device__ __forceinline__ float bf16_hi(uint32_t u) { return __builtin_bit_cast(float, u & 0xffff0000u); }
__device__ __forceinline__ float bf16_to_f32(uint16_t b) {
  return __builtin_bit_cast(float, static_cast<uint32_t>(b) << 16);
}

// Two fp32 values -> two bf16 (round to nearest even; v_cvt_pk_bf16_f32), low half first.
__device__ __forceinline__ uint32_t pack_bf16x2(float lo, float hi) {
  f32x2 v = {lo, hi};
  return __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
}
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
  return static_cast<uint16_t>(pack_bf16x2(f, 0.0f) & 0xffffu);
}

// Phase A on one 8-element chunk, ascending column order.
__device__ __forceinline__ float chunk_sumsq(u32x4 v, float acc) {
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    const float a = bf16_lo(v[e]);
    const float b = bf16_hi(v[e]);
    acc = __builtin_fmaf(a, a, acc);
    acc = __builtin_fmaf(b, b, acc);
  }
  return acc;
}

template <int CTRL>
__device__ __forceinline__ float dpp_move(float v) {
  return __builtin_bit_cast(
      float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF, false));
}

__device__ __forceinline__ float read_lane(float v, int lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}

// Sum over the 64 lanes; every lane must be active. Returns a wave-uniform value.
__device__ __forceinline__ float wave_sum(float v) {
  v = v + dpp_move<0xB1>(v);   // quad_perm [1,0,3,2]: lane pairs
  v = v + dpp_move<0x4E>(v);   // quad_perm [2,3,0,1]: quads
  v = v + dpp_move<0x141>(v);  // row_half_mirror: 8 lanes
  v = v + dpp_move<0x140>(v);  // row_mirror: 16 lanes
  const float r0 = read_lane(v, 0), r1 = read_lane(v, 16);
  const float r2 = read_lane(v, 32), r3 = read_lane(v, 48);
  return (r0 + r1) + (r2 + r3);
}

// Lanes 0..tp-1 fetch rank k's slot of token t; the slot `skip` (the rank's
// own, computed in this kernel) is not read.
__device__ __forceinline__ float load_slots(const float* partials, int64_t T, int64_t t,
                                            int lane, int tp, int skip) {
  float v = 0.0f;
  if (lane < tp && lane != skip) v = partials[static_cast<int64_t>(lane) * T + t];
  return v;
}

// Phase B reduction: S = P_0 + P_1 + ... + P_{tp-1}, left to right in fp32,
// with P_own taken from the register `own` (own < 0: every slot from memory).
__device__ __forceinline__ float combine_slots(float slots, float own, int tp, int own_rank) {
  float S = (own_rank == 0) ? own : read_lane(slots, 0);
  for (int k = 1; k < tp; ++k) {
    const float pk = (k == own_rank) ? own : read_lane(slots, k);
    S = S + pk;
  }
  return S;
}

// tp > 64: slot k lives on lane k % 64 of batch k / 64; batches are fetched in turn.
__device__ __forceinline__ float combine_slots_any(const float* partials, int64_t T, int64_t t,
                                                   int lane, int tp, float own, int own_rank) {
  float S = 0.0f;
  for (int k0 = 0; k0 < tp; k0 += kWave) {
    const int n = (tp - k0 < kWave) ? tp - k0 : kWave;
    const int skip = (own_rank >= k0 && own_rank < k0 + n) ? own_rank - k0 : -1;
    float v = 0.0f;
    if (lane < n && lane != skip) v = partials[static_cast<int64_t>(k0 + lane) * T + t];
    for (int i = 0; i < n; ++i) {
      const float pk = (i == skip) ? own : read_lane(v, i);
      S = (k0 == 0 && i == 0) ? pk : S + pk;
    }
  }
  return S;
}

__device__ __forceinline__ float rms_inverse(float S, float d_full, float eps) {
  return 1.0f / sqrtf(S / d_full + eps);
}

__device__ __forceinline__ int64_t wave_index() {
  const int w = static_cast<int>(blockIdx.x) * static_cast<int>(blockDim.x / kWave) +
                static_cast<int>(threadIdx.x / kWave);
  return __builtin_amdgcn_readfirstlane(w);
}

// ------------------------------------------------------------------ register path
//
// Every memory access of the register path is a raw buffer access whose
// descriptor covers exactly the valid bytes (built per row in scalar
// registers; the row base is wave-uniform). Lanes whose chunk lies past the end
// read zeros and their stores are dropped by the hardware range check, so no
// access sits behind a branch and the compiler can count outstanding requests
// exactly (a wait for the current token does not also wait for the next one).

typedef __amdgpu_buffer_rsrc_t Rsrc;
constexpr int kRsrcWord3 = 0x00020000;  // raw (untyped) buffer, gfx9 family
#ifndef QKN_LOAD_CPOL
#define QKN_LOAD_CPOL 2  // non-temporal
#endif
#ifndef QKN_STORE_CPOL
#define QKN_STORE_CPOL 18  // non-temporal, system scope (sc1 nt): measured best for y
#endif
constexpr int kLoadCpol = QKN_LOAD_CPOL;    // cache policy of the streamed x
constexpr int kStoreCpol = QKN_STORE_CPOL;  // cache policy of the streamed y

__device__ __forceinline__ Rsrc make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), static_cast<short>(0),
                                           static_cast<int>(bytes), kRsrcWord3);
}

// Descriptor of `bytes` bytes at base + byte offset `off`; an empty one when base is NULL.
__device__ __forceinline__ Rsrc make_rsrc_at(const void* base, int64_t off, uint32_t bytes) {
  const uintptr_t b = reinterpret_cast<uintptr_t>(base);
  return make_rsrc(reinterpret_cast<const void*>(b ? b + off : 0), b ? bytes : 0u);
}

__device__ __forceinline__ u32x4 ld16(Rsrc r, int off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}
__device__ __forceinline__ u32x4 ld16_nt(Rsrc r, int off) {
  return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kLoadCpol));
}
__device__ __forceinline__ void st16_nt(u32x4 v, Rsrc r, int off) {
  __builtin_amdgcn_raw_buffer_store_b128(
      __builtin_bit_cast(decltype(__builtin_amdgcn_raw_buffer_load_b128(r, 0, 0, 0)), v), r, off,
      0, kStoreCpol);
}
__device__ __forceinline__ float ld4f(Rsrc r, int off) {
  return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
}
// Lane 0 stores v at the descriptor's first word; other lanes are out of range.
__device__ __forceinline__ void st4f_lane0(float v, Rsrc r, int lane) {
  __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(uint32_t, v), r, lane == 0 ? 0 : 4, 0,
                                        0);
}

template <int N>
__device__ __forceinline__ void load_gamma(const DevSeg& s, int64_t col, int lane,
                                           f32x4 (&g)[N][2]) {
  const Rsrc r = make_rsrc(s.w + col, static_cast<uint32_t>(s.nchunks) * 32u);
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const int c = i * kWave + lane;
    g[i][0] = __builtin_bit_cast(f32x4, ld16(r, c * 32));
    g[i][1] = __builtin_bit_cast(f32x4, ld16(r, c * 32 + 16));
  }
}

// `live` false: an empty descriptor -- every lane reads zeros, nothing is fetched.
template <int N>
__device__ __forceinline__ void load_row(const DevSeg& s, int64_t col, int64_t t, int lane,
                                         u32x4 (&x)[N], bool live = true) {
  const Rsrc r = make_rsrc(s.x + t * s.ldx + col, live ? static_cast<uint32_t>(s.nchunks) * 16u : 0u);
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = ld16_nt(r, (i * kWave + lane) * 16);
}

// Lanes 0..tp-1 fetch rank k's statistic slot of token t (offset k*T words
// from slot t of rank 0); the rank's own slot `skip` and lanes >= tp are out of
// range and read 0. The register path requires tp * T * 4 < 2^31.
__device__ __forceinline__ float load_slots_buf(const float* partials, int64_t T, int64_t t,
                                                int lane, int tp, int skip, bool live = true) {
  const uint32_t nrec = static_cast<uint32_t>((tp - 1) * T * 4 + 4);
  const Rsrc r = make_rsrc_at(partials, t * 4, live ? nrec : 0u);
  const int off = (lane < tp && lane != skip) ? static_cast<int>(lane * T * 4)
                                              : static_cast<int>(nrec);
  return ld4f(r, off);
}

template <int N>
__device__ __forceinline__ float row_lane_sumsq(const u32x4 (&x)[N]) {
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < N; ++i) acc = chunk_sumsq(x[i], acc);
  return acc;
}

// Phase B compute path: z = x * gamma, elementwise in fp32.
template <int N>
__device__ __forceinline__ void times_gamma(const u32x4 (&x)[N], const f32x4 (&g)[N][2],
                                            float (&z)[N][8]) {
#pragma unroll
  for (int i = 0; i < N; ++i) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const f32x4& gg = g[i][e >> 1];
      z[i][2 * e] = bf16_lo(x[i][e]) * gg[(2 * e) & 3];
      z[i][2 * e + 1] = bf16_hi(x[i][e]) * gg[(2 * e + 1) & 3];
    }
  }
}

// Phase C: y = bf16(z * inv), non-temporal 128-bit stores.
template <int N>
__device__ __forceinline__ void store_scaled(const DevSeg& s, int64_t col, int64_t t, int lane,
                                             const float (&z)[N][8], float inv) {
  const Rsrc r = make_rsrc(s.y + t * s.ldy + col, static_cast<uint32_t>(s.nchunks) * 16u);
#pragma unroll
  for (int i = 0; i < N; ++i) {
    u32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = pack_bf16x2(z[i][2 * e] * inv, z[i][2 * e + 1] * inv);
    st16_nt(o, r, (i * kWave + lane) * 16);
  }
}

// ------------------------------------------------------------------ flagged slots
//
// A published statistic is one 8-byte word: fp32 bits in the low half, the
// round's epoch in the high half, written by a single aligned 64-bit store, so
// a reader that sees the epoch also sees the value (no separate flag or fence).

__device__ __forceinline__ void publish_slot(uint64_t* slot, float v, uint32_t epoch) {
  const uint64_t word = (static_cast<uint64_t>(epoch) << 32) | __builtin_bit_cast(uint32_t, v);
  __hip_atomic_store(slot, word, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Lanes 0..tp-1 other than `rank` poll rank k's slot of token t until it
// carries `epoch`, at most `limit` times (with a short sleep between polls).
// A lane that gives up, or any lane once `given_up` is set, returns NaN.
// `first` is the slot's word as read when the token's rows were requested (see
// poll_slots); only a lane whose slot was not ready yet polls again.
__device__ __forceinline__ float wait_slot(const uint64_t* slots, int64_t T, int64_t t, int lane,
                                           int tp, int rank, uint32_t epoch, int64_t limit,
                                           bool given_up, uint64_t first, bool& gave_up_now) {
  float v = 0.0f;
  if (lane < tp && lane != rank) {
    v = __builtin_nanf("");
    if (!given_up) {
      const uint64_t* slot = slots + static_cast<int64_t>(lane) * T + t;
      uint64_t word = first;
      for (int64_t n = 1;;) {
        if (static_cast<uint32_t>(word >> 32) == epoch) {
          v = __builtin_bit_cast(float, static_cast<uint32_t>(word));
          break;
        }
        if (n++ >= limit) {
          gave_up_now = true;
          break;
        }
        __builtin_amdgcn_s_sleep(1);
        word = __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
      }
    }
  }
  return v;
}

// First poll of the other ranks' slots of token t, issued with the token's rows:
// lanes 0..tp-1 (not `rank`) read slot lane*T + t with one 64-bit agent-coherent
// load each (the same single-copy-atomic access as the relaxed atomic load);
// other lanes are out of range and read 0, which no epoch matches.
constexpr int kCoherentCpol = 16;  // sc1: bypass the CU-local cache
__device__ __forceinline__ uint64_t poll_slots(const uint64_t* slots, int64_t T, int64_t t,
                                               int lane, int tp, int rank, bool live) {
  const uint32_t nrec = static_cast<uint32_t>(((tp - 1) * T + 1) * 8);
  const Rsrc r = make_rsrc_at(slots, t * 8, live ? nrec : 0u);
  const int off = (lane < tp && lane != rank) ? static_cast<int>(lane * T * 8)
                                              : static_cast<int>(nrec);
  return __builtin_bit_cast(uint64_t, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kCoherentCpol));
}

// The rank a wavefront computes and where that rank's slice sits: the launch's
// rank with no offsets, or, when one launch runs every rank of a group, rank
// w mod tp with its columns [rank*d_local, (rank+1)*d_local) of full tensors.
struct WaveSlice {
  int rank;
  int64_t col0, col1;  // column offset of the slice in segment 0 / 1
  int64_t inv_row;     // offset (in tokens) of this rank's factors in inv_rms
};

// Registers of one token in flight: its Q and K chunks and its statistic slots.
template <int N0, int M1>
struct TokenRegs {
  u32x4 x0[N0];
  u32x4 x1[M1];
  float slots0;
  float slots1;
  uint64_t word0;  // wait mode: first poll of the other ranks' slots
  uint64_t word1;
};

// `live` false (a pipelined request past the last token): nothing is fetched.
template <int N0, int N1, int MODE>
__device__ __forceinline__ void fetch_token(const KParams& p, const WaveSlice& ws, int64_t t,
                                            int lane, int own_rank,
                                            TokenRegs<N0, (N1 > 0 ? N1 : 1)>& r,
                                            bool live = true) {
  load_row<N0>(p.seg[0], ws.col0, t, lane, r.x0, live);
  if constexpr (N1 > 0) load_row<N1>(p.seg[1], ws.col1, t, lane, r.x1, live);
  r.slots0 = 0.0f;
  r.slots1 = 0.0f;
  if constexpr (MODE == kFused || MODE == kApply) {
    // with tp == 1 (fused) every lane is out of range: nothing is read
    r.slots0 = load_slots_buf(p.seg[0].partials, p.T, t, lane, p.tp, own_rank, live);
    if constexpr (N1 > 0)
      r.slots1 = load_slots_buf(p.seg[1].partials, p.T, t, lane, p.tp, own_rank, live);
  }
  if constexpr (MODE == kFusedWait) {
    r.word0 = poll_slots(p.slots[0], p.T, t, lane, p.tp, own_rank, live);
    r.word1 = 0;
    if constexpr (N1 > 0) r.word1 = poll_slots(p.slots[1], p.T, t, lane, p.tp, own_rank, live);
  }
}

// Phases A, B and C of token t, whose rows and slots are in `r`.
template <int N0, int N1, int MODE>
__device__ __forceinline__ void process_token(const KParams& p, const WaveSlice& ws, int64_t t,
                                              int lane, int own_rank, const f32x4 (&g0)[N0][2],
                                              const f32x4 (&g1)[(N1 > 0 ? N1 : 1)][2],
                                              const TokenRegs<N0, (N1 > 0 ? N1 : 1)>& r,
                                              bool& given_up) {
  constexpr int M1 = N1 > 0 ? N1 : 1;
  const DevSeg& s0 = p.seg[0];
  const DevSeg& s1 = p.seg[1];

  // Phase A: per-lane partial sums (not needed when every slot is given).
  float a0 = 0.0f, a1 = 0.0f;
  if constexpr (MODE != kApply) {
    a0 = row_lane_sumsq<N0>(r.x0);
    if constexpr (N1 > 0) a1 = row_lane_sumsq<N1>(r.x1);
  }

  if constexpr (MODE == kPartial) {
    const float own0 = wave_sum(a0);
    st4f_lane0(own0, make_rsrc_at(s0.partials, t * 4, 4u), lane);
  } else if constexpr (MODE == kPublish) {
    const float own0 = wave_sum(a0);
    if (lane == 0) publish_slot(p.slots[0] + t, own0, p.epoch);
  } else {
    float own0 = 0.0f, own1 = 0.0f;
    if constexpr (MODE == kFused || MODE == kFusedWait) {
      own0 = wave_sum(a0);
      if constexpr (N1 > 0) own1 = wave_sum(a1);
    }
    if constexpr (MODE == kFusedWait) {
      // publish this rank's statistics before waiting for the others'
      if (lane == 0) {
        publish_slot(p.slots[0] + static_cast<int64_t>(ws.rank) * p.T + t, own0, p.epoch);
        if constexpr (N1 > 0)
          publish_slot(p.slots[1] + static_cast<int64_t>(ws.rank) * p.T + t, own1, p.epoch);
      }
    }

    // Phase B, compute path: independent of the statistic.
    float z0[N0][8];
    float z1[M1][8];
    times_gamma<N0>(r.x0, g0, z0);
    if constexpr (N1 > 0) times_gamma<N1>(r.x1, g1, z1);

    // Phase B, reduction path.
    float slots0 = r.slots0, slots1 = r.slots1;
    if constexpr (MODE == kFusedWait) {
      bool gave_up = false;
      slots0 = wait_slot(p.slots[0], p.T, t, lane, p.tp, ws.rank, p.epoch, p.spin_limit, given_up,
                         r.word0, gave_up);
      if constexpr (N1 > 0)
        slots1 = wait_slot(p.slots[1], p.T, t, lane, p.tp, ws.rank, p.epoch, p.spin_limit,
                           given_up || gave_up, r.word1, gave_up);
      if (__ballot(gave_up) != 0) {
        if (!given_up && lane == 0)
          __hip_atomic_store(p.status, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
        given_up = true;  // later tokens of this wavefront do not wait again
      }
    }
    const float S0 = combine_slots(slots0, own0, p.tp, own_rank);
    const float inv0 = rms_inverse(S0, s0.d_full, p.eps);
    float inv1 = 0.0f;
    if constexpr (N1 > 0) {
      const float S1 = combine_slots(slots1, own1, p.tp, own_rank);
      inv1 = rms_inverse(S1, s1.d_full, p.eps);
    }

    // Phase C.
    store_scaled<N0>(s0, ws.col0, t, lane, z0, inv0);
    if constexpr (N1 > 0) store_scaled<N1>(s1, ws.col1, t, lane, z1, inv1);
    const int64_t own_slot = (static_cast<int64_t>(ws.rank) * p.T + t) * 4;
    if constexpr (MODE == kFused) {
      st4f_lane0(own0, make_rsrc_at(s0.partials, own_slot, 4u), lane);
      if constexpr (N1 > 0) st4f_lane0(own1, make_rsrc_at(s1.partials, own_slot, 4u), lane);
    }
    st4f_lane0(inv0, make_rsrc_at(s0.inv_rms, (ws.inv_row + t) * 4, 4u), lane);
    if constexpr (N1 > 0) st4f_lane0(inv1, make_rsrc_at(s1.inv_rms, (ws.inv_row + t) * 4, 4u), lane);
  }
}

// Persistent register-resident kernel. N0/N1: 16-byte chunks per lane of the
// two segments (N1 = 0: one segment). PF: software pipelining -- the next
// token's rows and slots are requested before the current token is reduced
// and written, so each wavefront keeps two tokens in flight. Two register sets
// alternate roles (the loop is unrolled by two) so that no copy forces a wait
// on the requests in flight; past the last token the request goes through an
// empty descriptor, so it is unconditional and fetches nothing.
template <int N0, int N1, int MODE, int SCHED>
__global__ __launch_bounds__(256) void qkn_rows(const KParams p) {
  constexpr bool PF = (SCHED == 1);
  constexpr int M1 = N1 > 0 ? N1 : 1;
  const int lane = static_cast<int>(threadIdx.x) & (kWave - 1);
  const int64_t nwaves = static_cast<int64_t>(gridDim.x) * (blockDim.x / kWave);
  bool given_up = false;
  int64_t w = wave_index();
  int64_t nw = nwaves;
  WaveSlice ws{p.rank, 0, 0, 0};
  if constexpr (MODE == kFusedWait) {
    if (p.group > 1) {  // the grid is a multiple of the group size
      ws.rank = static_cast<int>(w % p.group);
      w /= p.group;
      nw /= p.group;
      ws.col0 = static_cast<int64_t>(ws.rank) * p.seg[0].d;
      ws.col1 = static_cast<int64_t>(ws.rank) * p.seg[1].d;
      ws.inv_row = static_cast<int64_t>(ws.rank) * p.T;
    }
  }
  const int own_rank = (MODE == kFused || MODE == kFusedWait) ? ws.rank : -1;
  int64_t t, step, end;
  if (p.tok_chunk > 0) {
    t = w * p.tok_chunk;
    step = 1;
    end = (t + p.tok_chunk < p.T) ? t + p.tok_chunk : p.T;
  } else {
    t = w;
    step = nw;
    end = p.T;
  }
  if (t >= end) return;

  f32x4 g0[N0][2];
  f32x4 g1[M1][2];
  if constexpr (MODE != kPartial && MODE != kPublish) {
    load_gamma<N0>(p.seg[0], ws.col0, lane, g0);
    if constexpr (N1 > 0) load_gamma<N1>(p.seg[1], ws.col1, lane, g1);
  }

  TokenRegs<N0, M1> ra;
  fetch_token<N0, N1, MODE>(p, ws, t, lane, own_rank, ra);
  if constexpr (PF) {
    TokenRegs<N0, M1> rb;
    const int64_t last = end - 1;
    while (true) {
      int64_t tn = t + step;
      fetch_token<N0, N1, MODE>(p, ws, tn <= last ? tn : last, lane, own_rank, rb, tn <= last);
      process_token<N0, N1, MODE>(p, ws, t, lane, own_rank, g0, g1, ra, given_up);
      if (tn > last) break;
      t = tn;
      tn = t + step;
      fetch_token<N0, N1, MODE>(p, ws, tn <= last ? tn : last, lane, own_rank, ra, tn <= last);
      process_token<N0, N1, MODE>(p, ws, t, lane, own_rank, g0, g1, rb, given_up);
      if (tn > last) break;
      t = tn;
    }
  } else {
    while (true) {
      process_token<N0, N1, MODE>(p, ws, t, lane, own_rank, g0, g1, ra, given_up);
      t += step;
      if (t >= end) break;
      fetch_token<N0, N1, MODE>(p, ws, t, lane, own_rank, ra);
    }
  }
}

// ------------------------------------------------------------------ wide rows
//
// Slices wider than the register path holds with gamma (d_local in (4096,
// 16384], aligned as for the register path). One wavefront per token with
// both tensors' rows in VGPRs (N0 / N1 chunks per lane, all requested at
// once; the launcher puts the wide tensor in slot 0). gamma of both tensors is
// staged in LDS once per workgroup and read from there in Phase C, which forms
// (x * gamma) * factor -- the same operations, order and reduction tree as
// every other path.

// Phase C of one wide row from gamma in LDS: y = bf16((x * gamma) * inv).
template <int N>
__device__ __forceinline__ void store_scaled_lds(const DevSeg& s, int64_t t, int lane,
                                                 const u32x4 (&x)[N], const f32x4* g, float inv) {
  const Rsrc ry = make_rsrc(s.y + t * s.ldy, static_cast<uint32_t>(s.nchunks) * 16u);
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const int c = i * kWave + lane;
    const int cc = c < s.nchunks ? c : 0;  // masked lanes: any in-range gamma, store dropped
    const f32x4 ga = g[2 * cc], gb = g[2 * cc + 1];
    u32x4 o;
    o[0] = pack_bf16x2((bf16_lo(x[i][0]) * ga[0]) * inv, (bf16_hi(x[i][0]) * ga[1]) * inv);
    o[1] = pack_bf16x2((bf16_lo(x[i][1]) * ga[2]) * inv, (bf16_hi(x[i][1]) * ga[3]) * inv);
    o[2] = pack_bf16x2((bf16_lo(x[i][2]) * gb[0]) * inv, (bf16_hi(x[i][2]) * gb[1]) * inv);
    o[3] = pack_bf16x2((bf16_lo(x[i][3]) * gb[2]) * inv, (bf16_hi(x[i][3]) * gb[3]) * inv);
    st16_nt(o, ry, c * 16);
    // keep the scheduler from hoisting every chunk's gamma reads (register pressure)
    if ((i & 1) == 1) __builtin_amdgcn_sched_barrier(0);
  }
}

template <int N0, int N1, int MODE>
__global__ __launch_bounds__(256) void qkn_wide(const KParams p) {
  extern __shared__ __align__(16) float gamma_lds[];  // [d0 + d1] (fused / apply)
  constexpr int M1 = N1 > 0 ? N1 : 1;
  const int lane = static_cast<int>(threadIdx.x) & (kWave - 1);
  const int64_t nwaves = static_cast<int64_t>(gridDim.x) * (blockDim.x / kWave);
  const int own_rank = (MODE == kFused) ? p.rank : -1;
  const DevSeg& s0 = p.seg[0];
  const DevSeg& s1 = p.seg[1];

  if constexpr (MODE != kPartial) {
    // stage gamma: 16 bytes per thread per step, both tensors back to back
    const int n0 = s0.d / 4;
    const int n1 = (N1 > 0) ? s1.d / 4 : 0;
    f32x4* dst = reinterpret_cast<f32x4*>(gamma_lds);
    for (int i = static_cast<int>(threadIdx.x); i < n0 + n1; i += static_cast<int>(blockDim.x)) {
      dst[i] = (i < n0) ? reinterpret_cast<const f32x4*>(s0.w)[i]
                        : reinterpret_cast<const f32x4*>(s1.w)[i - n0];
    }
    __syncthreads();
  }
  const f32x4* g0 = reinterpret_cast<const f32x4*>(gamma_lds);
  const f32x4* g1 = g0 + s0.d / 4;

  for (int64_t t = wave_index(); t < p.T; t += nwaves) {
    u32x4 x0[N0];
    u32x4 x1[M1];
    load_row<N0>(s0, 0, t, lane, x0);
    if constexpr (N1 > 0) load_row<N1>(s1, 0, t, lane, x1);
    float sl0 = 0.0f, sl1 = 0.0f;
    if constexpr (MODE != kPartial) {
      sl0 = load_slots_buf(s0.partials, p.T, t, lane, p.tp, own_rank);
      if constexpr (N1 > 0) sl1 = load_slots_buf(s1.partials, p.T, t, lane, p.tp, own_rank);
    }
    float own0 = 0.0f, own1 = 0.0f;
    if constexpr (MODE != kApply) {
      own0 = wave_sum(row_lane_sumsq<N0>(x0));
      if constexpr (N1 > 0) own1 = wave_sum(row_lane_sumsq<N1>(x1));
    }
    if constexpr (MODE == kPartial) {
      st4f_lane0(own0, make_rsrc_at(s0.partials, t * 4, 4u), lane);
    } else {
      const float inv0 = rms_inverse(combine_slots(sl0, own0, p.tp, own_rank), s0.d_full, p.eps);
      float inv1 = 0.0f;
      if constexpr (N1 > 0)
        inv1 = rms_inverse(combine_slots(sl1, own1, p.tp, own_rank), s1.d_full, p.eps);
      // Re-derive the fp32 values from the packed rows instead of keeping the
      // unpacked ones alive from Phase A (an empty asm hides x's value; no code).
#pragma unroll
      for (int i = 0; i < N0; ++i) asm volatile("" : "+v"(x0[i]));
#pragma unroll
      for (int i = 0; i < M1; ++i) asm volatile("" : "+v"(x1[i]));
      store_scaled_lds<N0>(s0, t, lane, x0, g0, inv0);
      if constexpr (N1 > 0) store_scaled_lds<N1>(s1, t, lane, x1, g1, inv1);
      const int64_t own_slot = (static_cast<int64_t>(p.rank) * p.T + t) * 4;
      if constexpr (MODE == kFused) {
        st4f_lane0(own0, make_rsrc_at(s0.partials, own_slot, 4u), lane);
        if constexpr (N1 > 0) st4f_lane0(own1, make_rsrc_at(s1.partials, own_slot, 4u), lane);
      }
      st4f_lane0(inv0, make_rsrc_at(s0.inv_rms, t * 4, 4u), lane);
      if constexpr (N1 > 0) st4f_lane0(inv1, make_rsrc_at(s1.inv_rms, t * 4, 4u), lane);
    }
  }
}

// ------------------------------------------------------------------ general path
//
// Any width, stride or alignment. One wavefront per token; each segment in turn.
// Lane l handles chunks l, l+64, ... exactly as above (same tree, same bits).
// The row is staged in LDS between Phase A and Phase C when it fits; each lane
// reads back only the chunks it wrote, so no barrier is needed.

template <int MODE>
__global__ __launch_bounds__(64) void qkn_generic(const KParams p, int32_t stage_elems) {
  extern __shared__ __align__(16) uint16_t stage[];
  const int lane = static_cast<int>(threadIdx.x) & (kWave - 1);
  const int64_t nwaves = gridDim.x;
  const int own_rank = (MODE == kFused) ? p.rank : -1;

  for (int64_t t = wave_index(); t < p.T; t += nwaves) {
    for (int si = 0; si < p.nseg; ++si) {
      const DevSeg& s = p.seg[si];
      const uint16_t* xrow = s.x + t * s.ldx;
      const bool staged = (MODE == kFused) && (s.nchunks * kChunk <= stage_elems);

      float own = 0.0f;
      if constexpr (MODE != kApply) {
        float a = 0.0f;
        for (int c = lane; c < s.nchunks; c += kWave) {
          if (s.vec) {
            const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(xrow) + c);
            a = chunk_sumsq(v, a);
            if (staged) *reinterpret_cast<u32x4*>(stage + c * kChunk) = v;
          } else {
            for (int e = 0; e < kChunk; ++e) {
              const int j = c * kChunk + e;
              if (j < s.d) {
                const uint16_t b = xrow[j];
                const float f = bf16_to_f32(b);
                a = __builtin_fmaf(f, f, a);
                if (staged) stage[j] = b;
              }
            }
          }
        }
        own = wave_sum(a);
      }

      if constexpr (MODE == kPartial) {
        if (lane == 0) s.partials[t] = own;
        continue;
      } else {
        float S;
        if (p.tp <= kMaxFastTp) {
          const float slots = (p.tp > 1 || MODE == kApply)
                                  ? load_slots(s.partials, p.T, t, lane, p.tp, own_rank)
                                  : 0.0f;
          S = combine_slots(slots, own, p.tp, own_rank);
        } else {
          S = combine_slots_any(s.partials, p.T, t, lane, p.tp, own, own_rank);
        }
        const float inv = rms_inverse(S, s.d_full, p.eps);

        uint16_t* yrow = s.y + t * s.ldy;
        for (int c = lane; c < s.nchunks; c += kWave) {
          if (s.vec) {
            const u32x4 v = staged ? *reinterpret_cast<const u32x4*>(stage + c * kChunk)
                                   : __builtin_nontemporal_load(
                                         reinterpret_cast<const u32x4*>(xrow) + c);
            const f32x4* gp = reinterpret_cast<const f32x4*>(s.w) + 2 * c;
            const f32x4 ga = gp[0], gb = gp[1];
            u32x4 o;
            o[0] = pack_bf16x2((bf16_lo(v[0]) * ga[0]) * inv, (bf16_hi(v[0]) * ga[1]) * inv);
            o[1] = pack_bf16x2((bf16_lo(v[1]) * ga[2]) * inv, (bf16_hi(v[1]) * ga[3]) * inv);
            o[2] = pack_bf16x2((bf16_lo(v[2]) * gb[0]) * inv, (bf16_hi(v[2]) * gb[1]) * inv);
            o[3] = pack_bf16x2((bf16_lo(v[3]) * gb[2]) * inv, (bf16_hi(v[3]) * gb[3]) * inv);
            __builtin_nontemporal_store(o, reinterpret_cast<u32x4*>(yrow) + c);
          } else {
            for (int e = 0; e < kChunk; ++e) {
              const int j = c * kChunk + e;
              if (j < s.d) {
                const uint16_t b = staged ? stage[j] : xrow[j];
                const float z = bf16_to_f32(b) * s.w[j];
                yrow[j] = f32_to_bf16(z * inv);
              }
            }
          }
        }
        if (lane == 0) {
          if constexpr (MODE == kFused) {
            if (s.partials) s.partials[static_cast<int64_t>(p.rank) * p.T + t] = own;
          }
          if (s.inv_rms) s.inv_rms[t] = inv;
        }
      }
    }
  }
}

// ------------------------------------------------------------------ host side

typedef void (*RowsFn)(KParams);
typedef void (*GenericFn)(KParams, int32_t);

// Chunks per lane are rounded up to 1, 2, 4 or 8; unused chunks are masked.
constexpr int kNIdx[9] = {-1, 0, 1, 2, 2, 3, 3, 3, 3};  // chunks/lane -> table index
constexpr int kNVal[4] = {1, 2, 4, 8};

#define QKN_ROW_SET(M, A, S)                                                           \
  {qkn_rows<A, 0, M, S>, qkn_rows<A, 1, M, S>, qkn_rows<A, 2, M, S>, qkn_rows<A, 4, M, S>, \
   qkn_rows<A, 8, M, S>}
#define QKN_ONE_SET(M, S) \
  {qkn_rows<1, 0, M, S>, qkn_rows<2, 0, M, S>, qkn_rows<4, 0, M, S>, qkn_rows<8, 0, M, S>}
#define QKN_FULL_SET(M, S) \
  {QKN_ROW_SET(M, 1, S), QKN_ROW_SET(M, 2, S), QKN_ROW_SET(M, 4, S), QKN_ROW_SET(M, 8, S)}

// Schedules: 0 one token per step, 1 pipelined (next token requested early).
// [schedule][N0 index][N1 index: 0 = single segment, then 1, 2, 4, 8]
const RowsFn kFusedTable[2][4][5] = {QKN_FULL_SET(kFused, 0), QKN_FULL_SET(kFused, 1)};
const RowsFn kApplyTable[2][4] = {QKN_ONE_SET(kApply, 0), QKN_ONE_SET(kApply, 1)};
const RowsFn kPartialTable[2][4] = {QKN_ONE_SET(kPartial, 0), QKN_ONE_SET(kPartial, 1)};
const RowsFn kFusedWaitTable[2][4][5] = {QKN_FULL_SET(kFusedWait, 0),
                                         QKN_FULL_SET(kFusedWait, 1)};
const RowsFn kPublishTable[4] = QKN_ONE_SET(kPublish, 0);
const GenericFn kGenericTable[3] = {qkn_generic<kFused>, qkn_generic<kApply>,
                                    qkn_generic<kPartial>};
constexpr int kMaxWideChunks = 32;  // chunks per lane on the wide path (d_local <= 16384)
constexpr int kMaxWideLdsBytes = 64 * 1024;
#define QKN_WIDE_SET(A, M) \
  {qkn_wide<A, 0, M>, qkn_wide<A, 1, M>, qkn_wide<A, 2, M>, qkn_wide<A, 4, M>, qkn_wide<A, 8, M>}
// [wide N0: 16, 32][mode][N1 index: 0 = single segment, then 1, 2, 4, 8]
const RowsFn kWideTable[2][3][5] = {
    {QKN_WIDE_SET(16, kFused), QKN_WIDE_SET(16, kApply), QKN_WIDE_SET(16, kPartial)},
    {QKN_WIDE_SET(32, kFused), QKN_WIDE_SET(32, kApply), QKN_WIDE_SET(32, kPartial)}};

const char* const kModeName[5] = {"fused", "apply", "partial", "fused_wait", "publish"};

// Static names "rows<N0,N1>/mode" ("rows_pf<...>" when pipelined).
const char* rows_name(int mode, int sched, int i0, int i1) {
  static char names[5][2][4][5][40];
  static std::once_flag once;
  std::call_once(once, [] {
    const char* const prefix[2] = {"rows", "rows_pf"};
    for (int m = 0; m < 5; ++m)
      for (int f = 0; f < 2; ++f)
        for (int a = 0; a < 4; ++a)
          for (int b = 0; b < 5; ++b)
            snprintf(names[m][f][a][b], sizeof(names[m][f][a][b]), "%s<%d,%d>/%s", prefix[f],
                     kNVal[a], b == 0 ? 0 : kNVal[b - 1], kModeName[m]);
  });
  return names[mode][sched][i0][i1];
}
const char* const kGenericName[3] = {"generic/fused", "generic/apply", "generic/partial"};

// Static names "wide<N0,N1>/mode".
const char* wide_name(int mode, int i0, int i1) {
  static char names[3][2][5][40];
  static std::once_flag once;
  std::call_once(once, [] {
    for (int m = 0; m < 3; ++m)
      for (int a = 0; a < 2; ++a)
        for (int b = 0; b < 5; ++b)
          snprintf(names[m][a][b], sizeof(names[m][a][b]), "wide<%d,%d>/%s", a ? 32 : 16,
                   b == 0 ? 0 : kNVal[b - 1], kModeName[m]);
  });
  return names[mode][i0][i1];
}

// Options.
int64_t g_opt_waves_per_cu = 0;
int64_t g_opt_waves_per_block = 0;
int64_t g_opt_force_generic = 0;
int64_t g_opt_validate_only = 0;
int64_t g_opt_prefetch = 0;
int64_t g_opt_token_blocks = 0;
int64_t g_opt_balance = 0;

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

bool bad_eps(float eps) { return !(eps >= 0.0f) || !isfinite(eps); }

// A strided byte region: `rows` rows of `width` elements every `ld` elements.
struct Span {
  uintptr_t base;
  int64_t rows, ld, width, esz;
};

int64_t floor_div(int64_t a, int64_t b) {  // b > 0
  int64_t q = a / b;
  if ((a % b != 0) && ((a < 0) != (b < 0))) --q;
  return q;
}

bool spans_overlap(const Span& a, const Span& b) {
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

Span bf16_span(const void* p, int64_t rows, int64_t ld, int64_t width) {
  return Span{reinterpret_cast<uintptr_t>(p), rows, ld, width, 2};
}
Span f32_span(const void* p, int64_t n) {
  return Span{reinterpret_cast<uintptr_t>(p), 1, n, n, 4};
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

constexpr int64_t kMaxWidth = (int64_t{1} << 30);  // d_local and strides fit in int32 chunk math

struct Planned {
  KParams kp;
  int mode;
};

int check_seg_shape(const qkn_seg& s, int mode) {
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
int check_overlaps(const qkn_seg* segs, int nseg, int tp, int rank, int64_t T, int mode,
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
    const qkn_seg& s = segs[i];
    items[n++] = Item{bf16_span(s.x, T, s.ldx, s.d_local), false, i, 0};
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
    items[n++] = Item{bf16_span(s.y, T, s.ldy, s.d_local), true, i, 3};
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

bool seg_vec_ok(const qkn_seg& s, int mode) {
  if (!aligned16(s.x) || (s.ldx % kChunk) || (s.d_local % kChunk)) return false;
  if (mode != kPartial && mode != kPublish) {
    if (!aligned16(s.y) || !aligned16(s.w) || (s.ldy % kChunk)) return false;
  }
  return true;
}

DevSeg to_dev(const qkn_seg& s, int mode) {
  DevSeg d;
  d.x = s.x;
  d.w = s.w;
  d.partials = s.partials;
  d.y = s.y;
  d.inv_rms = s.inv_rms;
  d.ldx = s.ldx;
  d.ldy = (mode == kPartial || mode == kPublish) ? 0 : s.ldy;
  d.d = static_cast<int32_t>(s.d_local);
  d.nchunks = static_cast<int32_t>((s.d_local + kChunk - 1) / kChunk);
  d.d_full = static_cast<float>((mode == kPartial || mode == kPublish) ? s.d_local : s.d_full);
  d.vec = seg_vec_ok(s, mode) ? 1 : 0;
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

int launch(const qkn_seg* segs, int nseg, int tp, int rank, int64_t T, float eps, int mode,
           void* stream, const WaitArgs* wa = nullptr) {
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
  const bool buffer_ok = (g_opt_force_generic == 0) && tp <= kMaxFastTp &&
                         static_cast<__int128>(tp) * T * 4 < (static_cast<__int128>(1) << 31);
  bool fast = buffer_ok;
  bool wide = buffer_ok && !waits;
  int idx[2] = {0, 0};
  int max_chunks = 0, max_per_lane = 0;
  int64_t gamma_floats = 0;
  for (int i = 0; i < nseg; ++i) {
    kp.seg[i] = to_dev(segs[i], mode);
    const int per_lane = (kp.seg[i].nchunks + kWave - 1) / kWave;
    if (!kp.seg[i].vec || per_lane > kMaxRegChunks) fast = false;
    else idx[i] = kNIdx[per_lane];
    if (!kp.seg[i].vec || per_lane > kMaxWideChunks) wide = false;
    if (kp.seg[i].nchunks > max_chunks) max_chunks = kp.seg[i].nchunks;
    if (per_lane > max_per_lane) max_per_lane = per_lane;
    gamma_floats += kp.seg[i].d;
  }
  if (fast) wide = false;
  if (mode != kPartial && gamma_floats * 4 > kMaxWideLdsBytes) wide = false;
  int wide_i0 = 0, wide_i1 = 0;
  if (wide) {
    // the wider tensor goes first (slot 0 holds up to 32 chunks per lane, slot 1 up to 8)
    if (nseg == 2 && kp.seg[1].nchunks > kp.seg[0].nchunks) {
      const DevSeg tmp = kp.seg[0];
      kp.seg[0] = kp.seg[1];
      kp.seg[1] = tmp;
    }
    const int pl0 = (kp.seg[0].nchunks + kWave - 1) / kWave;
    wide_i0 = pl0 <= 16 ? 0 : 1;
    if (nseg == 2) {
      const int pl1 = (kp.seg[1].nchunks + kWave - 1) / kWave;
      if (pl1 > kMaxRegChunks) wide = false;  // both tensors wide: general path
      else wide_i1 = kNIdx[pl1] + 1;
    }
  }

  if (waits && !fast) return QKN_ENOTSUP;  // the flagged-slot modes exist on the register path only
  const void* fn;
  const char* name;
  int lds = 0;
  int32_t stage_elems = 0;
  if (wide) {
    fn = reinterpret_cast<const void*>(kWideTable[wide_i0][mode][wide_i1]);
    name = wide_name(mode, wide_i0, wide_i1);
    lds = (mode == kPartial) ? 0 : static_cast<int>(gamma_floats * 4);
  } else if (waits) {
    const int sched = (mode == kFusedWait && g_opt_prefetch) ? 1 : 0;
    if (mode == kFusedWait) fn = reinterpret_cast<const void*>(kFusedWaitTable[sched][idx[0]][nseg == 2 ? idx[1] + 1 : 0]);
    else fn = reinterpret_cast<const void*>(kPublishTable[idx[0]]);
    name = rows_name(mode, sched, idx[0], nseg == 2 ? idx[1] + 1 : 0);
  } else if (fast) {
    const int sched = g_opt_prefetch ? 1 : 0;
    if (mode == kFused) fn = reinterpret_cast<const void*>(kFusedTable[sched][idx[0]][nseg == 2 ? idx[1] + 1 : 0]);
    else if (mode == kApply) fn = reinterpret_cast<const void*>(kApplyTable[sched][idx[0]]);
    else fn = reinterpret_cast<const void*>(kPartialTable[sched][idx[0]]);
    name = rows_name(mode, sched, idx[0], nseg == 2 ? idx[1] + 1 : 0);
  } else {
    fn = reinterpret_cast<const void*>(kGenericTable[mode]);
    name = kGenericName[mode];
    if (mode == kFused && static_cast<int64_t>(max_chunks) * kChunk * 2 <= kMaxStageBytes) {
      stage_elems = max_chunks * kChunk;
      lds = stage_elems * 2;
    }
  }
  if (g_opt_validate_only) {  // arguments accepted and a kernel chosen; no HIP call
    t_last = qkn_launch_info{name, 0, 0, 0, lds};
    return QKN_OK;
  }

  int dev = 0, cus = 0;
  int rc = query_device(&dev, &cus);
  if (rc != QKN_OK) return rc;
  int wpb = 1;
  if (fast && !waits && g_opt_waves_per_block > 0) wpb = static_cast<int>(g_opt_waves_per_block);
  if (wide) wpb = 4;  // four wavefronts share the gamma staged in LDS
  const int block = wpb * kWave;
  int bpc = 0;
  rc = blocks_per_cu(dev, fn, block, lds, &bpc);
  if (rc != QKN_OK) return rc;
  // Persistent grid: enough wavefronts per CU to keep about kInFlightBytes of
  // rows requested per CU, at least kMinWavesPerCu, at most what fits.
  int64_t waves_per_cu = static_cast<int64_t>(bpc) * wpb;
  if ((fast || wide) && mode != kFusedWait) {  // a waiting launch keeps every resident slot
    int64_t token_bytes = 0;
    for (int i = 0; i < nseg; ++i) token_bytes += 2 * static_cast<int64_t>(kp.seg[i].d);
    int64_t want = (kInFlightBytes + token_bytes - 1) / token_bytes;
    if (want < kMinWavesPerCu) want = kMinWavesPerCu;
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

}  // namespace

extern "C" {

int qkn_partial_sumsq(const uint16_t* x, int64_t ldx, int64_t T, int64_t d_local,
                      float* partial_out, void* stream) {
  if (T < 0 || d_local < 1 || d_local > kMaxWidth || ldx < d_local) return QKN_EINVAL;
  if (T == 0) return QKN_OK;
  if (!x || !partial_out) return QKN_EINVAL;
  qkn_seg s;
  memset(&s, 0, sizeof(s));
  s.x = x;
  s.ldx = ldx;
  s.partials = partial_out;
  s.d_local = d_local;
  s.d_full = d_local;
  int rc = check_seg_shape(s, kPartial);
  if (rc != QKN_OK) return rc;
  rc = check_overlaps(&s, 1, 1, 0, T, kPartial);
  if (rc != QKN_OK) return rc;
  return launch(&s, 1, 1, 0, T, 0.0f, kPartial, stream);
}

int qkn_apply(const uint16_t* x, int64_t ldx, const float* w, const float* partials, int tp,
              int64_t T, int64_t d_local, int64_t d_full, float eps, uint16_t* y, int64_t ldy,
              float* inv_rms, void* stream) {
  int rc = validate_common(T, eps, tp, 0);
  if (rc != QKN_OK) return rc;
  qkn_seg s;
  s.x = x;
  s.ldx = ldx;
  s.w = w;
  s.partials = const_cast<float*>(partials);
  s.y = y;
  s.ldy = ldy;
  s.inv_rms = inv_rms;
  s.d_local = d_local;
  s.d_full = d_full;
  if (s.d_local < 1 || s.d_local > kMaxWidth || s.ldx < s.d_local || s.d_full < s.d_local ||
      s.ldy < s.d_local)
    return QKN_EINVAL;
  if (T == 0) return QKN_OK;
  rc = check_seg_shape(s, kApply);
  if (rc != QKN_OK) return rc;
  if (!partials) return QKN_EINVAL;
  rc = check_overlaps(&s, 1, tp, 0, T, kApply);
  if (rc != QKN_OK) return rc;
  return launch(&s, 1, tp, 0, T, eps, kApply, stream);
}

int qkn_fused_shard(const qkn_seg* segs, int nseg, int tp, int rank, int64_t T, float eps,
                    void* stream) {
  if (!segs || nseg < 1 || nseg > 2) return QKN_EINVAL;
  int rc = validate_common(T, eps, tp, rank);
  if (rc != QKN_OK) return rc;
  for (int i = 0; i < nseg; ++i) {
    const qkn_seg& s = segs[i];
    if (s.d_local < 1 || s.d_local > kMaxWidth || s.ldx < s.d_local || s.d_full < s.d_local ||
        s.ldy < s.d_local)
      return QKN_EINVAL;
  }
  if (T == 0) return QKN_OK;
  for (int i = 0; i < nseg; ++i) {
    rc = check_seg_shape(segs[i], kFused);
    if (rc != QKN_OK) return rc;
    if (tp > 1 && !segs[i].partials) return QKN_EINVAL;
  }
  rc = check_overlaps(segs, nseg, tp, rank, T, kFused);
  if (rc != QKN_OK) return rc;
  return launch(segs, nseg, tp, rank, T, eps, kFused, stream);
}

int qkn_publish_partials(const uint16_t* x, int64_t ldx, int64_t T, int64_t d_local,
                         uint64_t* slots_out, uint32_t epoch, void* stream) {
  if (T < 0 || d_local < 1 || d_local > kMaxWidth || ldx < d_local) return QKN_EINVAL;
  if (T == 0) return QKN_OK;
  if (!x || !slots_out || epoch == 0 || (reinterpret_cast<uintptr_t>(slots_out) & 7u))
    return QKN_EINVAL;
  qkn_seg s;
  memset(&s, 0, sizeof(s));
  s.x = x;
  s.ldx = ldx;
  s.d_local = d_local;
  s.d_full = d_local;
  const Span out{reinterpret_cast<uintptr_t>(slots_out), 1, T, T, 8};
  int rc = check_overlaps(&s, 1, 1, 0, T, kPublish, &out, 1);
  if (rc != QKN_OK) return rc;
  WaitArgs wa;
  memset(&wa, 0, sizeof(wa));
  wa.slots[0] = slots_out;
  wa.epoch = epoch;
  wa.spin_limit = 1;
  wa.co_resident = 1;
  wa.group = 1;
  return launch(&s, 1, 1, 0, T, 0.0f, kPublish, stream, &wa);
}

int qkn_fused_shard_wait(const qkn_seg* segs, int nseg, int tp, int rank, int64_t T, float eps,
                         const qkn_wait* wait, void* stream) {
  if (!segs || nseg < 1 || nseg > 2 || !wait) return QKN_EINVAL;
  int rc = validate_common(T, eps, tp, rank);
  if (rc != QKN_OK) return rc;
  if (wait->epoch == 0 || wait->spin_limit < 1 || wait->co_resident < 1) return QKN_EINVAL;
  for (int i = 0; i < nseg; ++i) {
    const qkn_seg& s = segs[i];
    if (s.d_local < 1 || s.d_local > kMaxWidth || s.ldx < s.d_local || s.d_full < s.d_local ||
        s.ldy < s.d_local)
      return QKN_EINVAL;
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
  rc = check_overlaps(segs, nseg, tp, rank, T, kFusedWait, extra, nextra);
  if (rc != QKN_OK) return rc;
  WaitArgs wa;
  wa.slots[0] = wait->slots[0];
  wa.slots[1] = nseg == 2 ? wait->slots[1] : nullptr;
  wa.status = wait->status;
  wa.spin_limit = wait->spin_limit;
  wa.epoch = wait->epoch;
  wa.co_resident = wait->co_resident;
  wa.group = 1;
  return launch(segs, nseg, tp, rank, T, eps, kFusedWait, stream, &wa);
}

int qkn_fused_group_wait(const qkn_seg* segs, int nseg, int tp, int64_t T, float eps,
                         const qkn_wait* wait, void* stream) {
  if (!segs || nseg < 1 || nseg > 2 || !wait) return QKN_EINVAL;
  int rc = validate_common(T, eps, tp, 0);
  if (rc != QKN_OK) return rc;
  if (wait->epoch == 0 || wait->spin_limit < 1 || wait->co_resident < 1) return QKN_EINVAL;
  qkn_seg view[2];  // the full tensors, for shape and overlap checks
  for (int i = 0; i < nseg; ++i) {
    const qkn_seg& s = segs[i];
    if (s.d_local < 1 || s.d_local > kMaxWidth || s.d_full != s.d_local * tp ||
        s.ldx < s.d_full || s.ldy < s.d_full)
      return QKN_EINVAL;
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
  rc = check_overlaps(view, nseg, tp, 0, T, kFusedWait, extra, nextra);
  if (rc != QKN_OK) return rc;
  WaitArgs wa;
  wa.slots[0] = wait->slots[0];
  wa.slots[1] = nseg == 2 ? wait->slots[1] : nullptr;
  wa.status = wait->status;
  wa.spin_limit = wait->spin_limit;
  wa.epoch = wait->epoch;
  wa.co_resident = wait->co_resident;
  wa.group = tp;
  return launch(segs, nseg, tp, 0, T, eps, kFusedWait, stream, &wa);
}

int qkn_full(const qkn_seg* segs, int nseg, int64_t T, float eps, void* stream) {
  if (!segs || nseg < 1 || nseg > 2) return QKN_EINVAL;
  for (int i = 0; i < nseg; ++i)
    if (segs[i].d_full != segs[i].d_local) return QKN_EINVAL;
  return qkn_fused_shard(segs, nseg, 1, 0, T, eps, stream);
}

const char* qkn_strerror(int status) {
  switch (status) {
    case QKN_OK: return "ok";
    case QKN_EINVAL: return "invalid argument";
    case QKN_EOVERLAP: return "output overlaps an input or another output";
    case QKN_EHIP: return "HIP runtime error";
    case QKN_ENOTSUP: return "shape or alignment not supported by this entry point";
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
  } else if (strcmp(key, "balance") == 0) {
    if (value != 0 && value != 1) return QKN_EINVAL;
    g_opt_balance = value;
  } else if (strcmp(key, "token_blocks") == 0) {
    if (value != 0 && value != 1) return QKN_EINVAL;
    g_opt_token_blocks = value;
  } else if (strcmp(key, "validate_only") == 0) {
    if (value != 0 && value != 1) return QKN_EINVAL;
    g_opt_validate_only = value;
  } else {
    return QKN_EINVAL;
  }
  return QKN_OK;
}

}  // extern "C"
