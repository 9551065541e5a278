// libqkn: device code of the sharded layerwise QK-Norm kernels for AMD MI355X
// (gfx950, CDNA4, wave64). The kernel tables that instantiate these templates
// are split over qkn_kern_*.hip (compiled in parallel); qkn.hip holds the host
// side (validation, path choice, launch).
//
// What is computed (SwiftQK, arXiv 2608.09160): RMSNorm of Eq. 1 (Sec. II-A)
// applied to each token's full projected Q and, separately, K vector, when the
// hidden dimension is split over tensor-parallel ranks (Sec. II-B). One rank's
// share follows the three phases of Sec. III / Alg. 1:
//   Phase A  partial sum of squares of the rank's slice, fp32;
//   Phase B  ascending-rank sum of all ranks' partials and the factor
//            1/sqrt(S/H_total + eps); independently of it, x * gamma;
//   Phase C  the scaled slice, rounded once to the activation format and written.
//
// Activations are bf16 or FP8-E4M3 (OCP e4m3fn, the FP8 format Sec. IV-C
// evaluates); all sums and products are fp32 in both cases.
//
// Design for gfx950 (the paper's warp/block layout is prior art, not reused):
//   * One wavefront owns one token at a time: its Q row and K row are spread
//     over the 64 lanes in 16-byte chunks (8 bf16 or 16 fp8), chunk c on lane
//     c % 64, so the row reduction needs no LDS and no barrier: four DPP row
//     steps and four readlanes.
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

#ifndef QKN_KERNELS_H
#define QKN_KERNELS_H

#include <hip/hip_runtime.h>

#include <math.h>
#include <stdint.h>

#include "qkn.h"

namespace qkn_dev {


typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kMaxFastTp = kWave;   // one statistic slot per lane
constexpr int kMaxStageBytes = 64 * 1024;
// Grid sizing of the register path (measured on MI355X: HBM throughput peaks
// with few, long-lived wavefronts per CU rather than full occupancy); the
// rows requested per CU at a time are set per activation format below.
constexpr int64_t kMinWavesPerCu = 6;

// kFusedWait: fused, with the other ranks' statistics published concurrently
// as flagged slots that the kernel waits for; kPublish: Phase A into flagged slots.
enum Mode { kFused = 0, kApply = 1, kPartial = 2, kFusedWait = 3, kPublish = 4 };

struct DevSeg {
  const void* x;    // activations (element type set by the kernel's format)
  const float* w;
  float* partials;  // [tp * T], rank-major
  void* y;
  float* inv_rms;   // optional [T]
  int64_t ldx;
  int64_t ldy;
  int32_t d;        // d_local
  int32_t nchunks;  // ceil(d_local / elements per chunk)
  float rcp_d_full; // 1 / H_total rounded to fp32 (the mean's divisor)
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

// Element formats. A 16-byte chunk holds kPer elements, element e of the chunk
// at byte e * sizeof(Elem) (little-endian). Decoding is exact; encoding rounds
// to nearest, ties to even.
struct FmtBf16 {
  using Elem = uint16_t;
  static constexpr int kPer = 8;
  __device__ static __forceinline__ void unpack(u32x4 v, float (&f)[8]) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[2 * e] = bf16_lo(v[e]);
      f[2 * e + 1] = bf16_hi(v[e]);
    }
  }
  __device__ static __forceinline__ u32x4 pack(const float (&f)[8]) {
    u32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) o[e] = pack_bf16x2(f[2 * e], f[2 * e + 1]);
    return o;
  }
  __device__ static __forceinline__ float decode(Elem b) { return bf16_to_f32(b); }
  __device__ static __forceinline__ Elem encode(float f) { return f32_to_bf16(f); }
};

// FP8-E4M3 (OCP e4m3fn) with the gfx950 conversions: v_cvt_pk_f32_fp8 decodes
// two bytes of a word, v_cvt_pk_fp8_f32 rounds two floats to nearest even into
// two bytes; a value that rounds beyond 448 becomes NaN (the format has no
// infinity), as in the usual cast to e4m3fn.
struct FmtFp8 {
  using Elem = uint8_t;
  static constexpr int kPer = 16;
  __device__ static __forceinline__ void unpack(u32x4 v, float (&f)[16]) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const f32x2 lo = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(v[e]), false);
      const f32x2 hi = __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(v[e]), true);
      f[4 * e] = lo[0];
      f[4 * e + 1] = lo[1];
      f[4 * e + 2] = hi[0];
      f[4 * e + 3] = hi[1];
    }
  }
  __device__ static __forceinline__ u32x4 pack(const float (&f)[16]) {
    u32x4 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      int w = __builtin_amdgcn_cvt_pk_fp8_f32(f[4 * e], f[4 * e + 1], 0, false);
      w = __builtin_amdgcn_cvt_pk_fp8_f32(f[4 * e + 2], f[4 * e + 3], w, true);
      o[e] = static_cast<uint32_t>(w);
    }
    return o;
  }
  __device__ static __forceinline__ float decode(Elem b) {
    return __builtin_amdgcn_cvt_pk_f32_fp8(static_cast<int>(b), false)[0];
  }
  __device__ static __forceinline__ Elem encode(float f) {
    return static_cast<Elem>(__builtin_amdgcn_cvt_pk_fp8_f32(f, 0.0f, 0, false) & 0xff);
  }
};

// Phase A on one chunk, ascending column order.
template <class F>
__device__ __forceinline__ float chunk_sumsq(u32x4 v, float acc) {
  float f[F::kPer];
  F::unpack(v, f);
#pragma unroll
  for (int e = 0; e < F::kPer; ++e) acc = __builtin_fmaf(f[e], f[e], acc);
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

// Phase B factor 1/sqrt(S/H_total + eps): the hardware reciprocal square root
// (v_rsq_f32, within 1 ulp) of fma(S, 1/H_total, eps) -- three fp32
// roundings in all, far below one step of the bf16 or FP8 output, and a
// fraction of the instructions of a correctly rounded divide and square root
// (which the per-token critical path of a wavefront measurably feels).
__device__ __forceinline__ float rms_inverse(float S, float rcp_d_full, float eps) {
  return __builtin_amdgcn_rsqf(__builtin_fmaf(S, rcp_d_full, eps));
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
// non-temporal (nt): the prefill shapes run as with sc1 nt (within 1 %), and
// decode-sized launches, whose stores end the launch, 5 % faster
#define QKN_STORE_CPOL 2
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

// gamma of a chunk: kPer floats, kPer / 4 float4 values.
template <class F>
constexpr int kGammaVecs = F::kPer / 4;

template <class F, int N>
__device__ __forceinline__ void load_gamma(const DevSeg& s, int64_t col, int lane,
                                           f32x4 (&g)[N][kGammaVecs<F>]) {
  constexpr int kG = kGammaVecs<F>;
  const Rsrc r = make_rsrc(s.w + col, static_cast<uint32_t>(s.nchunks) * (kG * 16u));
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const int c = i * kWave + lane;
#pragma unroll
    for (int j = 0; j < kG; ++j) g[i][j] = __builtin_bit_cast(f32x4, ld16(r, (c * kG + j) * 16));
  }
}

// Address of element (t, col) of a row-major tensor with leading dimension ld.
template <class F>
__device__ __forceinline__ const typename F::Elem* elem_at(const void* base, int64_t t, int64_t ld,
                                                           int64_t col) {
  return static_cast<const typename F::Elem*>(base) + t * ld + col;
}

// `live` false: an empty descriptor -- every lane reads zeros, nothing is fetched.
template <class F, int N>
__device__ __forceinline__ void load_row(const DevSeg& s, int64_t col, int64_t t, int lane,
                                         u32x4 (&x)[N], bool live = true) {
  const Rsrc r = make_rsrc(elem_at<F>(s.x, t, s.ldx, col),
                           live ? static_cast<uint32_t>(s.nchunks) * 16u : 0u);
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

template <class F, int N>
__device__ __forceinline__ float row_lane_sumsq(const u32x4 (&x)[N]) {
  float acc = 0.0f;
#pragma unroll
  for (int i = 0; i < N; ++i) acc = chunk_sumsq<F>(x[i], acc);
  return acc;
}

// Phase B compute path: z = x * gamma, elementwise in fp32.
template <class F, int N>
__device__ __forceinline__ void times_gamma(const u32x4 (&x)[N], const f32x4 (&g)[N][kGammaVecs<F>],
                                            float (&z)[N][F::kPer]) {
#pragma unroll
  for (int i = 0; i < N; ++i) {
    float f[F::kPer];
    F::unpack(x[i], f);
#pragma unroll
    for (int e = 0; e < F::kPer; ++e) z[i][e] = f[e] * g[i][e >> 2][e & 3];
  }
}

// Phase C: y = round(z * inv), non-temporal 128-bit stores.
template <class F, int N>
__device__ __forceinline__ void store_scaled(const DevSeg& s, int64_t col, int64_t t, int lane,
                                             const float (&z)[N][F::kPer], float inv) {
  const Rsrc r = make_rsrc(elem_at<F>(s.y, t, s.ldy, col), static_cast<uint32_t>(s.nchunks) * 16u);
#pragma unroll
  for (int i = 0; i < N; ++i) {
    float o[F::kPer];
#pragma unroll
    for (int e = 0; e < F::kPer; ++e) o[e] = z[i][e] * inv;
    st16_nt(F::pack(o), r, (i * kWave + lane) * 16);
  }
}

// ------------------------------------------------------------------ flagged slots
//
// A published statistic is one 8-byte word: fp32 bits in the low half, the
// round's epoch in the high half, written by a single aligned 64-bit store, so
// a reader that sees the epoch also sees the value (no separate flag or fence).

// The slots are written and read through buffer instructions with the sc1
// policy, the form the memory model gives agent-scope relaxed atomic loads and
// stores. (Not flat instructions: a flat access in flight makes the compiler
// wait for every outstanding load before the next use of any of them, which
// would undo the schedules that keep rows requested across a wait.)
constexpr int kCoherentCpol = 16;  // sc1: bypass the CU-local cache

typedef unsigned int B64 __attribute__((ext_vector_type(2)));  // the 64-bit buffer operand

// Lane 0 publishes `v` with `epoch` at byte address `at` (one aligned 64-bit store).
__device__ __forceinline__ void publish_slot_at(uintptr_t at, float v, uint32_t epoch, int lane) {
  const uint64_t word = (static_cast<uint64_t>(epoch) << 32) | __builtin_bit_cast(uint32_t, v);
  __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(B64, word),
                                        make_rsrc(reinterpret_cast<const void*>(at), 8),
                                        lane == 0 ? 0 : 8, 0, kCoherentCpol);
}

// Lanes 0..tp-1 other than `rank` poll rank k's slot of the token (byte
// address `at` + 8 k T, `nrec` bytes behind `at`) until it carries `epoch`, at
// most `limit` times (with a short sleep between polls). A lane that gives up,
// or any lane once `given_up` is set, returns NaN. `first` is the slot's word
// as read by the token's first poll; only a lane whose slot was not ready yet
// polls again.
__device__ __forceinline__ float wait_slot(uintptr_t at, uint32_t nrec, int64_t T, int lane,
                                           int tp, int rank, uint32_t epoch, int64_t limit,
                                           bool given_up, uint64_t first, bool& gave_up_now) {
  float v = 0.0f;
  if (lane < tp && lane != rank) {
    v = __builtin_nanf("");
    if (!given_up) {
      const Rsrc r = make_rsrc(reinterpret_cast<const void*>(at), nrec);
      const int off = static_cast<int>(lane * T * 8);
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
        word = __builtin_bit_cast(uint64_t,
                                  __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kCoherentCpol));
      }
    }
  }
  return v;
}

// Lane 0 sets the launch's status word (agent-coherent 32-bit store).
__device__ __forceinline__ void set_status(int* status, int value, int lane) {
  __builtin_amdgcn_raw_buffer_store_b32(static_cast<uint32_t>(value), make_rsrc(status, 4),
                                        lane == 0 ? 0 : 4, 0, kCoherentCpol);
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

// Byte addresses of one token's rows and slots for each segment, moved by a
// fixed stride per token, so that a token costs a 64-bit add per address
// instead of a 64-bit multiply (the scalar instructions of the address
// arithmetic sit on each wavefront's serial per-token path).
struct Cursor {
  uintptr_t x[2];    // token t's row of x at the slice's first column
  uintptr_t y[2];    // the same for y
  uintptr_t sl[2];   // rank 0's slot of token t (statistics or flagged slots)
  uintptr_t own[2];  // this rank's slot of token t
  uintptr_t inv[2];  // token t's factor (inv_rms + inv_row + t)
};

// Bytes behind each address, fixed per launch (0: nothing there; a descriptor
// of 0 bytes reads zeros and drops stores).
struct CursorBytes {
  uint32_t row[2];   // live row: nchunks * 16
  uint32_t sl[2];    // slot reads: (tp - 1) T words + 1
  uint32_t own[2];   // 4 when the own statistic is stored, else 0
  uint32_t inv[2];   // 4 when inv_rms is stored, else 0
};

__device__ __forceinline__ void advance(Cursor& c, const Cursor& step) {
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    c.x[i] += step.x[i];
    c.y[i] += step.y[i];
    c.sl[i] += step.sl[i];
    c.own[i] += step.own[i];
    c.inv[i] += step.inv[i];
  }
}

__device__ __forceinline__ Rsrc rsrc_of(uintptr_t at, uint32_t bytes) {
  return make_rsrc(reinterpret_cast<const void*>(at), bytes);
}

// `live` false: an empty descriptor -- every lane reads zeros, nothing is fetched.
template <int N>
__device__ __forceinline__ void load_row_at(uintptr_t row, uint32_t bytes, int lane, u32x4 (&x)[N],
                                            bool live = true) {
  const Rsrc r = rsrc_of(row, live ? bytes : 0u);
#pragma unroll
  for (int i = 0; i < N; ++i) x[i] = ld16_nt(r, (i * kWave + lane) * 16);
}

// Lanes 0..tp-1 other than `skip` read rank k's statistic of the token (k*T
// words after rank 0's); other lanes are out of range and read 0.
__device__ __forceinline__ float load_slots_at(uintptr_t at, uint32_t nrec, int64_t T, int lane,
                                               int tp, int skip, bool live = true) {
  const Rsrc r = rsrc_of(at, live ? nrec : 0u);
  const int off = (lane < tp && lane != skip) ? static_cast<int>(lane * T * 4)
                                              : static_cast<int>(nrec);
  return ld4f(r, off);
}

// First poll of the other ranks' flagged slots of the token, issued with the
// token's rows: lanes 0..tp-1 (not `rank`) read slot lane*T of the token with
// one 64-bit agent-coherent load each (the same single-copy-atomic access as
// the relaxed atomic load); other lanes are out of range and read 0, which no
// epoch matches.
__device__ __forceinline__ uint64_t poll_slots_at(uintptr_t at, uint32_t nrec, int64_t T, int lane,
                                                  int tp, int rank, bool live) {
  const Rsrc r = rsrc_of(at, live ? nrec : 0u);
  const int off = (lane < tp && lane != rank) ? static_cast<int>(lane * T * 8)
                                              : static_cast<int>(nrec);
  return __builtin_bit_cast(uint64_t, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, kCoherentCpol));
}

// Phase C: y = round(z * inv), non-temporal 128-bit stores.
template <class F, int N>
__device__ __forceinline__ void store_scaled_at(uintptr_t row, uint32_t bytes, int lane,
                                                const float (&z)[N][F::kPer], float inv) {
  const Rsrc r = rsrc_of(row, bytes);
#pragma unroll
  for (int i = 0; i < N; ++i) {
    float o[F::kPer];
#pragma unroll
    for (int e = 0; e < F::kPer; ++e) o[e] = z[i][e] * inv;
    st16_nt(F::pack(o), r, (i * kWave + lane) * 16);
  }
}

// `live` false (a pipelined request past the last token): nothing is fetched.
// POLL false (wait mode, publish-ahead schedule): the rows only; the first poll
// of the token's slots is issued later, once the other ranks have had time to
// publish.
template <class F, int N0, int N1, int MODE, bool POLL = true>
__device__ __forceinline__ void fetch_token(const KParams& p, const Cursor& c,
                                            const CursorBytes& nb, int lane, int own_rank,
                                            TokenRegs<N0, (N1 > 0 ? N1 : 1)>& r,
                                            bool live = true) {
  load_row_at<N0>(c.x[0], nb.row[0], lane, r.x0, live);
  if constexpr (N1 > 0) load_row_at<N1>(c.x[1], nb.row[1], lane, r.x1, live);
  r.slots0 = 0.0f;
  r.slots1 = 0.0f;
  if constexpr (MODE == kFused || MODE == kApply) {
    // with tp == 1 (fused) every lane is out of range: nothing is read
    r.slots0 = load_slots_at(c.sl[0], nb.sl[0], p.T, lane, p.tp, own_rank, live);
    if constexpr (N1 > 0) r.slots1 = load_slots_at(c.sl[1], nb.sl[1], p.T, lane, p.tp, own_rank, live);
  }
  r.word0 = 0;
  r.word1 = 0;
  if constexpr (MODE == kFusedWait && POLL) {
    r.word0 = poll_slots_at(c.sl[0], nb.sl[0], p.T, lane, p.tp, own_rank, live);
    if constexpr (N1 > 0) r.word1 = poll_slots_at(c.sl[1], nb.sl[1], p.T, lane, p.tp, own_rank, live);
  }
}

// Wait mode, Phase A of the token in `r`: the wavefront's statistics, which
// lane 0 publishes to this rank's flagged slots.
template <class F, int N0, int N1>
__device__ __forceinline__ void publish_token(const KParams& p, const Cursor& c, int lane,
                                              const TokenRegs<N0, (N1 > 0 ? N1 : 1)>& r,
                                              float& own0, float& own1) {
  own0 = wave_sum(row_lane_sumsq<F, N0>(r.x0));
  own1 = 0.0f;
  if constexpr (N1 > 0) own1 = wave_sum(row_lane_sumsq<F, N1>(r.x1));
  publish_slot_at(c.own[0], own0, p.epoch, lane);
  if constexpr (N1 > 0) publish_slot_at(c.own[1], own1, p.epoch, lane);
}

// Wait mode, Phases B and C of the token in `r` whose own statistics are
// published: x * gamma, then the other ranks' statistics (`word0/1`: the first
// poll of their slots; lanes whose slot was not ready poll again, bounded),
// the combination, the factor and the stores.
template <class F, int N0, int N1>
__device__ __forceinline__ void finish_waiting_token(
    const KParams& p, const Cursor& c, const CursorBytes& nb, int lane, int own_rank,
    const f32x4 (&g0)[N0][kGammaVecs<F>], const f32x4 (&g1)[(N1 > 0 ? N1 : 1)][kGammaVecs<F>],
    const TokenRegs<N0, (N1 > 0 ? N1 : 1)>& r, float own0, float own1, uint64_t word0,
    uint64_t word1, bool& given_up) {
  constexpr int M1 = N1 > 0 ? N1 : 1;
  // Phase B, compute path: independent of the statistics.
  float z0[N0][F::kPer];
  float z1[M1][F::kPer];
  times_gamma<F, N0>(r.x0, g0, z0);
  if constexpr (N1 > 0) times_gamma<F, N1>(r.x1, g1, z1);
  // Phase B, reduction path.
  bool gave_up = false;
  const float slots0 = wait_slot(c.sl[0], nb.sl[0], p.T, lane, p.tp, own_rank, p.epoch,
                                 p.spin_limit, given_up, word0, gave_up);
  float slots1 = 0.0f;
  if constexpr (N1 > 0)
    slots1 = wait_slot(c.sl[1], nb.sl[1], p.T, lane, p.tp, own_rank, p.epoch, p.spin_limit,
                       given_up || gave_up, word1, gave_up);
  if (__ballot(gave_up) != 0) {
    if (!given_up) set_status(p.status, 1, lane);
    given_up = true;  // later tokens of this wavefront do not wait again
  }
  const float inv0 = rms_inverse(combine_slots(slots0, own0, p.tp, own_rank), p.seg[0].rcp_d_full,
                                 p.eps);
  float inv1 = 0.0f;
  if constexpr (N1 > 0)
    inv1 = rms_inverse(combine_slots(slots1, own1, p.tp, own_rank), p.seg[1].rcp_d_full, p.eps);
  // Phase C.
  store_scaled_at<F, N0>(c.y[0], nb.row[0], lane, z0, inv0);
  if constexpr (N1 > 0) store_scaled_at<F, N1>(c.y[1], nb.row[1], lane, z1, inv1);
  st4f_lane0(inv0, rsrc_of(c.inv[0], nb.inv[0]), lane);
  if constexpr (N1 > 0) st4f_lane0(inv1, rsrc_of(c.inv[1], nb.inv[1]), lane);
}

// Phases A, B and C of the token at cursor `c`, whose rows and slots are in `r`.
template <class F, int N0, int N1, int MODE>
__device__ __forceinline__ void process_token(const KParams& p, const Cursor& c,
                                              const CursorBytes& nb, int lane, int own_rank,
                                              const f32x4 (&g0)[N0][kGammaVecs<F>],
                                              const f32x4 (&g1)[(N1 > 0 ? N1 : 1)][kGammaVecs<F>],
                                              const TokenRegs<N0, (N1 > 0 ? N1 : 1)>& r,
                                              bool& given_up) {
  constexpr int M1 = N1 > 0 ? N1 : 1;
  const DevSeg& s0 = p.seg[0];
  const DevSeg& s1 = p.seg[1];
  if constexpr (MODE == kFusedWait) {
    // publish this rank's statistics before waiting for the others'
    float own0, own1;
    publish_token<F, N0, N1>(p, c, lane, r, own0, own1);
    finish_waiting_token<F, N0, N1>(p, c, nb, lane, own_rank, g0, g1, r, own0, own1, r.word0,
                                    r.word1, given_up);
    return;
  }

  // Phase A: per-lane partial sums (not needed when every slot is given).
  float a0 = 0.0f, a1 = 0.0f;
  if constexpr (MODE != kApply) {
    a0 = row_lane_sumsq<F, N0>(r.x0);
    if constexpr (N1 > 0) a1 = row_lane_sumsq<F, N1>(r.x1);
  }

  if constexpr (MODE == kPartial) {
    const float own0 = wave_sum(a0);
    st4f_lane0(own0, rsrc_of(c.own[0], nb.own[0]), lane);
  } else if constexpr (MODE == kPublish) {
    const float own0 = wave_sum(a0);
    publish_slot_at(c.own[0], own0, p.epoch, lane);
  } else {
    float own0 = 0.0f, own1 = 0.0f;
    if constexpr (MODE == kFused) {
      own0 = wave_sum(a0);
      if constexpr (N1 > 0) own1 = wave_sum(a1);
    }

    // Phase B, compute path: independent of the statistic.
    float z0[N0][F::kPer];
    float z1[M1][F::kPer];
    times_gamma<F, N0>(r.x0, g0, z0);
    if constexpr (N1 > 0) times_gamma<F, N1>(r.x1, g1, z1);

    // Phase B, reduction path.
    const float slots0 = r.slots0, slots1 = r.slots1;
    const float S0 = combine_slots(slots0, own0, p.tp, own_rank);
    const float inv0 = rms_inverse(S0, s0.rcp_d_full, p.eps);
    float inv1 = 0.0f;
    if constexpr (N1 > 0) {
      const float S1 = combine_slots(slots1, own1, p.tp, own_rank);
      inv1 = rms_inverse(S1, s1.rcp_d_full, p.eps);
    }

    // Phase C.
    store_scaled_at<F, N0>(c.y[0], nb.row[0], lane, z0, inv0);
    if constexpr (N1 > 0) store_scaled_at<F, N1>(c.y[1], nb.row[1], lane, z1, inv1);
    if constexpr (MODE == kFused) {
      st4f_lane0(own0, rsrc_of(c.own[0], nb.own[0]), lane);
      if constexpr (N1 > 0) st4f_lane0(own1, rsrc_of(c.own[1], nb.own[1]), lane);
    }
    st4f_lane0(inv0, rsrc_of(c.inv[0], nb.inv[0]), lane);
    if constexpr (N1 > 0) st4f_lane0(inv1, rsrc_of(c.inv[1], nb.inv[1]), lane);
  }
}

// The cursors of token t and their per-token strides (`step` tokens apart).
template <class F, int MODE>
__device__ __forceinline__ void make_cursors(const KParams& p, const WaveSlice& ws, int64_t t,
                                             int64_t step, Cursor& c, Cursor& dc,
                                             CursorBytes& nb) {
  constexpr int64_t kEsz = sizeof(typename F::Elem);
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const DevSeg& s = p.seg[i];
    const int64_t col = i == 0 ? ws.col0 : ws.col1;
    const bool used = i < p.nseg;
    c.x[i] = reinterpret_cast<uintptr_t>(s.x) + (t * s.ldx + col) * kEsz;
    dc.x[i] = step * s.ldx * kEsz;
    c.y[i] = reinterpret_cast<uintptr_t>(s.y) + (t * s.ldy + col) * kEsz;
    dc.y[i] = step * s.ldy * kEsz;
    nb.row[i] = used ? static_cast<uint32_t>(s.nchunks) * 16u : 0u;
    const int64_t own_tok = static_cast<int64_t>(ws.rank) * p.T + t;
    if constexpr (MODE == kFusedWait || MODE == kPublish) {
      const uintptr_t base = reinterpret_cast<uintptr_t>(p.slots[i]);
      c.sl[i] = base + t * 8;
      c.own[i] = base + ((MODE == kPublish) ? t : own_tok) * 8;
      dc.sl[i] = dc.own[i] = step * 8;
      nb.sl[i] = static_cast<uint32_t>(((p.tp - 1) * p.T + 1) * 8);
      nb.own[i] = 8;
    } else {
      const uintptr_t base = reinterpret_cast<uintptr_t>(s.partials);
      const bool has = base != 0 && used;
      c.sl[i] = has ? base + t * 4 : 0;
      c.own[i] = has ? base + ((MODE == kPartial) ? t : own_tok) * 4 : 0;
      dc.sl[i] = dc.own[i] = has ? step * 4 : 0;
      nb.sl[i] = has ? static_cast<uint32_t>((p.tp - 1) * p.T * 4 + 4) : 0u;
      nb.own[i] = has ? 4u : 0u;
    }
    const uintptr_t ib = reinterpret_cast<uintptr_t>(s.inv_rms);
    const bool has_inv = ib != 0 && used;
    c.inv[i] = has_inv ? ib + (ws.inv_row + t) * 4 : 0;
    dc.inv[i] = has_inv ? step * 4 : 0;
    nb.inv[i] = has_inv ? 4u : 0u;
  }
}

// Persistent register-resident kernel. N0/N1: 16-byte chunks per lane of the
// two segments (N1 = 0: one segment). PF: software pipelining -- the next
// token's rows and slots are requested before the current token is reduced
// and written, so each wavefront keeps two tokens in flight. Two register sets
// alternate roles (the loop is unrolled by two) so that no copy forces a wait
// on the requests in flight; past the last token the request goes through an
// empty descriptor, so it is unconditional and fetches nothing.
template <class F, int N0, int N1, int MODE, int SCHED>
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

  f32x4 g0[N0][kGammaVecs<F>];
  f32x4 g1[M1][kGammaVecs<F>];
  if constexpr (MODE != kPartial && MODE != kPublish) {
    load_gamma<F, N0>(p.seg[0], ws.col0, lane, g0);
    if constexpr (N1 > 0) load_gamma<F, N1>(p.seg[1], ws.col1, lane, g1);
  }

  Cursor c, dc;
  CursorBytes nb;
  make_cursors<F, MODE>(p, ws, t, step, c, dc, nb);
  TokenRegs<N0, M1> ra;
  if constexpr (SCHED >= 2) {
    static_assert(MODE == kFusedWait, "the publish-ahead schedules are wait-mode schedules");
    // Publish ahead by D = SCHED - 1 tokens: a token's statistics are published
    // D tokens before it waits for the other ranks' (its rows requested D + 1
    // tokens before), so that by the time a wavefront polls, its peers --
    // which run the same schedule -- have usually published long since. A
    // step, with token X current: issue X's first poll, request the rows of
    // token X + D + 1 (after the poll, so that waiting for the poll, which the
    // in-order memory counter measures, does not wait for those rows), publish
    // token X + D, then wait for X's peers and finish X. D + 2 register sets
    // take the roles in turn (the steps are unrolled D + 2 at a time, so every
    // index is a constant and no copy waits on requests in flight). Waits move
    // only to tokens whose peers published them before waiting on anything
    // later, so with every wavefront resident no chain of waits can close.
    constexpr int D = SCHED - 1;
    constexpr int NS = D + 2;
    TokenRegs<N0, M1> r[NS];
    Cursor cur[NS];
    float o0[NS], o1[NS];
    const int64_t last = end - 1;
    cur[0] = c;
#pragma unroll
    for (int k = 1; k <= D; ++k) {
      cur[k] = cur[k - 1];
      advance(cur[k], dc);
    }
#pragma unroll
    for (int k = 0; k <= D; ++k)
      fetch_token<F, N0, N1, MODE, false>(p, cur[k], nb, lane, own_rank, r[k],
                                          t + k * step <= last);
#pragma unroll
    for (int k = 0; k < NS; ++k) o0[k] = o1[k] = 0.0f;
#pragma unroll
    for (int k = 0; k < D; ++k)
      if (t + k * step <= last) publish_token<F, N0, N1>(p, cur[k], lane, r[k], o0[k], o1[k]);
    bool more = true;
    while (more) {
#pragma unroll
      for (int k = 0; k < NS; ++k) {
        const int x = k, z = (k + D) % NS, w = (k + D + 1) % NS;
        const uint64_t w0 =
            poll_slots_at(cur[x].sl[0], nb.sl[0], p.T, lane, p.tp, own_rank, true);
        uint64_t w1 = 0;
        if constexpr (N1 > 0)
          w1 = poll_slots_at(cur[x].sl[1], nb.sl[1], p.T, lane, p.tp, own_rank, true);
        cur[w] = cur[z];
        advance(cur[w], dc);
        fetch_token<F, N0, N1, MODE, false>(p, cur[w], nb, lane, own_rank, r[w],
                                            t + (D + 1) * step <= last);
        if (t + D * step <= last) publish_token<F, N0, N1>(p, cur[z], lane, r[z], o0[z], o1[z]);
        finish_waiting_token<F, N0, N1>(p, cur[x], nb, lane, own_rank, g0, g1, r[x], o0[x],
                                        o1[x], w0, w1, given_up);
        if (t + step > last) {
          more = false;
          break;
        }
        t += step;
      }
    }
    return;
  } else {
    fetch_token<F, N0, N1, MODE>(p, c, nb, lane, own_rank, ra);
  }
  if constexpr (PF) {
    TokenRegs<N0, M1> rb;
    const int64_t last = end - 1;
    Cursor cn = c;
    while (true) {
      advance(cn, dc);  // token t + step (its requests go nowhere past the last token)
      int64_t tn = t + step;
      fetch_token<F, N0, N1, MODE>(p, cn, nb, lane, own_rank, rb, tn <= last);
      process_token<F, N0, N1, MODE>(p, c, nb, lane, own_rank, g0, g1, ra, given_up);
      if (tn > last) break;
      t = tn;
      c = cn;
      advance(cn, dc);
      tn = t + step;
      fetch_token<F, N0, N1, MODE>(p, cn, nb, lane, own_rank, ra, tn <= last);
      process_token<F, N0, N1, MODE>(p, c, nb, lane, own_rank, g0, g1, rb, given_up);
      if (tn > last) break;
      t = tn;
      c = cn;
    }
  } else {
    while (true) {
      process_token<F, N0, N1, MODE>(p, c, nb, lane, own_rank, g0, g1, ra, given_up);
      t += step;
      if (t >= end) break;
      advance(c, dc);
      fetch_token<F, N0, N1, MODE>(p, c, nb, lane, own_rank, ra);
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

// Phase C of one chunk: y = round((x * gamma) * inv), gamma from kGammaVecs<F> vectors.
template <class F>
__device__ __forceinline__ u32x4 scale_chunk(u32x4 v, const f32x4* g, float inv) {
  constexpr int kG = kGammaVecs<F>;
  f32x4 gq[kG];
#pragma unroll
  for (int j = 0; j < kG; ++j) gq[j] = g[j];
  float f[F::kPer];
  F::unpack(v, f);
  float o[F::kPer];
#pragma unroll
  for (int e = 0; e < F::kPer; ++e) o[e] = (f[e] * gq[e >> 2][e & 3]) * inv;
  return F::pack(o);
}

// Phase C of one wide row from gamma in LDS.
template <class F, int N>
__device__ __forceinline__ void store_scaled_lds(const DevSeg& s, int64_t t, int lane,
                                                 const u32x4 (&x)[N], const f32x4* g, float inv) {
  const Rsrc ry = make_rsrc(elem_at<F>(s.y, t, s.ldy, 0), static_cast<uint32_t>(s.nchunks) * 16u);
#pragma unroll
  for (int i = 0; i < N; ++i) {
    const int c = i * kWave + lane;
    const int cc = c < s.nchunks ? c : 0;  // masked lanes: any in-range gamma, store dropped
    st16_nt(scale_chunk<F>(x[i], g + kGammaVecs<F> * cc, inv), ry, c * 16);
    // keep the scheduler from hoisting every chunk's gamma reads (register pressure)
    if ((i & 1) == 1) __builtin_amdgcn_sched_barrier(0);
  }
}

template <class F, int N0, int N1, int MODE>
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
    load_row<F, N0>(s0, 0, t, lane, x0);
    if constexpr (N1 > 0) load_row<F, N1>(s1, 0, t, lane, x1);
    float sl0 = 0.0f, sl1 = 0.0f;
    if constexpr (MODE != kPartial) {
      sl0 = load_slots_buf(s0.partials, p.T, t, lane, p.tp, own_rank);
      if constexpr (N1 > 0) sl1 = load_slots_buf(s1.partials, p.T, t, lane, p.tp, own_rank);
    }
    float own0 = 0.0f, own1 = 0.0f;
    if constexpr (MODE != kApply) {
      own0 = wave_sum(row_lane_sumsq<F, N0>(x0));
      if constexpr (N1 > 0) own1 = wave_sum(row_lane_sumsq<F, N1>(x1));
    }
    if constexpr (MODE == kPartial) {
      st4f_lane0(own0, make_rsrc_at(s0.partials, t * 4, 4u), lane);
    } else {
      const float inv0 = rms_inverse(combine_slots(sl0, own0, p.tp, own_rank), s0.rcp_d_full, p.eps);
      float inv1 = 0.0f;
      if constexpr (N1 > 0)
        inv1 = rms_inverse(combine_slots(sl1, own1, p.tp, own_rank), s1.rcp_d_full, p.eps);
      // Re-derive the fp32 values from the packed rows instead of keeping the
      // unpacked ones alive from Phase A (an empty asm hides x's value; no code).
#pragma unroll
      for (int i = 0; i < N0; ++i) asm volatile("" : "+v"(x0[i]));
#pragma unroll
      for (int i = 0; i < M1; ++i) asm volatile("" : "+v"(x1[i]));
      store_scaled_lds<F, N0>(s0, t, lane, x0, g0, inv0);
      if constexpr (N1 > 0) store_scaled_lds<F, N1>(s1, t, lane, x1, g1, inv1);
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

template <class F, int MODE>
__global__ __launch_bounds__(64) void qkn_generic(const KParams p, int32_t stage_elems) {
  using E = typename F::Elem;
  constexpr int kPer = F::kPer;
  extern __shared__ __align__(16) unsigned char stage_raw[];
  E* const stage = reinterpret_cast<E*>(stage_raw);
  const int lane = static_cast<int>(threadIdx.x) & (kWave - 1);
  const int64_t nwaves = gridDim.x;
  const int own_rank = (MODE == kFused) ? p.rank : -1;

  for (int64_t t = wave_index(); t < p.T; t += nwaves) {
    for (int si = 0; si < p.nseg; ++si) {
      const DevSeg& s = p.seg[si];
      const E* xrow = elem_at<F>(s.x, t, s.ldx, 0);
      const bool staged = (MODE == kFused) && (s.nchunks * kPer <= stage_elems);

      float own = 0.0f;
      if constexpr (MODE != kApply) {
        float a = 0.0f;
        for (int c = lane; c < s.nchunks; c += kWave) {
          if (s.vec) {
            const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(xrow) + c);
            a = chunk_sumsq<F>(v, a);
            if (staged) *reinterpret_cast<u32x4*>(stage + c * kPer) = v;
          } else {
            for (int e = 0; e < kPer; ++e) {
              const int j = c * kPer + e;
              if (j < s.d) {
                const E b = xrow[j];
                const float f = F::decode(b);
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
        const float inv = rms_inverse(S, s.rcp_d_full, p.eps);

        E* yrow = const_cast<E*>(elem_at<F>(s.y, t, s.ldy, 0));
        for (int c = lane; c < s.nchunks; c += kWave) {
          if (s.vec) {
            const u32x4 v = staged ? *reinterpret_cast<const u32x4*>(stage + c * kPer)
                                   : __builtin_nontemporal_load(
                                         reinterpret_cast<const u32x4*>(xrow) + c);
            const f32x4* gp = reinterpret_cast<const f32x4*>(s.w) + kGammaVecs<F> * c;
            __builtin_nontemporal_store(scale_chunk<F>(v, gp, inv),
                                        reinterpret_cast<u32x4*>(yrow) + c);
          } else {
            for (int e = 0; e < kPer; ++e) {
              const int j = c * kPer + e;
              if (j < s.d) {
                const E b = staged ? stage[j] : xrow[j];
                const float z = F::decode(b) * s.w[j];
                yrow[j] = F::encode(z * inv);
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

typedef void (*RowsFn)(KParams);
typedef void (*GenericFn)(KParams, int32_t);

// Kernel tables. Each is defined, and its kernels instantiated, in exactly one
// translation unit (qkn_kern_*.hip); the host side picks entries from them.
// Register path, [schedule][N0 index][N1 index: 0 = single segment, then 1, 2, 4, 8]:
// schedules 0 one token per step, 1 pipelined (next token requested early);
// wait mode also 2 + d - 1 = publish d tokens ahead (d = 1, 2, 3).
extern const RowsFn kFusedTable[2][4][5];
extern const RowsFn kApplyTable[2][4];
extern const RowsFn kPartialTable[2][4];
extern const RowsFn kFusedWaitTable[5][4][5];
extern const RowsFn kPublishTable[4];
// fp8: [N0 index][N1 index] (up to 4 chunks per lane), the wait modes with [schedule] first
extern const RowsFn kFusedTable8[4][5];
extern const RowsFn kApplyTable8[4];
extern const RowsFn kPartialTable8[4];
extern const RowsFn kFusedWaitTable8[5][4][5];
extern const RowsFn kPublishTable8[4];
// general path [format][mode]; wide path [format][wide N0 index][mode][N1 index]
extern const GenericFn kGenericTable[2][3];
extern const RowsFn kWideTable[2][2][3][5];

#define QKN_ROW_SET(F, M, A, S)                                                     \
  {qkn_rows<F, A, 0, M, S>, qkn_rows<F, A, 1, M, S>, qkn_rows<F, A, 2, M, S>,       \
   qkn_rows<F, A, 4, M, S>, qkn_rows<F, A, 8, M, S>}
#define QKN_ONE_SET(F, M, S) \
  {qkn_rows<F, 1, 0, M, S>, qkn_rows<F, 2, 0, M, S>, qkn_rows<F, 4, 0, M, S>, qkn_rows<F, 8, 0, M, S>}
#define QKN_FULL_SET(F, M, S) \
  {QKN_ROW_SET(F, M, 1, S), QKN_ROW_SET(F, M, 2, S), QKN_ROW_SET(F, M, 4, S), QKN_ROW_SET(F, M, 8, S)}
#define QKN_ROW_SET8(M, A, S)                                                                  \
  {qkn_rows<FmtFp8, A, 0, M, S>, qkn_rows<FmtFp8, A, 1, M, S>, qkn_rows<FmtFp8, A, 2, M, S>, \
   qkn_rows<FmtFp8, A, 4, M, S>, nullptr}
#define QKN_FULL_SET8(M, S)                                                  \
  {QKN_ROW_SET8(M, 1, S), QKN_ROW_SET8(M, 2, S), QKN_ROW_SET8(M, 4, S), \
   {nullptr, nullptr, nullptr, nullptr, nullptr}}
#define QKN_ONE_SET8(M, S) \
  {qkn_rows<FmtFp8, 1, 0, M, S>, qkn_rows<FmtFp8, 2, 0, M, S>, qkn_rows<FmtFp8, 4, 0, M, S>, nullptr}
#define QKN_WIDE_SET(F, A, M)                                                            \
  {qkn_wide<F, A, 0, M>, qkn_wide<F, A, 1, M>, qkn_wide<F, A, 2, M>, qkn_wide<F, A, 4, M>, \
   qkn_wide<F, A, 8, M>}
#define QKN_WIDE_SET8(A, M)                                                                    \
  {qkn_wide<FmtFp8, A, 0, M>, qkn_wide<FmtFp8, A, 1, M>, qkn_wide<FmtFp8, A, 2, M>,           \
   qkn_wide<FmtFp8, A, 4, M>, nullptr}

}  // namespace qkn_dev

#endif  // QKN_KERNELS_H
