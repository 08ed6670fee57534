// Shared device/host helpers of the Tactic HIP library (gfx950, wave64).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace tactic {

constexpr int kHeadDim = 128;
constexpr int kWave = 64;

// ----------------------------------------------------------------------------
// Geometry of the exact head and the two sampling windows of a token list of
// length n (Sec. 4.4, Algorithm 1).  All fractions are integer basis points.
// ----------------------------------------------------------------------------
struct SelParams {
  float target_frac;
  int exact_bp, win_bp, win_min, p1_bp, p2_bp;
};

struct Geometry {
  int64_t n, N, s1, t1, s2, t2, samples;
  int exact;
};

__host__ __device__ inline int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Tokens of sequence b: its span [indptr[b], indptr[b+1]) or, with a length
// array, the first len[b] rows of that span.
__device__ __forceinline__ int64_t seq_tokens(const int64_t* indptr, const int64_t* len, int b) {
  const int64_t l = len ? len[b] : 0;  // issued before the span is formed, so the loads overlap
  const int64_t span = indptr[b + 1] - indptr[b];
  return len ? max((int64_t)0, min(l, span)) : span;
}

__host__ __device__ inline Geometry make_geometry(int64_t n, const SelParams& p) {
  Geometry g;
  g.n = n;
  int64_t N = ceil_div64(n * p.exact_bp, 10000);
  if (N < 1) N = 1;
  if (N > n) N = n;
  int64_t W = ceil_div64(n * p.win_bp, 10000);
  if (W < p.win_min) W = p.win_min;
  const int64_t c1 = (n * p.p1_bp + 5000) / 10000;
  const int64_t c2 = (n * p.p2_bp + 5000) / 10000;
  int64_t s1 = c1 - W / 2;
  if (s1 < N + 1) s1 = N + 1;
  int64_t t1 = s1 + W - 1;
  if (t1 > n) t1 = n;
  int64_t s2 = c2 - W / 2;
  if (s2 < N + 1) s2 = N + 1;
  int64_t t2 = s2 + W - 1;
  if (t2 > n) t2 = n;
  g.N = N;
  g.s1 = s1;
  g.t1 = t1;
  g.s2 = s2;
  g.t2 = t2;
  g.exact = (N == n) || (s1 > t1) || (s2 > t2) || (t1 >= s2);
  g.samples = g.exact ? n : N + (t1 - s1 + 1) + (t2 - s2 + 1);
  return g;
}

// ----------------------------------------------------------------------------
// bf16 helpers (bf16 is the upper half of an fp32)
// ----------------------------------------------------------------------------
__device__ __forceinline__ float bf16lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ __forceinline__ float bf16hi(uint32_t w) { return __uint_as_float(w & 0xffff0000u); }

// 2^x with the hardware instruction (v_exp_f32; results below 2^-126 flush
// to zero, which is harmless for softmax weights); 2^-inf = 0
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

typedef short short2_t __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

// 16-byte streaming load (non-temporal hint: the data is read once)
__device__ __forceinline__ uint4 load_stream16(const uint16_t* p) {
  const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4*>(p));
  return make_uint4(v.x, v.y, v.z, v.w);
}

// a.x*b.x + a.y*b.y + c on bf16 pairs, fp32 accumulate (v_dot2_f32_bf16)
__device__ __forceinline__ float dot2_bf16(uint32_t a, uint32_t b, float c) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(short2_t, a),
                                         __builtin_bit_cast(short2_t, b), c, false);
}

// ----------------------------------------------------------------------------
// Cross-lane reductions within groups of 16 lanes (one DPP row)
// ----------------------------------------------------------------------------
template <int CTRL>
__device__ __forceinline__ float dpp(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(0, __builtin_bit_cast(int, v), CTRL, 0xF, 0xF,
                                                               false));
}

// Sum over the 16 lanes of a DPP row, bitwise identical in every lane: each
// step adds a lane and its mirror partner (row_mirror, row_half_mirror, then
// quad swaps), so both partners compute the same commutative sum.
__device__ __forceinline__ float sum16(float v) {
  v += dpp<0x140>(v);  // row_mirror: lane i + lane 15-i
  v += dpp<0x141>(v);  // row_half_mirror: lane i + lane 7-i within each half
  v += dpp<0x4E>(v);   // quad_perm [2,3,0,1]
  v += dpp<0xB1>(v);   // quad_perm [1,0,3,2]
  return v;
}

template <int CTRL>
__device__ __forceinline__ double dpp(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const int lo = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)u, CTRL, 0xF, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp(0, (int)(uint32_t)(u >> 32), CTRL, 0xF, 0xF, false);
  return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

// fp64 sum over the 16 lanes of a DPP row, bitwise identical in every lane
// (the same mirror-partner steps as sum16)
__device__ __forceinline__ double sum16d(double v) {
  v += dpp<0x140>(v);
  v += dpp<0x141>(v);
  v += dpp<0x4E>(v);
  v += dpp<0xB1>(v);
  return v;
}

// Lane shift / broadcast by DPP with zero fill: lanes whose source lies
// outside their row (row_shr) or whose row is masked off (row_bcast) get 0.
template <int CTRL, int RM>
__device__ __forceinline__ uint32_t dpp_zero(uint32_t v) {
  return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, RM, 0xF, true);
}
template <int CTRL, int RM>
__device__ __forceinline__ uint64_t dpp_zero(uint64_t v) {
  return ((uint64_t)dpp_zero<CTRL, RM>((uint32_t)(v >> 32)) << 32) | dpp_zero<CTRL, RM>((uint32_t)v);
}
template <int CTRL, int RM>
__device__ __forceinline__ int dpp_zero(int v) {
  return __builtin_amdgcn_update_dpp(0, v, CTRL, RM, 0xF, true);
}
template <int CTRL, int RM>
__device__ __forceinline__ int64_t dpp_zero(int64_t v) {
  return (int64_t)dpp_zero<CTRL, RM>((uint64_t)v);
}
template <int CTRL, int RM>
__device__ __forceinline__ float dpp_zero(float v) {
  return __builtin_bit_cast(float, dpp_zero<CTRL, RM>(__builtin_bit_cast(uint32_t, v)));
}
template <int CTRL, int RM>
__device__ __forceinline__ double dpp_zero(double v) {
  return __builtin_bit_cast(double, dpp_zero<CTRL, RM>(__builtin_bit_cast(uint64_t, v)));
}

// Inclusive scan over the 16 lanes of each DPP row (row_shr 1, 2, 4, 8).
template <typename T>
__device__ __forceinline__ T row_incl_scan(T v) {
  v += dpp_zero<0x111, 0xF>(v);
  v += dpp_zero<0x112, 0xF>(v);
  v += dpp_zero<0x114, 0xF>(v);
  v += dpp_zero<0x118, 0xF>(v);
  return v;
}

// Inclusive scan over the 64 lanes of a wave without LDS: the row scans, then
// lane 15 of rows 0 and 2 added to rows 1 and 3 (row_bcast:15) and lane 31 to
// rows 2 and 3 (row_bcast:31).
template <typename T>
__device__ __forceinline__ T wave_incl_scan(T v) {
  v = row_incl_scan(v);
  v += dpp_zero<0x142, 0xA>(v);
  v += dpp_zero<0x143, 0xC>(v);
  return v;
}

// Inclusive max-scan over the 64 lanes of a wave of non-negative values (the
// zero fill of the shifts is neutral): the same steps as wave_incl_scan.
__device__ __forceinline__ int wave_incl_max(int v) {
  v = max(v, dpp_zero<0x111, 0xF>(v));
  v = max(v, dpp_zero<0x112, 0xF>(v));
  v = max(v, dpp_zero<0x114, 0xF>(v));
  v = max(v, dpp_zero<0x118, 0xF>(v));
  v = max(v, dpp_zero<0x142, 0xA>(v));
  v = max(v, dpp_zero<0x143, 0xC>(v));
  return v;
}

// Lane shift / broadcast by DPP that keeps the lane's own value where the
// source lies outside its row or the row is masked off (neutral for max/min).
template <int CTRL, int RM>
__device__ __forceinline__ float dpp_self(float v) {
  return __builtin_bit_cast(float, __builtin_amdgcn_update_dpp(__builtin_bit_cast(int, v), __builtin_bit_cast(int, v),
                                                               CTRL, RM, 0xF, false));
}
template <int CTRL, int RM>
__device__ __forceinline__ double dpp_self(double v) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const int lo = __builtin_amdgcn_update_dpp((int)(uint32_t)u, (int)(uint32_t)u, CTRL, RM, 0xF, false);
  const int hi = __builtin_amdgcn_update_dpp((int)(uint32_t)(u >> 32), (int)(uint32_t)(u >> 32), CTRL, RM, 0xF, false);
  return __builtin_bit_cast(double, ((uint64_t)(uint32_t)hi << 32) | (uint32_t)lo);
}

__device__ __forceinline__ float readlane_f(float v, int lane) {
  return __builtin_bit_cast(float, __builtin_amdgcn_readlane(__builtin_bit_cast(int, v), lane));
}
__device__ __forceinline__ double readlane_d(double v, int lane) {
  const uint64_t u = __builtin_bit_cast(uint64_t, v);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), lane);
  return __builtin_bit_cast(double, ((uint64_t)hi << 32) | lo);
}

// Wave-wide reductions without LDS, the same value in every lane: the DPP
// inclusive scan (sum) or max/min scan, read from the last lane.
template <typename T>
__device__ __forceinline__ T wave_scan_max(T v) {
  v = fmax(v, dpp_self<0x111, 0xF>(v));
  v = fmax(v, dpp_self<0x112, 0xF>(v));
  v = fmax(v, dpp_self<0x114, 0xF>(v));
  v = fmax(v, dpp_self<0x118, 0xF>(v));
  v = fmax(v, dpp_self<0x142, 0xA>(v));
  v = fmax(v, dpp_self<0x143, 0xC>(v));
  return v;
}
template <typename T>
__device__ __forceinline__ T wave_scan_min(T v) {
  v = fmin(v, dpp_self<0x111, 0xF>(v));
  v = fmin(v, dpp_self<0x112, 0xF>(v));
  v = fmin(v, dpp_self<0x114, 0xF>(v));
  v = fmin(v, dpp_self<0x118, 0xF>(v));
  v = fmin(v, dpp_self<0x142, 0xA>(v));
  v = fmin(v, dpp_self<0x143, 0xC>(v));
  return v;
}
__device__ __forceinline__ double wave_allsum_d(double v) { return readlane_d(wave_incl_scan(v), kWave - 1); }
__device__ __forceinline__ double wave_allmax_d(double v) { return readlane_d(wave_scan_max(v), kWave - 1); }
__device__ __forceinline__ float wave_allsum_f(float v) { return readlane_f(wave_incl_scan(v), kWave - 1); }
__device__ __forceinline__ float wave_allmax_f(float v) { return readlane_f(wave_scan_max(v), kWave - 1); }
__device__ __forceinline__ float wave_allmin_f(float v) { return readlane_f(wave_scan_min(v), kWave - 1); }


}  // namespace tactic
