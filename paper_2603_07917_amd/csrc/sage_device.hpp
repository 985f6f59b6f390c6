// Device-side helpers shared by the gfx950 kernels of the scheduling path.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace sage {

constexpr int kWave = 64;

// ---------------------------------------------------------------------------
// Neighbour keys. A candidate (similarity s, history index n) is packed into
// one 64-bit key whose unsigned order is the neighbour order of the
// predictor: larger similarity first, and for equal similarity the lower
// history index first. High word: the fp32 bits made monotone (negative
// values bit-flipped, positive ones with the sign bit set); low word: ~n.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t f32_order_bits(float s) {
  uint32_t u = __float_as_uint(s);
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}
__device__ __forceinline__ float f32_from_order_bits(uint32_t o) {
  uint32_t u = (o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o;
  return __uint_as_float(u);
}
__device__ __forceinline__ uint64_t make_key(float s, uint32_t n) {
  return ((uint64_t)f32_order_bits(s) << 32) | (uint64_t)(~n);
}
// Largest float below x (x finite or -inf; -inf maps to itself).
__device__ __forceinline__ float float_below(float x) {
  if (x == -__builtin_inff()) return x;
  if (x == 0.0f) return -1.401298464e-45f;            // below both zeros
  const uint32_t u = __float_as_uint(x);
  return __uint_as_float(x > 0.0f ? u - 1u : u + 1u);
}

// Padding key: similarity -inf, index -1. Every real candidate beats it.
constexpr uint64_t kPadKey = (uint64_t)0x007FFFFFu << 32;

__device__ __forceinline__ float key_sim(uint64_t k) { return f32_from_order_bits((uint32_t)(k >> 32)); }
__device__ __forceinline__ int32_t key_id(uint64_t k) { return (int32_t)(~(uint32_t)k); }

// ---------------------------------------------------------------------------
// Cross-lane moves within a 64-wide wavefront (ds_bpermute based).
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t lane_id() { return __lane_id(); }

__device__ __forceinline__ uint64_t shfl_u64(uint64_t v, int src_lane) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  lo = (uint32_t)__shfl((int)lo, src_lane, kWave);
  hi = (uint32_t)__shfl((int)hi, src_lane, kWave);
  return ((uint64_t)hi << 32) | lo;
}
__device__ __forceinline__ uint64_t shfl_xor_u64(uint64_t v, int mask) {
  uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32);
  lo = (uint32_t)__shfl_xor((int)lo, mask, kWave);
  hi = (uint32_t)__shfl_xor((int)hi, mask, kWave);
  return ((uint64_t)hi << 32) | lo;
}

// Compare-exchange with the lane `stride` away: the lane whose `stride` bit
// is clear keeps the larger key when `desc`, the smaller one otherwise.
__device__ __forceinline__ uint64_t cx_lanes(uint64_t v, int stride, bool desc) {
  uint64_t o = shfl_xor_u64(v, stride);
  bool low = (lane_id() & stride) == 0;
  bool keep_max = (low == desc);
  uint64_t mx = v > o ? v : o;
  uint64_t mn = v > o ? o : v;
  return keep_max ? mx : mn;
}

// Sort the wave's 64 keys (one per lane) into descending order across lanes
// (lane 0 holds the largest): bitonic sorting network.
__device__ __forceinline__ uint64_t wave_sort_desc64(uint64_t v) {
  const int lane = (int)lane_id();
#pragma unroll
  for (int size = 2; size <= 64; size <<= 1) {
    const bool desc_block = (lane & size) == 0;   // always true at size 64
#pragma unroll
    for (int stride = size >> 1; stride > 0; stride >>= 1) v = cx_lanes(v, stride, desc_block);
  }
  return v;
}

// ---------------------------------------------------------------------------
// Wave reductions / scans.
// ---------------------------------------------------------------------------
__device__ __forceinline__ double wave_incl_scan_f64(double x) {
  const int lane = (int)lane_id();
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    double y = __shfl_up(x, off, kWave);
    if (lane >= off) x += y;
  }
  return x;
}
// Sum over lanes strictly below this one (no subtraction: shift, then scan).
__device__ __forceinline__ double wave_excl_scan_f64(double x) {
  const int lane = (int)lane_id();
  double v = __shfl_up(x, 1, kWave);
  if (lane == 0) v = 0.0;
  return wave_incl_scan_f64(v);
}
// Sum over lanes strictly above this one (no subtraction: shift, then scan).
__device__ __forceinline__ double wave_excl_suffix_f64(double x) {
  const int lane = (int)lane_id();
  double v = __shfl_down(x, 1, kWave);
  if (lane == kWave - 1) v = 0.0;
#pragma unroll
  for (int off = 1; off < kWave; off <<= 1) {
    double y = __shfl_down(v, off, kWave);
    if (lane + off < kWave) v += y;
  }
  return v;
}

__device__ __forceinline__ int wave_sum_i32(int x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, kWave);
  return x;
}

}  // namespace sage
