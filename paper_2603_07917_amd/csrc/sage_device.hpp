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
// Cross-lane moves within a 64-wide wavefront: DPP and the lane-swap
// instructions for fixed strides, readlane for a fixed lane.
// ---------------------------------------------------------------------------
__device__ __forceinline__ uint32_t lane_id() { return __lane_id(); }

// Value held by lane (lane ^ S), for a stride S fixed at compile time, with
// no LDS round trip: DPP within a row of 16 lanes (S = 1, 2: quad
// permutes; S = 4: row half-mirror then quad reverse, i -> 7 - i -> i ^ 4;
// S = 8: row rotate by 8), and the lane-swap instructions across rows
// (S = 16, 32). permlane16_swap on two copies of v leaves v[lane - 16] in
// the first copy's odd rows and v[lane + 16] in the second copy's even rows;
// permlane32_swap does the same for the two halves of the wave.
template <int S>
__device__ __forceinline__ uint32_t xor_lane_u32(uint32_t v) {
  if constexpr (S == 1) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);
  } else if constexpr (S == 2) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);
  } else if constexpr (S == 4) {
    const int t = __builtin_amdgcn_mov_dpp((int)v, 0x141, 0xF, 0xF, false);
    return (uint32_t)__builtin_amdgcn_mov_dpp(t, 0x1B, 0xF, 0xF, false);
  } else if constexpr (S == 8) {
    return (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x128, 0xF, 0xF, false);
  } else if constexpr (S == 16) {
    const auto r = __builtin_amdgcn_permlane16_swap(v, v, false, false);
    return (__lane_id() & 16) ? r[0] : r[1];
  } else {
    static_assert(S == 32, "stride must be a power of two below 64");
    const auto r = __builtin_amdgcn_permlane32_swap(v, v, false, false);
    return (__lane_id() & 32) ? r[0] : r[1];
  }
}
template <int S>
__device__ __forceinline__ uint64_t xor_lane_u64(uint64_t v) {
  const uint32_t lo = xor_lane_u32<S>((uint32_t)v), hi = xor_lane_u32<S>((uint32_t)(v >> 32));
  return ((uint64_t)hi << 32) | lo;
}
// The same for a stride known only after unrolling (folds to one case).
__device__ __forceinline__ uint64_t xor_lane_u64(uint64_t v, int stride) {
  switch (stride) {
    case 1: return xor_lane_u64<1>(v);
    case 2: return xor_lane_u64<2>(v);
    case 4: return xor_lane_u64<4>(v);
    case 8: return xor_lane_u64<8>(v);
    case 16: return xor_lane_u64<16>(v);
    default: return xor_lane_u64<32>(v);
  }
}

// Key of a fixed lane, in every lane.
__device__ __forceinline__ uint64_t lane_value_u64(uint64_t v, int src_lane) {
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, src_lane);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(v >> 32), src_lane);
  return ((uint64_t)hi << 32) | lo;
}

// Compare-exchange with the lane `stride` away (stride a power of two below
// 64): the lane whose `stride` bit is clear keeps the larger key when
// `desc`, the smaller one otherwise.
__device__ __forceinline__ uint64_t cx_lanes(uint64_t v, int stride, bool desc) {
  const uint64_t o = xor_lane_u64(v, stride);
  const bool keep_max = ((lane_id() & stride) == 0) == desc;
  return ((v > o) == keep_max) ? v : o;
}

// Sort the wave's 64 keys (one per lane) across lanes with a bitonic
// sorting network: descending (lane 0 holds the largest) or ascending.
__device__ __forceinline__ uint64_t wave_sort64(uint64_t v, bool descending) {
  const int lane = (int)lane_id();
#pragma unroll
  for (int size = 2; size <= 64; size <<= 1) {
    const bool desc_block = ((lane & size) == 0) == descending;   // the whole wave at size 64
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

// ---------------------------------------------------------------------------
// DPP cross-lane moves (gfx9 wave64 encodings): no LDS round trip.
// ---------------------------------------------------------------------------
constexpr int kDppRowShr1 = 0x111, kDppRowShr2 = 0x112, kDppRowShr4 = 0x114, kDppRowShr8 = 0x118;
constexpr int kDppWaveShr1 = 0x138, kDppRowMirror = 0x140, kDppRowHalfMirror = 0x141;
constexpr int kDppRowBcast15 = 0x142, kDppRowBcast31 = 0x143;
constexpr int kDppQuadXor1 = 0xB1, kDppQuadXor2 = 0x4E;     // quad_perm [1,0,3,2], [2,3,0,1]

// Lanes whose source is outside the pattern, or whose row is not in
// kRowMask, receive `old`.
template <int kCtrl, int kRowMask = 0xf>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t old, uint32_t x) {
  return (uint32_t)__builtin_amdgcn_update_dpp((int)old, (int)x, kCtrl, kRowMask, 0xf, false);
}
template <int kCtrl, int kRowMask = 0xf>
__device__ __forceinline__ double dpp_f64(double old, double x) {
  const uint64_t o = (uint64_t)__double_as_longlong(old), v = (uint64_t)__double_as_longlong(x);
  const uint32_t lo = dpp_u32<kCtrl, kRowMask>((uint32_t)o, (uint32_t)v);
  const uint32_t hi = dpp_u32<kCtrl, kRowMask>((uint32_t)(o >> 32), (uint32_t)(v >> 32));
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Inclusive prefix sum over the 64 lanes (rows of 16 first, then across rows).
__device__ __forceinline__ double wave_incl_scan_dpp_f64(double x) {
  x += dpp_f64<kDppRowShr1>(0.0, x);
  x += dpp_f64<kDppRowShr2>(0.0, x);
  x += dpp_f64<kDppRowShr4>(0.0, x);
  x += dpp_f64<kDppRowShr8>(0.0, x);
  x += dpp_f64<kDppRowBcast15, 0xa>(0.0, x);
  x += dpp_f64<kDppRowBcast31, 0xc>(0.0, x);
  return x;
}
// Lane 63's value, in every lane.
__device__ __forceinline__ double last_lane_f64(double x) {
  const uint64_t u = (uint64_t)__double_as_longlong(x);
  const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, kWave - 1);
  const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), kWave - 1);
  return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}
// The inclusive value of the lane below (0 for lane 0): an exclusive prefix.
__device__ __forceinline__ double wave_shift_up_dpp_f64(double x) { return dpp_f64<kDppWaveShr1>(0.0, x); }

// Sum over the 64 lanes, returned as a wave-uniform value (DPP row scans,
// then lane 63).
__device__ __forceinline__ uint32_t wave_sum_dpp_u32(uint32_t x) {
  x += dpp_u32<kDppRowShr1>(0u, x);
  x += dpp_u32<kDppRowShr2>(0u, x);
  x += dpp_u32<kDppRowShr4>(0u, x);
  x += dpp_u32<kDppRowShr8>(0u, x);
  x += dpp_u32<kDppRowBcast15, 0xa>(0u, x);
  x += dpp_u32<kDppRowBcast31, 0xc>(0u, x);
  return (uint32_t)__builtin_amdgcn_readlane((int)x, kWave - 1);
}

// Maximum and minimum over the 64 lanes, wave-uniform.
__device__ __forceinline__ uint32_t wave_max_dpp_u32(uint32_t x) {
  x = max(x, dpp_u32<kDppRowShr1>(x, x));
  x = max(x, dpp_u32<kDppRowShr2>(x, x));
  x = max(x, dpp_u32<kDppRowShr4>(x, x));
  x = max(x, dpp_u32<kDppRowShr8>(x, x));
  x = max(x, dpp_u32<kDppRowBcast15, 0xa>(x, x));
  x = max(x, dpp_u32<kDppRowBcast31, 0xc>(x, x));
  return (uint32_t)__builtin_amdgcn_readlane((int)x, kWave - 1);
}
__device__ __forceinline__ uint32_t wave_min_dpp_u32(uint32_t x) {
  x = min(x, dpp_u32<kDppRowShr1>(x, x));
  x = min(x, dpp_u32<kDppRowShr2>(x, x));
  x = min(x, dpp_u32<kDppRowShr4>(x, x));
  x = min(x, dpp_u32<kDppRowShr8>(x, x));
  x = min(x, dpp_u32<kDppRowBcast15, 0xa>(x, x));
  x = min(x, dpp_u32<kDppRowBcast31, 0xc>(x, x));
  return (uint32_t)__builtin_amdgcn_readlane((int)x, kWave - 1);
}

__device__ __forceinline__ int wave_sum_i32(int x) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) x += __shfl_xor(x, off, kWave);
  return x;
}

}  // namespace sage
