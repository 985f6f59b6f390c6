// The semantic-unaware history-based predictor of the predictor ablation
// (Sec. 4.3): a request's neighbours are the history records whose input
// length is most similar to its own, instead of those whose prompt is. The
// similarity of input lengths I and L is s = min(I, L) / max(I, L), the fp32
// quotient (correctly rounded), so that the predictor's threshold (0.8)
// keeps its meaning; lengths below 1 count as 1, stored lengths above
// max_len as max_len. Neighbours are the k largest s, ties to the lower
// history index, and go through the same histogram as the semantic
// predictor's.
//
// With max_len <= 2^20, two stored lengths on the same side of I never share
// an fp32 similarity (neighbouring quotients differ by far more than their
// rounding), so each side holds at most one length run at a given level.
//
// Length index (built once per store): the record indices sorted by input
// length (ties by index: the stable rank of the lengths), the sorted lengths,
// and off[L] = the first sorted position with length >= L (L = 0..max_len+1).
// Records with s >= sigma are those whose length lies in one interval
// [Lmin(sigma), Lmax(sigma)] around the query's length (s rises up to L = I
// and falls after it), so their number is off[Lmax + 1] - off[Lmin].
//
// Query (one wavefront each): the k-th largest similarity level sigma* is
// found by a 64-way search over the fp32 bit patterns of sigma in [0, 1]
// (each lane counts the records at or above one candidate, five rounds).
// The records above sigma* (fewer than k) are one contiguous range of the
// sorted positions; those at sigma* sit in at most one length run on each
// side, each sorted by index, so the lowest indices are the first ones of
// each run. At most 2k keys (similarity bits, ~index) are then sorted in
// LDS and the first k written.
#include "sage_device.hpp"
#include "sage_internal.hpp"

namespace sage {
namespace {

constexpr int kThreads = 256;
constexpr int kMaxKeys = 512;                      // 2 SAGE_MAX_K

__device__ __forceinline__ int clamp_len(int L, int max_len) { return min(max(L, 1), max_len); }

// fp32 similarity of input lengths I and L (both >= 1), IEEE division.
__device__ __forceinline__ float len_sim(int I, int L) {
  const int a = min(I, L), b = max(I, L);
  return __fdiv_rn((float)a, (float)b);
}

// [Lmin, Lmax] of lengths in [1, max_len] with len_sim >= sigma; Lmin > Lmax
// when none. P = min(I, max_len) has the largest similarity.
__device__ __forceinline__ int2 level_range(float sigma, int I, int max_len) {
  const int P = min(I, max_len);
  if (!(len_sim(I, P) >= sigma)) return make_int2(1, 0);
  int lo = 1, hi = P;                              // smallest L in [1, P] with s >= sigma
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (len_sim(I, mid) >= sigma) hi = mid; else lo = mid + 1;
  }
  const int lmin = lo;
  lo = P;
  hi = max_len;                                    // largest L in [P, max_len] with s >= sigma
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (len_sim(I, mid) >= sigma) lo = mid; else hi = mid - 1;
  }
  return make_int2(lmin, lo);
}

__device__ __forceinline__ int count_range(const int32_t* off, int2 r) {
  return r.x > r.y ? 0 : off[r.y + 1] - off[r.x];
}

__global__ void length_keys_kernel(const int32_t* __restrict__ len, int N, int max_len, float* __restrict__ key) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < N) key[i] = (float)clamp_len(len[i], max_len);
}

__global__ void length_sorted_kernel(const int32_t* __restrict__ len, const int32_t* __restrict__ by_len, int N,
                                     int max_len, int32_t* __restrict__ sorted_len) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i < N) sorted_len[i] = clamp_len(len[by_len[i]], max_len);
}

// off[L] = first position p with sorted_len[p] >= L (N if none), L = 0..max_len+1.
__global__ void length_offsets_kernel(const int32_t* __restrict__ sorted_len, int N, int max_len,
                                      int32_t* __restrict__ off) {
  const int L = blockIdx.x * blockDim.x + threadIdx.x;
  if (L > max_len + 1) return;
  int lo = 0, hi = N;
  while (lo < hi) {
    const int mid = (lo + hi) >> 1;
    if (sorted_len[mid] >= L) hi = mid; else lo = mid + 1;
  }
  off[L] = lo;
}

__global__ void __launch_bounds__(kThreads) length_neighbours_kernel(
    const int32_t* __restrict__ prompt_len, int Q, const int32_t* __restrict__ by_len,
    const int32_t* __restrict__ sorted_len, const int32_t* __restrict__ off, int max_len, int N, int k,
    int32_t* __restrict__ ids, float* __restrict__ sims) {
  __shared__ uint64_t keys_s[kThreads / kWave][kMaxKeys];
  const int lane = (int)lane_id();
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  const int q = blockIdx.x * (kThreads / kWave) + w;
  if (q >= Q) return;                               // whole wavefronts; no workgroup barrier below
  uint64_t* keys = keys_s[w];
  const int I = max(prompt_len[q], 1);
  const int total = off[max_len + 1] - off[1];      // every record (lengths are clamped to [1, max_len])

  // Ranges of positions to gather: all of [mb, me), and the first r of
  // [lb, le) and of [rb, re).
  int mb = off[1], me = off[max_len + 1], lb = 0, le = 0, rb = 0, re = 0, r = 0;
  if (total > k) {
    // Largest sigma (as fp32 bits) with at least k records at or above it.
    uint32_t lo = 0u, hi = 0x3F800001u;             // count(lo) = total >= k; count(hi) = 0 < k
    while (hi - lo > 1u) {
      const uint32_t p = lo + (uint32_t)(((uint64_t)(hi - lo) * (uint64_t)(lane + 1)) / 65u);
      const bool enough = count_range(off, level_range(__uint_as_float(p), I, max_len)) >= k;
      const uint64_t m = __ballot(enough);
      if (m == 0) {
        hi = __shfl(p, 0, kWave);
      } else {
        const int j = 63 - __clzll(m);              // the counts fall with sigma: the ballot is a prefix
        const uint32_t pj = __shfl(p, j, kWave);
        hi = j == kWave - 1 ? hi : __shfl(p, j + 1, kWave);
        lo = pj;
      }
    }
    const int2 at = level_range(__uint_as_float(lo), I, max_len);      // s >= sigma*
    const int2 above = level_range(__uint_as_float(hi), I, max_len);   // s > sigma*
    const int P = min(I, max_len);
    int split_lo, split_hi;                         // length runs at sigma*: [at.x, split_lo), (split_hi, at.y]
    if (above.x <= above.y) {
      mb = off[above.x];
      me = off[above.y + 1];
      split_lo = above.x;
      split_hi = above.y;
    } else {
      mb = me = 0;
      split_lo = min(P, at.y) + 1;
      split_hi = min(P, at.y);
    }
    lb = off[at.x];
    le = off[split_lo];
    rb = off[split_hi + 1];
    re = off[at.y + 1];
    r = k - (me - mb);
  }
  // Gather the keys: the range above sigma*, then the first r of each run.
  const int n_mid = me - mb, n_l = min(r, le - lb), n_r = min(r, re - rb);
  const int n_keys = n_mid + n_l + n_r;             // <= 2k (or every record when total <= k)
  int n_pow = kWave;                               // a power of two holding the keys and the k outputs
  while (n_pow < n_keys || n_pow < k) n_pow <<= 1;
  for (int i = lane; i < n_pow; i += kWave) {
    uint64_t key = kPadKey;
    if (i < n_keys) {
      const int p = i < n_mid ? mb + i : (i < n_mid + n_l ? lb + (i - n_mid) : rb + (i - n_mid - n_l));
      key = make_key(len_sim(I, sorted_len[p]), (uint32_t)by_len[p]);
    }
    keys[i] = key;
  }
  __builtin_amdgcn_wave_barrier();
  // Bitonic sort of the n_pow keys in LDS, descending (one wave).
  for (int size = 2; size <= n_pow; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int i = lane; i < n_pow / 2; i += kWave) {
        const int a = 2 * stride * (i / stride) + (i % stride), b = a + stride;
        const bool desc = (a & size) == 0;
        const uint64_t x = keys[a], y = keys[b];
        if ((x < y) == desc) { keys[a] = y; keys[b] = x; }
      }
      __builtin_amdgcn_wave_barrier();
    }
  }
  for (int i = lane; i < k; i += kWave) {
    const uint64_t key = keys[i];
    ids[(size_t)q * k + i] = key == kPadKey ? -1 : key_id(key);
    sims[(size_t)q * k + i] = key == kPadKey ? -__builtin_inff() : key_sim(key);
  }
}

}  // namespace

size_t length_index_workspace_bytes(int N) {
  return ((size_t)N * sizeof(float) + 255) / 256 * 256 + rank_workspace_bytes(N);
}

hipError_t launch_length_index(const int32_t* hist_prompt_len, int N, int max_len, int32_t* by_len,
                               int32_t* sorted_len, int32_t* off, void* ws, hipStream_t stream) {
  float* key = static_cast<float*>(ws);
  void* rank_ws = static_cast<char*>(ws) + ((size_t)N * sizeof(float) + 255) / 256 * 256;
  LaunchScope scope("length_index", stream);
  hipLaunchKernelGGL(length_keys_kernel, dim3((N + 255) / 256), dim3(256), 0, stream, hist_prompt_len, N, max_len,
                     key);
  hipError_t e = launch_rank(key, N, by_len, rank_ws, stream);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL(length_sorted_kernel, dim3((N + 255) / 256), dim3(256), 0, stream, hist_prompt_len, by_len,
                     N, max_len, sorted_len);
  hipLaunchKernelGGL(length_offsets_kernel, dim3((max_len + 2 + 255) / 256), dim3(256), 0, stream, sorted_len, N,
                     max_len, off);
  return hipGetLastError();
}

hipError_t launch_length_neighbours(const int32_t* prompt_len, int Q, const int32_t* by_len,
                                    const int32_t* sorted_len, const int32_t* off, int max_len, int N, int k,
                                    int32_t* ids, float* sims, hipStream_t stream) {
  if (Q == 0) return hipSuccess;
  if (k > kMaxKeys / 2) return hipErrorInvalidValue;
  LaunchScope scope("length_neighbours", stream);
  hipLaunchKernelGGL(length_neighbours_kernel, dim3((Q + 3) / 4), dim3(kThreads), 0, stream, prompt_len, Q, by_len,
                     sorted_len, off, max_len, N, k, ids, sims);
  return hipGetLastError();
}

}  // namespace sage
