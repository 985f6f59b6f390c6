// Predicted output-length distribution of each request from its neighbours:
// counts per log-spaced length bin and the similarity-weighted mass.
#include "sage_device.hpp"
#include "sage_internal.hpp"

namespace sage {
namespace {

// Fixed-point scale for the weights: every fp32 weight >= 2^-20 is an integer
// multiple of 2^-43, so w * 2^43 is an exact integer; weights below 2^11 keep
// a sum of up to 256 of them below 2^63. Integer sums are order independent.
constexpr double kWeightScale = 8796093022208.0;  // 2^43

// Largest b in [0, B-1] with edges[b] <= L (0 when L < edges[0]).
__device__ __forceinline__ int length_bin(const double* __restrict__ edges, int B, int L) {
  const double x = (double)L;
  int lo = 0, hi = B;   // invariant: edges[lo] <= x or lo == 0; the answer is < hi
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (edges[mid] <= x) lo = mid; else hi = mid;
  }
  return lo;
}

// One wavefront per request; QPB requests per workgroup share nothing but
// the launch. LDS per wave: B int32 counts + B uint64 fixed-point weights.
// A neighbour at or above tau weighs its similarity, or 1 when `uniform`
// (the paper's unweighted form).
template <int QPB>
__global__ void __launch_bounds__(64 * QPB) hist_kernel(
    const int32_t* __restrict__ ids, const float* __restrict__ sims, int Q, int k,
    const int32_t* __restrict__ hist_len, int N, float tau, const double* __restrict__ edges, int B,
    int uniform, int32_t* __restrict__ counts, float* __restrict__ mass) {
  extern __shared__ __align__(16) unsigned char smem[];
  const int w = threadIdx.x / kWave;
  const int lane = (int)lane_id();
  uint64_t* wsum = reinterpret_cast<uint64_t*>(smem) + (size_t)w * B;
  uint32_t* cnt = reinterpret_cast<uint32_t*>(reinterpret_cast<uint64_t*>(smem) + (size_t)QPB * B) +
                  (size_t)w * B;
  const int q = blockIdx.x * QPB + w;
  const bool active = q < Q;

  for (int b = lane; b < B; b += kWave) { cnt[b] = 0u; wsum[b] = 0ull; }
  __syncthreads();

  uint64_t wtot = 0;
  int m = 0;
  if (active) {
    const size_t row = (size_t)q * (size_t)k;
    for (int i = lane; i < k; i += kWave) {
      const int32_t id = ids[row + i];
      if (id < 0 || id >= N) continue;
      const int b = length_bin(edges, B, hist_len[id]);
      atomicAdd(&cnt[b], 1u);
      ++m;
      const float s = sims[row + i];
      if (s >= tau) {
        const uint64_t fx = (uint64_t)((uniform ? 1.0 : (double)s) * kWeightScale);
        atomicAdd(reinterpret_cast<unsigned long long*>(&wsum[b]), (unsigned long long)fx);
        wtot += fx;
      }
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    wtot += (uint64_t)__shfl_xor((unsigned long long)wtot, off, kWave);
    m += __shfl_xor(m, off, kWave);
  }
  __syncthreads();
  if (!active) return;
  const size_t out = (size_t)q * (size_t)B;
  const double inv_m = m > 0 ? 1.0 / (double)m : 0.0;
  for (int b = lane; b < B; b += kWave) {
    const uint32_t c = cnt[b];
    counts[out + b] = (int32_t)c;
    float v;
    if (wtot > 0) v = (float)((double)wsum[b] / (double)wtot);
    else v = (float)((double)c * inv_m);
    mass[out + b] = v;
  }
}

}  // namespace

hipError_t launch_hist(const int32_t* ids, const float* sims, int Q, int k, const int32_t* hist_len,
                       int N, float tau, const double* edges, int B, int uniform, int32_t* counts,
                       float* mass, hipStream_t stream) {
  if (Q == 0) return hipSuccess;
  LaunchScope scope("hist", stream);
  if (B <= 1024) {
    constexpr int qpb = 4;
    const size_t lds = (size_t)qpb * B * 12;
    hipLaunchKernelGGL(hist_kernel<qpb>, dim3((Q + qpb - 1) / qpb), dim3(64 * qpb), lds, stream, ids,
                       sims, Q, k, hist_len, N, tau, edges, B, uniform, counts, mass);
  } else {
    const size_t lds = (size_t)B * 12;
    hipLaunchKernelGGL(hist_kernel<1>, dim3(Q), dim3(64), lds, stream, ids, sims, Q, k, hist_len,
                       N, tau, edges, B, uniform, counts, mass);
  }
  return hipGetLastError();
}

}  // namespace sage
