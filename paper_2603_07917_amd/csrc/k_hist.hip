// Predicted output-length distribution of each request from its neighbours:
// counts per log-spaced length bin and the similarity-weighted mass.
#include "sage_device.hpp"
#include "sage_internal.hpp"

#include <algorithm>

namespace sage {
namespace {

// Fixed-point scale for the weights: every fp32 weight >= 2^-20 is an integer
// multiple of 2^-43, so w * 2^43 is an exact integer; weights below 2^11 keep
// a sum of up to 256 of them below 2^63. Integer sums are order independent.
constexpr double kWeightScale = 8796093022208.0;  // 2^43

// Largest b in [0, B-1] with edges[b] <= L (0 when L < edges[0]); edges in LDS.
__device__ __forceinline__ int length_bin(const double* edges, int B, int L) {
  const double x = (double)L;
  int lo = 0, hi = B;   // invariant: edges[lo] <= x or lo == 0; the answer is < hi
  while (hi - lo > 1) {
    const int mid = (lo + hi) >> 1;
    if (edges[mid] <= x) lo = mid; else hi = mid;
  }
  return lo;
}

constexpr int kMaxNbr = 256;   // SAGE_MAX_K

// WPR wavefronts per request and QPB requests per workgroup. LDS: the bin
// edges when kEdgesLds (shared by the workgroup; otherwise they are read from
// global memory through L1), then per request B uint64 fixed-point weights,
// B int32 counts and the request's totals. A neighbour at or above tau weighs
// its similarity, or 1 when `uniform` (the paper's unweighted form). With kVec
// (B % 4 == 0) each thread writes 4 consecutive bins with 16-byte stores.
template <int QPB, int WPR, bool kVec, bool kEdgesLds>
__global__ void __launch_bounds__(64 * QPB * WPR) hist_kernel(
    const int32_t* __restrict__ ids, const float* __restrict__ sims, int Q, int k,
    const int32_t* __restrict__ hist_len, int N, float tau, const double* __restrict__ edges, int B,
    int uniform, int32_t* __restrict__ counts, float* __restrict__ mass) {
  constexpr int kThreads = kWave * WPR;             // threads per request
  constexpr int kPer = kMaxNbr / kThreads;          // neighbours per thread at most
  extern __shared__ __align__(16) unsigned char smem[];
  const int r = threadIdx.x / kThreads;             // request within the workgroup
  const int t = threadIdx.x % kThreads;
  // LDS layout (8-byte words): edges [n_edges] | totals [QPB][2] | weights [QPB][B] | counts
  const int n_edges = kEdgesLds ? (B + 2) & ~1 : 0;  // B + 1 edges, padded to 16 bytes
  double* edges_s = reinterpret_cast<double*>(smem);
  uint64_t* tot = reinterpret_cast<uint64_t*>(smem) + n_edges + 2 * r;           // wtot, m
  uint64_t* wsum = reinterpret_cast<uint64_t*>(smem) + n_edges + 2 * QPB + (size_t)r * B;
  uint32_t* cnt = reinterpret_cast<uint32_t*>(reinterpret_cast<uint64_t*>(smem) + n_edges + 2 * QPB +
                                               (size_t)QPB * B) + (size_t)r * B;
  const double* edge = kEdgesLds ? edges_s : edges;
  const int q = blockIdx.x * QPB + r;
  const bool active = q < Q;

  // Neighbour lists first, so that their latency overlaps the LDS set-up.
  int32_t id[kPer];
  float sim[kPer];
  const size_t row = (size_t)q * (size_t)k;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    const int i = t + j * kThreads;
    const bool in = active && i < k;
    id[j] = in ? ids[row + i] : -1;
    sim[j] = in ? sims[row + i] : 0.0f;
  }
  if (kEdgesLds)
    for (int i = threadIdx.x; i <= B; i += blockDim.x) edges_s[i] = edges[i];
  for (int b = t; b < B; b += kThreads) { cnt[b] = 0u; wsum[b] = 0ull; }
  if (t < 2) tot[t] = 0ull;
  int32_t len[kPer];
#pragma unroll
  for (int j = 0; j < kPer; ++j) len[j] = (id[j] >= 0 && id[j] < N) ? hist_len[id[j]] : 0;
  __syncthreads();

  uint64_t wtot = 0;
  int m = 0;
#pragma unroll
  for (int j = 0; j < kPer; ++j) {
    if (id[j] < 0 || id[j] >= N) continue;
    const int b = length_bin(edge, B, len[j]);
    atomicAdd(&cnt[b], 1u);
    ++m;
    if (sim[j] >= tau) {
      const uint64_t fx = (uint64_t)((uniform ? 1.0 : (double)sim[j]) * kWeightScale);
      atomicAdd(reinterpret_cast<unsigned long long*>(&wsum[b]), (unsigned long long)fx);
      wtot += fx;
    }
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    wtot += (uint64_t)__shfl_xor((unsigned long long)wtot, off, kWave);
    m += __shfl_xor(m, off, kWave);
  }
  if (WPR > 1 && (t % kWave) == 0) {
    atomicAdd(reinterpret_cast<unsigned long long*>(&tot[0]), (unsigned long long)wtot);
    atomicAdd(reinterpret_cast<unsigned long long*>(&tot[1]), (unsigned long long)m);
  }
  __syncthreads();
  if (!active) return;
  if (WPR > 1) {
    wtot = tot[0];
    m = (int)tot[1];
  }
  const size_t out = (size_t)q * (size_t)B;
  const bool weighted = wtot > 0;
  const double scale = weighted ? 1.0 / (double)wtot : (m > 0 ? 1.0 / (double)m : 0.0);
  auto share = [&](uint32_t c, uint64_t ws) -> float {
    return (float)((weighted ? (double)ws : (double)c) * scale);
  };
  if (kVec) {
    for (int b = t * 4; b < B; b += 4 * kThreads) {
      const uint4 c = *reinterpret_cast<const uint4*>(cnt + b);
      const ulonglong2 s01 = *reinterpret_cast<const ulonglong2*>(wsum + b);
      const ulonglong2 s23 = *reinterpret_cast<const ulonglong2*>(wsum + b + 2);
      *reinterpret_cast<int4*>(counts + out + b) = make_int4((int)c.x, (int)c.y, (int)c.z, (int)c.w);
      *reinterpret_cast<float4*>(mass + out + b) =
          make_float4(share(c.x, s01.x), share(c.y, s01.y), share(c.z, s23.x), share(c.w, s23.y));
    }
  } else {
    for (int b = t; b < B; b += kThreads) {
      const uint32_t c = cnt[b];
      counts[out + b] = (int32_t)c;
      mass[out + b] = share(c, wsum[b]);
    }
  }
}

// Persistent waves, each with a private LDS region: wave v takes requests
// v, v + W, v + 2W, ... (W waves in the grid). While request r is binned, the
// lengths of request r + W are already being gathered and the neighbour
// lists of request r + 2W loaded, so a wave has three requests' memory
// traffic in flight and the chain lists -> lengths -> bins is paid once per
// wave rather than once per request. The only workgroup barrier is after
// the edges are staged; the per-request phases (clear, LDS atomics, read
// back) are ordered within the wave. Lane l holds neighbour slots
// l + 64 j (j < KPL = ceil(k / 64)). Weights as in hist_kernel (exact fixed
// point, order independent); kVec: B % 4 == 0, 16-byte stores of 4 bins.
template <int KPL, bool kVec>
__global__ void __launch_bounds__(256) hist_wave_kernel(
    const int32_t* __restrict__ ids, const float* __restrict__ sims, int Q, int k,
    const int32_t* __restrict__ hist_len, int N, float tau, const double* __restrict__ edges, int B,
    int uniform, int32_t* __restrict__ counts, float* __restrict__ mass) {
  extern __shared__ __align__(16) unsigned char smem[];
  constexpr int kWaves = 4;
  const int lane = (int)lane_id();
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  // LDS (8-byte words): edges [n_edges] | weights [4][B] | counts [4][B] (4-byte)
  const int n_edges = (B + 2) & ~1;
  double* edges_s = reinterpret_cast<double*>(smem);
  uint64_t* wsum = reinterpret_cast<uint64_t*>(smem) + n_edges + (size_t)w * B;
  uint32_t* cnt = reinterpret_cast<uint32_t*>(reinterpret_cast<uint64_t*>(smem) + n_edges + (size_t)kWaves * B) +
                  (size_t)w * B;
  for (int i = threadIdx.x; i <= B; i += blockDim.x) edges_s[i] = edges[i];

  const int W = gridDim.x * kWaves;
  const int q0 = blockIdx.x * kWaves + w;
  auto load_lists = [&](int q, int32_t (&id)[KPL], float (&sim)[KPL]) {
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      const int i = lane + j * kWave;
      const bool in = q < Q && i < k;
      id[j] = in ? ids[(size_t)q * k + i] : -1;
      sim[j] = in ? sims[(size_t)q * k + i] : 0.0f;
    }
  };
  auto gather = [&](const int32_t (&id)[KPL], int32_t (&len)[KPL]) {
#pragma unroll
    for (int j = 0; j < KPL; ++j) len[j] = (id[j] >= 0 && id[j] < N) ? hist_len[id[j]] : 0;
  };
  int32_t id_a[KPL], id_b[KPL], len_a[KPL];
  float sim_a[KPL], sim_b[KPL];
  load_lists(q0, id_a, sim_a);
  load_lists(q0 + W, id_b, sim_b);
  gather(id_a, len_a);
  __syncthreads();                                    // edges staged

  for (int q = q0; q < Q; q += W) {
    // In flight while request q is binned: lengths of q + W, lists of q + 2W.
    int32_t len_b[KPL], id_c[KPL];
    float sim_c[KPL];
    gather(id_b, len_b);
    load_lists(q + 2 * W, id_c, sim_c);
    for (int b = lane; b < B; b += kWave) { cnt[b] = 0u; wsum[b] = 0ull; }
    __builtin_amdgcn_wave_barrier();
    uint64_t wtot = 0;
    int m = 0;
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      if (id_a[j] < 0 || id_a[j] >= N) continue;
      const int b = length_bin(edges_s, B, len_a[j]);
      atomicAdd(&cnt[b], 1u);
      ++m;
      if (sim_a[j] >= tau) {
        const uint64_t fx = (uint64_t)((uniform ? 1.0 : (double)sim_a[j]) * kWeightScale);
        atomicAdd(reinterpret_cast<unsigned long long*>(&wsum[b]), (unsigned long long)fx);
        wtot += fx;
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      wtot += (uint64_t)__shfl_xor((unsigned long long)wtot, off, kWave);
      m += __shfl_xor(m, off, kWave);
    }
    __builtin_amdgcn_wave_barrier();
    const size_t out = (size_t)q * (size_t)B;
    const bool weighted = wtot > 0;
    const double scale = weighted ? 1.0 / (double)wtot : (m > 0 ? 1.0 / (double)m : 0.0);
    auto share = [&](uint32_t c, uint64_t ws) -> float {
      return (float)((weighted ? (double)ws : (double)c) * scale);
    };
    if (kVec) {
      for (int b = lane * 4; b < B; b += 4 * kWave) {
        const uint4 c = *reinterpret_cast<const uint4*>(cnt + b);
        const ulonglong2 s01 = *reinterpret_cast<const ulonglong2*>(wsum + b);
        const ulonglong2 s23 = *reinterpret_cast<const ulonglong2*>(wsum + b + 2);
        *reinterpret_cast<int4*>(counts + out + b) = make_int4((int)c.x, (int)c.y, (int)c.z, (int)c.w);
        *reinterpret_cast<float4*>(mass + out + b) =
            make_float4(share(c.x, s01.x), share(c.y, s01.y), share(c.z, s23.x), share(c.w, s23.y));
      }
    } else {
      for (int b = lane; b < B; b += kWave) {
        const uint32_t c = cnt[b];
        counts[out + b] = (int32_t)c;
        mass[out + b] = share(c, wsum[b]);
      }
    }
    __builtin_amdgcn_wave_barrier();                  // read back before the next clear
#pragma unroll
    for (int j = 0; j < KPL; ++j) {
      id_a[j] = id_b[j]; sim_a[j] = sim_b[j]; len_a[j] = len_b[j];
      id_b[j] = id_c[j]; sim_b[j] = sim_c[j];
    }
  }
}

}  // namespace

hipError_t launch_hist(const int32_t* ids, const float* sims, int Q, int k, const int32_t* hist_len,
                       int N, float tau, const double* edges, int B, int uniform, int32_t* counts,
                       float* mass, hipStream_t stream) {
  if (Q == 0) return hipSuccess;
  if (k > kMaxNbr) return hipErrorInvalidValue;
  LaunchScope scope("hist", stream);
  const bool vec = B % 4 == 0;
  // LDS bytes: edges (when staged) + per request 12 B per bin + 16 B of totals
#define SAGE_HIST_LAUNCH(QPB, WPR, VEC, ELDS)                                                        \
  hipLaunchKernelGGL((hist_kernel<QPB, WPR, VEC, ELDS>), dim3((Q + QPB - 1) / QPB),                 \
                     dim3(64 * QPB * WPR),                                                           \
                     (ELDS ? (size_t)((B + 2) & ~1) * 8 : 0) + (size_t)QPB * (B * 12 + 16), stream,  \
                     ids, sims, Q, k, hist_len, N, tau, edges, B, uniform, counts, mass)
  if (B <= 1024) {               // persistent waves, edges and per-wave bins in LDS
    // LDS: edges + 4 waves x 12 B per bin; about 8 workgroups per CU at B = 256.
    const size_t lds = (size_t)((B + 2) & ~1) * 8 + (size_t)4 * B * 12;
    const int per_cu = (int)std::min<size_t>(8, (160u << 10) / lds);
    const int blocks = (int)std::min<long long>((Q + 3) / 4, 256LL * per_cu);
#define SAGE_HIST_WAVE(KPL, VEC)                                                                        \
  hipLaunchKernelGGL((hist_wave_kernel<KPL, VEC>), dim3(blocks), dim3(256), lds, stream, ids, sims, Q, k, \
                     hist_len, N, tau, edges, B, uniform, counts, mass)
    const int kpl = (k + 63) / 64;
    if (vec) {
      if (kpl == 1) SAGE_HIST_WAVE(1, true); else if (kpl == 2) SAGE_HIST_WAVE(2, true); else SAGE_HIST_WAVE(4, true);
    } else {
      if (kpl == 1) SAGE_HIST_WAVE(1, false); else if (kpl == 2) SAGE_HIST_WAVE(2, false); else SAGE_HIST_WAVE(4, false);
    }
#undef SAGE_HIST_WAVE
  } else {                       // four waves per request, edges through L1
    if (vec) SAGE_HIST_LAUNCH(1, 4, true, false); else SAGE_HIST_LAUNCH(1, 4, false, false);
  }
#undef SAGE_HIST_LAUNCH
  return hipGetLastError();
}

}  // namespace sage
