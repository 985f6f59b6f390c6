// Gittins index scan (with the cost model fused in) and the radix-sort rank.
#include "sage_device.hpp"
#include "sage_internal.hpp"

namespace sage {
namespace {

// ---------------------------------------------------------------------------
// Index scan. One wavefront per request row; lane l owns the C consecutive
// bins [l*C, l*C + C), so a wave reads its row as one contiguous span.
//   F_b = sum_{j<=b} p_j, S_b = sum_{j<=b} p_j x_j, T_b = sum_{j>b} p_j,
//   G = min over b with F_b > 0 of (S_b + T_b x_b) / F_b.
// Candidates are compared by cross-multiplication (N_b F* < N* F_b), so a row
// costs one fp64 division. All sums are fp64.
// ---------------------------------------------------------------------------
template <int C>
__global__ void __launch_bounds__(256) index_kernel(const float* __restrict__ mass,
                                                    const float* __restrict__ cost,
                                                    const int32_t* __restrict__ prompt_len,
                                                    const double* __restrict__ repr, int Q, int B,
                                                    float* __restrict__ index,
                                                    int32_t* __restrict__ argmin) {
  constexpr bool kCacheRepr = C <= 16;
  const int lane = (int)lane_id();
  const int wave = (int)(blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave);
  const int n_waves = (int)(gridDim.x * (blockDim.x / kWave));
  const int b0 = lane * C;
  const bool fused = cost == nullptr;
  const bool full = b0 + C <= B;
  const bool vec = full && (C % 4 == 0) && (B % 4 == 0);

  double r_c[kCacheRepr ? C : 1], h_c[kCacheRepr ? C : 1];
  if (kCacheRepr && fused) {
#pragma unroll
    for (int j = 0; j < C; ++j) {
      const int b = b0 + j;
      const double r = b < B ? repr[b] : 0.0;
      r_c[j] = r;
      h_c[j] = r * r * 0.5;
    }
  }

  for (int q = wave; q < Q; q += n_waves) {
    const size_t row = (size_t)q * (size_t)B;
    float p[C];
    if (vec) {
#pragma unroll
      for (int j = 0; j < C; j += 4) {
        const float4 v = *reinterpret_cast<const float4*>(mass + row + b0 + j);
        p[j] = v.x; p[j + 1] = v.y; p[j + 2] = v.z; p[j + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int j = 0; j < C; ++j) p[j] = (b0 + j < B) ? mass[row + b0 + j] : 0.0f;
    }
    const double I = fused ? (double)prompt_len[q] : 0.0;

    // Lane-local suffix masses and totals.
    double t_loc[C];
    double lane_f = 0.0;
#pragma unroll
    for (int j = C - 1; j >= 0; --j) {
      t_loc[j] = lane_f;
      lane_f += (double)p[j];
    }
    double lane_s = 0.0;
    double x[C];
#pragma unroll
    for (int j = 0; j < C; ++j) {
      const int b = b0 + j;
      double xv;
      if (fused) {
        if (kCacheRepr) {
          xv = fma(I, r_c[j], h_c[j]);
        } else {
          const double r = b < B ? repr[b] : 0.0;
          xv = fma(I, r, r * r * 0.5);
        }
      } else {
        xv = b < B ? (double)cost[row + b] : 0.0;
      }
      x[j] = xv;
      lane_s = fma((double)p[j], xv, lane_s);
    }
    const double f_base = wave_excl_scan_f64(lane_f);
    const double s_base = wave_excl_scan_f64(lane_s);
    const double t_base = wave_excl_suffix_f64(lane_f);

    double best_n = 0.0, best_f = 0.0;
    int best_b = -1;
    double f_run = f_base, s_run = s_base;
#pragma unroll
    for (int j = 0; j < C; ++j) {
      f_run += (double)p[j];
      s_run = fma((double)p[j], x[j], s_run);
      const int b = b0 + j;
      if (f_run > 0.0 && b < B) {
        const double n = fma(t_base + t_loc[j], x[j], s_run);
        if (best_b < 0 || n * best_f < best_n * f_run) {
          best_n = n; best_f = f_run; best_b = b;
        }
      }
    }
    // Wave-wide minimum of n/f; ties keep the smaller bin.
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const double on = __shfl_xor(best_n, off, kWave);
      const double of = __shfl_xor(best_f, off, kWave);
      const int ob = __shfl_xor(best_b, off, kWave);
      bool take = false;
      if (ob >= 0) {
        if (best_b < 0) {
          take = true;
        } else {
          const double lhs = on * best_f, rhs = best_n * of;
          take = lhs < rhs || (lhs == rhs && ob < best_b);
        }
      }
      if (take) { best_n = on; best_f = of; best_b = ob; }
    }
    if (lane == 0) {
      index[q] = best_b >= 0 ? (float)(best_n / best_f) : __builtin_inff();
      if (argmin) argmin[q] = best_b;
    }
  }
}

template <int C>
hipError_t launch_index_c(const float* mass, const float* cost, const int32_t* prompt_len,
                          const double* repr, int Q, int B, float* index, int32_t* argmin,
                          hipStream_t stream) {
  const int waves_per_block = 4;
  const int rows_per_wave = 4;
  long waves = ((long)Q + rows_per_wave - 1) / rows_per_wave;
  long blocks = (waves + waves_per_block - 1) / waves_per_block;
  if (blocks > 65535) blocks = 65535;
  if (blocks < 1) blocks = 1;
  hipLaunchKernelGGL(index_kernel<C>, dim3((unsigned)blocks), dim3(64 * waves_per_block), 0, stream,
                     mass, cost, prompt_len, repr, Q, B, index, argmin);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Rank: stable least-significant-digit radix sort of the index keys (fp32
// bits made monotone, -0 folded onto +0), 8-bit digits, 4 passes. Each pass:
// per-tile digit counts, one exclusive scan over (digit, tile), then a stable
// scatter where each wave ranks equal digits with ballots.
// ---------------------------------------------------------------------------
constexpr int kRankThreads = 256;
constexpr int kRankItems = 8;
constexpr int kRankTile = kRankThreads * kRankItems;

__device__ __forceinline__ uint32_t index_key(float g) {
  uint32_t u = __float_as_uint(g);
  if (u == 0x80000000u) u = 0u;      // -0 sorts with +0
  return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__global__ void __launch_bounds__(kRankThreads) rank_hist_kernel(const float* __restrict__ g_in,
                                                                 const uint32_t* __restrict__ k_in,
                                                                 int Q, int shift, int n_tiles,
                                                                 uint32_t* __restrict__ hist) {
  __shared__ uint32_t cnt[256];
  cnt[threadIdx.x] = 0;
  __syncthreads();
  const int base = blockIdx.x * kRankTile;
#pragma unroll
  for (int it = 0; it < kRankItems; ++it) {
    const int i = base + it * kRankThreads + threadIdx.x;
    if (i < Q) {
      const uint32_t key = k_in ? k_in[i] : index_key(g_in[i]);
      atomicAdd(&cnt[(key >> shift) & 255u], 1u);
    }
  }
  __syncthreads();
  hist[threadIdx.x * n_tiles + blockIdx.x] = cnt[threadIdx.x];
}

// Exclusive scan of n entries in one workgroup of 1024 threads.
__global__ void __launch_bounds__(1024) rank_scan_kernel(uint32_t* __restrict__ a, int n) {
  __shared__ uint32_t part[1024];
  const int t = threadIdx.x;
  const int per = (n + 1023) / 1024;
  const int s = t * per;
  const int e = min(n, s + per);
  uint32_t sum = 0;
  for (int i = s; i < e; ++i) sum += a[i];
  part[t] = sum;
  __syncthreads();
  for (int off = 1; off < 1024; off <<= 1) {
    uint32_t v = t >= off ? part[t - off] : 0u;
    __syncthreads();
    part[t] += v;
    __syncthreads();
  }
  uint32_t run = part[t] - sum;
  for (int i = s; i < e; ++i) {
    const uint32_t v = a[i];
    a[i] = run;
    run += v;
  }
}

__global__ void __launch_bounds__(kRankThreads) rank_scatter_kernel(
    const float* __restrict__ g_in, const uint32_t* __restrict__ k_in,
    const uint32_t* __restrict__ v_in, int Q, int shift, int n_tiles,
    const uint32_t* __restrict__ offsets, uint32_t* __restrict__ k_out,
    uint32_t* __restrict__ v_out) {
  constexpr int kWaves = kRankThreads / kWave;
  __shared__ uint32_t base_off[256];
  __shared__ uint32_t running[256];
  __shared__ uint32_t wave_cnt[kWaves][256];
  const int t = threadIdx.x;
  const int lane = (int)lane_id();
  const int w = t / kWave;
  base_off[t] = offsets[t * n_tiles + blockIdx.x];
  running[t] = 0;
#pragma unroll
  for (int i = 0; i < kWaves; ++i) wave_cnt[i][t] = 0;
  __syncthreads();
  const int tile0 = blockIdx.x * kRankTile;
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  for (int it = 0; it < kRankItems; ++it) {
    const int i = tile0 + it * kRankThreads + t;
    const bool valid = i < Q;
    uint32_t key = 0, val = 0;
    if (valid) {
      key = k_in ? k_in[i] : index_key(g_in[i]);
      val = v_in ? v_in[i] : (uint32_t)i;
    }
    const uint32_t digit = (key >> shift) & 255u;
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int bit = 0; bit < 8; ++bit) {
      const bool on = (digit >> bit) & 1u;
      const uint64_t m = __ballot(on);
      peers &= on ? m : ~m;
    }
    const uint32_t rank_in_wave = (uint32_t)__popcll(peers & lt_mask);
    if (valid && rank_in_wave == 0) wave_cnt[w][digit] = (uint32_t)__popcll(peers);
    __syncthreads();
    uint32_t pos = 0;
    if (valid) {
      pos = base_off[digit] + running[digit] + rank_in_wave;
      for (int ww = 0; ww < w; ++ww) pos += wave_cnt[ww][digit];
    }
    __syncthreads();
    uint32_t add = 0;
#pragma unroll
    for (int ww = 0; ww < kWaves; ++ww) { add += wave_cnt[ww][t]; wave_cnt[ww][t] = 0; }
    running[t] += add;
    if (valid) {
      if (k_out) k_out[pos] = key;
      v_out[pos] = val;
    }
    __syncthreads();
  }
}

// Rank of a small queue (Q <= kRankSmallMax) in one workgroup of 1024
// threads: the same stable LSD radix sort (8-bit digits, 4 passes), with the
// keys and request ids kept in registers and scattered through LDS. Element
// e = 1024 r + t is item r of thread t, so rounds r run in index order. Per
// pass: digit totals (wave ballots), their exclusive scan, then per round the
// per-wave digit counts and a stable scatter.
constexpr int kRankSmallMax = 16384;
constexpr int kRankSmallThreads = 1024;
constexpr int kRankSmallItems = kRankSmallMax / kRankSmallThreads;

__global__ void __launch_bounds__(kRankSmallThreads) rank_small_kernel(const float* __restrict__ g_in, int Q,
                                                                       int32_t* __restrict__ order) {
  constexpr int kWaves = kRankSmallThreads / kWave;
  __shared__ uint32_t kbuf[kRankSmallMax];
  __shared__ uint32_t vbuf[kRankSmallMax];
  __shared__ uint32_t wave_cnt[kWaves][256];
  __shared__ uint32_t base[256];
  const int t = threadIdx.x;
  const int lane = (int)lane_id();
  const int w = t / kWave;
  const int rounds = (Q + kRankSmallThreads - 1) / kRankSmallThreads;
  const uint64_t lt_mask = (1ull << lane) - 1ull;
  uint32_t key[kRankSmallItems], val[kRankSmallItems];
#pragma unroll
  for (int r = 0; r < kRankSmallItems; ++r) {
    const int e = r * kRankSmallThreads + t;
    key[r] = e < Q ? index_key(g_in[e]) : 0u;
    val[r] = (uint32_t)e;
  }
  for (int i = t; i < kWaves * 256; i += kRankSmallThreads) (&wave_cnt[0][0])[i] = 0;
  __syncthreads();
  for (int shift = 0; shift < 32; shift += 8) {
    // digit totals (wave_cnt is all zero here)
#pragma unroll
    for (int r = 0; r < kRankSmallItems; ++r) {
      if (r >= rounds) break;
      const bool valid = r * kRankSmallThreads + t < Q;
      const uint32_t digit = (key[r] >> shift) & 255u;
      uint64_t peers = __ballot(valid);
#pragma unroll
      for (int bit = 0; bit < 8; ++bit) {
        const bool on = (digit >> bit) & 1u;
        const uint64_t m = __ballot(on);
        peers &= on ? m : ~m;
      }
      if (valid && __popcll(peers & lt_mask) == 0) wave_cnt[w][digit] += (uint32_t)__popcll(peers);
    }
    __syncthreads();
    if (t < 256) {                                     // read and clear column t
      uint32_t tot = 0;
#pragma unroll
      for (int i = 0; i < kWaves; ++i) { tot += wave_cnt[i][t]; wave_cnt[i][t] = 0; }
      base[t] = tot;
    }
    __syncthreads();
    if (t < kWave) {                                   // exclusive scan of 256 totals, 4 per lane
      uint32_t c[4], run = 0;
#pragma unroll
      for (int j = 0; j < 4; ++j) { c[j] = run; run += base[4 * t + j]; }
      uint32_t incl = run;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const uint32_t y = __shfl_up(incl, o, kWave);
        if (lane >= o) incl += y;
      }
      const uint32_t before = incl - run;
#pragma unroll
      for (int j = 0; j < 4; ++j) base[4 * t + j] = before + c[j];
    }
    __syncthreads();
    // stable scatter, round by round
#pragma unroll
    for (int r = 0; r < kRankSmallItems; ++r) {
      if (r >= rounds) break;
      const bool valid = r * kRankSmallThreads + t < Q;
      const uint32_t digit = (key[r] >> shift) & 255u;
      uint64_t peers = __ballot(valid);
#pragma unroll
      for (int bit = 0; bit < 8; ++bit) {
        const bool on = (digit >> bit) & 1u;
        const uint64_t m = __ballot(on);
        peers &= on ? m : ~m;
      }
      const uint32_t rank_in_wave = (uint32_t)__popcll(peers & lt_mask);
      if (valid && rank_in_wave == 0) wave_cnt[w][digit] = (uint32_t)__popcll(peers);
      __syncthreads();
      if (valid) {
        uint32_t pos = base[digit] + rank_in_wave;
        for (int i = 0; i < w; ++i) pos += wave_cnt[i][digit];
        kbuf[pos] = key[r];
        vbuf[pos] = val[r];
      }
      __syncthreads();
      if (t < 256) {                                   // advance column t, clear it for the next round
        uint32_t add = 0;
#pragma unroll
        for (int i = 0; i < kWaves; ++i) { add += wave_cnt[i][t]; wave_cnt[i][t] = 0; }
        base[t] += add;
      }
      __syncthreads();
    }
#pragma unroll
    for (int r = 0; r < kRankSmallItems; ++r) {
      const int e = r * kRankSmallThreads + t;
      if (e < Q) {
        key[r] = kbuf[e];
        val[r] = vbuf[e];
      }
    }
    __syncthreads();
  }
#pragma unroll
  for (int r = 0; r < kRankSmallItems; ++r) {
    const int e = r * kRankSmallThreads + t;
    if (e < Q) order[e] = (int32_t)val[r];
  }
}

}  // namespace

size_t rank_workspace_bytes(int Q) {
  if (Q <= 0) return 0;
  const size_t tiles = ((size_t)Q + kRankTile - 1) / kRankTile;
  return 4 * (size_t)Q * sizeof(uint32_t) + 256 * tiles * sizeof(uint32_t) + 256;
}

hipError_t launch_index(const float* mass, const float* cost, const int32_t* prompt_len,
                        const double* bin_repr, int Q, int B, float* index, int32_t* argmin,
                        hipStream_t stream) {
  if (Q == 0) return hipSuccess;
  LaunchScope scope("index_scan", stream);
  const int per_lane = (B + kWave - 1) / kWave;
  if (per_lane <= 1) return launch_index_c<1>(mass, cost, prompt_len, bin_repr, Q, B, index, argmin, stream);
  if (per_lane <= 2) return launch_index_c<2>(mass, cost, prompt_len, bin_repr, Q, B, index, argmin, stream);
  if (per_lane <= 4) return launch_index_c<4>(mass, cost, prompt_len, bin_repr, Q, B, index, argmin, stream);
  if (per_lane <= 8) return launch_index_c<8>(mass, cost, prompt_len, bin_repr, Q, B, index, argmin, stream);
  if (per_lane <= 16) return launch_index_c<16>(mass, cost, prompt_len, bin_repr, Q, B, index, argmin, stream);
  if (per_lane <= 32) return launch_index_c<32>(mass, cost, prompt_len, bin_repr, Q, B, index, argmin, stream);
  return launch_index_c<64>(mass, cost, prompt_len, bin_repr, Q, B, index, argmin, stream);
}

hipError_t launch_rank(const float* index, int Q, int32_t* order, void* ws, hipStream_t stream) {
  if (Q == 0) return hipSuccess;
  if (Q <= kRankSmallMax) {
    LaunchScope scope("rank_small", stream);
    hipLaunchKernelGGL(rank_small_kernel, dim3(1), dim3(kRankSmallThreads), 0, stream, index, Q, order);
    return hipGetLastError();
  }
  const int n_tiles = (Q + kRankTile - 1) / kRankTile;
  uint32_t* kA = static_cast<uint32_t*>(ws);
  uint32_t* vA = kA + Q;
  uint32_t* kB = vA + Q;
  uint32_t* vB = kB + Q;
  uint32_t* hist = vB + Q;
  const uint32_t* k_in = nullptr;
  const uint32_t* v_in = nullptr;
  for (int pass = 0; pass < 4; ++pass) {
    const int shift = 8 * pass;
    const bool last = pass == 3;
    uint32_t* k_out = last ? nullptr : (pass % 2 == 0 ? kA : kB);
    uint32_t* v_out = last ? reinterpret_cast<uint32_t*>(order) : (pass % 2 == 0 ? vA : vB);
    {
      LaunchScope scope("rank_hist", stream);
      hipLaunchKernelGGL(rank_hist_kernel, dim3(n_tiles), dim3(kRankThreads), 0, stream, index, k_in,
                         Q, shift, n_tiles, hist);
    }
    {
      LaunchScope scope("rank_scan", stream);
      hipLaunchKernelGGL(rank_scan_kernel, dim3(1), dim3(1024), 0, stream, hist, 256 * n_tiles);
    }
    {
      LaunchScope scope("rank_scatter", stream);
      hipLaunchKernelGGL(rank_scatter_kernel, dim3(n_tiles), dim3(kRankThreads), 0, stream, index,
                         k_in, v_in, Q, shift, n_tiles, hist, k_out, v_out);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    k_in = k_out;
    v_in = v_out;
  }
  return hipSuccess;
}

}  // namespace sage
