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
template <int C, bool kFull>
__device__ __forceinline__ void load_row(const float* __restrict__ mass, size_t row, int b0, int B,
                                         float (&p)[C]) {
  if (kFull && C % 4 == 0) {
#pragma unroll
    for (int j = 0; j < C; j += 4) {
      const float4 v = *reinterpret_cast<const float4*>(mass + row + b0 + j);
      p[j] = v.x; p[j + 1] = v.y; p[j + 2] = v.z; p[j + 3] = v.w;
    }
  } else {
#pragma unroll
    for (int j = 0; j < C; ++j) p[j] = (kFull || b0 + j < B) ? mass[row + b0 + j] : 0.0f;
  }
}

// kFull: B == 64 C, so every lane owns C real bins (no guards, vector loads).
// kMode: kGivenCost takes the support from the cost matrix; kFused computes
// it from the prompt length and the representatives (kept in LDS);
// kAttained also refreshes running requests: with o = bucket *
// floor(generated / bucket) tokens served, a = o^2 / 2 + I o, the bins with
// x <= a are ruled out and the rest are shifted down by a, so the result is
// the index of the remaining cost. kVariant takes the cost model, the kind
// of index (Gittins or mean) and a uniform-mixing weight at run time.
// kTable: kAttained for every row at each level o = lv * bucket (lv < levels).
enum IndexMode { kGivenCost = 0, kFused = 1, kAttained = 2, kVariant = 3, kTable = 4 };
// Workgroups per CU the register budget is tuned for (4 waves each).
template <int C> struct IndexOcc { static constexpr int value = C <= 8 ? 4 : (C == 16 ? 3 : 1); };

constexpr int kNoBin = 0x7fffffff;   // a lane without a candidate bin

template <int C, bool kFull, int kMode, bool kArg>
__global__ void __launch_bounds__(256, IndexOcc<C>::value) index_kernel(const float* __restrict__ mass,
                                                    const float* __restrict__ cost,
                                                    const int32_t* __restrict__ prompt_len,
                                                    const double* __restrict__ repr,
                                                    const int32_t* __restrict__ generated, int bucket,
                                                    int Q, int B, float* __restrict__ index,
                                                    int32_t* __restrict__ argmin, IndexVariant var) {
  constexpr bool kFused = kMode != kGivenCost;
  extern __shared__ double repr_s[];               // [B] representatives (fused cost only)
  const int lane = (int)lane_id();
  const int wave = (int)(blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave);
  const int n_waves = (int)(gridDim.x * (blockDim.x / kWave));
  const int b0 = lane * C;
  if (kFused) {
    for (int b = threadIdx.x; b < B; b += blockDim.x) repr_s[b] = repr[b];
    __syncthreads();
  }

  float p[C], p_next[C];
  // Refresh table (kTable): every row at each level o = lv * bucket, from
  // one read of the row; index[lv * Q + q]. One level in every other mode.
  constexpr bool kAtt = kMode == kAttained || kMode == kTable;
  const int n_lv = kMode == kTable ? var.levels : 1;
  if (wave < Q) load_row<C, kFull>(mass, (size_t)wave * B, b0, B, p_next);
  for (int q = wave; q < Q; q += n_waves) {
    const size_t row = (size_t)q * (size_t)B;
#pragma unroll
    for (int j = 0; j < C; ++j) p[j] = p_next[j];
    if (q + n_waves < Q) load_row<C, kFull>(mass, row + (size_t)n_waves * B, b0, B, p_next);   // prefetch
    const double I = kFused ? (double)prompt_len[q] : 0.0;
   for (int lv = 0; lv < n_lv; ++lv) {
    const size_t out = (size_t)lv * (size_t)Q + (size_t)q;
    double a = 0.0;                                 // service already received
    if (kAtt) {
      const double o = kMode == kTable ? (double)lv * (double)bucket
                                       : (double)((max(generated[q], 0) / bucket) * bucket);
      a = o * fma(0.5, o, I);
    }

    // Support x_j = r (I + r / 2) (or the given cost); recomputed where used,
    // which keeps the register count (and so the occupancy) down.
    auto support = [&](int j) -> double {
      const int b = b0 + j;
      const bool in = kFull || b < B;
      if (kMode == kVariant) {
        const double r = in ? repr_s[b] : 0.0;
        if (var.cost_model == 1) return r;                       // output length
        if (var.cost_model == 2) return fma(2.0, r, I);          // input + 2 output
        return r * fma(0.5, r, I);
      }
      if (kFused) {
        const double r = in ? repr_s[b] : 0.0;
        return r * fma(0.5, r, I);
      }
      return in ? (double)cost[row + b] : 0.0;
    };
    if (kMode == kVariant && var.noise > 0.0f) {     // p' = (1 - w) p / sum(p) + w / B
      double raw = 0.0;
#pragma unroll
      for (int j = 0; j < C; ++j) raw += (double)p[j];
      const double tot = last_lane_f64(wave_incl_scan_dpp_f64(raw));
      if (tot > 0.0) {
        const double keep = (1.0 - (double)var.noise) / tot, spread = (double)var.noise / (double)B;
#pragma unroll
        for (int j = 0; j < C; ++j)
          if (kFull || b0 + j < B) p[j] = (float)fma(keep, (double)p[j], spread);
      }
    }
    // The mass of bin j; with attained service, the outcomes already passed
    // (x <= a) are ruled out (p itself is kept for the next level).
    auto pm = [&](int j) -> double {
      if (kAtt && !(support(j) > a)) return 0.0;
      return (double)p[j];
    };
    double lane_f = 0.0, lane_s = 0.0;
#pragma unroll
    for (int j = 0; j < C; ++j) {
      lane_f += pm(j);
      lane_s = fma(pm(j), support(j) - a, lane_s);
    }
    // Prefix sums over lanes (DPP); the mass above this lane is the row total
    // minus the inclusive prefix (fp64, so its rounding is ~1e-16 of the total).
    const double f_incl = wave_incl_scan_dpp_f64(lane_f);
    const double f_base = wave_shift_up_dpp_f64(f_incl);
    const double s_base = wave_shift_up_dpp_f64(wave_incl_scan_dpp_f64(lane_s));
    const double f_total = last_lane_f64(f_incl);
    const double t_base = f_total - f_incl;
    if (kMode == kVariant && var.kind == 1) {        // the mean: sum p x / sum p
      const double s_incl = s_base + lane_s;
      if (lane == kWave - 1) {
        index[out] = f_total > 0.0 ? (float)(s_incl / f_total) : __builtin_inff();
        if (kArg) argmin[out] = -1;
      }
      continue;
    }

    // Branch-free running minimum of n / f by cross-multiplication; the
    // start values (n, f) = (1, 0) lose to the first bin with f > 0 (f never
    // decreases, so no bin with f = 0 can win later), and a later bin must be
    // strictly smaller to win (ties keep the lower bin).
    double best_n = 1.0, best_f = 0.0;
    int best_b = kNoBin;
    double f_run = f_base, s_run = s_base, t_run = f_total - f_base;
#pragma unroll
    for (int j = 0; j < C; ++j) {
      const double pj = pm(j);
      const double xj = support(j) - a;
      f_run += pj;
      s_run = fma(pj, xj, s_run);
      t_run -= pj;                                  // mass strictly above bin j
      const double n = fma(t_run, xj, s_run);
      const bool take = (kFull || b0 + j < B) && n * best_f < best_n * f_run;
      best_n = take ? n : best_n;
      best_f = take ? f_run : best_f;
      if (kArg) best_b = take ? b0 + j : best_b;
    }
    // One division per lane, then the wave-wide minimum of the ratios
    // (ties keep the smaller bin when the argmin is wanted): butterflies within
    // rows of 16 (quads, half rows, rows), then rows 0+1 -> 1, 2+3 -> 3 and
    // 1 -> 3; lane 63 ends with the row's result. Lanes without a candidate
    // carry +inf and lose every tie.
    double r = best_f > 0.0 ? best_n / best_f : __builtin_inf();
    if (kArg) {
      auto combine = [&](double orr, int ob) {
        const bool take = orr < r || (orr == r && ob < best_b);
        r = take ? orr : r;
        best_b = take ? ob : best_b;
      };
#define SAGE_ARGMIN_STEP(CTRL, ROWS) \
      combine(dpp_f64<CTRL, ROWS>(r, r), (int)dpp_u32<CTRL, ROWS>((uint32_t)best_b, (uint32_t)best_b))
      SAGE_ARGMIN_STEP(kDppQuadXor1, 0xf);
      SAGE_ARGMIN_STEP(kDppQuadXor2, 0xf);
      SAGE_ARGMIN_STEP(kDppRowHalfMirror, 0xf);
      SAGE_ARGMIN_STEP(kDppRowMirror, 0xf);
      SAGE_ARGMIN_STEP(kDppRowBcast15, 0xa);
      SAGE_ARGMIN_STEP(kDppRowBcast31, 0xc);
#undef SAGE_ARGMIN_STEP
    } else {
      r = fmin(r, dpp_f64<kDppQuadXor1, 0xf>(r, r));
      r = fmin(r, dpp_f64<kDppQuadXor2, 0xf>(r, r));
      r = fmin(r, dpp_f64<kDppRowHalfMirror, 0xf>(r, r));
      r = fmin(r, dpp_f64<kDppRowMirror, 0xf>(r, r));
      r = fmin(r, dpp_f64<kDppRowBcast15, 0xa>(r, r));
      r = fmin(r, dpp_f64<kDppRowBcast31, 0xc>(r, r));
    }
    if (lane == kWave - 1) {
      const bool found = r < __builtin_inf();
      index[out] = found ? (float)r : __builtin_inff();
      if (kArg) argmin[out] = found ? best_b : -1;
    }
   }
  }
}

template <int C, bool kFull, int kMode>
hipError_t launch_index_v(const float* mass, const float* cost, const int32_t* prompt_len,
                          const double* repr, const int32_t* generated, int bucket, int Q, int B,
                          float* index, int32_t* argmin, hipStream_t stream, IndexVariant var) {
  const int waves_per_block = 4;
  const int rows_per_wave = 4;
  long waves = ((long)Q + rows_per_wave - 1) / rows_per_wave;
  long blocks = (waves + waves_per_block - 1) / waves_per_block;
  if (blocks > 65535) blocks = 65535;
  if (blocks < 1) blocks = 1;
  const size_t lds = kMode != kGivenCost ? (size_t)B * sizeof(double) : 0;   // representatives
  if (argmin)
    hipLaunchKernelGGL((index_kernel<C, kFull, kMode, true>), dim3((unsigned)blocks),
                       dim3(64 * waves_per_block), lds, stream, mass, cost, prompt_len, repr, generated,
                       bucket, Q, B, index, argmin, var);
  else
    hipLaunchKernelGGL((index_kernel<C, kFull, kMode, false>), dim3((unsigned)blocks),
                       dim3(64 * waves_per_block), lds, stream, mass, cost, prompt_len, repr, generated,
                       bucket, Q, B, index, argmin, var);
  return hipGetLastError();
}

template <int C>
hipError_t launch_index_c(const float* mass, const float* cost, const int32_t* prompt_len,
                          const double* repr, const int32_t* generated, int bucket, int Q, int B,
                          float* index, int32_t* argmin, hipStream_t stream, const IndexVariant* variant) {
  const bool full = B == 64 * C;
  const int mode = (variant && variant->levels > 0) ? kTable
                   : variant ? kVariant : (generated ? kAttained : (cost ? kGivenCost : kFused));
  const IndexVariant var = variant ? *variant : IndexVariant();
#define SAGE_INDEX_LAUNCH(FULL, MODE)                                                               \
  return launch_index_v<C, FULL, MODE>(mass, cost, prompt_len, repr, generated, bucket, Q, B, index, \
                                       argmin, stream, var)
  if (mode == kVariant) {
    if (full) SAGE_INDEX_LAUNCH(true, kVariant);
    SAGE_INDEX_LAUNCH(false, kVariant);
  }
  if (mode == kTable) {
    if (full) SAGE_INDEX_LAUNCH(true, kTable);
    SAGE_INDEX_LAUNCH(false, kTable);
  }
  if (full) {
    if (mode == kAttained) SAGE_INDEX_LAUNCH(true, kAttained);
    if (mode == kFused) SAGE_INDEX_LAUNCH(true, kFused);
    SAGE_INDEX_LAUNCH(true, kGivenCost);
  }
  if (mode == kAttained) SAGE_INDEX_LAUNCH(false, kAttained);
  if (mode == kFused) SAGE_INDEX_LAUNCH(false, kFused);
  SAGE_INDEX_LAUNCH(false, kGivenCost);
#undef SAGE_INDEX_LAUNCH
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
// Per-digit exclusive scan over the tiles: workgroup d scans hist[d][0..n_tiles)
// in place (contiguous, 256 counts per turn) and leaves the digit's total in
// total[d]. The scatter adds the exclusive scan of the 256 totals.
__global__ void __launch_bounds__(256) rank_scan_kernel(uint32_t* __restrict__ hist, int n_tiles,
                                                        uint32_t* __restrict__ total) {
  __shared__ uint32_t wsum[4];
  const int t = threadIdx.x;
  const int lane = (int)lane_id();
  const int w = t / kWave;
  uint32_t* row = hist + (size_t)blockIdx.x * n_tiles;
  uint32_t carry = 0;
  for (int base = 0; base < n_tiles; base += 256) {
    const int i = base + t;
    const uint32_t v = i < n_tiles ? row[i] : 0u;
    uint32_t incl = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const uint32_t y = (uint32_t)__shfl_up((int)incl, o, kWave);
      if (lane >= o) incl += y;
    }
    if (lane == kWave - 1) wsum[w] = incl;
    __syncthreads();
    uint32_t before = carry;
    for (int ww = 0; ww < w; ++ww) before += wsum[ww];
    if (i < n_tiles) row[i] = before + incl - v;
    carry += wsum[0] + wsum[1] + wsum[2] + wsum[3];
    __syncthreads();
  }
  if (t == 0) total[blockIdx.x] = carry;
}

__global__ void __launch_bounds__(kRankThreads) rank_scatter_kernel(
    const float* __restrict__ g_in, const uint32_t* __restrict__ k_in,
    const uint32_t* __restrict__ v_in, int Q, int shift, int n_tiles,
    const uint32_t* __restrict__ offsets, const uint32_t* __restrict__ digit_total, int fused,
    uint32_t* __restrict__ k_out, uint32_t* __restrict__ v_out) {
  constexpr int kWaves = kRankThreads / kWave;
  __shared__ uint32_t base_off[256];
  __shared__ uint32_t running[256];
  __shared__ uint32_t wave_cnt[kWaves][256];
  const int t = threadIdx.x;
  const int lane = (int)lane_id();
  const int w = t / kWave;
  {
    // exclusive scan of the 256 digit totals (one per thread), plus this
    // tile's offset within the digit. `fused` (few tiles): both from the raw
    // per-tile counts, offsets[digit][tile], read here (no scan kernel).
    uint32_t v, tile_off;
    if (fused) {
      const uint32_t* row = offsets + (size_t)t * n_tiles;
      v = 0;
      tile_off = 0;
      for (int i = 0; i < n_tiles; ++i) {
        const uint32_t c = row[i];
        if (i == (int)blockIdx.x) tile_off = v;
        v += c;
      }
    } else {
      v = digit_total[t];
      tile_off = offsets[t * n_tiles + blockIdx.x];
    }
    uint32_t incl = v;
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const uint32_t y = (uint32_t)__shfl_up((int)incl, o, kWave);
      if (lane >= o) incl += y;
    }
    if (lane == kWave - 1) running[w] = incl;           // wave totals (running is reset below)
    __syncthreads();
    uint32_t before = 0;
    for (int ww = 0; ww < w; ++ww) before += running[ww];
    base_off[t] = before + incl - v + tile_off;
    __syncthreads();
  }
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

// Rank of a small queue (Q <= kRankSmallMax) by counting: the position of
// request i in the stable ascending order is
//   rank(i) = #{j : key_j < key_i} + #{j < i : key_j == key_i},
// the same permutation the radix sort gives. Workgroup b owns TI requests
// i0 = TI b ... and counts over all Q keys, held in LDS: its 16 waves take
// 64-key chunks in turn, and within a wave S = 64 / TI lane groups take
// TI-key sub-blocks of each chunk (lane l: request i0 + l % TI, sub-block
// l / TI). A chunk wholly below i0 counts key_j <= key_i, one wholly past
// the workgroup's requests counts key_j < key_i, and only the chunk holding
// them takes the exact rule. Q^2 compares, one compare and one add each:
// at these sizes a few microseconds spread over the whole chip, where the
// four-pass radix sort in one workgroup ran serially.
constexpr int kRankSmallMax = 16384;
constexpr int kRankCountThreads = 1024;
constexpr int kRankCountWaves = kRankCountThreads / kWave;

template <int TI>
__global__ void __launch_bounds__(kRankCountThreads) rank_count_kernel(const float* __restrict__ g_in, int Q,
                                                                       int32_t* __restrict__ order) {
  constexpr int S = kWave / TI;
  __shared__ __align__(16) uint32_t keys[kRankSmallMax];
  __shared__ uint32_t part[kRankCountWaves][TI];
  const int tid = threadIdx.x;
  const int lane = (int)lane_id();
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);     // wave-uniform: scalar loop control
  const int n_chunks = (Q + kWave - 1) / kWave;
  {
    // All loads in flight at once, then the LDS writes; padding never counts.
    constexpr int kItems = kRankSmallMax / kRankCountThreads;
    float g[kItems];
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
      const int e = r * kRankCountThreads + tid;
      g[r] = e < Q ? g_in[e] : 0.0f;
    }
#pragma unroll
    for (int r = 0; r < kItems; ++r) {
      const int e = r * kRankCountThreads + tid;
      if (e < n_chunks * kWave) keys[e] = e < Q ? index_key(g[r]) : 0xFFFFFFFFu;
    }
  }
  __syncthreads();
  const int i0 = blockIdx.x * TI;
  const int il = lane % TI, sub = lane / TI;
  const int i = i0 + il;
  const uint32_t ki = keys[min(i, Q - 1)];
  const int c_lo = i0 / kWave;                                // chunk holding the requests
  uint32_t cnt = 0;
  for (int c = w; c < n_chunks; c += kRankCountWaves) {
    const int j0 = c * kWave + sub * TI;
    const uint4* kp = reinterpret_cast<const uint4*>(&keys[j0]);
    if (c < c_lo) {
#pragma unroll
      for (int m = 0; m < TI / 4; ++m) {
        const uint4 k4 = kp[m];
        cnt += (k4.x <= ki) + (k4.y <= ki) + (k4.z <= ki) + (k4.w <= ki);
      }
    } else if (c > c_lo) {
#pragma unroll
      for (int m = 0; m < TI / 4; ++m) {
        const uint4 k4 = kp[m];
        cnt += (k4.x < ki) + (k4.y < ki) + (k4.z < ki) + (k4.w < ki);
      }
    } else {
#pragma unroll
      for (int m = 0; m < TI; ++m) {
        const uint32_t kj = keys[j0 + m];
        cnt += (kj < ki || (kj == ki && j0 + m < i)) ? 1u : 0u;
      }
    }
  }
#pragma unroll
  for (int o = TI; o < kWave; o <<= 1) cnt += __shfl_xor(cnt, o, kWave);
  if (sub == 0) part[w][il] = cnt;
  __syncthreads();
  if (tid < TI && i < Q) {
    uint32_t r = 0;
#pragma unroll
    for (int ww = 0; ww < kRankCountWaves; ++ww) r += part[ww][tid];
    order[r] = i;
  }
}

}  // namespace

size_t rank_workspace_bytes(int Q) {
  if (Q <= 0) return 0;
  const size_t tiles = ((size_t)Q + kRankTile - 1) / kRankTile;
  return 4 * (size_t)Q * sizeof(uint32_t) + 256 * (tiles + 1) * sizeof(uint32_t) + 256;
}

hipError_t launch_index(const float* mass, const float* cost, const int32_t* prompt_len,
                        const double* bin_repr, const int32_t* generated, int bucket, int Q, int B,
                        float* index, int32_t* argmin, hipStream_t stream, const IndexVariant* variant) {
  if (Q == 0) return hipSuccess;
  LaunchScope scope(variant ? (variant->levels > 0 ? "index_attained_table" : "index_variant")
                            : (generated ? "index_attained" : "index_scan"),
                    stream);
  const int per_lane = (B + kWave - 1) / kWave;
#define SAGE_INDEX_C(CC) \
  return launch_index_c<CC>(mass, cost, prompt_len, bin_repr, generated, bucket, Q, B, index, argmin, stream, \
                            variant)
  if (per_lane <= 1) SAGE_INDEX_C(1);
  if (per_lane <= 2) SAGE_INDEX_C(2);
  if (per_lane <= 4) SAGE_INDEX_C(4);
  if (per_lane <= 8) SAGE_INDEX_C(8);
  if (per_lane <= 16) SAGE_INDEX_C(16);
  if (per_lane <= 32) SAGE_INDEX_C(32);
  SAGE_INDEX_C(64);
#undef SAGE_INDEX_C
}

hipError_t launch_rank(const float* index, int Q, int32_t* order, void* ws, hipStream_t stream) {
  if (Q == 0) return hipSuccess;
  if (Q <= kRankSmallMax) {
    // Requests per workgroup: the fewest that still leave >= 256 workgroups
    // (one per CU), so small queues spread over the chip.
    LaunchScope scope("rank_small", stream);
    if (Q <= 4096)
      hipLaunchKernelGGL(rank_count_kernel<16>, dim3((Q + 15) / 16), dim3(kRankCountThreads), 0, stream, index, Q, order);
    else if (Q <= 8192)
      hipLaunchKernelGGL(rank_count_kernel<32>, dim3((Q + 31) / 32), dim3(kRankCountThreads), 0, stream, index, Q, order);
    else
      hipLaunchKernelGGL(rank_count_kernel<64>, dim3((Q + 63) / 64), dim3(kRankCountThreads), 0, stream, index, Q, order);
    return hipGetLastError();
  }
  const int n_tiles = (Q + kRankTile - 1) / kRankTile;
  uint32_t* kA = static_cast<uint32_t*>(ws);
  uint32_t* vA = kA + Q;
  uint32_t* kB = vA + Q;
  uint32_t* vB = kB + Q;
  uint32_t* hist = vB + Q;
  uint32_t* totals = hist + 256 * (size_t)n_tiles;
  // With few tiles each scatter workgroup sums the per-tile counts itself
  // (n_tiles loads per digit) and the scan launch is skipped.
  const bool fused = n_tiles <= 64;
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
    if (!fused) {
      LaunchScope scope("rank_scan", stream);
      hipLaunchKernelGGL(rank_scan_kernel, dim3(256), dim3(256), 0, stream, hist, n_tiles, totals);
    }
    {
      LaunchScope scope("rank_scatter", stream);
      hipLaunchKernelGGL(rank_scatter_kernel, dim3(n_tiles), dim3(kRankThreads), 0, stream, index,
                         k_in, v_in, Q, shift, n_tiles, hist, totals, fused ? 1 : 0, k_out, v_out);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    k_in = k_out;
    v_in = v_out;
  }
  return hipSuccess;
}

}  // namespace sage
