// Fused similarity search + streaming top-k (the predictor's neighbour search,
// Sec. 3.1: brute-force cosine similarity of prompt embeddings against the
// history store; unit vectors make it an inner product).
//
// GEMM core (shared by the two kernels below). A workgroup of 4 wavefronts
// multiplies one step of 256 history rows by a tile of BQ queries:
// S^T[256 x BQ] = H_step[256 x d] * Q_tile^T with v_mfma_f32_32x32x16_bf16
// (fp32 accumulate). Wave w owns history rows [64w, 64w + 64) of the step and
// all BQ queries. The d axis is walked in 64-wide slices (128-byte row
// pieces) staged through LDS (rows padded to 144 bytes, which keeps the
// 16-byte MFMA operand reads free of bank conflicts); the next slice is
// fetched into registers while the current one is multiplied. The scores of
// a step depend only on (step, query tile), so both kernels compute
// bit-identical scores for the same (query, row) pair.
//
// threshold_sample_kernel: for every query, the maxima of disjoint 16-row
//   groups over a sample of steps (every SR-th step). The k-th largest
//   group maximum is a score reached by k distinct history rows, hence a
//   valid lower bound theta0 on the query's k-th best score.
// sim_topk_kernel: one workgroup owns a query tile and a chunk of history
//   rows. After each step, a lane compares its scores with the query's
//   thresholds (>= theta0, and > the k-th key of the chunk list so far: rows
//   come in index order, so a later equal score loses the tie), appends the
//   survivors as 64-bit keys (monotone score bits, then ~index) to a per-query
//   LDS buffer at deterministic positions (in rounds of 64 with merges in
//   between when a step brings more), and the wave owning the query folds
//   full buffers into the query's descending list with a bitonic merge. The
//   lists end in the partial buffer [Q][chunks][KL].
#include <atomic>

#include "sage_device.hpp"
#include "sage_internal.hpp"

namespace sage {
namespace {

typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;

constexpr int kThreads = 256;
constexpr int kStepRows = 256;     // history rows per step (64 per wave)
constexpr int kKT = 64;            // d elements per LDS slice
constexpr int kRowE = kKT + 8;     // padded LDS row: 72 bf16 = 144 bytes
// Per-query candidate buffer: 64 keys, or 32 for 128-query tiles (LDS budget).
template <int NQT> struct CapOf { static constexpr int value = NQT >= 4 ? 32 : 64; };

template <int NQT>
struct Core {
  static constexpr int BQ = 32 * NQT;
  static constexpr int A_LD = kStepRows * kKT / 8 / kThreads;    // 16-byte loads / thread
  static constexpr int B_CHUNKS = BQ * kKT / 8;
  static constexpr int B_LD = (B_CHUNKS + kThreads - 1) / kThreads;
  uint4 ra[A_LD];
  uint4 rb[B_LD];

  // Loads are unconditional (rows clamped into range) so that no branch sits
  // around them; only the zero-fill of columns past d is a select. Rows past
  // h_end and queries past Q carry real but unused data (masked later).
  __device__ __forceinline__ void load(const EmbView& hist, int h0, int h_last, const EmbView& queries,
                                       int q0, int q_last, int d, int kt) {
    const int tid = threadIdx.x;
    const int k0 = kt * kKT;
#pragma unroll
    for (int c = 0; c < A_LD; ++c) {
      const int f = c * kThreads + tid;
      const int row = f >> 3, col = k0 + (f & 7) * 8;
      const int h = min(h0 + row, h_last);
      const uint4 v = *reinterpret_cast<const uint4*>(emb_at(hist, h, min(col, d - 8)));
      ra[c] = col < d ? v : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int c = 0; c < B_LD; ++c) {
      const int f = min(c * kThreads + tid, B_CHUNKS - 1);
      const int row = f >> 3, col = k0 + (f & 7) * 8;
      const int q = min(q0 + row, q_last);
      const uint4 v = *reinterpret_cast<const uint4*>(emb_at(queries, q, min(col, d - 8)));
      rb[c] = col < d ? v : make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void store(uint16_t* a_tile, uint16_t* b_tile) const {
    const int tid = threadIdx.x;
#pragma unroll
    for (int c = 0; c < A_LD; ++c) {
      const int f = c * kThreads + tid;
      *reinterpret_cast<uint4*>(a_tile + (f >> 3) * kRowE + (f & 7) * 8) = ra[c];
    }
#pragma unroll
    for (int c = 0; c < B_LD; ++c) {
      const int f = c * kThreads + tid;
      if (B_CHUNKS % kThreads == 0 || f < B_CHUNKS)
        *reinterpret_cast<uint4*>(b_tile + (f >> 3) * kRowE + (f & 7) * 8) = rb[c];
    }
  }
};

template <int NQT>
__device__ __forceinline__ void mfma_slice(floatx16 (&acc)[2][NQT], const uint16_t* a_tile,
                                           const uint16_t* b_tile, int w, int l32, int half) {
  const uint16_t* as = a_tile + (64 * w + l32) * kRowE + half * 8;
  const uint16_t* bs = b_tile + l32 * kRowE + half * 8;
#pragma unroll
  for (int kk = 0; kk < kKT / 16; ++kk) {
    bf16x8 af[2], bfr[NQT];
#pragma unroll
    for (int u = 0; u < 2; ++u) af[u] = *reinterpret_cast<const bf16x8*>(as + 32 * u * kRowE + kk * 16);
#pragma unroll
    for (int t = 0; t < NQT; ++t) bfr[t] = *reinterpret_cast<const bf16x8*>(bs + 32 * t * kRowE + kk * 16);
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int t = 0; t < NQT; ++t)
        acc[u][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[u], bfr[t], acc[u][t], 0, 0, 0);
  }
}

// Scores of one step: acc[u][t][v] = S[h][q] with
//   h = h0 + 64w + 32u + 8(v/4) + 4*half + (v%4),  q = q0 + 32t + l32.
template <int NQT>
__device__ __forceinline__ void gemm_step(floatx16 (&acc)[2][NQT], const EmbView& hist, int h0, int h_end,
                                          const EmbView& queries, int q0, int Q, int d, uint16_t* a_tile,
                                          uint16_t* b_tile) {
  const int lane = (int)lane_id();
  const int w = threadIdx.x / kWave;
  const int l32 = lane & 31, half = lane >> 5;
#pragma unroll
  for (int u = 0; u < 2; ++u)
#pragma unroll
    for (int t = 0; t < NQT; ++t)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[u][t][v] = 0.0f;
  const int nk = (d + kKT - 1) / kKT;
  const int h_last = h_end - 1, q_last = Q - 1;
  Core<NQT> core;
  core.load(hist, h0, h_last, queries, q0, q_last, d, 0);
  for (int kt = 0; kt + 1 < nk; ++kt) {
    __syncthreads();
    core.store(a_tile, b_tile);
    __syncthreads();
    core.load(hist, h0, h_last, queries, q0, q_last, d, kt + 1);
    mfma_slice<NQT>(acc, a_tile, b_tile, w, l32, half);
  }
  __syncthreads();
  core.store(a_tile, b_tile);
  __syncthreads();
  mfma_slice<NQT>(acc, a_tile, b_tile, w, l32, half);
}

__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }
__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a > b ? b : a; }

// Fold `n_buf` (<= 64) unsorted keys of `buf` into the descending list of KL
// keys and return the list key at position k-1 (the same value in every lane).
template <int KL>
__device__ uint64_t merge_into_list(uint64_t* list, const uint64_t* buf, int n_buf, int k) {
  constexpr int S = KL / 64;
  const int lane = (int)lane_id();
  uint64_t lv[S];
#pragma unroll
  for (int s = 0; s < S; ++s) lv[s] = list[s * 64 + lane];
  uint64_t b = lane < n_buf ? buf[lane] : kPadKey;
  const uint64_t br = wave_sort64(b, false);          // ascending along the lanes
  lv[S - 1] = umax64(lv[S - 1], br);                  // bitonic over the KL positions
#pragma unroll
  for (int st = S / 2; st >= 1; st >>= 1) {
#pragma unroll
    for (int s = 0; s < S; ++s) {
      if ((s & st) == 0) {
        const uint64_t x = lv[s], y = lv[s + st];
        lv[s] = umax64(x, y);
        lv[s + st] = umin64(x, y);
      }
    }
  }
#pragma unroll
  for (int s = 0; s < S; ++s) {
#pragma unroll
    for (int stride = 32; stride > 0; stride >>= 1) lv[s] = cx_lanes(lv[s], stride, true);
    list[s * 64 + lane] = lv[s];
  }
  const int ks = (k - 1) >> 6, kl = (k - 1) & 63;
  uint64_t sel = lv[0];
#pragma unroll
  for (int s = 1; s < S; ++s) if (s == ks) sel = lv[s];
  return lane_value_u64(sel, kl);
}

// ------------------------------------------------------------------------
// Sampled group maxima: one workgroup per (query tile, sampled step).
// gm[q][s][g] for the 16 groups of 16 rows of a step; -inf past N.
// ------------------------------------------------------------------------
template <int NQT>
__global__ void __launch_bounds__(kThreads, 1) threshold_sample_kernel(
    EmbView queries, int Q, EmbView hist, int N, int d,
    int sample_every, int n_samples, float* __restrict__ gm) {
  constexpr int BQ = 32 * NQT;
  __shared__ __align__(16) uint16_t a_tile[kStepRows * kRowE];
  __shared__ __align__(16) uint16_t b_tile[BQ * kRowE];
  const int q0 = blockIdx.x * BQ;
  const int s = blockIdx.y;
  const int h0 = s * sample_every * kStepRows;
  const int h_end = min(N, h0 + kStepRows);
  floatx16 acc[2][NQT];
  gemm_step<NQT>(acc, hist, h0, h_end, queries, q0, Q, d, a_tile, b_tile);

  const int lane = (int)lane_id();
  const int w = threadIdx.x / kWave;
  const int l32 = lane & 31, half = lane >> 5;
#pragma unroll
  for (int t = 0; t < NQT; ++t) {
    const int q = q0 + 32 * t + l32;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      float m = -__builtin_inff();
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        const int h = h0 + 64 * w + 32 * u + 8 * (v >> 2) + 4 * half + (v & 3);
        if (h < h_end) m = fmaxf(m, acc[u][t][v]);
      }
      if (q < Q) gm[((size_t)q * n_samples + s) * 16 + w * 4 + half * 2 + u] = m;
    }
  }
}

// ------------------------------------------------------------------------
// Main kernel.
// ------------------------------------------------------------------------
template <int NQT, int KL>
struct TopkSmem {
  static constexpr int BQ = 32 * NQT;
  static constexpr int kCap = CapOf<NQT>::value;
  uint64_t list[BQ * KL];
  uint64_t buf[BQ * kCap];
  uint16_t a_tile[kStepRows * kRowE];
  uint16_t b_tile[BQ * kRowE];
  float theta[BQ];
  float theta0[BQ];
  int fill[BQ];
  int tot[BQ];
  int cnt[BQ * 8];
  int rounds;
};

// One (query tile, history chunk) of the list search.
template <int NQT, int KL>
__device__ __forceinline__ void list_tile(TopkSmem<NQT, KL>& sm, EmbView queries, int Q, EmbView hist, int N,
                                          int d, int k, int chunk_rows, int n_chunks, int q_tiles,
                                          const float* __restrict__ theta0, const int* __restrict__ only_flagged,
                                          uint64_t* __restrict__ partial, const int b) {
  constexpr int BQ = 32 * NQT;
  constexpr int QPW = BQ / 4;              // queries merged by each wave
  constexpr int kCap = CapOf<NQT>::value;

  // Block -> (query tile, chunk). When the chunks split evenly over the 8
  // XCDs, the query tiles of one chunk are dispatched to the same XCD so that
  // its history rows are shared through that XCD's L2.
  int qt, chunk;
  if (n_chunks % 8 == 0) {
    const int x = b & 7, slot = b >> 3;
    chunk = x + 8 * (slot / q_tiles);
    qt = slot % q_tiles;
  } else {
    chunk = b / q_tiles;
    qt = b % q_tiles;
  }
  const int tid = threadIdx.x;
  const int lane = (int)lane_id();
  const int w = tid / kWave;
  const int l32 = lane & 31, half = lane >> 5;
  const int q0 = qt * BQ;
  const int h_begin = chunk * chunk_rows;
  const int h_end = min(N, h_begin + chunk_rows);

  // As the exact fallback of the filtered path, only tiles holding a flagged
  // query do any work.
  if (only_flagged) {
    if (tid == 0) sm.rounds = 0;
    __syncthreads();
    if (tid < BQ && q0 + tid < Q && only_flagged[q0 + tid]) sm.rounds = 1;
    __syncthreads();
    if (sm.rounds == 0) return;
  }

  for (int i = tid; i < BQ * KL; i += kThreads) sm.list[i] = kPadKey;
  for (int i = tid; i < BQ; i += kThreads) {
    sm.theta[i] = -__builtin_inff();
    sm.theta0[i] = (theta0 && q0 + i < Q) ? theta0[q0 + i] : -__builtin_inff();
    sm.fill[i] = 0;
  }

  for (int h0 = h_begin; h0 < h_end; h0 += kStepRows) {
    floatx16 acc[2][NQT];
    const int step_end = min(h_end, h0 + kStepRows);
    gemm_step<NQT>(acc, hist, h0, step_end, queries, q0, Q, d, sm.a_tile, sm.b_tile);

    // ---------------- filter, rank, append, merge ----------------
    // One compare per score: s >= theta0 and s > theta  <=>  s > max(below(theta0), theta),
    // where below(x) is the largest float under x. Rows past the chunk end
    // (only in a chunk's last step) are masked out of the candidate bits.
    const bool full_step = step_end == h0 + kStepRows;
    float thr[NQT];
    uint32_t bits[NQT];
    int my_cnt[NQT];
#pragma unroll
    for (int t = 0; t < NQT; ++t) {
      const int ql = 32 * t + l32;
      thr[t] = fmaxf(float_below(sm.theta0[ql]), sm.theta[ql]);
      // Bit i = [s_i > thr] is the sign bit of thr - s_i, shifted in with
      // one funnel shift per score.
      uint32_t m = 0;
#pragma unroll
      for (int u = 1; u >= 0; --u)
#pragma unroll
        for (int v = 15; v >= 0; --v)
          m = __builtin_amdgcn_alignbit(m, __float_as_uint(thr[t] - acc[u][t][v]), 31);
      if (!full_step) {
        // Bit i = 16 u + v is row h0 + 64 w + 4 half + 8 (i / 4) + i % 4:
        // rows grow with i, so the rows inside the step are the lowest bits.
        const int c = min(max(step_end - h0 - 64 * w - 4 * half, 0), 64);
        const int n_in = 4 * (c >> 3) + min(c & 7, 4);
        m &= n_in >= 32 ? ~0u : (1u << n_in) - 1u;
      }
      if (q0 + ql >= Q) m = 0;
      bits[t] = m;
      my_cnt[t] = __popc(m);
      sm.cnt[ql * 8 + 2 * w + half] = my_cnt[t];
    }
    if (tid == 0) sm.rounds = 1;
    __syncthreads();
    if (tid < BQ) {
      int s = sm.fill[tid];
#pragma unroll
      for (int j = 0; j < 8; ++j) s += sm.cnt[tid * 8 + j];
      sm.tot[tid] = s;
      const int r = (s + kCap - 1) / kCap;
      if (r > 1) atomicMax(&sm.rounds, r);
    }
    __syncthreads();
    const int rounds = sm.rounds;
    int base[NQT];
#pragma unroll
    for (int t = 0; t < NQT; ++t) {
      const int ql = 32 * t + l32;
      int bb = sm.fill[ql];
      for (int j = 0; j < 2 * w + half; ++j) bb += sm.cnt[ql * 8 + j];
      base[t] = bb;
    }
    for (int r = 0; r < rounds; ++r) {
      const int lo = r * kCap, hi = lo + kCap;
#pragma unroll
      for (int t = 0; t < NQT; ++t) {
        const int ql = 32 * t + l32;
        if (my_cnt[t] == 0 || base[t] + my_cnt[t] <= lo || base[t] >= hi) continue;
        int g = base[t];
        uint32_t m = bits[t];
        while (m) {
          const int i = __ffs(m) - 1;
          m &= m - 1;
          if (g >= lo && g < hi) {
            const int u = i >> 4, v = i & 15;
            const int h = h0 + 64 * w + 32 * u + 8 * (v >> 2) + 4 * half + (v & 3);
            float sv = 0.0f;
#pragma unroll
            for (int uu = 0; uu < 2; ++uu)
#pragma unroll
              for (int vv = 0; vv < 16; ++vv)
                if (16 * uu + vv == i) sv = acc[uu][t][vv];
            sm.buf[ql * kCap + (g - lo)] = make_key(sv, (uint32_t)h);
          }
          ++g;
        }
      }
      __syncthreads();
      if (r + 1 < rounds) {
        for (int j = 0; j < QPW; ++j) {
          const int ql = w * QPW + j;
          if (sm.tot[ql] > hi) {
            const uint64_t kth = merge_into_list<KL>(&sm.list[ql * KL], &sm.buf[ql * kCap], kCap, k);
            if (lane == 0) sm.theta[ql] = key_sim(kth);
          }
        }
        __syncthreads();
      }
    }
    if (tid < BQ) {
      const int s = sm.tot[tid];
      sm.fill[tid] = s > 0 ? s - kCap * ((s - 1) / kCap) : 0;
    }
    // theta / fill are next read after the following step's barriers.
  }

  __syncthreads();
  for (int j = 0; j < QPW; ++j) {
    const int ql = w * QPW + j;
    const int f = sm.fill[ql];
    if (f > 0) merge_into_list<KL>(&sm.list[ql * KL], &sm.buf[ql * kCap], f, k);
  }
  __syncthreads();
  for (int i = tid; i < BQ * KL; i += kThreads) {
    const int ql = i / KL, e = i - ql * KL;
    const int q = q0 + ql;
    if (q < Q) partial[((size_t)q * n_chunks + chunk) * KL + e] = sm.list[i];
  }
}

template <int NQT, int KL>
__global__ void __launch_bounds__(kThreads, 1) sim_topk_kernel(
    EmbView queries, int Q, EmbView hist, int N, int d,
    int k, int chunk_rows, int n_chunks, int q_tiles, const float* __restrict__ theta0,
    const int* __restrict__ only_flagged, const uint32_t* __restrict__ flag_word,
    uint64_t* __restrict__ partial) {
  __shared__ __align__(16) TopkSmem<NQT, KL> sm;
  // As the exact fallback: nothing to do unless a query of this call was
  // flagged (the flagging kernel set the word).
  if (only_flagged && *flag_word == 0u) return;
  // Tiles b = blockIdx.x, + gridDim.x, ... (one each for the full search).
  for (int b = blockIdx.x; b < q_tiles * n_chunks; b += gridDim.x) {
    __syncthreads();                         // the previous tile's LDS reads are done
    list_tile<NQT, KL>(sm, queries, Q, hist, N, d, k, chunk_rows, n_chunks, q_tiles, theta0, only_flagged,
                       partial, b);
  }
}



// Descending order of a bitonic sequence held one key per lane (half-cleaners).
__device__ __forceinline__ uint64_t wave_bitonic_clean_desc64(uint64_t v) {
#pragma unroll
  for (int stride = 32; stride > 0; stride >>= 1) v = cx_lanes(v, stride, true);
  return v;
}

// Folds 64 keys (one per lane, any order) into the wave's descending list of
// its 64 largest keys: skipped when no key beats the list's last one,
// otherwise a wave bitonic sort, C_i = max(A_i, B_{63-i}) and half-cleaners.
__device__ __forceinline__ uint64_t fold_group(uint64_t list, uint64_t key) {
  if (!__any(key > lane_value_u64(list, kWave - 1))) return list;
  const uint64_t asc = wave_sort64(key, false);       // B_{63-i} of the descending order
  return wave_bitonic_clean_desc64(list > asc ? list : asc);
}

// theta0: the k-th largest of a query's m (<= 512 * 16) group maxima, held
// in registers as monotone key bits (VPL per lane; past m: key 0, below every
// real score). theta0 is the largest key T with at least k keys >= T, built
// bit by bit from the top: each bit costs one compare per key and a sum. That
// T is exactly the k-th largest key. Every key lies in [lo, hi], and so does
// the answer: the bits above the highest one where lo and hi differ are fixed
// from the start.
//
// WAVES = 1: one wavefront per query, four queries per workgroup (many
// queries). WAVES > 1: one workgroup of WAVES wavefronts per query, the sums
// completed through LDS (few queries, where one wave per query would leave
// the chip idle and each wave latency-bound).
template <int VPL, int WAVES>
__global__ void __launch_bounds__(256 * (WAVES > 1 ? WAVES / 4 : 1)) threshold_select_kernel(
    const float* __restrict__ gm, int Q, int m, int k, float* __restrict__ theta0, int* __restrict__ clear) {
  __shared__ uint32_t part[2][WAVES > 1 ? WAVES : 1];
  __shared__ uint32_t ext[2][WAVES > 1 ? WAVES : 1];
  const int lane = (int)lane_id();
  const int w = (int)(threadIdx.x / kWave);
  const int q = WAVES > 1 ? (int)blockIdx.x : (int)(blockIdx.x * (blockDim.x / kWave) + w);
  if (q >= Q) return;                                   // whole wavefronts (WAVES = 1 only)
  const float* src = gm + (size_t)q * m;
  const int first = WAVES > 1 ? w * VPL * kWave : 0;    // this wave's keys: first + i * 64 + lane
  uint32_t key[VPL];
  uint32_t kmax = 0, kmin = 0xffffffffu;
#pragma unroll
  for (int i = 0; i < VPL; ++i) {
    const int e = first + i * kWave + lane;
    key[i] = e < m ? f32_order_bits(src[e]) : 0u;
    kmax = max(kmax, key[i]);
    if (e < m) kmin = min(kmin, key[i]);
  }
  uint32_t hi = wave_max_dpp_u32(kmax), lo = wave_min_dpp_u32(kmin);
  if (WAVES > 1) {
    if (lane == 0) { ext[0][w] = hi; ext[1][w] = lo; }
    __syncthreads();
#pragma unroll
    for (int i = 0; i < WAVES; ++i) { hi = max(hi, ext[0][i]); lo = min(lo, ext[1][i]); }
  }
  const int top = hi == lo ? -1 : 31 - __clz(hi ^ lo);
  uint32_t T = top < 0 ? hi : hi & ~((2u << top) - 1u);
  for (int bit = top; bit >= 0; --bit) {
    const uint32_t c = T | (1u << bit);
    uint32_t n0 = 0, n1 = 0;
#pragma unroll
    for (int i = 0; i < VPL; i += 2) {
      n0 += key[i] >= c ? 1u : 0u;
      if (i + 1 < VPL) n1 += key[i + 1] >= c ? 1u : 0u;
    }
    uint32_t n = wave_sum_dpp_u32(n0 + n1);
    if (WAVES > 1) {                                    // partials alternate buffers: one barrier per bit
      if (lane == 0) part[bit & 1][w] = n;
      __syncthreads();
      n = 0;
#pragma unroll
      for (int i = 0; i < WAVES; ++i) n += part[bit & 1][i];
    }
    if (n >= (uint32_t)k) T = c;
  }
  if (lane == 0 && (WAVES == 1 || w == 0)) {
    theta0[q] = k <= m ? f32_from_order_bits(T) : -__builtin_inff();
    if (clear) clear[q] = 0;                            // the next kernel's per-query counter
  }
}
// ========================================================================
// Filtered path for k <= 64.
//
// Ring core: a workgroup multiplies 256 history rows by 256 queries per
// step; wave w = 2*wh + wq owns the 128 x 128 block of rows wh and queries
// wq (4 x 4 MFMA 32x32x16 tiles, 256 accumulators). The d axis is walked in
// 32-wide slices held in a ring of four LDS stages (512 rows x 64 bytes
// each). Stages are filled by direct global->LDS loads (16 bytes per lane,
// no registers): waves 0-1 move history rows, waves 2-3 query rows, three
// slices ahead of the MFMAs and straight across step boundaries, so the
// pipeline never drains between steps. One barrier per slice.
// ========================================================================
namespace ring {

constexpr int kKT = 32;                          // bf16 columns per slice
constexpr int kStages = 4;                       // a power of two (stage = g & (kStages - 1))
constexpr int kStageBytes = 512 * kKT * 2;       // 32 KiB
constexpr int kBQ = 256;                         // queries per tile
constexpr int kLoads = 8;                        // 16-byte loads per lane per slice
constexpr int kAhead = kStages - 1;              // slices in flight

// 16-byte chunk c (0..3) of LDS row r (64 bytes) is stored at position
// c ^ swz(r). An MFMA operand read has 16 lanes reading one chunk of 16
// consecutive rows per cycle; four rows fill the 64 four-byte banks, and
// swz = (r / 4) % 4 gives the four rows that share banks four different
// positions (measured: no bank conflicts, against one in three LDS cycles
// for the unswizzled layout).
__device__ __forceinline__ int swz(int r) { return (r >> 2) & 3; }

// LDS[m0 + 16*lane] = 16 bytes at base + off (gfx950 global_load_lds_dwordx4).
// Issued from inline assembly so that the compiler does not serialise LDS
// reads of other stages behind it; completion is tracked with wait_loads.
__device__ __forceinline__ void load_to_lds(const void* base, uint32_t off, uint32_t m0) {
  asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, %1"
               :: "v"(off), "s"(base), "s"(m0) : "memory", "m0");
}
// The same when the wave-uniform `enabled` is non-zero, else nothing. The
// test is a branch inside the assembly, which keeps the surrounding MFMA
// sequence in one basic block.
__device__ __forceinline__ void load_to_lds_if(const void* base, uint32_t off, uint32_t m0, int enabled) {
  asm volatile("s_cmp_eq_u32 %3, 0\n\ts_cbranch_scc1 1f\n\ts_mov_b32 m0, %2\n\ts_nop 0\n\t"
               "global_load_lds_dwordx4 %0, %1\n1:"
               :: "v"(off), "s"(base), "s"(m0), "s"(enabled) : "memory", "m0", "scc");
}
template <int N>
__device__ __forceinline__ void wait_loads() { asm volatile("s_waitcnt vmcnt(%0)" :: "n"(N) : "memory"); }
// Waits until at most n slices (n * kLoads loads) of this wave are in flight.
__device__ __forceinline__ void wait_slices(int n) {
  if (n <= 0) wait_loads<0>();
  else if (n == 1) wait_loads<kLoads>();
  else if (n == 2) wait_loads<2 * kLoads>();
  else wait_loads<3 * kLoads>();
}
// Workgroup barrier that first retires this wave's LDS reads. The wait is the
// compiler's own instruction (lgkmcnt(0), other counters untouched), so its
// bookkeeping of outstanding LDS reads stays exact after the barrier.
__device__ __forceinline__ void barrier() {
  __builtin_amdgcn_s_waitcnt(0xC07F);
  asm volatile("s_barrier" ::: "memory");
}

struct Frags {
  bf16x8 a[4], b[4];
};

// Keeps a tile in accumulator registers up to this point of the program, so
// that epilogues copy tiles out one at a time (bounded register use).
__device__ __forceinline__ void pin(floatx16& x) { asm volatile("" : "+a"(x)); }

// Runs steps h0 = h_first + j * h_stride (j < n_steps) of query tile q0 and
// calls epi(acc, h0, step_end) after each, step_end = min(h_limit, h0 + 256),
// with acc[u][t][v] = S[h][q] for
//   h = h0 + 128 wh + 32 u + 8 (v / 4) + 4 half + v % 4,  q = q0 + 128 wq + 32 t + l32.
// Rows past N - 1 and queries past Q - 1 are read clamped (their scores are
// meaningless and must be masked by the caller). Requires d % 32 == 0.
template <class Epi>
__device__ __forceinline__ void sweep(const EmbView& hist, int N, int h_first, int h_stride, int n_steps,
                                      int h_limit, const EmbView& queries, int Q, int q0, int d, char* lds,
                                      Epi& epi) {
  const int lane = (int)lane_id();
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int wh = w >> 1, wq = w & 1;
  const int l32 = lane & 31, half = lane >> 5;
  const int nk = d / kKT;
  const int total = n_steps * nk;
  const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char*)lds;

  // Loader: slot (8w + i) * 64 + lane of a stage holds chunk (lane & 3) ^ swz
  // of LDS row 16 (8w + i) + lane / 4, i.e. row r0 + 16 i (r0 = 128 (w & 1) +
  // lane / 4) of this wave's operand: the history step for w < 2, the query
  // tile otherwise. swz of that row depends on lane and on i only via i % 2.
  // swz of those rows is (lane / 16) % 4 for every i.
  const bool hist_side = w < 2;
  const int r0 = 128 * (w & 1) + (lane >> 2);
  const uint32_t cb = (uint32_t)(((lane & 3) ^ swz(lane >> 2)) * 16);
  // Bytes between rows of this wave's operand and between its 32-column slices.
  const uint32_t row_bytes = (uint32_t)((hist_side ? hist.row : queries.row) * 2);
  const long long slice_bytes = (hist_side ? hist.panel : queries.panel) * 2;
  int ld_step = 0, ld_kt = 0;
  const char* src = nullptr;                  // source of slice ld_kt of step ld_step
  uint32_t off[kLoads];                       // per-lane byte offsets within a slice
  auto next_source = [&]() {                  // at the first slice of step ld_step
    int last;
    if (hist_side) {
      const int base_row = h_first + ld_step * h_stride;
      src = reinterpret_cast<const char*>(emb_at(hist, base_row, 0));
      last = N - 1 - base_row;
    } else {
      src = reinterpret_cast<const char*>(emb_at(queries, q0, 0));
      last = Q - 1 - q0;
    }
#pragma unroll
    for (int i = 0; i < kLoads; ++i) off[i] = (uint32_t)min(r0 + 16 * i, last) * row_bytes + cb;
  };
  // Load i (0..7) of slice g into its stage; then advance to the next slice.
  auto issue_one = [&](int g, int i, int enabled) {
    const uint32_t m0 = lds0 + (uint32_t)((g & (kStages - 1)) * kStageBytes + (w * kLoads + i) * 1024);
    load_to_lds_if(src, off[i], __builtin_amdgcn_readfirstlane(m0), __builtin_amdgcn_readfirstlane(enabled));
  };
  auto issue_always = [&](int g, int i) {
    const uint32_t m0 = lds0 + (uint32_t)((g & (kStages - 1)) * kStageBytes + (w * kLoads + i) * 1024);
    load_to_lds(src, off[i], __builtin_amdgcn_readfirstlane(m0));
  };
  auto advance = [&]() {
    src += slice_bytes;
    if (++ld_kt == nk) {
      ld_kt = 0;
      ++ld_step;
      if (ld_step < n_steps) next_source();
    }
  };
  auto issue = [&](int g) {
#pragma unroll
    for (int i = 0; i < kLoads; ++i) issue_one(g, i, 1);
    advance();
  };
  next_source();

  // Operand reads: A = history rows 128 wh + 32 u + l32, B = query rows
  // 256 + 128 wq + 32 t + l32; k chunk 2 kk + half of the slice.
  uint32_t a_off[2], b_off[2];
#pragma unroll
  for (int kk = 0; kk < 2; ++kk) {
    const uint32_t pos = (uint32_t)(((2 * kk + half) ^ swz(l32)) * 16);
    a_off[kk] = (uint32_t)((128 * wh + l32) * 64) + pos;
    b_off[kk] = (uint32_t)((256 + 128 * wq + l32) * 64) + pos;
  }
  auto read = [&](int g, int kk, Frags& f) {
    const char* stage = lds + (g & (kStages - 1)) * kStageBytes;
#pragma unroll
    for (int u = 0; u < 4; ++u) f.a[u] = *reinterpret_cast<const bf16x8*>(stage + a_off[kk] + u * 2048);
#pragma unroll
    for (int t = 0; t < 4; ++t) f.b[t] = *reinterpret_cast<const bf16x8*>(stage + b_off[kk] + t * 2048);
  };
  // Piece p of the fragments: A tile p (p < 4) or B tile p - 4.
  auto read_piece = [&](int g, int kk, int p, Frags& f) {
    const char* stage = lds + (g & (kStages - 1)) * kStageBytes;
    if (p < 4) f.a[p] = *reinterpret_cast<const bf16x8*>(stage + a_off[kk] + p * 2048);
    else f.b[p - 4] = *reinterpret_cast<const bf16x8*>(stage + b_off[kk] + (p - 4) * 2048);
  };

  __syncthreads();                              // earlier users of the LDS are done
  const int pre = min(kAhead, total);
  for (int g = 0; g < pre; ++g) issue(g);
  wait_slices(pre - 1);                         // slice 0 has landed
  barrier();
  Frags f0, f1;
  read(0, 0, f0);
  int g = 0;
  for (int step = 0; step < n_steps; ++step) {
    floatx16 acc[4][4];
    // One slice: f0 holds its first 16 columns on entry; on exit f0 holds the
    // first 16 columns of slice g + 1 (past the last slice those reads fetch
    // a stale stage, which is never used).
    //  * The fragment reads are spread over the MFMAs, one after each of the
    //    first eight of a half, pinned there with scheduling groups: issued
    //    as one burst next to their consumers, the compiler waits on them and
    //    the matrix pipe drains (measured: 1.4 PF/s for a burst schedule
    //    against 2.0 PF/s interleaved, MFMA + LDS only). A read never
    //    overwrites a fragment that an MFMA still in the pipe reads: the
    //    previous users of f1 (f0) were issued a half-slice earlier.
    //  * The eight loads of slice g + kAhead (whose stage was last read in
    //    slice g - 1) go out four in each half, which keeps the address unit
    //    evenly busy.
    auto slice = [&](bool first, bool steady) {
      const int more = steady ? 1 : (g + kAhead < total);
      const floatx16 zero = {};
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int u = j >> 2, t = j & 3;
        acc[u][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f0.a[u], f0.b[t], first ? zero : acc[u][t], 0, 0, 0);
        if (j < 8) read_piece(g, 1, j, f1);
        if (t == 3) {
          if (steady) issue_always(g + kAhead, u);
          else issue_one(g + kAhead, u, more);
        }
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
      // The half's last eight MFMAs stay before the barrier (left alone, the
      // compiler sinks seven of them past it), so the matrix pipe has work
      // queued while the wave waits for its reads and for the other waves.
      __builtin_amdgcn_sched_barrier(0);
      if (steady) {
        wait_loads<kLoads + kLoads / 2>();
      } else {
        const int after = (g + 2 < total ? kLoads : 0) + (more ? kLoads / 2 : 0);
        if (after == 0) wait_loads<0>();
        else if (after == kLoads / 2) wait_loads<kLoads / 2>();
        else if (after == kLoads) wait_loads<kLoads>();
        else wait_loads<kLoads + kLoads / 2>();
      }
      barrier();
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        const int u = j >> 2, t = j & 3;
        acc[u][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(f1.a[u], f1.b[t], acc[u][t], 0, 0, 0);
        if (j < 8) read_piece(g + 1, 0, j, f0);
        if (t == 3) {
          if (steady) issue_always(g + kAhead, kLoads / 2 + u);
          else issue_one(g + kAhead, kLoads / 2 + u, more);
        }
      }
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
      }
      __builtin_amdgcn_sched_group_barrier(0x008, 8, 0);
      if (more) advance();
      ++g;
    };
    // Every slice of a step before the last has its look-ahead slice inside
    // the sweep (when a step has at least kAhead slices): no conditions.
    if (nk >= kAhead && step + 1 < n_steps) {
      slice(true, true);
      for (int kt = 1; kt < nk; ++kt) slice(false, true);
    } else {
      slice(true, false);
      for (int kt = 1; kt < nk; ++kt) slice(false, false);
    }
    const int h0 = h_first + step * h_stride;
    epi(acc, h0, min(h_limit, h0 + 256));
  }
}

}  // namespace ring

// Sampled group maxima with the ring core (the same scores as the filter
// kernel): block (tile, y) runs samples y * spb .. of the sample list,
// sample s being step s * sample_every; every sampled step is whole.
__global__ void __launch_bounds__(kThreads, 1) threshold_sample_ring_kernel(
    EmbView queries, int Q, EmbView hist, int N, int d,
    int sample_every, int n_samples, int spb, float* __restrict__ gm) {
  __shared__ __align__(16) char lds[ring::kStages * ring::kStageBytes];
  const int q0 = blockIdx.x * ring::kBQ;
  const int s0 = blockIdx.y * spb;
  const int n_steps = min(spb, n_samples - s0);
  const int lane = (int)lane_id();
  const int w = threadIdx.x / kWave;
  const int wh = w >> 1, wq = w & 1;
  const int l32 = lane & 31, half = lane >> 5;
  const int stride = sample_every * kStepRows;
  // Sampled steps are whole (256 rows inside the store): no row masking.
  auto epi = [&](floatx16 (&acc)[4][4], int h0, int) {
    const int s = h0 / stride;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
      const int q = q0 + 128 * wq + 32 * t + l32;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        ring::pin(acc[u][t]);
        float m = acc[u][t][0];
#pragma unroll
        for (int v = 1; v < 16; ++v) m = fmaxf(m, acc[u][t][v]);
        if (q < Q) gm[((size_t)q * n_samples + s) * 16 + wh * 8 + half * 4 + u] = m;
      }
    }
  };
  ring::sweep(hist, N, s0 * stride, stride, n_steps, N, queries, Q, q0, d, lds, epi);
}

// Filter kernel: every score >= theta0[q] is written as a key to the
// segment [q][chunk][0..seg_cap) (position from an LDS counter); the true
// count goes to seg_count[q][chunk] even when the segment overflows.
__global__ void __launch_bounds__(kThreads, 1) sim_filter_kernel(
    EmbView queries, int Q, EmbView hist, int N, int d,
    int chunk_rows, int n_chunks, int q_tiles, int q_groups, const float* __restrict__ theta0,
    int seg_cap, uint64_t* __restrict__ seg, int* __restrict__ seg_count, uint32_t* __restrict__ flag_word) {
  __shared__ __align__(16) char lds[ring::kStages * ring::kStageBytes];
  if (blockIdx.x == 0 && threadIdx.x == 0) *flag_word = 0u;     // set again by the select if it flags a query
  __shared__ int cnt[ring::kBQ];
  // Per-lane rows for reading survivors back by a lane-varying index (16
  // scores each, padded to 80 bytes so that the 16-byte writes of 16 lanes
  // fall on distinct banks).
  __shared__ __align__(16) float stage_rows[4][kWave][20];
  int qt, chunk;
  const int b = blockIdx.x;
  if (q_groups > 0) {
    // Workgroup b runs on XCD b % 8. XCD x owns query-tile group x % q_groups
    // and chunk group x / q_groups: its L2 keeps that group's query tiles
    // resident while the chunks stream through.
    const int x = b & 7, slot = b >> 3;
    const int per_group = q_tiles / q_groups;
    const int chunks_per_group = n_chunks / (8 / q_groups);
    qt = (x % q_groups) * per_group + slot % per_group;
    chunk = (x / q_groups) * chunks_per_group + slot / per_group;
  } else if (n_chunks % 8 == 0) {
    const int x = b & 7, slot = b >> 3;
    chunk = x + 8 * (slot / q_tiles);
    qt = slot % q_tiles;
  } else {
    chunk = b / q_tiles;
    qt = b % q_tiles;
  }
  const int tid = threadIdx.x;
  const int lane = (int)lane_id();
  const int w = tid / kWave;
  const int wh = w >> 1, wq = w & 1;
  const int l32 = lane & 31, half = lane >> 5;
  const int q0 = qt * ring::kBQ;
  const int h_begin = chunk * chunk_rows;
  const int h_end = min(N, h_begin + chunk_rows);
  cnt[tid] = 0;
  float thr[4];
#pragma unroll
  for (int t = 0; t < 4; ++t) {
    const int q = q0 + 128 * wq + 32 * t + l32;
    thr[t] = q < Q ? float_below(theta0 ? theta0[q] : -__builtin_inff()) : __builtin_inff();
  }
  // Score acc[u][t][v] of this lane is row h0 + 128 wh + 4 half + r(i) for
  // bit i = 16 u + v, r(i) = 32 (i / 16) + 8 ((i / 4) % 4) + i % 4.
  float* row = &stage_rows[w][lane][0];
  auto epi = [&](floatx16 (&acc)[4][4], int h0, int step_end) {
    const int lim = step_end - h0 - 128 * wh - 4 * half;     // r(i) < lim: row inside the step
    const int hl = h0 + 128 * wh + 4 * half;
    // Rows inside the step: all of them but in a sweep's last, partial step,
    // where r(i) grows with i, so they are the lowest bits (bits 4g..4g+3 are
    // rows 8g..8g+3, hence the count below).
    uint64_t in_step = ~0ull;
    if (step_end - h0 < kStepRows) {
      const int c = min(max(lim, 0), 128);
      const int n_in = 4 * (c >> 3) + min(c & 7, 4);
      in_step = n_in >= 64 ? ~0ull : (1ull << n_in) - 1ull;
    }
    // Column t's survivors are written one column later, so that its LDS
    // atomic (the segment position) is in flight during the next column's
    // compare. Per tile, the lane's first survivor is picked from the
    // registers by a select tree on its index; a lane with two or more
    // survivors in one tile (rare) takes the rest through its LDS row.
    uint64_t m_prev = 0;
    int base_prev = 0;
    uint32_t f_prev = 0;
    float fv_prev[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    auto write_column = [&](int t, uint64_t m, int base, uint32_t fidx, const float (&fv)[4]) {
      const int ql = 128 * wq + 32 * t + l32;
      uint64_t* dst = seg + ((size_t)(q0 + ql) * n_chunks + chunk) * seg_cap;
      uint64_t rest = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const uint32_t bits = (uint32_t)(m >> (16 * u)) & 0xffffu;
        if (bits != 0) {
          const int f = (int)((fidx >> (4 * u)) & 15u);
          const int i = 16 * u + f;
          const int j = base + __popcll(m & ((1ull << i) - 1ull));     // rank among the lane's survivors
          if (j < seg_cap) dst[j] = make_key(fv[u], (uint32_t)(hl + 32 * u + 8 * (f >> 2) + (f & 3)));
          rest |= (uint64_t)(bits & (bits - 1u)) << (16 * u);
        }
      }
      if (!__any(rest != 0)) return;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        uint32_t bits = (uint32_t)(rest >> (16 * u)) & 0xffffu;
        if (!__any(bits != 0)) continue;
#pragma unroll
        for (int c = 0; c < 4; ++c)
          *reinterpret_cast<float4*>(row + 4 * c) =
              make_float4(acc[u][t][4 * c], acc[u][t][4 * c + 1], acc[u][t][4 * c + 2], acc[u][t][4 * c + 3]);
        while (bits) {
          const int v = __ffs(bits) - 1;
          bits &= bits - 1;
          const int i = 16 * u + v;
          const int j = base + __popcll(m & ((1ull << i) - 1ull));
          if (j < seg_cap) dst[j] = make_key(row[v], (uint32_t)(hl + 32 * u + 8 * (v >> 2) + (v & 3)));
        }
      }
    };
#pragma unroll
    for (int t = 0; t < 4; ++t) {
#pragma unroll
      for (int u = 0; u < 4; ++u) ring::pin(acc[u][t]);
      // Bit v of mk[u] = [acc[u][t][v] > thr]: the sign of thr - s, shifted
      // in with one funnel shift (no compare, so no serialisation on VCC).
      // For finite scores the sign of the rounded difference is exact: -0
      // only arises from a negative difference.
      uint32_t mk[4] = {0u, 0u, 0u, 0u};
      float fv[4] = {0.0f, 0.0f, 0.0f, 0.0f};
      uint32_t fidx = 0;
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        // The tile is copied out whole before use, so the 16 register reads
        // and differences are independent rather than one chain through a
        // single temporary.
        floatx16 tv = acc[u][t];
        asm volatile("" : "+v"(tv));
        uint32_t sg[16];
#pragma unroll
        for (int v = 0; v < 16; ++v) sg[v] = __float_as_uint(thr[t] - tv[v]);
#pragma unroll
        for (int v = 15; v >= 0; --v) mk[u] = __builtin_amdgcn_alignbit(mk[u], sg[v], 31);
        mk[u] &= (uint32_t)(in_step >> (16 * u)) & 0xffffu;
        if (__any(mk[u] != 0)) {
          // Select tree on the bits of f, as bitwise selects under all-ones
          // / all-zeros masks (one v_bfi each). The masks are opaque to the
          // compiler, which would otherwise fold the tree into a dynamically
          // indexed array and send it through memory.
          const int f = (__ffs(mk[u]) - 1) & 15;
          uint32_t sel[4];
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            sel[k] = 0u - (uint32_t)((f >> k) & 1);
            asm volatile("" : "+v"(sel[k]));
          }
          auto pick = [](uint32_t mask, uint32_t hi, uint32_t lo) { return (hi & mask) | (lo & ~mask); };
          uint32_t a[8], b[4], c[2];
#pragma unroll
          for (int v = 0; v < 8; ++v) a[v] = pick(sel[0], __float_as_uint(tv[2 * v + 1]), __float_as_uint(tv[2 * v]));
#pragma unroll
          for (int v = 0; v < 4; ++v) b[v] = pick(sel[1], a[2 * v + 1], a[2 * v]);
#pragma unroll
          for (int v = 0; v < 2; ++v) c[v] = pick(sel[2], b[2 * v + 1], b[2 * v]);
          fv[u] = __uint_as_float(pick(sel[3], c[1], c[0]));
          fidx |= (uint32_t)f << (4 * u);
        }
      }
      const uint32_t lo = mk[0] | (mk[1] << 16), hi = mk[2] | (mk[3] << 16);
      const uint64_t m = ((uint64_t)hi << 32) | lo;
      const int ql = 128 * wq + 32 * t + l32;
      const int base = m != 0 ? atomicAdd(&cnt[ql], __popcll(m)) : 0;
      if (t > 0 && __any(m_prev != 0)) write_column(t - 1, m_prev, base_prev, f_prev, fv_prev);
      m_prev = m;
      base_prev = base;
      f_prev = fidx;
#pragma unroll
      for (int u = 0; u < 4; ++u) fv_prev[u] = fv[u];
    }
    if (__any(m_prev != 0)) write_column(3, m_prev, base_prev, f_prev, fv_prev);
  };
  const int n_steps = (h_end - h_begin + kStepRows - 1) / kStepRows;
  ring::sweep(hist, N, h_begin, kStepRows, n_steps, h_end, queries, Q, q0, d, lds, epi);
  __syncthreads();
  if (q0 + tid < Q) seg_count[(size_t)(q0 + tid) * n_chunks + chunk] = cnt[tid];
}

// Select kernel: one wavefront per query, four queries per workgroup. The
// wave reads the query's candidate keys straight from global memory (its
// segments form one index range; kPre groups of 64 keys in flight at once)
// and keeps its best 64 keys as a descending list across lanes: keys that
// beat the list's last key are gathered in LDS, and each 64 of them are
// sorted (wave bitonic sort) and folded in with C_i = max(A_i, B_{63-i}) and
// six half-cleaner stages. One list per query means only the keys that beat
// the query's running 64th are sorted (about k (1 + ln(n / k)) of n), not
// those of four partial lists. A query with an overflowed segment, or with
// fewer than min(k, N) candidates in all, is flagged for the exact fallback
// and left untouched here. Waves work independently (no workgroup barrier).
__global__ void __launch_bounds__(256) select_kernel(const uint64_t* __restrict__ seg,
                                                     const int* __restrict__ seg_count, int Q, int n_chunks,
                                                     int seg_cap, int k, int need, int* __restrict__ flags,
                                                     uint32_t* __restrict__ flag_word,
                                                     int32_t* __restrict__ ids, float* __restrict__ sims) {
  __shared__ int off_s[4][kWave + 1];
  __shared__ uint64_t pend[4][2 * kWave];
  const int lane = (int)lane_id();
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  const int q = blockIdx.x * 4 + w;
  if (q >= Q) return;
  int* off = off_s[w];
  // Segment c (one per lane; n_chunks <= 64) starts at off[c] of the range.
  const int n = lane < n_chunks ? seg_count[(size_t)q * n_chunks + lane] : 0;
  const int c = min(n, seg_cap);
  int incl = c;
#pragma unroll
  for (int o = 1; o < kWave; o <<= 1) {
    const int y = __shfl_up(incl, o, kWave);
    if (lane >= o) incl += y;
  }
  off[lane] = incl - c;
  if (lane == kWave - 1) off[kWave] = incl;
  const int total = __shfl(incl, kWave - 1, kWave);
  // Flag the query when a segment overflowed, or when fewer than min(k, N)
  // keys beat theta0: the pre-pass scores are the filter's own, bit for
  // bit, so the latter only follows from a raised threshold.
  if (__any(n > seg_cap) || total < need) {
    if (lane == 0) {
      flags[q] = 1;
      *flag_word = 1u;
    }
    return;
  }
  if (lane == 0) flags[q] = 0;
  __builtin_amdgcn_wave_barrier();                    // off[] written before it is read
  const uint64_t* src = seg + (size_t)q * n_chunks * seg_cap;
  uint64_t* buf = pend[w];
  uint64_t list = kPadKey;
  int n_buf = 0;                                      // keys waiting in buf (wave-uniform, < 64)
  auto take = [&](uint64_t cur) {
    const uint64_t tail = lane_value_u64(list, kWave - 1);
    const bool keep = cur > tail;
    const uint64_t mask = __ballot(keep);
    if (mask == 0) return;
    const int pos = n_buf + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                            __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
    if (keep) buf[pos] = cur;
    n_buf += __popcll(mask);
    __builtin_amdgcn_wave_barrier();
    if (n_buf >= kWave) {                             // fold 64, keep the rest (< 64) at the front
      list = fold_group(list, buf[lane]);
      n_buf -= kWave;
      const uint64_t rest = lane < n_buf ? buf[kWave + lane] : kPadKey;
      __builtin_amdgcn_wave_barrier();
      if (lane < n_buf) buf[lane] = rest;
      __builtin_amdgcn_wave_barrier();
    }
  };
  constexpr int kPre = 8;
  for (int e0 = 0; e0 < total; e0 += kWave * kPre) {
    uint64_t cur[kPre];
#pragma unroll
    for (int j = 0; j < kPre; ++j) {
      const int e = e0 + kWave * j + lane;
      cur[j] = kPadKey;
      if (e < total) {
        int lo = 0, hi = n_chunks - 1;                // the last segment c with off[c] <= e
        while (lo < hi) {
          const int mid = (lo + hi + 1) >> 1;
          if (off[mid] <= e) lo = mid; else hi = mid - 1;
        }
        cur[j] = src[(size_t)lo * seg_cap + (e - off[lo])];
      }
    }
#pragma unroll
    for (int j = 0; j < kPre; ++j) take(cur[j]);
  }
  if (n_buf > 0) list = fold_group(list, lane < n_buf ? buf[lane] : kPadKey);
  if (lane < k) {
    ids[(size_t)q * k + lane] = list == kPadKey ? -1 : key_id(list);
    sims[(size_t)q * k + lane] = list == kPadKey ? -__builtin_inff() : key_sim(list);
  }
}

template <int NQT, int KL>
hipError_t launch_lists(EmbView queries, int Q, EmbView hist, int N, int d, int k,
                        const SimTopkPlan& p, const float* theta0, const Flagged* only_flagged,
                        uint64_t* partial, hipStream_t stream) {
  LaunchScope scope(only_flagged ? "sim_topk_fallback" : "sim_topk", stream);
  // The fallback runs as one round of workgroups (one per CU) that loop over
  // the tiles, and return at once when no query of the call was flagged.
  const int tiles = p.q_tiles * p.n_chunks;
  hipLaunchKernelGGL((sim_topk_kernel<NQT, KL>), dim3(only_flagged ? std::min(tiles, 256) : tiles), dim3(kThreads),
                     0, stream, queries, Q, hist, N, d, k, p.chunk_rows, p.n_chunks, p.q_tiles, theta0,
                     only_flagged ? only_flagged->flags : nullptr, only_flagged ? only_flagged->word : nullptr,
                     partial);
  return hipGetLastError();
}

// Which kernel scores the sampled steps: each search path samples with the
// arithmetic of its own search, so the sampled scores are the search's own.
enum class Sampler { ring, list, stream };

// Threshold floor for tests of the exact fallback (sage_debug_theta_floor):
// theta0 = max(theta0, floor) before the search.
__global__ void theta_floor_kernel(float* __restrict__ theta0, int Q, float floor) {
  const int q = blockIdx.x * blockDim.x + threadIdx.x;
  if (q < Q) theta0[q] = fmaxf(theta0[q], floor);
}

hipError_t launch_theta(EmbView queries, int Q, EmbView hist, int N, int d, int k,
                        const SimTopkPlan& p, int q_tiles, Sampler sampler, float* gm, float* theta0,
                        int* clear, hipStream_t stream) {
  {
    LaunchScope scope("threshold_sample", stream);
    const dim3 grid(q_tiles, p.n_samples);
    if (sampler == Sampler::stream) {
      const hipError_t e = launch_stream_sample(queries, Q, hist, N, d, p.sample_every, p.n_samples, gm, stream);
      if (e != hipSuccess) return e;
    } else if (sampler == Sampler::ring) {
      const int spb = p.f_spb;
      const dim3 rgrid(q_tiles, (p.n_samples + spb - 1) / spb);
      hipLaunchKernelGGL(threshold_sample_ring_kernel, rgrid, dim3(kThreads), 0, stream, queries, Q,
                         hist, N, d, p.sample_every, p.n_samples, spb, gm);
    } else if (p.list_len == 128) {              // the same core as sim_topk_kernel<2, 128>
      hipLaunchKernelGGL((threshold_sample_kernel<2>), grid, dim3(kThreads), 0, stream, queries, Q,
                         hist, N, d, p.sample_every, p.n_samples, gm);
    } else {                                     // the same core as sim_topk_kernel<1, 256>
      hipLaunchKernelGGL((threshold_sample_kernel<1>), grid, dim3(kThreads), 0, stream, queries, Q,
                         hist, N, d, p.sample_every, p.n_samples, gm);
    }
  }
  const int m = p.n_samples * 16;
  LaunchScope scope("threshold_select", stream);
  if (Q < 512) {                                       // one 16-wave workgroup per query
    if (m <= 2 * 16 * kWave)
      hipLaunchKernelGGL((threshold_select_kernel<2, 16>), dim3(Q), dim3(1024), 0, stream, gm, Q, m, k, theta0, clear);
    else
      hipLaunchKernelGGL((threshold_select_kernel<8, 16>), dim3(Q), dim3(1024), 0, stream, gm, Q, m, k, theta0, clear);
  } else {                                             // four queries (wavefronts) per workgroup
    const dim3 grid((Q + 3) / 4);
    if (m <= 16 * kWave)
      hipLaunchKernelGGL((threshold_select_kernel<16, 1>), grid, dim3(256), 0, stream, gm, Q, m, k, theta0, clear);
    else if (m <= 32 * kWave)
      hipLaunchKernelGGL((threshold_select_kernel<32, 1>), grid, dim3(256), 0, stream, gm, Q, m, k, theta0, clear);
    else if (m <= 64 * kWave)
      hipLaunchKernelGGL((threshold_select_kernel<64, 1>), grid, dim3(256), 0, stream, gm, Q, m, k, theta0, clear);
    else
      hipLaunchKernelGGL((threshold_select_kernel<128, 1>), grid, dim3(256), 0, stream, gm, Q, m, k, theta0, clear);
  }
  const float floor = debug_theta_floor();
  if (sampler != Sampler::list && floor > -__builtin_inff())   // only the paths with a guarded fallback
    hipLaunchKernelGGL(theta_floor_kernel, dim3((Q + 255) / 256), dim3(256), 0, stream, theta0, Q, floor);
  return hipGetLastError();
}

size_t align256(size_t x) { return (x + 255) & ~(size_t)255; }

void chunking(int q_tiles, int N, int target_blocks, int max_chunks, int* chunk_rows, int* n_chunks) {
  const long steps = ((long)N + kStepRows - 1) / kStepRows;
  long want = ((long)target_blocks + q_tiles - 1) / (long)(q_tiles > 0 ? q_tiles : 1);
  if (want >= 8) want = (want + 7) / 8 * 8;            // whole chunks per XCD
  if (want < 1) want = 1;
  if (want > max_chunks) want = max_chunks;
  if (want > steps) want = steps;
  long rows = ((long)N + want - 1) / want;
  rows = (rows + kStepRows - 1) / kStepRows * kStepRows;
  *chunk_rows = (int)rows;
  *n_chunks = (int)(((long)N + rows - 1) / rows);
}

}  // namespace


SimTopkPlan plan_sim_topk(int Q, int N, int d, int k) {
  SimTopkPlan p{};
  int L = 64;
  while (L < k) L <<= 1;
  p.list_len = L;
  p.q_tile = L == 64 ? 128 : (L == 128 ? 64 : 32);
  p.q_tiles = (Q + p.q_tile - 1) / p.q_tile;
  chunking(p.q_tiles, N, 1024, 1 << 20, &p.chunk_rows, &p.n_chunks);
  // Threshold pre-pass: every SR-th step, >= 4k group maxima, at most 8192.
  // SR <= 16 on the filtered path (every candidate above theta0 is written
  // out there, so a tighter bound pays for the larger sample), else <= 32.
  // The sample costs about Q N d / SR and the candidates about Q k SR, so the
  // best SR grows with the square root of N d: from N d = 2^29 on (1M keys
  // of d = 1024) the filtered path also samples every 32nd step.
  // Only whole steps are sampled.
  const long steps = (long)N / kStepRows;
  if (steps * 16 >= 8L * k) {
    // The stream path (few queries) reads the whole store anyway and pays for
    // candidates only in its select: it samples every 128th step at most
    // (streaming workload: pre-pass 44 -> 16 us, select 16 -> 25 us, call -1.5%).
    const bool wide = Q > kStreamMaxQ && (long)N * d >= (1L << 29);
    const bool few = Q <= kStreamMaxQ && d <= kStreamMaxD && k <= 256;     // the stream path's shapes
    const long sr_max = few ? 128 : (L == 64 && !wide ? 16 : 32);
    long sr = steps * 16 / (4L * k);
    if (sr > sr_max) sr = sr_max;
    if (sr < 1) sr = 1;
    while ((steps + sr - 1) / sr > 512) ++sr;
    p.sample_every = (int)sr;
    p.n_samples = (int)((steps + sr - 1) / sr);
  }
  // Filtered path (k <= 64): 256-query tiles, segments of 8192 keys per query in all.
  p.fast = L == 64;
  if (p.fast) {
    p.f_q_tiles = (Q + ring::kBQ - 1) / ring::kBQ;
    // samples per sampling block: about one block per CU
    p.f_spb = 1;
    while (p.n_samples > 0 && (long)p.f_q_tiles * ((p.n_samples + 2 * p.f_spb - 1) / (2 * p.f_spb)) >= 256)
      p.f_spb *= 2;
    chunking(p.f_q_tiles, N, 512, 64, &p.f_chunk_rows, &p.f_n_chunks);
    // Query-tile groups per XCD: the fewest (of 1, 2, 4, 8) whose tiles take at
    // most 3 MiB of an XCD's 4 MiB L2 (0: no grouping). Each history chunk is
    // then read from HBM by as many XCDs as there are groups (two on the mid
    // workload; four groups measured no faster and read the store twice as
    // often).
    p.f_q_groups = 0;
    for (int a = 1; a <= 8; a *= 2) {
      if (p.f_q_tiles % a != 0 || p.f_n_chunks % (8 / a) != 0) continue;
      if ((size_t)(p.f_q_tiles / a) * ring::kBQ * d * 2 <= ((size_t)3 << 20)) { p.f_q_groups = a; break; }
    }
    p.seg_cap = 1;                                   // power of two, n_chunks * cap <= 8192
    while (p.seg_cap * 2 * p.f_n_chunks <= 8192) p.seg_cap *= 2;
  }
  // Few queries against a large store: the stream path (one pass over the
  // store, bound by HBM), given a threshold pre-pass. About k * SR keys
  // beat theta0 per query; the array holds four times that.
  p.stream = Q <= kStreamMaxQ && d <= kStreamMaxD && k <= 256 && p.n_samples > 0;
  if (p.stream) {
    p.fast = false;
    long rows = ((long)N + 511) / 512;                   // about two workgroups per CU
    rows = (rows + 63) / 64 * 64;
    p.s_chunk_rows = (int)rows;
    p.s_cap = 4096;
    while (p.s_cap < 4L * k * p.sample_every) p.s_cap *= 2;
  }
  size_t o = 0;
  p.off_partial = o; o = align256(o + (size_t)Q * p.n_chunks * L * sizeof(uint64_t));
  const int groups = merge_groups(Q, p.n_chunks, L);
  p.off_merge = o;   o = align256(o + (groups > 1 ? (size_t)Q * groups * L * sizeof(uint64_t) : 0));
  p.off_gm = o;      o = align256(o + (size_t)Q * p.n_samples * 16 * sizeof(float));
  p.off_theta = o;   o = align256(o + (size_t)Q * sizeof(float));
  if (p.fast) {
    p.off_seg = o;    o = align256(o + (size_t)Q * p.f_n_chunks * p.seg_cap * sizeof(uint64_t));
    p.off_segcnt = o; o = align256(o + (size_t)Q * p.f_n_chunks * sizeof(int));
    p.off_flags = o;  o = align256(o + (size_t)Q * sizeof(int));
    p.off_flag_word = o; o = align256(o + sizeof(uint32_t));
  }
  if (p.stream) {
    p.off_cand = o;   o = align256(o + (size_t)Q * p.s_cap * sizeof(uint64_t));
    p.off_ccount = o; o = align256(o + (size_t)Q * sizeof(int));
    p.off_flags = o;  o = align256(o + (size_t)Q * sizeof(int));
    p.off_flag_word = o; o = align256(o + sizeof(uint32_t));
  }
  p.total_bytes = o;
  return p;
}

hipError_t launch_neighbours(EmbView queries, int Q, EmbView hist, int N, int d, int k,
                             const SimTopkPlan& p, void* workspace, int32_t* ids, float* sims,
                             hipStream_t stream) {
  if (Q == 0) return hipSuccess;
  char* ws = static_cast<char*>(workspace);
  uint64_t* partial = reinterpret_cast<uint64_t*>(ws + p.off_partial);
  uint64_t* merge_lists = reinterpret_cast<uint64_t*>(ws + p.off_merge);
  float* gm = reinterpret_cast<float*>(ws + p.off_gm);
  float* theta0 = reinterpret_cast<float*>(ws + p.off_theta);
  hipError_t e;
  if (p.fast) {
    if (p.n_samples > 0) {
      e = launch_theta(queries, Q, hist, N, d, k, p, p.f_q_tiles, Sampler::ring, gm, theta0, nullptr, stream);
      if (e != hipSuccess) return e;
    }
    uint64_t* seg = reinterpret_cast<uint64_t*>(ws + p.off_seg);
    int* segcnt = reinterpret_cast<int*>(ws + p.off_segcnt);
    const Flagged fl{reinterpret_cast<int*>(ws + p.off_flags), reinterpret_cast<uint32_t*>(ws + p.off_flag_word)};
    {
      LaunchScope scope("sim_topk", stream);
      hipLaunchKernelGGL(sim_filter_kernel, dim3(p.f_q_tiles * p.f_n_chunks), dim3(kThreads), 0, stream,
                         queries, Q, hist, N, d, p.f_chunk_rows, p.f_n_chunks, p.f_q_tiles, p.f_q_groups,
                         p.n_samples > 0 ? theta0 : nullptr, p.seg_cap, seg, segcnt, fl.word);
    }
    {
      LaunchScope scope("topk_select", stream);
      hipLaunchKernelGGL(select_kernel, dim3((Q + 3) / 4), dim3(256), 0, stream, seg, segcnt, Q,
                         p.f_n_chunks, p.seg_cap, k, min(k, N), fl.flags, fl.word, ids, sims);
    }
    // Exact fallback for queries whose candidates overflowed (no work otherwise).
    e = launch_lists<4, 64>(queries, Q, hist, N, d, k, p, nullptr, &fl, partial, stream);
    if (e != hipSuccess) return e;
    return launch_topk_merge(partial, Q, p.n_chunks, p.list_len, k, &fl, merge_lists, ids, sims, stream);
  }
  if (p.stream) {
    uint64_t* cand = reinterpret_cast<uint64_t*>(ws + p.off_cand);
    int* ccount = reinterpret_cast<int*>(ws + p.off_ccount);
    const Flagged fl{reinterpret_cast<int*>(ws + p.off_flags), reinterpret_cast<uint32_t*>(ws + p.off_flag_word)};
    e = launch_theta(queries, Q, hist, N, d, k, p, 1, Sampler::stream, gm, theta0, ccount, stream);
    if (e != hipSuccess) return e;
    e = launch_stream_search(queries, Q, hist, N, d, k, p.s_chunk_rows, theta0, p.s_cap, cand, ccount, fl,
                             ids, sims, stream);
    if (e != hipSuccess) return e;
    // Exact fallback for queries whose candidates overflowed (no work otherwise).
    if (p.list_len == 64) e = launch_lists<4, 64>(queries, Q, hist, N, d, k, p, nullptr, &fl, partial, stream);
    else if (p.list_len == 128) e = launch_lists<2, 128>(queries, Q, hist, N, d, k, p, nullptr, &fl, partial, stream);
    else e = launch_lists<1, 256>(queries, Q, hist, N, d, k, p, nullptr, &fl, partial, stream);
    if (e != hipSuccess) return e;
    return launch_topk_merge(partial, Q, p.n_chunks, p.list_len, k, &fl, merge_lists, ids, sims, stream);
  }
  if (p.n_samples > 0) {
    e = launch_theta(queries, Q, hist, N, d, k, p, p.q_tiles, Sampler::list, gm, theta0, nullptr, stream);
    if (e != hipSuccess) return e;
  }
  const float* th = p.n_samples > 0 ? theta0 : nullptr;
  if (p.list_len == 128) e = launch_lists<2, 128>(queries, Q, hist, N, d, k, p, th, nullptr, partial, stream);
  else e = launch_lists<1, 256>(queries, Q, hist, N, d, k, p, th, nullptr, partial, stream);
  if (e != hipSuccess) return e;
  return launch_topk_merge(partial, Q, p.n_chunks, p.list_len, k, nullptr, merge_lists, ids, sims, stream);
}

}  // namespace sage
