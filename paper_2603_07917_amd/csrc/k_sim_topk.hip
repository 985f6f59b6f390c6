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
#include "sage_device.hpp"
#include "sage_internal.hpp"

namespace sage {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
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
  __device__ __forceinline__ void load(const uint16_t* __restrict__ hist, int h0, int h_last,
                                       const uint16_t* __restrict__ queries, int q0, int q_last,
                                       int d, int kt) {
    const int tid = threadIdx.x;
    const int k0 = kt * kKT;
#pragma unroll
    for (int c = 0; c < A_LD; ++c) {
      const int f = c * kThreads + tid;
      const int row = f >> 3, col = k0 + (f & 7) * 8;
      const int h = min(h0 + row, h_last);
      const uint4 v = *reinterpret_cast<const uint4*>(hist + (size_t)h * d + min(col, d - 8));
      ra[c] = col < d ? v : make_uint4(0, 0, 0, 0);
    }
#pragma unroll
    for (int c = 0; c < B_LD; ++c) {
      const int f = min(c * kThreads + tid, B_CHUNKS - 1);
      const int row = f >> 3, col = k0 + (f & 7) * 8;
      const int q = min(q0 + row, q_last);
      const uint4 v = *reinterpret_cast<const uint4*>(queries + (size_t)q * d + min(col, d - 8));
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
__device__ __forceinline__ void gemm_step(floatx16 (&acc)[2][NQT], const uint16_t* __restrict__ hist,
                                          int h0, int h_end, const uint16_t* __restrict__ queries,
                                          int q0, int Q, int d, uint16_t* a_tile, uint16_t* b_tile) {
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
  b = wave_sort_desc64(b);
  const uint64_t br = shfl_u64(b, 63 - lane);         // ascending along the lanes
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
  return shfl_u64(sel, kl);
}

// ------------------------------------------------------------------------
// Sampled group maxima: one workgroup per (query tile, sampled step).
// gm[q][s][g] for the 16 groups of 16 rows of a step; -inf past N.
// ------------------------------------------------------------------------
template <int NQT>
__global__ void __launch_bounds__(kThreads, 1) threshold_sample_kernel(
    const uint16_t* __restrict__ queries, int Q, const uint16_t* __restrict__ hist, int N, int d,
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

// theta0[q] = k-th largest of the query's m group maxima (-inf when fewer
// than k exist): bitonic sort in LDS, one workgroup per query.
__global__ void __launch_bounds__(256) threshold_select_kernel(const float* __restrict__ gm, int m,
                                                               int m_pow2, int k,
                                                               float* __restrict__ theta0) {
  extern __shared__ float vals[];
  const int q = blockIdx.x;
  const float* src = gm + (size_t)q * m;
  for (int i = threadIdx.x; i < m_pow2; i += 256) vals[i] = i < m ? src[i] : -__builtin_inff();
  __syncthreads();
  for (int size = 2; size <= m_pow2; size <<= 1) {
    for (int stride = size >> 1; stride > 0; stride >>= 1) {
      for (int e = threadIdx.x; e < m_pow2 / 2; e += 256) {
        const int i = (e / stride) * (2 * stride) + (e % stride);
        const int j = i + stride;
        const bool desc = (i & size) == 0;
        const float a = vals[i], b = vals[j];
        if ((a < b) == desc) { vals[i] = b; vals[j] = a; }
      }
      __syncthreads();
    }
  }
  if (threadIdx.x == 0) theta0[q] = k <= m ? vals[k - 1] : -__builtin_inff();
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

template <int NQT, int KL>
__global__ void __launch_bounds__(kThreads, 1) sim_topk_kernel(
    const uint16_t* __restrict__ queries, int Q, const uint16_t* __restrict__ hist, int N, int d,
    int k, int chunk_rows, int n_chunks, int q_tiles, const float* __restrict__ theta0,
    uint64_t* __restrict__ partial) {
  constexpr int BQ = 32 * NQT;
  constexpr int QPW = BQ / 4;              // queries merged by each wave
  constexpr int kCap = CapOf<NQT>::value;
  __shared__ __align__(16) TopkSmem<NQT, KL> sm;

  // Block -> (query tile, chunk). When the chunks split evenly over the 8
  // XCDs, the query tiles of one chunk are dispatched to the same XCD so that
  // its history rows are shared through that XCD's L2.
  int qt, chunk;
  const int b = blockIdx.x;
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
      uint32_t m = 0;
#pragma unroll
      for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int v = 0; v < 16; ++v) m |= (acc[u][t][v] > thr[t] ? 1u : 0u) << (16 * u + v);
      if (!full_step) {
        uint32_t valid = 0;
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int h = h0 + 64 * w + 32 * u + 8 * (v >> 2) + 4 * half + (v & 3);
            valid |= (h < step_end ? 1u : 0u) << (16 * u + v);
          }
        m &= valid;
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
hipError_t launch_t(const uint16_t* queries, int Q, const uint16_t* hist, int N, int d, int k,
                    const SimTopkPlan& plan, uint64_t* partial, float* gm, float* theta0,
                    hipStream_t stream) {
  if (plan.n_samples > 0) {
    {
      LaunchScope scope("threshold_sample", stream);
      hipLaunchKernelGGL((threshold_sample_kernel<NQT>), dim3(plan.q_tiles, plan.n_samples),
                         dim3(kThreads), 0, stream, queries, Q, hist, N, d, plan.sample_every,
                         plan.n_samples, gm);
    }
    const int m = plan.n_samples * 16;
    int m2 = 1;
    while (m2 < m) m2 <<= 1;
    {
      LaunchScope scope("threshold_select", stream);
      hipLaunchKernelGGL(threshold_select_kernel, dim3(Q), dim3(256), m2 * sizeof(float), stream, gm,
                         m, m2, k, theta0);
    }
  }
  LaunchScope scope("sim_topk", stream);
  hipLaunchKernelGGL((sim_topk_kernel<NQT, KL>), dim3(plan.q_tiles * plan.n_chunks), dim3(kThreads), 0,
                     stream, queries, Q, hist, N, d, k, plan.chunk_rows, plan.n_chunks, plan.q_tiles,
                     plan.n_samples > 0 ? theta0 : nullptr, partial);
  return hipGetLastError();
}

}  // namespace

SimTopkPlan plan_sim_topk(int Q, int N, int d, int k) {
  (void)d;
  SimTopkPlan p{};
  int L = 64;
  while (L < k) L <<= 1;
  p.list_len = L;
  p.q_tile = L == 64 ? 128 : (L == 128 ? 64 : 32);
  p.q_tiles = (Q + p.q_tile - 1) / p.q_tile;
  const long steps = ((long)N + kStepRows - 1) / kStepRows;
  long want = (1024 + (long)p.q_tiles - 1) / (long)(p.q_tiles > 0 ? p.q_tiles : 1);
  if (want >= 8) want = (want + 7) / 8 * 8;            // whole chunks per XCD
  if (want < 1) want = 1;
  if (want > steps) want = steps;
  long rows = ((long)N + want - 1) / want;
  rows = (rows + kStepRows - 1) / kStepRows * kStepRows;
  p.chunk_rows = (int)rows;
  p.n_chunks = (int)(((long)N + rows - 1) / rows);
  // Sample every SR-th step: at least 4k group maxima, at most 8192, SR <= 32.
  p.sample_every = 0;
  p.n_samples = 0;
  if (steps * 16 >= 8L * k) {
    long sr = steps * 16 / (4L * k);
    if (sr > 32) sr = 32;
    if (sr < 1) sr = 1;
    while ((steps + sr - 1) / sr > 512) ++sr;
    p.sample_every = (int)sr;
    p.n_samples = (int)((steps + sr - 1) / sr);
  }
  p.partial_bytes = (size_t)Q * (size_t)p.n_chunks * (size_t)L * sizeof(uint64_t);
  p.gm_bytes = (size_t)Q * (size_t)p.n_samples * 16 * sizeof(float);
  p.theta_bytes = (size_t)Q * sizeof(float);
  return p;
}

hipError_t launch_sim_topk(const uint16_t* queries, int Q, const uint16_t* hist, int N, int d,
                           int k, const SimTopkPlan& plan, void* workspace, hipStream_t stream) {
  if (Q == 0) return hipSuccess;
  char* ws = static_cast<char*>(workspace);
  uint64_t* partial = reinterpret_cast<uint64_t*>(ws);
  float* gm = reinterpret_cast<float*>(ws + plan.partial_bytes);
  float* theta0 = reinterpret_cast<float*>(ws + plan.partial_bytes + plan.gm_bytes);
  switch (plan.list_len) {
    case 64: return launch_t<4, 64>(queries, Q, hist, N, d, k, plan, partial, gm, theta0, stream);
    case 128: return launch_t<2, 128>(queries, Q, hist, N, d, k, plan, partial, gm, theta0, stream);
    default: return launch_t<1, 256>(queries, Q, hist, N, d, k, plan, partial, gm, theta0, stream);
  }
}

}  // namespace sage
