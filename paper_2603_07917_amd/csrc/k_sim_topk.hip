// Fused similarity search + streaming top-k (the predictor's neighbour search,
// Sec. 3.1: brute-force cosine similarity of prompt embeddings against the
// history store; unit vectors make it an inner product).
//
// One workgroup (4 wavefronts) owns a tile of BQ queries and a contiguous
// chunk of history rows, and walks the chunk in steps of 256 rows:
//
//  * MFMA: S^T[256 x BQ] = H_step[256 x d] * Q_tile^T with
//    v_mfma_f32_32x32x16_bf16 (fp32 accumulate). Both operands are staged
//    through LDS in 64-wide d slices; the next slice is fetched into
//    registers while the current one is multiplied. Wave w computes history
//    rows [64w, 64w + 64) of the step against all BQ queries. Scores stay in
//    registers; nothing of S reaches HBM.
//  * Filter: a lane owns (query, 16 rows) pieces of the accumulator tile and
//    compares each score with the query's threshold theta (the k-th best key
//    of the query's list so far; -inf until k keys exist). History indices
//    grow along the walk, so a later row with the same score loses the tie:
//    a strict ">" is exact.
//  * Append: survivors are packed as 64-bit keys (score bits made monotone,
//    then ~index) and appended to a per-query buffer of 64 keys in LDS at a
//    deterministic position (prefix over lanes). When a step brings more
//    survivors than the buffer holds, the append runs in rounds of 64 with a
//    merge between rounds.
//  * Merge: the wave owning a query sorts the buffer (bitonic, across lanes)
//    and folds it into the query's descending list of KL keys with one
//    bitonic merge; theta becomes the list's k-th key.
//
// At the end of the chunk every list is written to the partial buffer
// [Q][chunks][KL]; a second kernel merges a query's lists across chunks.
#include "sage_device.hpp"
#include "sage_internal.hpp"

namespace sage {
namespace {

typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float floatx16;

constexpr int kThreads = 256;
constexpr int kStepRows = 256;     // history rows per step (64 per wave)
constexpr int kKT = 64;            // d elements per LDS slice
constexpr int kLdsRow = kKT + 8;   // padded LDS row (bf16 elements): 144 bytes
constexpr int kCap = 64;           // per-query candidate buffer

template <int NQT, int KL>
struct Smem {
  static constexpr int BQ = 32 * NQT;
  uint64_t list[BQ * KL];
  uint64_t buf[BQ * kCap];
  uint16_t a_tile[kStepRows * kLdsRow];
  uint16_t b_tile[BQ * kLdsRow];
  float theta[BQ];
  int fill[BQ];
  int tot[BQ];
  int cnt[BQ * 8];
  int rounds;
};

__device__ __forceinline__ uint64_t umax64(uint64_t a, uint64_t b) { return a > b ? a : b; }
__device__ __forceinline__ uint64_t umin64(uint64_t a, uint64_t b) { return a > b ? b : a; }

// Fold `n_buf` unsorted keys of `buf` into the descending list of KL keys and
// return the key at position k-1 (broadcast to every lane).
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

template <int NQT, int KL>
__global__ void __launch_bounds__(kThreads, 1) sim_topk_kernel(
    const uint16_t* __restrict__ queries, int Q, const uint16_t* __restrict__ hist, int N, int d,
    int k, int chunk_rows, int n_chunks, uint64_t* __restrict__ partial) {
  constexpr int BQ = 32 * NQT;
  constexpr int QPW = BQ / 4;                // queries owned (merged) by each wave
  constexpr int A_CHUNKS = kStepRows * kKT / 8 / kThreads;   // 16-byte loads per thread
  constexpr int B_CHUNKS = (BQ * kKT / 8 + kThreads - 1) / kThreads;
  __shared__ Smem<NQT, KL> sm;

  const int tid = threadIdx.x;
  const int lane = (int)lane_id();
  const int w = tid / kWave;
  const int half = lane >> 5;
  const int l32 = lane & 31;
  const int q0 = blockIdx.x * BQ;
  const int chunk = blockIdx.y;
  const int h_begin = chunk * chunk_rows;
  const int h_end = min(N, h_begin + chunk_rows);

  for (int i = tid; i < BQ * KL; i += kThreads) sm.list[i] = kPadKey;
  for (int i = tid; i < BQ; i += kThreads) {
    sm.theta[i] = -__builtin_inff();
    sm.fill[i] = 0;
  }

  const int n_kt = (d + kKT - 1) / kKT;
  uint4 ra[A_CHUNKS];
  uint4 rb[B_CHUNKS];

  for (int h0 = h_begin; h0 < h_end; h0 += kStepRows) {
    floatx16 acc[2][NQT];
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
      for (int t = 0; t < NQT; ++t)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[u][t][v] = 0.0f;

    auto load_slice = [&](int kt) {
      const int k0 = kt * kKT;
#pragma unroll
      for (int c = 0; c < A_CHUNKS; ++c) {
        const int flat = c * kThreads + tid;
        const int row = flat >> 3, col = (flat & 7) * 8;
        const int h = h0 + row;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (h < h_end && k0 + col < d)
          v = *reinterpret_cast<const uint4*>(hist + (size_t)h * d + k0 + col);
        ra[c] = v;
      }
#pragma unroll
      for (int c = 0; c < B_CHUNKS; ++c) {
        const int flat = c * kThreads + tid;
        uint4 v = make_uint4(0, 0, 0, 0);
        if (flat < BQ * kKT / 8) {
          const int row = flat >> 3, col = (flat & 7) * 8;
          const int q = q0 + row;
          if (q < Q && k0 + col < d)
            v = *reinterpret_cast<const uint4*>(queries + (size_t)q * d + k0 + col);
        }
        rb[c] = v;
      }
    };
    auto store_slice = [&]() {
#pragma unroll
      for (int c = 0; c < A_CHUNKS; ++c) {
        const int flat = c * kThreads + tid;
        const int row = flat >> 3, col = (flat & 7) * 8;
        *reinterpret_cast<uint4*>(&sm.a_tile[row * kLdsRow + col]) = ra[c];
      }
#pragma unroll
      for (int c = 0; c < B_CHUNKS; ++c) {
        const int flat = c * kThreads + tid;
        if (flat < BQ * kKT / 8) {
          const int row = flat >> 3, col = (flat & 7) * 8;
          *reinterpret_cast<uint4*>(&sm.b_tile[row * kLdsRow + col]) = rb[c];
        }
      }
    };

    load_slice(0);
    for (int kt = 0; kt < n_kt; ++kt) {
      __syncthreads();
      store_slice();
      __syncthreads();
      if (kt + 1 < n_kt) load_slice(kt + 1);
#pragma unroll
      for (int kk = 0; kk < kKT / 16; ++kk) {
        const int kofs = kk * 16 + half * 8;
        bf16x8 af[2], bfr[NQT];
#pragma unroll
        for (int u = 0; u < 2; ++u)
          af[u] = *reinterpret_cast<const bf16x8*>(&sm.a_tile[(64 * w + 32 * u + l32) * kLdsRow + kofs]);
#pragma unroll
        for (int t = 0; t < NQT; ++t)
          bfr[t] = *reinterpret_cast<const bf16x8*>(&sm.b_tile[(32 * t + l32) * kLdsRow + kofs]);
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int t = 0; t < NQT; ++t)
            acc[u][t] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af[u], bfr[t], acc[u][t], 0, 0, 0);
      }
    }

    // ---------------- epilogue: filter, rank, append, merge ----------------
    // acc[u][t][v] holds S[h][q] with q = 32t + l32 and
    // h = h0 + 64w + 32u + 8(v/4) + 4*half + (v%4).
    float th[NQT];
    int my_cnt[NQT];
#pragma unroll
    for (int t = 0; t < NQT; ++t) {
      const int ql = 32 * t + l32;
      th[t] = sm.theta[ql];
      int c = 0;
      if (q0 + ql < Q) {
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int h = h0 + 64 * w + 32 * u + 8 * (v >> 2) + 4 * half + (v & 3);
            c += (h < h_end && acc[u][t][v] > th[t]) ? 1 : 0;
          }
      }
      my_cnt[t] = c;
      sm.cnt[ql * 8 + 2 * w + half] = c;
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
      int b = sm.fill[ql];
      for (int j = 0; j < 2 * w + half; ++j) b += sm.cnt[ql * 8 + j];
      base[t] = b;
    }
    for (int r = 0; r < rounds; ++r) {
      const int lo = r * kCap, hi = lo + kCap;
#pragma unroll
      for (int t = 0; t < NQT; ++t) {
        const int ql = 32 * t + l32;
        if (my_cnt[t] == 0 || base[t] + my_cnt[t] <= lo || base[t] >= hi) continue;
        int g = base[t];
#pragma unroll
        for (int u = 0; u < 2; ++u)
#pragma unroll
          for (int v = 0; v < 16; ++v) {
            const int h = h0 + 64 * w + 32 * u + 8 * (v >> 2) + 4 * half + (v & 3);
            const float s = acc[u][t][v];
            if (h < h_end && s > th[t]) {
              if (g >= lo && g < hi) sm.buf[ql * kCap + (g - lo)] = make_key(s, (uint32_t)h);
              ++g;
            }
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
                    const SimTopkPlan& plan, uint64_t* partial, hipStream_t stream) {
  dim3 grid(plan.q_tiles, plan.n_chunks);
  hipLaunchKernelGGL((sim_topk_kernel<NQT, KL>), grid, dim3(kThreads), 0, stream, queries, Q, hist,
                     N, d, k, plan.chunk_rows, plan.n_chunks, partial);
  return hipGetLastError();
}

}  // namespace

SimTopkPlan plan_sim_topk(int Q, int N, int d, int k) {
  (void)d;
  SimTopkPlan p{};
  int L = 64;
  while (L < k) L <<= 1;
  p.list_len = L;
  p.q_tile = L <= 128 ? 64 : 32;
  p.q_tiles = (Q + p.q_tile - 1) / p.q_tile;
  const long max_chunks = ((long)N + kStepRows - 1) / kStepRows;
  long want = (1024 + (long)p.q_tiles - 1) / (long)(p.q_tiles > 0 ? p.q_tiles : 1);
  if (want < 1) want = 1;
  if (want > max_chunks) want = max_chunks;
  long rows = ((long)N + want - 1) / want;
  rows = (rows + kStepRows - 1) / kStepRows * kStepRows;
  p.chunk_rows = (int)rows;
  p.n_chunks = (int)(((long)N + rows - 1) / rows);
  p.partial_bytes = (size_t)Q * (size_t)p.n_chunks * (size_t)L * sizeof(uint64_t);
  return p;
}

hipError_t launch_sim_topk(const uint16_t* queries, int Q, const uint16_t* hist, int N, int d,
                           int k, const SimTopkPlan& plan, uint64_t* partial, hipStream_t stream) {
  if (Q == 0) return hipSuccess;
  LaunchScope scope("sim_topk", stream);
  switch (plan.list_len) {
    case 64: return launch_t<2, 64>(queries, Q, hist, N, d, k, plan, partial, stream);
    case 128: return launch_t<2, 128>(queries, Q, hist, N, d, k, plan, partial, stream);
    default: return launch_t<1, 256>(queries, Q, hist, N, d, k, plan, partial, stream);
  }
}

}  // namespace sage
