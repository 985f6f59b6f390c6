// Few-query neighbour search (Sec. 3.1 predictor, a handful of new arrivals
// against a large history store): at most 16 queries, any k <= 256.
//
// With so few queries the search is a single pass over the store, bound by
// HBM, not by the matrix cores. Each wave streams its own 16-row tiles of the
// store straight into registers (no LDS staging, no barriers): a ring of 16
// one-kilobyte loads per wave stays in flight, and each tile's 16 x 16 scores
// against all queries come from d / 32 chained v_mfma_f32_16x16x32_bf16,
// whose query operands sit in LDS. A score above the query's threshold (the
// pre-pass lower bound theta0 on its k-th best score) becomes a candidate
// key; a workgroup gathers its candidates per query in LDS and appends them
// to the query's candidate array with one global atomic per query. The
// select kernel then folds each query's candidates into its top k.
//
// The pre-pass (stream_sample_kernel) scores its sampled rows with this
// kernel's own MFMA chain, so theta0 is a score that k distinct rows reach
// in the search itself, bit for bit: every true neighbour scores >= theta0
// and is a candidate. A workgroup whose LDS slots for a query fill up (a
// store with similar rows side by side) sends the rest to the array one
// atomic at a time; a query whose candidates overflow the array, or that
// ends with fewer than min(k, N) of them (which the bit-identity above rules
// out, so only a raised threshold can cause it), is flagged and answered by
// the exact list path instead.
#include "sage_device.hpp"
#include "sage_internal.hpp"

namespace sage {
namespace {

typedef __attribute__((__vector_size__(4 * sizeof(float)))) float floatx4;

constexpr int kThreads = 256;
constexpr int kWaves = kThreads / kWave;
constexpr int kRows = 16;            // history rows per MFMA tile
constexpr int kRing = 16;            // k-block loads in flight per wave
constexpr int kLCap = 64;            // LDS candidate slots per query and workgroup

__device__ __forceinline__ bf16x8 as_bf16x8(uint4 v) { return __builtin_bit_cast(bf16x8, v); }

// Query operands of the 16x16x32 chain, in LDS: slot j * 64 + l holds query
// l % 16, columns 32 j + 8 (l / 16) .. + 7 (zeros for queries past Q).
__device__ __forceinline__ void load_query_frags(uint4* qfrag, const EmbView& queries, int Q, int KB) {
  for (int i = threadIdx.x; i < KB * kWave; i += kThreads) {
    const int j = i / kWave, l = i % kWave, q = l % 16;
    uint4 v = make_uint4(0u, 0u, 0u, 0u);
    if (q < Q) v = *reinterpret_cast<const uint4*>(emb_at(queries, q, 32 * j + 8 * (l / 16)));
    qfrag[i] = v;
  }
}

// Threshold pre-pass of this path: the maximum of each disjoint 16-row group
// of every sample_every-th 256-row step, gm[q][s][g] (g: the group within
// the step). A group is scored exactly as the search below scores a tile:
// d / 32 chained v_mfma_f32_16x16x32_bf16 from a zero accumulator, column
// blocks in order, row r at operand row r % 16 (tiles start at multiples of
// 16 in both kernels), query q at operand column q. Each maximum is thus the
// search's own fp32 score of one row, and the k-th largest of them (theta0)
// is reached by k distinct rows in the search. Sampled steps are whole.
__global__ void __launch_bounds__(kThreads) stream_sample_kernel(EmbView queries, int Q, EmbView hist, int N,
                                                                 int d, int sample_every, int n_samples,
                                                                 float* __restrict__ gm) {
  extern __shared__ uint4 qfrag[];                  // d / 32 KiB, sized at launch
  const int lane = (int)lane_id();
  const int w = __builtin_amdgcn_readfirstlane((int)(threadIdx.x / kWave));
  const int KB = d / 32;
  load_query_frags(qfrag, queries, Q, KB);
  __syncthreads();
  const int tile = blockIdx.x * kWaves + w;         // 16 tiles per sampled step
  if (tile >= n_samples * 16) return;
  const int s = tile >> 4, g = tile & 15;
  const int row = min(s * sample_every * 256 + 16 * g + (lane & 15), N - 1);
  const uint16_t* p = emb_at(hist, row, 8 * (lane >> 4));
  floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  constexpr int kBatch = 8;                          // loads in flight per wave
  for (int j0 = 0; j0 < KB; j0 += kBatch) {
    uint4 a[kBatch];
#pragma unroll
    for (int i = 0; i < kBatch; ++i)
      if (j0 + i < KB) a[i] = *reinterpret_cast<const uint4*>(p + (long long)(j0 + i) * hist.panel);
#pragma unroll
    for (int i = 0; i < kBatch; ++i)
      if (j0 + i < KB)
        acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a[i]), as_bf16x8(qfrag[(j0 + i) * kWave + lane]),
                                                      acc, 0, 0, 0);
  }
  // Lane l holds rows 4 (l / 16) .. + 3 of query l % 16: the group maximum
  // over the lanes l, l ^ 16, l ^ 32, l ^ 48 (exact: no rounding in a max).
  float m = fmaxf(fmaxf(acc[0], acc[1]), fmaxf(acc[2], acc[3]));
  m = fmaxf(m, __uint_as_float(xor_lane_u32<16>(__float_as_uint(m))));
  m = fmaxf(m, __uint_as_float(xor_lane_u32<32>(__float_as_uint(m))));
  if (lane < Q) gm[((size_t)lane * n_samples + s) * 16 + g] = m;
}

// Workgroup b scans rows [b * chunk_rows, ...); wave w takes the chunk's
// 16-row tiles w, w + 4, ... Lane l of a tile: A operand = row l % 16,
// columns 8 (l / 16) .. + 7 of each 32-column block; B operand = query l % 16,
// the same columns; accumulator i = score of row 4 (l / 16) + i and query
// l % 16.
__global__ void __launch_bounds__(kThreads) sim_stream_kernel(
    EmbView queries, int Q, EmbView hist, int N, int d, int chunk_rows, const float* __restrict__ theta0,
    int cap, uint64_t* __restrict__ cand, int* __restrict__ cand_count, uint32_t* __restrict__ flag_word) {
  extern __shared__ uint4 qfrag[];                  // d / 32 KiB, sized at launch
  if (blockIdx.x == 0 && threadIdx.x == 0) *flag_word = 0u;     // set again by the select if it flags a query
  __shared__ uint64_t lbuf[kStreamMaxQ][kLCap];
  __shared__ int lcnt[kStreamMaxQ];
  __shared__ int gbase[kStreamMaxQ];
  const int tid = threadIdx.x;
  const int lane = (int)lane_id();
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int KB = d / 32;
  load_query_frags(qfrag, queries, Q, KB);
  if (tid < kStreamMaxQ) lcnt[tid] = 0;
  const int ql = lane & 15;
  const float thr = ql < Q ? float_below(theta0[ql]) : __builtin_inff();
  __syncthreads();

  const int h_begin = blockIdx.x * chunk_rows;
  const int h_end = min(N, h_begin + chunk_rows);
  const int n_tiles = (h_end - h_begin + kRows - 1) / kRows;
  const int my_tiles = n_tiles > w ? (n_tiles - w + kWaves - 1) / kWaves : 0;
  const int n_items = my_tiles * KB;                 // item i: tile i / KB, column block i % KB
  const int col = 8 * (lane >> 4);

  // Next item to load: (tile ld_t, column block ld_j) at ld_ptr; rows past
  // the store are clamped to its last row (their scores are dropped).
  int ld_t = 0, ld_j = 0;
  auto tile_ptr = [&](int t) {
    return emb_at(hist, min(h_begin + (w + kWaves * t) * kRows + (lane & 15), N - 1), col);
  };
  const uint16_t* ld_ptr = tile_ptr(0);
  auto load_next = [&](uint4& slot) {
    slot = *reinterpret_cast<const uint4*>(ld_ptr);
    ld_ptr += hist.panel;                            // the next 32 columns
    if (++ld_j == KB) {
      ld_j = 0;
      ld_ptr = tile_ptr(++ld_t);
    }
  };
  auto epilogue = [&](int t, const floatx4& acc) {
    const int r0 = h_begin + (w + kWaves * t) * kRows + 4 * (lane >> 4);
    uint32_t bits = 0;
#pragma unroll
    for (int i = 0; i < 4; ++i) bits |= (acc[i] > thr && r0 + i < h_end ? 1u : 0u) << i;
    if (!__any(bits != 0)) return;
    if (bits == 0) return;
    int pos = atomicAdd(&lcnt[ql], __popc(bits));
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if ((bits >> i) & 1u) {
        const uint64_t key = make_key(acc[i], (uint32_t)(r0 + i));
        if (pos < kLCap) {
          lbuf[ql][pos] = key;
        } else {                                   // slots full (clustered store): straight to the array
          const int gpos = atomicAdd(&cand_count[ql], 1);
          if (gpos < cap) cand[(size_t)ql * cap + gpos] = key;
        }
        ++pos;
      }
    }
  };

  uint4 ring[kRing];
  floatx4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
  int cu_t = 0, cu_j = 0;
  auto consume = [&](const uint4& a) {
    const uint4 b = qfrag[cu_j * kWave + lane];
    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(a), as_bf16x8(b), acc, 0, 0, 0);
    if (++cu_j == KB) {
      epilogue(cu_t, acc);
      acc = floatx4{0.0f, 0.0f, 0.0f, 0.0f};
      cu_j = 0;
      ++cu_t;
    }
  };
  int base = 0;
  if (n_items >= 2 * kRing) {
    // Steady state: every slot is consumed and reloaded, all unconditional
    // (prologue included), so the wait before each use is for the oldest
    // of the kRing loads in flight rather than for all of them.
    // (In slot order: the scheduler must not reorder them, or the first
    // wait would have to be for all of them.)
#pragma unroll
    for (int s = 0; s < kRing; ++s) {
      load_next(ring[s]);
      __builtin_amdgcn_sched_barrier(0);
    }
    for (; base + 2 * kRing <= n_items; base += kRing) {
#pragma unroll
      for (int s = 0; s < kRing; ++s) {
        consume(ring[s]);         // then the slot's next load reuses its registers
        load_next(ring[s]);
      }
    }
  } else {
#pragma unroll
    for (int s = 0; s < kRing; ++s)
      if (s < n_items) load_next(ring[s]);
  }
  // The last one or two turns: reload only what exists.
  for (; base < n_items; base += kRing) {
#pragma unroll
    for (int s = 0; s < kRing; ++s) {
      if (base + s < n_items) {
        consume(ring[s]);
        if (base + s + kRing < n_items) load_next(ring[s]);
      }
    }
  }

  // Append this workgroup's candidates: one global atomic per query for its
  // LDS slots (keys past them went to the array one by one). A query whose
  // count passes the array's capacity is flagged for the exact path.
  __syncthreads();
  if (tid < Q) {
    const int n = min(lcnt[tid], kLCap);
    gbase[tid] = n == 0 ? 0 : atomicAdd(&cand_count[tid], n);
  }
  __syncthreads();
  for (int i = tid; i < Q * kLCap; i += kThreads) {
    const int q = i / kLCap, e = i % kLCap;
    if (e < min(lcnt[q], kLCap) && gbase[q] + e < cap) cand[(size_t)q * cap + gbase[q] + e] = lbuf[q][e];
  }
}

// The list of a wave's S * 64 best keys, descending over positions
// p = 64 s + lane (register s, lane). Half-cleaners sort a bitonic list.
template <int S>
__device__ __forceinline__ void list_clean(uint64_t (&lv)[S]) {
#pragma unroll
  for (int st = S / 2; st >= 1; st >>= 1)
#pragma unroll
    for (int s = 0; s < S; ++s)
      if ((s & st) == 0) {
        const uint64_t x = lv[s], y = lv[s + st];
        lv[s] = x > y ? x : y;
        lv[s + st] = x > y ? y : x;
      }
#pragma unroll
  for (int s = 0; s < S; ++s)
#pragma unroll
    for (int stride = 32; stride > 0; stride >>= 1) lv[s] = cx_lanes(lv[s], stride, true);
}
// Fold 64 keys (one per lane, any order) into the list: sorted ascending
// they are the reversed tail of a descending list, so max(A_p, B_(KL-1-p))
// touches the last register only and leaves a bitonic list.
template <int S>
__device__ __forceinline__ void list_fold(uint64_t (&lv)[S], uint64_t key) {
  const uint64_t asc = wave_sort64(key, false);
  lv[S - 1] = lv[S - 1] > asc ? lv[S - 1] : asc;
  list_clean<S>(lv);
}

// One workgroup of 16 waves per query; a query with more candidates than the
// array holds, or fewer than min(k, N), is flagged for the exact path and
// left untouched. Wave w takes candidates
// 64 w + lane + 1024 i; keys that beat its list's last key are gathered in
// LDS and folded 64 at a time. The 16 lists are then merged pairwise in a
// tree, and wave 0 writes the first k.
template <int S>
__global__ void __launch_bounds__(1024) select_few_kernel(const uint64_t* __restrict__ cand,
                                                          const int* __restrict__ cand_count, int cap, int k,
                                                          int need, int* __restrict__ flags,
                                                          uint32_t* __restrict__ flag_word,
                                                          int32_t* __restrict__ ids, float* __restrict__ sims) {
  constexpr int KL = 64 * S;
  constexpr int W = 16;
  __shared__ uint64_t lists[W][KL];
  __shared__ uint64_t pend[W][2 * kWave];
  const int q = blockIdx.x;
  const int tid = threadIdx.x;
  const int lane = (int)lane_id();
  const int w = __builtin_amdgcn_readfirstlane(tid / kWave);
  const int n = cand_count[q];
  if (n > cap || n < need) {                         // need = min(k, N)
    if (tid == 0) {
      flags[q] = 1;
      *flag_word = 1u;
    }
    return;
  }
  if (tid == 0) flags[q] = 0;
  const uint64_t* src = cand + (size_t)q * cap;
  uint64_t lv[S];
#pragma unroll
  for (int s = 0; s < S; ++s) lv[s] = kPadKey;
  uint64_t* buf = pend[w];
  int n_buf = 0;
  auto take = [&](uint64_t cur) {
    const bool keep = cur > lane_value_u64(lv[S - 1], kWave - 1);
    const uint64_t mask = __ballot(keep);
    if (mask == 0) return;
    const int pos = n_buf + (int)__builtin_amdgcn_mbcnt_hi((uint32_t)(mask >> 32),
                                                            __builtin_amdgcn_mbcnt_lo((uint32_t)mask, 0u));
    if (keep) buf[pos] = cur;
    n_buf += __popcll(mask);
    __builtin_amdgcn_wave_barrier();
    if (n_buf >= kWave) {
      list_fold<S>(lv, buf[lane]);
      n_buf -= kWave;
      const uint64_t rest = lane < n_buf ? buf[kWave + lane] : kPadKey;
      __builtin_amdgcn_wave_barrier();
      if (lane < n_buf) buf[lane] = rest;
      __builtin_amdgcn_wave_barrier();
    }
  };
  constexpr int kPre = 4;                            // loads in flight per wave
  for (int b0 = w * kWave; b0 < n; b0 += kPre * W * kWave) {
    uint64_t cur[kPre];
#pragma unroll
    for (int j = 0; j < kPre; ++j) {
      const int e = b0 + j * W * kWave + lane;
      cur[j] = e < n ? src[e] : kPadKey;
    }
#pragma unroll
    for (int j = 0; j < kPre; ++j) take(cur[j]);
  }
  if (n_buf > 0) list_fold<S>(lv, lane < n_buf ? buf[lane] : kPadKey);
#pragma unroll
  for (int s = 0; s < S; ++s) lists[w][64 * s + lane] = lv[s];
  __syncthreads();
  for (int h = 1; h < W; h <<= 1) {
    if ((w & (2 * h - 1)) == 0) {
      // C_p = max(A_p, B_(KL-1-p)) is bitonic and holds the KL best of both.
#pragma unroll
      for (int s = 0; s < S; ++s) {
        const uint64_t o = lists[w + h][64 * (S - 1 - s) + (kWave - 1 - lane)];
        lv[s] = lv[s] > o ? lv[s] : o;
      }
      list_clean<S>(lv);
#pragma unroll
      for (int s = 0; s < S; ++s) lists[w][64 * s + lane] = lv[s];
    }
    __syncthreads();
  }
  if (w != 0) return;
#pragma unroll
  for (int s = 0; s < S; ++s) {
    const int p = 64 * s + lane;
    if (p < k) {
      ids[(size_t)q * k + p] = lv[s] == kPadKey ? -1 : key_id(lv[s]);
      sims[(size_t)q * k + p] = lv[s] == kPadKey ? -__builtin_inff() : key_sim(lv[s]);
    }
  }
}

}  // namespace

hipError_t launch_stream_sample(EmbView queries, int Q, EmbView hist, int N, int d, int sample_every,
                                int n_samples, float* gm, hipStream_t stream) {
  if (Q <= 0 || Q > kStreamMaxQ || d % 32 != 0 || d > kStreamMaxD || n_samples <= 0 || sample_every <= 0 ||
      (long long)(n_samples - 1) * sample_every * 256 + 256 > N)
    return hipErrorInvalidValue;
  const int blocks = (n_samples * 16 + kWaves - 1) / kWaves;
  const size_t lds = (size_t)(d / 32) * kWave * sizeof(uint4);
  hipLaunchKernelGGL(stream_sample_kernel, dim3(blocks), dim3(kThreads), lds, stream, queries, Q, hist, N, d,
                     sample_every, n_samples, gm);
  return hipGetLastError();
}

hipError_t launch_stream_search(EmbView queries, int Q, EmbView hist, int N, int d, int k, int chunk_rows,
                                const float* theta0, int cap, uint64_t* cand, int* cand_count, Flagged fl,
                                int32_t* ids, float* sims, hipStream_t stream) {
  if (Q <= 0 || Q > kStreamMaxQ || d % 32 != 0 || d > kStreamMaxD || k > 256 || N <= 0 || chunk_rows <= 0)
    return hipErrorInvalidValue;
  {
    LaunchScope scope("sim_topk", stream);
    const int blocks = (N + chunk_rows - 1) / chunk_rows;
    const size_t lds = (size_t)(d / 32) * kWave * sizeof(uint4);   // sized to d: more workgroups per CU
    hipLaunchKernelGGL(sim_stream_kernel, dim3(blocks), dim3(kThreads), lds, stream, queries, Q, hist, N, d,
                       chunk_rows, theta0, cap, cand, cand_count, fl.word);
  }
  LaunchScope scope("topk_select", stream);
  if (k <= 64)
    hipLaunchKernelGGL((select_few_kernel<1>), dim3(Q), dim3(1024), 0, stream, cand, cand_count, cap, k,
                       min(k, N), fl.flags, fl.word, ids, sims);
  else if (k <= 128)
    hipLaunchKernelGGL((select_few_kernel<2>), dim3(Q), dim3(1024), 0, stream, cand, cand_count, cap, k,
                       min(k, N), fl.flags, fl.word, ids, sims);
  else
    hipLaunchKernelGGL((select_few_kernel<4>), dim3(Q), dim3(1024), 0, stream, cand, cand_count, cap, k,
                       min(k, N), fl.flags, fl.word, ids, sims);
  return hipGetLastError();
}

}  // namespace sage
