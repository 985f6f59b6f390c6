// Merge of the per-stream neighbour lists into each request's final top-k.
//
// The fused similarity kernel leaves, for every request, one descending list
// of `list_len` neighbour keys per history chunk. Here one workgroup per
// request folds those lists together with bitonic merges in LDS: two
// descending lists A, B of length L give C_i = max(A_i, B_{L-1-i}), a bitonic
// sequence holding exactly the L largest keys of A and B, which log2(L)
// half-cleaner stages sort back into descending order.
#include "sage_device.hpp"
#include "sage_internal.hpp"

namespace sage {
namespace {

constexpr int kMergeThreads = 256;
constexpr int kMergeKeys = 4096;   // LDS capacity in keys (32 KiB)

// Workgroup (q, y) merges lists [y * per_group, ...) of query q (all of them
// when gridDim.y == 1). With `out_lists` it writes the merged list of L keys
// to out_lists[q][y] (first level of a two-level merge); otherwise the first
// k entries as ids and similarities.
__device__ __forceinline__ void merge_query(uint64_t* slot, int q, const uint64_t* __restrict__ partial,
                                            int n_lists, int list_len, int k, int per_group,
                                            uint64_t* __restrict__ out_lists, int32_t* __restrict__ ids,
                                            float* __restrict__ sims) {
  const int L = list_len;
  const int G = kMergeKeys / L;                 // lists per LDS batch (power of two)
  const int first = blockIdx.y * per_group;
  const int count = min(per_group, n_lists - first);
  const uint64_t* src = partial + ((size_t)q * n_lists + first) * L;
  const int t = threadIdx.x;

  bool have_result = false;
  for (int base = 0; base < count || !have_result;) {
    const int s0 = have_result ? 1 : 0;
    const int n_load = min(G - s0, count - base);
    int n_used = s0 + n_load;
    int n_tree = 1;
    while (n_tree < n_used) n_tree <<= 1;
    // Load the batch (slot 0 keeps the running result) and pad to n_tree lists.
    for (int i = t; i < n_load * L; i += kMergeThreads) slot[s0 * L + i] = src[(size_t)base * L + i];
    for (int i = n_used * L + t; i < n_tree * L; i += kMergeThreads) slot[i] = kPadKey;
    __syncthreads();
    for (int width = 1; width < n_tree; width <<= 1) {
      const int pairs = n_tree / (2 * width);
      // C_i = max(A_i, B_{L-1-i}) for every pair (A in slot j, B in slot j + width).
      for (int e = t; e < pairs * L; e += kMergeThreads) {
        const int p = e / L, i = e - p * L;
        const int a = (2 * p) * width, b = a + width;
        const uint64_t va = slot[a * L + i], vb = slot[b * L + (L - 1 - i)];
        slot[a * L + i] = va > vb ? va : vb;
      }
      __syncthreads();
      for (int stride = L >> 1; stride > 0; stride >>= 1) {
        for (int e = t; e < pairs * (L >> 1); e += kMergeThreads) {
          const int p = e / (L >> 1), r = e - p * (L >> 1);
          const int a = (2 * p) * width;
          const int i = (r / stride) * (2 * stride) + (r % stride);
          uint64_t* s = slot + a * L;
          const uint64_t x = s[i], y = s[i + stride];
          if (y > x) { s[i] = y; s[i + stride] = x; }
        }
        __syncthreads();
      }
    }
    have_result = true;
    base += n_load;
  }
  if (out_lists) {
    uint64_t* dst = out_lists + ((size_t)q * gridDim.y + blockIdx.y) * L;
    for (int i = t; i < L; i += kMergeThreads) dst[i] = slot[i];
    return;
  }
  for (int i = t; i < k; i += kMergeThreads) {
    const uint64_t key = slot[i];
    ids[(size_t)q * k + i] = key == kPadKey ? -1 : key_id(key);
    sims[(size_t)q * k + i] = key == kPadKey ? -__builtin_inff() : key_sim(key);
  }
}

// Queries q = blockIdx.x, + gridDim.x, ... As the exact fallback (with
// only_flagged) it returns at once unless a query of this call was flagged,
// and merges only the flagged queries.
__global__ void __launch_bounds__(kMergeThreads) topk_merge_kernel(
    const uint64_t* __restrict__ partial, int Q, int n_lists, int list_len, int k, int per_group,
    const int* __restrict__ only_flagged, const uint32_t* __restrict__ flag_word,
    uint64_t* __restrict__ out_lists, int32_t* __restrict__ ids, float* __restrict__ sims) {
  __shared__ uint64_t slot[kMergeKeys];
  if (only_flagged && *flag_word == 0u) return;
  for (int q = blockIdx.x; q < Q; q += gridDim.x) {
    if (only_flagged && only_flagged[q] == 0) continue;
    __syncthreads();                            // the previous query's LDS reads are done
    merge_query(slot, q, partial, n_lists, list_len, k, per_group, out_lists, ids, sims);
  }
}

}  // namespace

hipError_t launch_topk_merge(const uint64_t* partial, int Q, int n_lists, int list_len, int k,
                             const Flagged* only_flagged, uint64_t* scratch_lists, int32_t* ids, float* sims,
                             hipStream_t stream) {
  if (Q == 0) return hipSuccess;
  LaunchScope scope(only_flagged ? "topk_merge_fallback" : "topk_merge", stream);
  const int* flags = only_flagged ? only_flagged->flags : nullptr;
  const uint32_t* word = only_flagged ? only_flagged->word : nullptr;
  // One workgroup per query; as the fallback, at most 1024 that loop over the queries.
  const int gx = only_flagged ? std::min(Q, 1024) : Q;
  const int groups = merge_groups(Q, n_lists, list_len);
  if (groups > 1 && scratch_lists) {
    // Few queries with many lists: merge groups of lists in parallel first.
    const int per_group = (n_lists + groups - 1) / groups;
    hipLaunchKernelGGL(topk_merge_kernel, dim3(gx, groups), dim3(kMergeThreads), 0, stream, partial, Q,
                       n_lists, list_len, k, per_group, flags, word, scratch_lists, nullptr, nullptr);
    hipLaunchKernelGGL(topk_merge_kernel, dim3(gx), dim3(kMergeThreads), 0, stream, scratch_lists, Q, groups,
                       list_len, k, groups, flags, word, nullptr, ids, sims);
  } else {
    hipLaunchKernelGGL(topk_merge_kernel, dim3(gx), dim3(kMergeThreads), 0, stream, partial, Q, n_lists,
                       list_len, k, n_lists, flags, word, nullptr, ids, sims);
  }
  return hipGetLastError();
}

int merge_groups(int Q, int n_lists, int list_len) {
  const int per_batch = kMergeKeys / list_len;
  if (Q >= 1024 || n_lists <= per_batch) return 1;
  return (n_lists + per_batch - 1) / per_batch;   // one LDS batch of lists per first-level group
}

}  // namespace sage
