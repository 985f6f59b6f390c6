// Host-side internals of libsage: launchers of the gfx950 kernels and the
// per-launch timing hook. Not part of the public C ABI.
#pragma once
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace sage {

// Records a start/stop event pair around one kernel launch when a stage timer
// is attached to the calling thread; a no-op otherwise.
struct LaunchScope {
  LaunchScope(const char* name, hipStream_t stream);
  ~LaunchScope();
  LaunchScope(const LaunchScope&) = delete;
  LaunchScope& operator=(const LaunchScope&) = delete;
 private:
  int slot_ = -1;
  hipStream_t stream_;
};

// A matrix of bf16 embeddings (raw bits), `rows` x d: element (r, c) sits at
// base[(c / 32) * panel + r * row + c % 32]. Row-major [rows, d]: panel = 32,
// row = d. Panel-major [d / 32][rows][32]: panel = 32 * rows, row = 32; one
// 32-column slice of consecutive rows is then contiguous, so a load of 16
// rows of a slice covers whole 128-byte lines.
struct EmbView {
  const uint16_t* base;
  long long panel;
  long long row;
};
inline EmbView rows_view(const uint16_t* base, int d) { return EmbView{base, 32, (long long)d}; }
inline EmbView panels_view(const uint16_t* base, int rows) { return EmbView{base, 32LL * rows, 32}; }
// Address of element (r, c) of an embedding matrix in either layout.
__device__ __forceinline__ const uint16_t* emb_at(const EmbView& m, int r, int c) {
  return m.base + (long long)(c >> 5) * m.panel + (long long)r * m.row + (c & 31);
}
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;

// Launch plan of the neighbour search (threshold pre-pass, search, merge).
struct SimTopkPlan {
  // exact per-chunk lists (the path for k > 64, and the fallback of the filtered path)
  int list_len;     // list length: next power of two >= k, at least 64
  int q_tile;       // queries per workgroup
  int q_tiles;      // workgroups along the query axis
  int chunk_rows;   // history rows per workgroup (multiple of 256)
  int n_chunks;     // workgroups along the history axis (= lists per query)
  // threshold pre-pass: every sample_every-th 256-row step (0 samples: none)
  int sample_every;
  int n_samples;
  // filtered path (k <= 64)
  bool fast;
  int f_q_tiles, f_chunk_rows, f_n_chunks;
  int f_spb;        // sampled steps per threshold-sampling workgroup
  int f_q_groups;   // query-tile groups across the 8 XCDs (0: plain mapping)
  int seg_cap;      // candidate keys per (query, chunk) segment
  // few-query stream path (Q <= kStreamMaxQ, any k <= 256)
  bool stream;
  int s_chunk_rows; // history rows per workgroup
  int s_cap;        // candidate keys per query
  // workspace layout (byte offsets, 256-aligned)
  size_t off_partial, off_merge, off_gm, off_theta, off_seg, off_segcnt, off_flags, off_flag_word, off_cand, off_ccount,
      total_bytes;
  size_t workspace_bytes() const { return total_bytes; }
};
SimTopkPlan plan_sim_topk(int Q, int N, int d, int k);
// Few-query stream path: limits, and the search + candidate select.
constexpr int kStreamMaxQ = 16;
constexpr int kStreamMaxD = 2048;
// Threshold pre-pass of the stream path (group maxima of the sampled steps).
hipError_t launch_stream_sample(EmbView queries, int Q, EmbView hist, int N, int d, int sample_every,
                                int n_samples, float* gm, hipStream_t stream);
// Test hook (sage_debug_theta_floor): a floor on the pre-pass threshold of the
// filtered and stream paths; -inf when unset.
float debug_theta_floor();
// Queries sent to the exact fallback: flags[q] = 1 for each, and *word = 1
// once any query is flagged. The search's first kernel that always runs (the
// filter kernel, the stream search) clears the word, so that the fallback
// kernels return at once when it is still 0; nothing here depends on the
// call, so a captured graph replays it as it stands.
struct Flagged {
  int* flags;
  uint32_t* word;
};

hipError_t launch_stream_search(EmbView queries, int Q, EmbView hist, int N, int d, int k, int chunk_rows,
                                const float* theta0, int cap, uint64_t* cand, int* cand_count, Flagged fl,
                                int32_t* ids, float* sims, hipStream_t stream);

// Launchers: each enqueues kernels on `stream` and returns the HIP status of
// the launch (hipSuccess or the first error).
hipError_t launch_ingest_bf16(const float* src, size_t n, uint16_t* dst, hipStream_t stream);
// [rows, d] -> panel-major bf16: from fp32 (rounded to nearest even) or from bf16 bits.
hipError_t launch_ingest_panels(const float* src, int rows, int d, uint16_t* dst, hipStream_t stream);
hipError_t launch_panels_from_rows(const uint16_t* src, int rows, int d, uint16_t* dst, hipStream_t stream);
hipError_t launch_store_insert(const float* emb, const int32_t* out_len, int n, int d, long long total,
                               int cap, uint16_t* ring_emb, int32_t* ring_len, hipStream_t stream);
hipError_t launch_queue_admit(const int64_t* free_slots, int batch, const float* new_mass,
                              const int32_t* new_plen, int B, long long next_request, int slots, float* mass,
                              int32_t* plen, int64_t* request, hipStream_t stream);
hipError_t launch_queue_dispatch(const int32_t* order, int batch, const int64_t* request, int slots,
                                 int64_t* free_slots, int64_t* dispatched, hipStream_t stream);
// Device check of the bin and prompt-length preconditions (bitmask to *status).
hipError_t launch_check_inputs(const double* edges, int n_edges, const double* repr, int B, const int32_t* plen,
                               int Q, int32_t* status, hipStream_t stream);
hipError_t launch_cost(const int32_t* prompt_len, int Q, const double* bin_repr, int B,
                       float* cost, hipStream_t stream);
hipError_t launch_mix_uniform(const float* mass, int Q, int B, float weight, float* out,
                              hipStream_t stream);
// Index variants: cost model (0 resource, 1 output length, 2 input + 2 output),
// kind (0 Gittins, 1 mean) and a uniform mixing weight in [0, 1).
struct IndexVariant {
  int cost_model = 0;
  int kind = 0;
  float noise = 0.0f;
  int levels = 0;     // > 0: the refreshed index at o = 0, bucket, ..., (levels - 1) * bucket
};
hipError_t launch_index(const float* mass, const float* cost, const int32_t* prompt_len,
                        const double* bin_repr, const int32_t* generated, int bucket, int Q, int B,
                        float* index, int32_t* argmin, hipStream_t stream,
                        const IndexVariant* variant = nullptr);
size_t rank_workspace_bytes(int Q);
hipError_t launch_rank(const float* index, int Q, int32_t* order, void* ws, hipStream_t stream);
// Neighbours of every query: ids [Q, k] and sims [Q, k] (sorted, padded).
hipError_t launch_neighbours(EmbView queries, int Q, EmbView hist, int N, int d, int k,
                             const SimTopkPlan& plan, void* workspace, int32_t* ids, float* sims,
                             hipStream_t stream);
// Merge of per-chunk lists; with `only_flagged`, queries whose flag is 0 are skipped.
// Number of first-level groups of the list merge (1: single level).
int merge_groups(int Q, int n_lists, int list_len);
hipError_t launch_topk_merge(const uint64_t* partial, int Q, int n_lists, int list_len, int k,
                             const Flagged* only_flagged, uint64_t* scratch_lists, int32_t* ids, float* sims,
                             hipStream_t stream);
hipError_t launch_hist(const int32_t* ids, const float* sims, int Q, int k, const int32_t* hist_len,
                       int N, float tau, const double* edges, int B, int uniform, int32_t* counts,
                       float* mass, hipStream_t stream);


// Semantic-unaware predictor: the store's length index and the neighbours by
// input-length similarity.
constexpr int kLengthMaxLen = 1 << 20;
size_t length_index_workspace_bytes(int N);
hipError_t launch_length_index(const int32_t* hist_prompt_len, int N, int max_len, int32_t* by_len,
                               int32_t* sorted_len, int32_t* off, void* ws, hipStream_t stream);
hipError_t launch_length_neighbours(const int32_t* prompt_len, int Q, const int32_t* by_len,
                                    const int32_t* sorted_len, const int32_t* off, int max_len, int N, int k,
                                    int32_t* ids, float* sims, hipStream_t stream);

// Host event loop of sage_simulate (inputs already validated); 0 on success.
int simulate_queue(const double* arrival, const int32_t* prompt_len, const int32_t* output_len, int R,
                   const int32_t* order, int levels, int informed, int bucket, int servers,
                   double rate, int queue_cap, double* finish, int32_t* preemptions);

}  // namespace sage
