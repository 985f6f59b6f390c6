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

// Launch-configuration choice of the fused similarity/top-k kernel.
struct SimTopkPlan {
  int list_len;     // per-stream list length: next power of two >= k, at least 64
  int q_tile;       // queries per workgroup
  int chunk_rows;   // history rows per workgroup (multiple of the step size)
  int n_chunks;     // workgroups along the history axis (= streams per query)
  int q_tiles;      // workgroups along the query axis
  int sample_every; // threshold pre-pass: every sample_every-th 256-row step
  int n_samples;    // sampled steps (0: no pre-pass, thresholds start at -inf)
  size_t partial_bytes;  // workspace: per-stream lists [Q][n_chunks][list_len] keys
  size_t gm_bytes;       //            sampled group maxima [Q][n_samples][16] f32
  size_t theta_bytes;    //            per-query threshold [Q] f32
  size_t workspace_bytes() const { return partial_bytes + gm_bytes + theta_bytes; }
};
SimTopkPlan plan_sim_topk(int Q, int N, int d, int k);

// Launchers: each enqueues kernels on `stream` and returns the HIP status of
// the launch (hipSuccess or the first error).
hipError_t launch_ingest_bf16(const float* src, size_t n, uint16_t* dst, hipStream_t stream);
hipError_t launch_cost(const int32_t* prompt_len, int Q, const double* bin_repr, int B,
                       float* cost, hipStream_t stream);
hipError_t launch_index(const float* mass, const float* cost, const int32_t* prompt_len,
                        const double* bin_repr, int Q, int B, float* index, int32_t* argmin,
                        hipStream_t stream);
size_t rank_workspace_bytes(int Q);
hipError_t launch_rank(const float* index, int Q, int32_t* order, void* ws, hipStream_t stream);
hipError_t launch_sim_topk(const uint16_t* queries, int Q, const uint16_t* hist, int N, int d,
                           int k, const SimTopkPlan& plan, void* workspace, hipStream_t stream);
hipError_t launch_topk_merge(const uint64_t* partial, int Q, int n_lists, int list_len, int k,
                             int32_t* ids, float* sims, hipStream_t stream);
hipError_t launch_hist(const int32_t* ids, const float* sims, int Q, int k, const int32_t* hist_len,
                       int N, float tau, const double* edges, int B, int32_t* counts, float* mass,
                       hipStream_t stream);

}  // namespace sage
