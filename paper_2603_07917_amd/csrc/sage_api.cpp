// C ABI of libsage: argument validation, workspace sizing, device checks and
// dispatch to the gfx950 kernels. Nothing here allocates device memory.
#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "sage.h"
#include "sage_internal.hpp"

#define SAGE_API extern "C" __attribute__((visibility("default")))

namespace {

thread_local std::string g_last_error;
thread_local sage_timer* g_timer = nullptr;

int fail(int status, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int status, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return status;
}

int ok() {
  g_last_error.clear();
  return SAGE_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

// Device check, cached per device ordinal: the kernels are built for gfx950.
int check_device() {
  static std::mutex mu;
  static std::vector<int> arch_state;   // 0 unknown, 1 ok, -1 unsupported
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SAGE_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  std::lock_guard<std::mutex> lock(mu);
  if ((int)arch_state.size() <= dev) arch_state.resize(dev + 1, 0);
  if (arch_state[dev] == 0) {
    hipDeviceProp_t prop;
    e = hipGetDeviceProperties(&prop, dev);
    if (e != hipSuccess) return fail(SAGE_EHIP, "hipGetDeviceProperties: %s", hipGetErrorString(e));
    arch_state[dev] = std::strncmp(prop.gcnArchName, "gfx950", 6) == 0 ? 1 : -1;
    if (arch_state[dev] < 0)
      return fail(SAGE_EUNSUPPORTED, "device %d is %s, the library is built for gfx950", dev,
                  prop.gcnArchName);
  }
  if (arch_state[dev] < 0) return fail(SAGE_EUNSUPPORTED, "device %d is not gfx950", dev);
  return SAGE_OK;
}

int hip_status(hipError_t e, const char* what) {
  if (e != hipSuccess) return fail(SAGE_EHIP, "%s: %s", what, hipGetErrorString(e));
  return ok();
}

constexpr float kMinTau = 9.5367431640625e-07f;   // 2^-20

int check_bins(const double* edges, int B) {
  if (B < 1 || B > SAGE_MAX_BINS) return fail(SAGE_EINVAL, "B=%d outside [1, %d]", B, SAGE_MAX_BINS);
  if (!edges) return fail(SAGE_EINVAL, "bin_edges is NULL");
  if (!aligned16(edges)) return fail(SAGE_EINVAL, "bin_edges is not 16-byte aligned");
  return SAGE_OK;
}

int check_tau(float tau) {
  if (!(tau >= kMinTau && tau <= 1.0f)) return fail(SAGE_EINVAL, "tau=%g outside [2^-20, 1]", (double)tau);
  return SAGE_OK;
}

}  // namespace

// ------------------------------------------------------------------ timer
struct sage_timer {
  int capacity = 0;
  int used = 0;
  std::vector<hipEvent_t> start, stop;
  std::vector<const char*> name;
  std::string only;          // when set, only launches of this name are timed
};

namespace sage {
LaunchScope::LaunchScope(const char* name, hipStream_t stream) : stream_(stream) {
  sage_timer* t = g_timer;
  if (!t || t->used >= t->capacity || (!t->only.empty() && t->only != name)) return;
  slot_ = t->used++;
  t->name[slot_] = name;
  (void)hipEventRecord(t->start[slot_], stream);
}
LaunchScope::~LaunchScope() {
  sage_timer* t = g_timer;
  if (slot_ < 0 || !t) return;
  (void)hipEventRecord(t->stop[slot_], stream_);
}
}  // namespace sage

SAGE_API int sage_timer_create(int capacity, sage_timer** out) {
  if (!out || capacity < 1) return fail(SAGE_EINVAL, "sage_timer_create: bad arguments");
  sage_timer* t = new sage_timer;
  t->capacity = capacity;
  t->start.resize(capacity);
  t->stop.resize(capacity);
  t->name.resize(capacity, nullptr);
  for (int i = 0; i < capacity; ++i) {
    hipError_t e1 = hipEventCreate(&t->start[i]);
    hipError_t e2 = hipEventCreate(&t->stop[i]);
    if (e1 != hipSuccess || e2 != hipSuccess) {
      t->capacity = i;
      sage_timer_destroy(t);
      return fail(SAGE_EHIP, "hipEventCreate failed");
    }
  }
  *out = t;
  return ok();
}

SAGE_API int sage_timer_destroy(sage_timer* t) {
  if (!t) return ok();
  if (g_timer == t) g_timer = nullptr;
  for (int i = 0; i < t->capacity; ++i) {
    (void)hipEventDestroy(t->start[i]);
    (void)hipEventDestroy(t->stop[i]);
  }
  delete t;
  return ok();
}

SAGE_API int sage_timer_attach(sage_timer* t) {
  g_timer = t;
  return ok();
}

SAGE_API int sage_timer_only(sage_timer* t, const char* label) {
  if (!t) return fail(SAGE_EINVAL, "timer is NULL");
  t->only = label ? label : "";
  return ok();
}

SAGE_API int sage_timer_reset(sage_timer* t) {
  if (!t) return fail(SAGE_EINVAL, "timer is NULL");
  t->used = 0;
  return ok();
}

namespace {
std::vector<const char*> timer_names(sage_timer* t) {
  std::vector<const char*> names;
  for (int i = 0; i < t->used; ++i) {
    bool seen = false;
    for (const char* n : names) seen = seen || std::strcmp(n, t->name[i]) == 0;
    if (!seen) names.push_back(t->name[i]);
  }
  return names;
}
}  // namespace

SAGE_API int sage_timer_count(sage_timer* t) {
  if (!t) return 0;
  return (int)timer_names(t).size();
}

SAGE_API int sage_timer_get(sage_timer* t, int i, const char** name, int* launches, double* total_ms) {
  if (!t || !name || !launches || !total_ms) return fail(SAGE_EINVAL, "sage_timer_get: NULL argument");
  std::vector<const char*> names = timer_names(t);
  if (i < 0 || i >= (int)names.size()) return fail(SAGE_EINVAL, "timer index %d out of range", i);
  int n = 0;
  double ms = 0.0;
  for (int j = 0; j < t->used; ++j) {
    if (std::strcmp(t->name[j], names[i]) != 0) continue;
    float e = 0.f;
    hipError_t err = hipEventElapsedTime(&e, t->start[j], t->stop[j]);
    if (err != hipSuccess) return fail(SAGE_EHIP, "hipEventElapsedTime: %s", hipGetErrorString(err));
    ms += e;
    ++n;
  }
  *name = names[i];
  *launches = n;
  *total_ms = ms;
  return ok();
}

// -------------------------------------------------------------- status
SAGE_API const char* sage_status_string(int status) {
  switch (status) {
    case SAGE_OK: return "SAGE_OK";
    case SAGE_EINVAL: return "SAGE_EINVAL: invalid argument";
    case SAGE_EWORKSPACE: return "SAGE_EWORKSPACE: workspace too small";
    case SAGE_EUNSUPPORTED: return "SAGE_EUNSUPPORTED: device is not gfx950";
    case SAGE_EHIP: return "SAGE_EHIP: HIP runtime error";
    default: return "unknown sage status";
  }
}

SAGE_API const char* sage_last_error(void) { return g_last_error.c_str(); }

// ------------------------------------------------------------- ingest
SAGE_API int sage_ingest_bf16(const float* src, size_t n, uint16_t* dst, sage_stream_t stream) {
  if (n == 0) return ok();
  if (!src || !dst) return fail(SAGE_EINVAL, "sage_ingest_bf16: NULL pointer");
  if (!aligned16(src) || !aligned16(dst)) return fail(SAGE_EINVAL, "sage_ingest_bf16: misaligned pointer");
  const char* s0 = reinterpret_cast<const char*>(src);
  const char* d0 = reinterpret_cast<const char*>(dst);
  if (s0 < d0 + n * sizeof(uint16_t) && d0 < s0 + n * sizeof(float))
    return fail(SAGE_EINVAL, "sage_ingest_bf16: src and dst overlap");
  int st = check_device();
  if (st != SAGE_OK) return st;
  return hip_status(sage::launch_ingest_bf16(src, n, dst, (hipStream_t)stream), "ingest_bf16 launch");
}

namespace {
int check_panels_args(const char* fn, const void* src, int rows, int d, const void* dst) {
  if (rows < 0) return fail(SAGE_EINVAL, "%s: rows=%d is negative", fn, rows);
  if (rows >= (1 << 29)) return fail(SAGE_EINVAL, "%s: rows=%d not below 2^29", fn, rows);
  if (d < 32 || d % 32 != 0) return fail(SAGE_EINVAL, "%s: d=%d must be a positive multiple of 32", fn, d);
  if (rows == 0) return SAGE_OK;
  if (!src || !dst) return fail(SAGE_EINVAL, "%s: NULL pointer", fn);
  if (!aligned16(src) || !aligned16(dst)) return fail(SAGE_EINVAL, "%s: misaligned pointer", fn);
  return SAGE_OK;
}
}  // namespace

SAGE_API int sage_ingest_bf16_panels(const float* src, int rows, int d, uint16_t* dst, sage_stream_t stream) {
  int st = check_panels_args("sage_ingest_bf16_panels", src, rows, d, dst);
  if (st != SAGE_OK || rows == 0) return st == SAGE_OK ? ok() : st;
  const char* s0 = reinterpret_cast<const char*>(src);
  const char* d0 = reinterpret_cast<const char*>(dst);
  const size_t n = (size_t)rows * d;
  if (s0 < d0 + n * sizeof(uint16_t) && d0 < s0 + n * sizeof(float))
    return fail(SAGE_EINVAL, "sage_ingest_bf16_panels: src and dst overlap");
  if ((st = check_device()) != SAGE_OK) return st;
  return hip_status(sage::launch_ingest_panels(src, rows, d, dst, (hipStream_t)stream), "ingest_panels launch");
}

SAGE_API int sage_panels_from_rows(const uint16_t* src, int rows, int d, uint16_t* dst, sage_stream_t stream) {
  int st = check_panels_args("sage_panels_from_rows", src, rows, d, dst);
  if (st != SAGE_OK || rows == 0) return st == SAGE_OK ? ok() : st;
  const char* s0 = reinterpret_cast<const char*>(src);
  const char* d0 = reinterpret_cast<const char*>(dst);
  const size_t bytes = (size_t)rows * d * sizeof(uint16_t);
  if (s0 < d0 + bytes && d0 < s0 + bytes) return fail(SAGE_EINVAL, "sage_panels_from_rows: src and dst overlap");
  if ((st = check_device()) != SAGE_OK) return st;
  return hip_status(sage::launch_panels_from_rows(src, rows, d, dst, (hipStream_t)stream),
                    "panels_from_rows launch");
}

SAGE_API int sage_store_insert(const float* emb, const int32_t* out_len, int n, int d, long long total,
                               int capacity, uint16_t* ring_emb, int32_t* ring_len, sage_stream_t stream) {
  if (n < 0) return fail(SAGE_EINVAL, "n=%d is negative", n);
  if (d < 32 || d % 32 != 0) return fail(SAGE_EINVAL, "d=%d must be a positive multiple of 32", d);
  if (capacity < 1) return fail(SAGE_EINVAL, "capacity=%d must be >= 1", capacity);
  if (total < 0) return fail(SAGE_EINVAL, "total=%lld is negative", total);
  if (n == 0) return ok();
  const void* ptrs[] = {emb, out_len, ring_emb, ring_len};
  for (const void* p : ptrs) {
    if (!p) return fail(SAGE_EINVAL, "sage_store_insert: NULL pointer");
    if (!aligned16(p)) return fail(SAGE_EINVAL, "sage_store_insert: misaligned pointer");
  }
  int st = check_device();
  if (st != SAGE_OK) return st;
  return hip_status(sage::launch_store_insert(emb, out_len, n, d, total, capacity, ring_emb, ring_len,
                                              (hipStream_t)stream),
                    "store_insert launch");
}

// ------------------------------------------------------------- queue
SAGE_API int sage_queue_admit(const int64_t* free_slots, int batch, const float* new_mass,
                              const int32_t* new_plen, int B, long long next_request, int slots, float* mass,
                              int32_t* plen, int64_t* request, sage_stream_t stream) {
  if (batch < 0) return fail(SAGE_EINVAL, "batch=%d is negative", batch);
  if (B < 1 || B > SAGE_MAX_BINS) return fail(SAGE_EINVAL, "B=%d outside [1, %d]", B, SAGE_MAX_BINS);
  if (slots < batch) return fail(SAGE_EINVAL, "slots=%d is smaller than batch=%d", slots, batch);
  if (next_request < 0) return fail(SAGE_EINVAL, "next_request=%lld is negative", next_request);
  if (batch == 0) return ok();
  const void* ptrs[] = {free_slots, new_mass, new_plen, mass, plen, request};
  for (const void* p : ptrs) {
    if (!p) return fail(SAGE_EINVAL, "sage_queue_admit: NULL pointer");
    if (!aligned16(p)) return fail(SAGE_EINVAL, "sage_queue_admit: misaligned pointer");
  }
  int st = check_device();
  if (st != SAGE_OK) return st;
  return hip_status(sage::launch_queue_admit(free_slots, batch, new_mass, new_plen, B, next_request, slots, mass,
                                             plen, request, (hipStream_t)stream),
                    "queue_admit launch");
}

SAGE_API int sage_queue_dispatch(const int32_t* order, int batch, const int64_t* request, int slots,
                                 int64_t* free_slots, int64_t* dispatched, sage_stream_t stream) {
  if (batch < 0) return fail(SAGE_EINVAL, "batch=%d is negative", batch);
  if (slots < batch) return fail(SAGE_EINVAL, "slots=%d is smaller than batch=%d", slots, batch);
  if (batch == 0) return ok();
  const void* ptrs[] = {order, request, free_slots, dispatched};
  for (const void* p : ptrs) {
    if (!p) return fail(SAGE_EINVAL, "sage_queue_dispatch: NULL pointer");
    if (!aligned16(p)) return fail(SAGE_EINVAL, "sage_queue_dispatch: misaligned pointer");
  }
  int st = check_device();
  if (st != SAGE_OK) return st;
  return hip_status(sage::launch_queue_dispatch(order, batch, request, slots, free_slots, dispatched,
                                                (hipStream_t)stream),
                    "queue_dispatch launch");
}

// ------------------------------------------------------------- predict
namespace {
int check_predict_sizes(int Q, int N, int d, int k, int B) {
  if (Q < 0) return fail(SAGE_EINVAL, "Q=%d is negative", Q);
  if (N < 1) return fail(SAGE_EINVAL, "N=%d must be >= 1", N);
  if (d < 32 || d % 32 != 0) return fail(SAGE_EINVAL, "d=%d must be a positive multiple of 32", d);
  if (k < 1 || k > SAGE_MAX_K) return fail(SAGE_EINVAL, "k=%d outside [1, %d]", k, SAGE_MAX_K);
  if (B < 1 || B > SAGE_MAX_BINS) return fail(SAGE_EINVAL, "B=%d outside [1, %d]", B, SAGE_MAX_BINS);
  return SAGE_OK;
}
}  // namespace

SAGE_API size_t sage_predict_workspace_bytes(int Q, int N, int d, int k, int B) {
  std::string keep = g_last_error;
  if (check_predict_sizes(Q, N, d, k, B) != SAGE_OK) return 0;
  g_last_error = keep;
  if (Q == 0) return 0;
  return sage::plan_sim_topk(Q, N, d, k).workspace_bytes();
}

SAGE_API int sage_predict_layout(const uint16_t* queries, int query_layout, int Q, const uint16_t* hist_emb,
                                 int hist_layout, const int32_t* hist_len, int N, int d, int k, float tau,
                                 const double* bin_edges, int B, int32_t* nbr_ids, float* nbr_sims,
                                 int32_t* counts, float* mass, void* workspace, size_t workspace_bytes,
                                 sage_stream_t stream) {
  for (int layout : {query_layout, hist_layout})
    if (layout != SAGE_LAYOUT_ROWS && layout != SAGE_LAYOUT_PANELS)
      return fail(SAGE_EINVAL, "layout=%d is not a SAGE_LAYOUT_* value", layout);
  int st = check_predict_sizes(Q, N, d, k, B);
  if (st != SAGE_OK) return st;
  if ((st = check_tau(tau)) != SAGE_OK) return st;
  if (Q == 0) return ok();
  if ((st = check_bins(bin_edges, B)) != SAGE_OK) return st;
  const void* ptrs[] = {queries, hist_emb, hist_len, nbr_ids, nbr_sims, counts, mass};
  const char* names[] = {"queries", "hist_emb", "hist_len", "nbr_ids", "nbr_sims", "counts", "mass"};
  for (int i = 0; i < 7; ++i) {
    if (!ptrs[i]) return fail(SAGE_EINVAL, "sage_predict: %s is NULL", names[i]);
    if (!aligned16(ptrs[i])) return fail(SAGE_EINVAL, "sage_predict: %s is not 16-byte aligned", names[i]);
  }
  const sage::SimTopkPlan plan = sage::plan_sim_topk(Q, N, d, k);
  if (workspace_bytes < plan.workspace_bytes() || !workspace)
    return fail(SAGE_EWORKSPACE, "sage_predict: workspace of %zu bytes, %zu needed", workspace_bytes,
                plan.workspace_bytes());
  if (!aligned16(workspace)) return fail(SAGE_EINVAL, "sage_predict: workspace is not 16-byte aligned");
  if ((st = check_device()) != SAGE_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  const sage::EmbView qv = query_layout == SAGE_LAYOUT_PANELS ? sage::panels_view(queries, Q)
                                                              : sage::rows_view(queries, d);
  const sage::EmbView hv = hist_layout == SAGE_LAYOUT_PANELS ? sage::panels_view(hist_emb, N)
                                                             : sage::rows_view(hist_emb, d);
  hipError_t e = sage::launch_neighbours(qv, Q, hv, N, d, k, plan, workspace, nbr_ids, nbr_sims, s);
  if (e != hipSuccess) return hip_status(e, "neighbour search launch");
  e = sage::launch_hist(nbr_ids, nbr_sims, Q, k, hist_len, N, tau, bin_edges, B, 0, counts, mass, s);
  return hip_status(e, "hist launch");
}

// ------------------------------------------------ predict, no allocation
// Workspace of sage_predict_noalloc: a file-scope device array, one copy per
// GPU, held until the process ends. Host code never passes its name to a
// kernel (on the host the name is only a stand-in); it uses the device
// address from hipGetSymbolAddress, looked up once per device with that
// device current.
static __device__ __align__(256) unsigned char scratch[SAGE_NOALLOC_SCRATCH_BYTES];

namespace {
int scratch_address(void** out) {
  static std::mutex mu;
  static std::vector<void*> addr;                    // per device ordinal, NULL until looked up
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(SAGE_EHIP, "hipGetDevice: %s", hipGetErrorString(e));
  std::lock_guard<std::mutex> lock(mu);
  if ((int)addr.size() <= dev) addr.resize(dev + 1, nullptr);
  if (!addr[dev]) {
    void* p = nullptr;
    e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    if (e != hipSuccess || !p)
      return fail(SAGE_EHIP, "hipGetSymbolAddress(scratch): %s", hipGetErrorString(e));
    addr[dev] = p;
  }
  *out = addr[dev];
  return SAGE_OK;
}
}  // namespace

SAGE_API int sage_predict_noalloc(const uint16_t* queries, int query_layout, int Q, const uint16_t* hist_emb,
                                  int hist_layout, const int32_t* hist_len, int N, int d, int k, float tau,
                                  const double* bin_edges, int B, int32_t* nbr_ids, float* nbr_sims,
                                  int32_t* counts, float* mass, sage_stream_t stream) {
  int st = check_predict_sizes(Q, N, d, k, B);
  if (st != SAGE_OK) return st;
  if (Q == 0) return sage_predict_layout(queries, query_layout, 0, hist_emb, hist_layout, hist_len, N, d, k, tau,
                                         bin_edges, B, nbr_ids, nbr_sims, counts, mass, nullptr, 0, stream);
  const size_t need = sage::plan_sim_topk(Q, N, d, k).workspace_bytes();
  if (need > (size_t)SAGE_NOALLOC_SCRATCH_BYTES)
    return fail(SAGE_EWORKSPACE, "sage_predict_noalloc: this search needs %zu bytes of scratch, the static "
                "array holds %zu (use sage_predict_layout with a workspace)", need,
                (size_t)SAGE_NOALLOC_SCRATCH_BYTES);
  if ((st = check_device()) != SAGE_OK) return st;
  void* ws = nullptr;
  if ((st = scratch_address(&ws)) != SAGE_OK) return st;
  return sage_predict_layout(queries, query_layout, Q, hist_emb, hist_layout, hist_len, N, d, k, tau, bin_edges, B,
                             nbr_ids, nbr_sims, counts, mass, ws, (size_t)SAGE_NOALLOC_SCRATCH_BYTES, stream);
}

SAGE_API int sage_predict_stats(const void* workspace, size_t workspace_bytes, int Q, int N, int d, int k, int B,
                               long long* stats, sage_stream_t stream) {
  int st = check_predict_sizes(Q, N, d, k, B);
  if (st != SAGE_OK) return st;
  if (!stats) return fail(SAGE_EINVAL, "sage_predict_stats: stats is NULL");
  for (int i = 0; i < 5; ++i) stats[i] = 0;
  if (Q == 0) return ok();
  const sage::SimTopkPlan plan = sage::plan_sim_topk(Q, N, d, k);
  if (!workspace || workspace_bytes < plan.workspace_bytes())
    return fail(SAGE_EWORKSPACE, "sage_predict_stats: workspace of %zu bytes, %zu needed", workspace_bytes,
                plan.workspace_bytes());
  if ((st = check_device()) != SAGE_OK) return st;
  const char* ws = static_cast<const char*>(workspace);
  hipStream_t s = (hipStream_t)stream;
  std::vector<int32_t> counts, flags;
  int per_query = 0, cap = 0;
  if (plan.fast) {
    stats[0] = 1;
    per_query = plan.f_n_chunks;
    cap = plan.seg_cap;
  } else if (plan.stream) {
    stats[0] = 2;
    per_query = 1;
    cap = plan.s_cap;
  } else {
    stats[0] = 0;
    stats[1] = (long long)Q * plan.n_chunks * plan.list_len;
    stats[3] = plan.n_chunks;
    stats[4] = plan.list_len;
    return ok();
  }
  counts.resize((size_t)Q * per_query);
  flags.resize(Q);
  hipError_t e = hipMemcpyAsync(counts.data(), ws + (plan.fast ? plan.off_segcnt : plan.off_ccount),
                                counts.size() * sizeof(int32_t), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess)
    e = hipMemcpyAsync(flags.data(), ws + plan.off_flags, flags.size() * sizeof(int32_t), hipMemcpyDeviceToHost, s);
  if (e == hipSuccess) e = hipStreamSynchronize(s);
  if (e != hipSuccess) return hip_status(e, "sage_predict_stats copy");
  long long keys = 0, flagged = 0;
  for (int32_t c : counts) keys += c < cap ? c : cap;
  for (int32_t f : flags) flagged += f != 0;
  stats[1] = keys;
  stats[2] = flagged;
  stats[3] = per_query;
  stats[4] = cap;
  return ok();
}

SAGE_API int sage_predict(const uint16_t* queries, int Q, const uint16_t* hist_emb,
                          const int32_t* hist_len, int N, int d, int k, float tau,
                          const double* bin_edges, int B, int32_t* nbr_ids, float* nbr_sims,
                          int32_t* counts, float* mass, void* workspace, size_t workspace_bytes,
                          sage_stream_t stream) {
  return sage_predict_layout(queries, SAGE_LAYOUT_ROWS, Q, hist_emb, SAGE_LAYOUT_ROWS, hist_len, N, d, k, tau,
                             bin_edges, B, nbr_ids, nbr_sims, counts, mass, workspace, workspace_bytes, stream);
}

static int histogram_impl(const int32_t* nbr_ids, const float* nbr_sims, int Q, int k,
                          const int32_t* hist_len, int N, float tau, const double* bin_edges, int B,
                          int weighting, int32_t* counts, float* mass, sage_stream_t stream) {
  if (weighting != SAGE_WEIGHT_SIMILARITY && weighting != SAGE_WEIGHT_UNIFORM)
    return fail(SAGE_EINVAL, "weighting=%d is not a SAGE_WEIGHT_* value", weighting);
  if (Q < 0) return fail(SAGE_EINVAL, "Q=%d is negative", Q);
  if (k < 1 || k > SAGE_MAX_K) return fail(SAGE_EINVAL, "k=%d outside [1, %d]", k, SAGE_MAX_K);
  if (N < 1) return fail(SAGE_EINVAL, "N=%d must be >= 1", N);
  int st = check_tau(tau);
  if (st != SAGE_OK) return st;
  if (B < 1 || B > SAGE_MAX_BINS) return fail(SAGE_EINVAL, "B=%d outside [1, %d]", B, SAGE_MAX_BINS);
  if (Q == 0) return ok();
  if ((st = check_bins(bin_edges, B)) != SAGE_OK) return st;
  const void* ptrs[] = {nbr_ids, nbr_sims, hist_len, counts, mass};
  for (const void* p : ptrs) {
    if (!p) return fail(SAGE_EINVAL, "sage_histogram: NULL pointer");
    if (!aligned16(p)) return fail(SAGE_EINVAL, "sage_histogram: misaligned pointer");
  }
  if ((st = check_device()) != SAGE_OK) return st;
  return hip_status(sage::launch_hist(nbr_ids, nbr_sims, Q, k, hist_len, N, tau, bin_edges, B, weighting,
                                      counts, mass, (hipStream_t)stream),
                    "hist launch");
}

SAGE_API int sage_histogram(const int32_t* nbr_ids, const float* nbr_sims, int Q, int k,
                            const int32_t* hist_len, int N, float tau, const double* bin_edges, int B,
                            int32_t* counts, float* mass, sage_stream_t stream) {
  return histogram_impl(nbr_ids, nbr_sims, Q, k, hist_len, N, tau, bin_edges, B, SAGE_WEIGHT_SIMILARITY,
                        counts, mass, stream);
}

SAGE_API int sage_histogram_variant(const int32_t* nbr_ids, const float* nbr_sims, int Q, int k,
                                    const int32_t* hist_len, int N, float tau, const double* bin_edges,
                                    int B, int weighting, int32_t* counts, float* mass,
                                    sage_stream_t stream) {
  return histogram_impl(nbr_ids, nbr_sims, Q, k, hist_len, N, tau, bin_edges, B, weighting, counts, mass,
                        stream);
}

// ------------------------------------------ predict by input length
SAGE_API size_t sage_length_index_workspace_bytes(int N) {
  return N > 0 ? sage::length_index_workspace_bytes(N) : 0;
}

SAGE_API int sage_length_index(const int32_t* hist_prompt_len, int N, int max_len, int32_t* by_len,
                               int32_t* sorted_len, int32_t* len_off, void* workspace, size_t workspace_bytes,
                               sage_stream_t stream) {
  if (N < 1) return fail(SAGE_EINVAL, "N=%d must be >= 1", N);
  if (max_len < 1 || max_len > sage::kLengthMaxLen)
    return fail(SAGE_EINVAL, "max_len=%d outside [1, %d]", max_len, sage::kLengthMaxLen);
  const void* ptrs[] = {hist_prompt_len, by_len, sorted_len, len_off};
  for (const void* p : ptrs) {
    if (!p) return fail(SAGE_EINVAL, "sage_length_index: NULL pointer");
    if (!aligned16(p)) return fail(SAGE_EINVAL, "sage_length_index: misaligned pointer");
  }
  const size_t need = sage::length_index_workspace_bytes(N);
  if (!workspace || workspace_bytes < need)
    return fail(SAGE_EWORKSPACE, "sage_length_index: workspace of %zu bytes, %zu needed", workspace_bytes, need);
  if (!aligned16(workspace)) return fail(SAGE_EINVAL, "sage_length_index: workspace is not 16-byte aligned");
  int st = check_device();
  if (st != SAGE_OK) return st;
  return hip_status(sage::launch_length_index(hist_prompt_len, N, max_len, by_len, sorted_len, len_off, workspace,
                                              (hipStream_t)stream),
                    "length index launch");
}

SAGE_API int sage_predict_by_length(const int32_t* prompt_len, int Q, const int32_t* by_len,
                                    const int32_t* sorted_len, const int32_t* len_off, int max_len,
                                    const int32_t* hist_len, int N, int k, float tau, const double* bin_edges, int B,
                                    int32_t* nbr_ids, float* nbr_sims, int32_t* counts, float* mass,
                                    sage_stream_t stream) {
  if (Q < 0) return fail(SAGE_EINVAL, "Q=%d is negative", Q);
  if (N < 1) return fail(SAGE_EINVAL, "N=%d must be >= 1", N);
  if (k < 1 || k > SAGE_MAX_K) return fail(SAGE_EINVAL, "k=%d outside [1, %d]", k, SAGE_MAX_K);
  if (B < 1 || B > SAGE_MAX_BINS) return fail(SAGE_EINVAL, "B=%d outside [1, %d]", B, SAGE_MAX_BINS);
  if (max_len < 1 || max_len > sage::kLengthMaxLen)
    return fail(SAGE_EINVAL, "max_len=%d outside [1, %d]", max_len, sage::kLengthMaxLen);
  int st = check_tau(tau);
  if (st != SAGE_OK) return st;
  if (Q == 0) return ok();
  if ((st = check_bins(bin_edges, B)) != SAGE_OK) return st;
  const void* ptrs[] = {prompt_len, by_len, sorted_len, len_off, hist_len, nbr_ids, nbr_sims, counts, mass};
  for (const void* p : ptrs) {
    if (!p) return fail(SAGE_EINVAL, "sage_predict_by_length: NULL pointer");
    if (!aligned16(p)) return fail(SAGE_EINVAL, "sage_predict_by_length: misaligned pointer");
  }
  if ((st = check_device()) != SAGE_OK) return st;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = sage::launch_length_neighbours(prompt_len, Q, by_len, sorted_len, len_off, max_len, N, k, nbr_ids,
                                                nbr_sims, s);
  if (e != hipSuccess) return hip_status(e, "length neighbours launch");
  e = sage::launch_hist(nbr_ids, nbr_sims, Q, k, hist_len, N, tau, bin_edges, B, SAGE_WEIGHT_SIMILARITY, counts,
                        mass, s);
  return hip_status(e, "hist launch");
}

// --------------------------------------------------------- cost / index
SAGE_API int sage_cost(const int32_t* prompt_len, int Q, const double* bin_repr, int B, float* cost,
                       sage_stream_t stream) {
  if (Q < 0) return fail(SAGE_EINVAL, "Q=%d is negative", Q);
  if (B < 1 || B > SAGE_MAX_BINS) return fail(SAGE_EINVAL, "B=%d outside [1, %d]", B, SAGE_MAX_BINS);
  if (Q == 0) return ok();
  if (!prompt_len || !bin_repr || !cost) return fail(SAGE_EINVAL, "sage_cost: NULL pointer");
  if (!aligned16(prompt_len) || !aligned16(bin_repr) || !aligned16(cost))
    return fail(SAGE_EINVAL, "sage_cost: misaligned pointer");
  int st = check_device();
  if (st != SAGE_OK) return st;
  return hip_status(sage::launch_cost(prompt_len, Q, bin_repr, B, cost, (hipStream_t)stream), "cost launch");
}

SAGE_API int sage_index(const float* mass, const float* cost, const int32_t* prompt_len,
                        const double* bin_repr, int Q, int B, float* index, int32_t* argmin_bin,
                        sage_stream_t stream) {
  if (Q < 0) return fail(SAGE_EINVAL, "Q=%d is negative", Q);
  if (B < 1 || B > SAGE_MAX_BINS) return fail(SAGE_EINVAL, "B=%d outside [1, %d]", B, SAGE_MAX_BINS);
  if (Q == 0) return ok();
  if (!mass || !index) return fail(SAGE_EINVAL, "sage_index: mass or index is NULL");
  if (!cost && (!prompt_len || !bin_repr))
    return fail(SAGE_EINVAL, "sage_index: cost is NULL, so prompt_len and bin_repr are required");
  const void* ptrs[] = {mass, cost, prompt_len, bin_repr, index, argmin_bin};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return fail(SAGE_EINVAL, "sage_index: misaligned pointer");
  int st = check_device();
  if (st != SAGE_OK) return st;
  return hip_status(sage::launch_index(mass, cost, prompt_len, bin_repr, nullptr, 1, Q, B, index, argmin_bin,
                                       (hipStream_t)stream),
                    "index launch");
}

SAGE_API int sage_index_variant(const float* mass, const int32_t* prompt_len, const double* bin_repr, int Q,
                                int B, int cost_model, int index_kind, float noise_weight, float* index,
                                int32_t* argmin_bin, sage_stream_t stream) {
  if (Q < 0) return fail(SAGE_EINVAL, "Q=%d is negative", Q);
  if (B < 1 || B > SAGE_MAX_BINS) return fail(SAGE_EINVAL, "B=%d outside [1, %d]", B, SAGE_MAX_BINS);
  if (cost_model < SAGE_COST_RESOURCE || cost_model > SAGE_COST_OVERALL)
    return fail(SAGE_EINVAL, "cost_model=%d is not a SAGE_COST_* value", cost_model);
  if (index_kind != SAGE_INDEX_GITTINS && index_kind != SAGE_INDEX_MEAN)
    return fail(SAGE_EINVAL, "index_kind=%d is not a SAGE_INDEX_* value", index_kind);
  if (!(noise_weight >= 0.0f && noise_weight < 1.0f))
    return fail(SAGE_EINVAL, "noise_weight=%g outside [0, 1)", (double)noise_weight);
  if (Q == 0) return ok();
  if (!mass || !prompt_len || !bin_repr || !index)
    return fail(SAGE_EINVAL, "sage_index_variant: NULL required pointer");
  const void* ptrs[] = {mass, prompt_len, bin_repr, index, argmin_bin};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return fail(SAGE_EINVAL, "sage_index_variant: misaligned pointer");
  int st = check_device();
  if (st != SAGE_OK) return st;
  sage::IndexVariant v;
  v.cost_model = cost_model;
  v.kind = index_kind;
  v.noise = noise_weight;
  return hip_status(sage::launch_index(mass, nullptr, prompt_len, bin_repr, nullptr, 1, Q, B, index,
                                       argmin_bin, (hipStream_t)stream, &v),
                    "index launch");
}

SAGE_API int sage_mix_uniform(const float* mass, int Q, int B, float weight, float* out,
                              sage_stream_t stream) {
  if (Q < 0) return fail(SAGE_EINVAL, "Q=%d is negative", Q);
  if (B < 1 || B > SAGE_MAX_BINS) return fail(SAGE_EINVAL, "B=%d outside [1, %d]", B, SAGE_MAX_BINS);
  if (!(weight >= 0.0f && weight <= 1.0f))
    return fail(SAGE_EINVAL, "weight=%g outside [0, 1]", (double)weight);
  if (Q == 0) return ok();
  if (!mass || !out) return fail(SAGE_EINVAL, "sage_mix_uniform: NULL pointer");
  if (!aligned16(mass) || !aligned16(out)) return fail(SAGE_EINVAL, "sage_mix_uniform: misaligned pointer");
  const char* a = reinterpret_cast<const char*>(mass);
  const char* o = reinterpret_cast<const char*>(out);
  const size_t bytes = (size_t)Q * (size_t)B * sizeof(float);
  if (a != o && a < o + bytes && o < a + bytes)
    return fail(SAGE_EINVAL, "sage_mix_uniform: out overlaps mass without being the same buffer");
  int st = check_device();
  if (st != SAGE_OK) return st;
  return hip_status(sage::launch_mix_uniform(mass, Q, B, weight, out, (hipStream_t)stream), "mix launch");
}

SAGE_API int sage_index_attained(const float* mass, const int32_t* prompt_len, const double* bin_repr,
                                 const int32_t* generated, int bucket, int Q, int B, float* index,
                                 int32_t* argmin_bin, sage_stream_t stream) {
  if (Q < 0) return fail(SAGE_EINVAL, "Q=%d is negative", Q);
  if (B < 1 || B > SAGE_MAX_BINS) return fail(SAGE_EINVAL, "B=%d outside [1, %d]", B, SAGE_MAX_BINS);
  if (bucket < 1) return fail(SAGE_EINVAL, "bucket=%d must be >= 1", bucket);
  if (Q == 0) return ok();
  if (!mass || !prompt_len || !bin_repr || !generated || !index)
    return fail(SAGE_EINVAL, "sage_index_attained: NULL required pointer");
  const void* ptrs[] = {mass, prompt_len, bin_repr, generated, index, argmin_bin};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return fail(SAGE_EINVAL, "sage_index_attained: misaligned pointer");
  int st = check_device();
  if (st != SAGE_OK) return st;
  return hip_status(sage::launch_index(mass, nullptr, prompt_len, bin_repr, generated, bucket, Q, B, index,
                                       argmin_bin, (hipStream_t)stream),
                    "index launch");
}

SAGE_API int sage_index_attained_table(const float* mass, const int32_t* prompt_len, const double* bin_repr,
                                       int bucket, int levels, int Q, int B, float* index, sage_stream_t stream) {
  if (Q < 0) return fail(SAGE_EINVAL, "Q=%d is negative", Q);
  if (B < 1 || B > SAGE_MAX_BINS) return fail(SAGE_EINVAL, "B=%d outside [1, %d]", B, SAGE_MAX_BINS);
  if (bucket < 1) return fail(SAGE_EINVAL, "bucket=%d must be >= 1", bucket);
  if (levels < 1) return fail(SAGE_EINVAL, "levels=%d must be >= 1", levels);
  if ((double)levels * (double)bucket > 2147483647.0)
    return fail(SAGE_EINVAL, "levels * bucket = %.0f exceeds the int32 token range", (double)levels * bucket);
  if (Q == 0) return ok();
  if (!mass || !prompt_len || !bin_repr || !index)
    return fail(SAGE_EINVAL, "sage_index_attained_table: NULL required pointer");
  const void* ptrs[] = {mass, prompt_len, bin_repr, index};
  for (const void* p : ptrs)
    if (!aligned16(p)) return fail(SAGE_EINVAL, "sage_index_attained_table: misaligned pointer");
  int st = check_device();
  if (st != SAGE_OK) return st;
  sage::IndexVariant table;
  table.levels = levels;
  return hip_status(sage::launch_index(mass, nullptr, prompt_len, bin_repr, nullptr, bucket, Q, B, index, nullptr,
                                       (hipStream_t)stream, &table),
                    "index table launch");
}

// --------------------------------------------------------- input check
SAGE_API int sage_check_inputs(const double* bin_edges, const double* bin_repr, int B, const int32_t* prompt_len,
                               int Q, int32_t* status, sage_stream_t stream) {
  if (B < 1 || B > SAGE_MAX_BINS) return fail(SAGE_EINVAL, "B=%d outside [1, %d]", B, SAGE_MAX_BINS);
  if (Q < 0) return fail(SAGE_EINVAL, "Q=%d is negative", Q);
  if (!status) return fail(SAGE_EINVAL, "sage_check_inputs: status is NULL");
  const void* ptrs[] = {bin_edges, bin_repr, prompt_len, status};
  for (const void* p : ptrs)
    if (p && !aligned16(p)) return fail(SAGE_EINVAL, "sage_check_inputs: misaligned pointer");
  int st = check_device();
  if (st != SAGE_OK) return st;
  return hip_status(sage::launch_check_inputs(bin_edges, B + 1, bin_repr, B, prompt_len, Q, status,
                                              (hipStream_t)stream),
                    "check_inputs launch");
}

// ---------------------------------------------------------- test hook
namespace {
std::atomic<uint32_t> g_theta_floor_bits{0xff800000u};   // -inf: off
}  // namespace

namespace sage {
float debug_theta_floor() {
  const uint32_t b = g_theta_floor_bits.load(std::memory_order_relaxed);
  float f;
  std::memcpy(&f, &b, sizeof f);
  return f;
}
}  // namespace sage

SAGE_API int sage_debug_theta_floor(float floor) {
  if (std::isnan(floor)) return fail(SAGE_EINVAL, "sage_debug_theta_floor: NaN");
  uint32_t b;
  std::memcpy(&b, &floor, sizeof b);
  g_theta_floor_bits.store(b, std::memory_order_relaxed);
  return ok();
}

// ----------------------------------------------------------------- rank
SAGE_API size_t sage_rank_workspace_bytes(int Q) { return Q > 0 ? sage::rank_workspace_bytes(Q) : 0; }

SAGE_API int sage_rank(const float* index, int Q, int32_t* order, void* workspace,
                       size_t workspace_bytes, sage_stream_t stream) {
  if (Q < 0) return fail(SAGE_EINVAL, "Q=%d is negative", Q);
  if (Q == 0) return ok();
  if (!index || !order) return fail(SAGE_EINVAL, "sage_rank: NULL pointer");
  if (!aligned16(index) || !aligned16(order)) return fail(SAGE_EINVAL, "sage_rank: misaligned pointer");
  const size_t need = sage::rank_workspace_bytes(Q);
  if (!workspace || workspace_bytes < need)
    return fail(SAGE_EWORKSPACE, "sage_rank: workspace of %zu bytes, %zu needed", workspace_bytes, need);
  if (!aligned16(workspace)) return fail(SAGE_EINVAL, "sage_rank: workspace is not 16-byte aligned");
  int st = check_device();
  if (st != SAGE_OK) return st;
  return hip_status(sage::launch_rank(index, Q, order, workspace, (hipStream_t)stream), "rank launch");
}

// ------------------------------------------------------------ simulate
SAGE_API int sage_simulate(const double* arrival, const int32_t* prompt_len, const int32_t* output_len,
                           int R, const int32_t* order, int levels, int informed, int bucket,
                           int servers, double rate, int queue_cap, double* finish,
                           int32_t* preemptions) {
  if (R < 0) return fail(SAGE_EINVAL, "R=%d is negative", R);
  if (levels < 1) return fail(SAGE_EINVAL, "levels=%d must be >= 1", levels);
  if ((long long)levels * R > 0x7fffffffLL)
    return fail(SAGE_EINVAL, "levels * R = %lld exceeds 2^31 - 1", (long long)levels * R);
  if (informed < 0 || (long long)informed > (long long)levels * R)
    return fail(SAGE_EINVAL, "informed=%d outside [0, levels * R]", informed);
  if (bucket < 0) return fail(SAGE_EINVAL, "bucket=%d is negative", bucket);
  if (bucket == 0 && levels != 1) return fail(SAGE_EINVAL, "levels=%d without refreshing (bucket 0)", levels);
  if (servers < 1) return fail(SAGE_EINVAL, "servers=%d must be >= 1", servers);
  if (!(rate > 0.0) || !std::isfinite(rate)) return fail(SAGE_EINVAL, "rate=%g must be positive and finite", rate);
  if (queue_cap < 0) return fail(SAGE_EINVAL, "queue_cap=%d is negative", queue_cap);
  if (R == 0) return ok();
  if (!arrival || !prompt_len || !output_len || !order || !finish)
    return fail(SAGE_EINVAL, "sage_simulate: NULL pointer");
  for (int r = 0; r < R; ++r) {
    if (!std::isfinite(arrival[r])) return fail(SAGE_EINVAL, "arrival[%d] is not finite", r);
    if (r > 0 && arrival[r] < arrival[r - 1]) return fail(SAGE_EINVAL, "arrivals decrease at %d", r);
    if (prompt_len[r] < 0) return fail(SAGE_EINVAL, "prompt_len[%d]=%d is negative", r, prompt_len[r]);
    if (output_len[r] < 1) return fail(SAGE_EINVAL, "output_len[%d]=%d must be >= 1", r, output_len[r]);
    if (bucket > 0 && (output_len[r] - 1) / bucket >= levels)
      return fail(SAGE_EINVAL, "request %d (O=%d) needs %d levels, %d given", r, output_len[r],
                  (output_len[r] - 1) / bucket + 1, levels);
  }
  const size_t n = (size_t)levels * R;
  std::vector<unsigned char> seen(n, 0);
  for (size_t i = 0; i < n; ++i) {
    const int32_t e = order[i];
    if (e < 0 || (size_t)e >= n || seen[e]) return fail(SAGE_EINVAL, "order is not a permutation (at %zu)", i);
    seen[e] = 1;
  }
  if (sage::simulate_queue(arrival, prompt_len, output_len, R, order, levels, informed, bucket, servers,
                           rate, queue_cap, finish, preemptions) != 0)
    return fail(SAGE_EINVAL, "sage_simulate: event loop stalled");
  return ok();
}
