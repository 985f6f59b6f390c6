// Elementwise kernels: bf16 ingest of the embeddings and the materialised
// cost support (the index scan computes the same cost inline).
#include "sage_device.hpp"
#include "sage_internal.hpp"

namespace sage {
namespace {

// fp32 -> bf16, round to nearest, ties to even: add half of the dropped
// 16-bit range plus the kept part's lowest bit, then truncate.
__device__ __forceinline__ uint16_t bf16_rne(float x) {
  uint32_t u = __float_as_uint(x);
  u += 0x7FFFu + ((u >> 16) & 1u);
  return (uint16_t)(u >> 16);
}

__global__ void __launch_bounds__(256) ingest_bf16_kernel(const float* __restrict__ src, size_t n,
                                                          uint16_t* __restrict__ dst) {
  const size_t n4 = n / 4;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  const float4* s4 = reinterpret_cast<const float4*>(src);
  ushort4* d4 = reinterpret_cast<ushort4*>(dst);
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride) {
    float4 v = s4[i];
    d4[i] = make_ushort4(bf16_rne(v.x), bf16_rne(v.y), bf16_rne(v.z), bf16_rne(v.w));
  }
  for (size_t i = n4 * 4 + (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < n; i += stride)
    dst[i] = bf16_rne(src[i]);
}

// [rows, d] fp32 -> panel-major bf16 [d / 32][rows][32] (RNE). Block row y
// walks panels y, y + gridDim.y, ...; a thread writes one 16-byte piece (8
// values) of a panel row and reads the matching 32 bytes of the source row,
// so four consecutive threads read one whole 128-byte line.
__global__ void __launch_bounds__(256) ingest_panels_kernel(const float* __restrict__ src, int rows, int d,
                                                            uint16_t* __restrict__ dst) {
  const int pieces = rows * 4;
  for (int p = blockIdx.y; p < d / 32; p += gridDim.y) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < pieces; i += gridDim.x * blockDim.x) {
      const float* s = src + (size_t)(i >> 2) * d + p * 32 + (i & 3) * 8;
      const float4 a = *reinterpret_cast<const float4*>(s);
      const float4 b = *reinterpret_cast<const float4*>(s + 4);
      ushort4* out = reinterpret_cast<ushort4*>(dst + ((size_t)p * pieces + i) * 8);
      out[0] = make_ushort4(bf16_rne(a.x), bf16_rne(a.y), bf16_rne(a.z), bf16_rne(a.w));
      out[1] = make_ushort4(bf16_rne(b.x), bf16_rne(b.y), bf16_rne(b.z), bf16_rne(b.w));
    }
  }
}

// The same rearrangement of bf16 bits already rounded.
__global__ void __launch_bounds__(256) panels_from_rows_kernel(const uint16_t* __restrict__ src, int rows,
                                                               int d, uint16_t* __restrict__ dst) {
  const int pieces = rows * 4;
  for (int p = blockIdx.y; p < d / 32; p += gridDim.y) {
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < pieces; i += gridDim.x * blockDim.x) {
      const uint4 v = *reinterpret_cast<const uint4*>(src + (size_t)(i >> 2) * d + p * 32 + (i & 3) * 8);
      *reinterpret_cast<uint4*>(dst + ((size_t)p * pieces + i) * 8) = v;
    }
  }
}

// FIFO insert into the history ring: record i of the batch (only the last
// `cap` of the batch survive) goes to slot (total + i) mod cap, embedding
// rounded to bf16 (RNE), length copied. One thread per 8 embedding values.
__global__ void __launch_bounds__(256) store_insert_kernel(const float* __restrict__ emb,
                                                           const int32_t* __restrict__ out_len, int n, int d,
                                                           int first, long long total, int cap,
                                                           uint16_t* __restrict__ ring_emb,
                                                           int32_t* __restrict__ ring_len) {
  const int per_row = d / 8;
  const size_t work = (size_t)(n - first) * per_row;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t w = (size_t)blockIdx.x * blockDim.x + threadIdx.x; w < work; w += stride) {
    const int i = first + (int)(w / per_row);
    const int c = (int)(w % per_row) * 8;
    const size_t slot = (size_t)((total + i) % cap);
    const float4 a = *reinterpret_cast<const float4*>(emb + (size_t)i * d + c);
    const float4 b = *reinterpret_cast<const float4*>(emb + (size_t)i * d + c + 4);
    ushort4* dst = reinterpret_cast<ushort4*>(ring_emb + slot * d + c);
    dst[0] = make_ushort4(bf16_rne(a.x), bf16_rne(a.y), bf16_rne(a.z), bf16_rne(a.w));
    dst[1] = make_ushort4(bf16_rne(b.x), bf16_rne(b.y), bf16_rne(b.z), bf16_rne(b.w));
    if (c == 0) ring_len[slot] = out_len[i];
  }
}

// A deliberately inaccurate prediction: each row merged with the uniform
// distribution, out = (1 - w) p / sum(p) + w / B in fp64, rounded to fp32; a
// row with no mass stays zero. One wavefront per row; the row sum is complete
// before any element is written, so out may alias mass.
__global__ void __launch_bounds__(256) mix_uniform_kernel(const float* mass, int Q, int B, float w,
                                                          float* out) {
  const int lane = (int)lane_id();
  const int n_waves = (int)(gridDim.x * (blockDim.x / kWave));
  for (int q = (int)(blockIdx.x * (blockDim.x / kWave) + threadIdx.x / kWave); q < Q; q += n_waves) {
    const size_t row = (size_t)q * (size_t)B;
    double sum = 0.0;
    for (int b = lane; b < B; b += kWave) sum += (double)mass[row + b];
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) sum += __shfl_xor(sum, off, kWave);
    const bool empty = !(sum > 0.0);
    const double keep = empty ? 0.0 : (1.0 - (double)w) / sum;
    const double spread = empty ? 0.0 : (double)w / (double)B;
    for (int b = lane; b < B; b += kWave) out[row + b] = (float)fma(keep, (double)mass[row + b], spread);
  }
}

// x[q, b] = r_b^2 / 2 + I_q * r_b in fp64, rounded once to fp32.
__global__ void __launch_bounds__(256) cost_kernel(const int32_t* __restrict__ prompt_len, int Q,
                                                   const double* __restrict__ repr, int B,
                                                   float* __restrict__ cost) {
  const size_t total = (size_t)Q * (size_t)B;
  const size_t stride = (size_t)gridDim.x * blockDim.x;
  for (size_t i = (size_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += stride) {
    const int q = (int)(i / (size_t)B);
    const int b = (int)(i - (size_t)q * B);
    const double r = repr[b];
    cost[i] = (float)fma((double)prompt_len[q], r, r * r * 0.5);
  }
}

int grid_for(size_t work, int block, int cap = 4096) {
  size_t g = (work + block - 1) / block;
  if (g < 1) g = 1;
  if (g > (size_t)cap) g = cap;
  return (int)g;
}

}  // namespace

// Preconditions of the binning and the index scan, checked on the device:
// edges strictly increasing and finite (the histogram's binary search), the
// representatives finite, non-negative and non-decreasing, and prompt
// lengths non-negative (together they make the cost support r (I + r / 2)
// non-decreasing along a row, which the index scan relies on). One
// workgroup; bit SAGE_CHECK_* of *status is set for each failed condition,
// 0 when all hold. Every thread reaches the barrier; thread 0 writes.
__global__ void __launch_bounds__(1024) check_inputs_kernel(const double* __restrict__ edges, int n_edges,
                                                            const double* __restrict__ repr, int B,
                                                            const int32_t* __restrict__ plen, int Q,
                                                            int32_t* __restrict__ status) {
  __shared__ int bad;
  if (threadIdx.x == 0) bad = 0;
  __syncthreads();
  int mine = 0;
  for (int i = threadIdx.x; edges && i < n_edges; i += blockDim.x) {
    const double e = edges[i];
    if (!__builtin_isfinite(e) || (i + 1 < n_edges && !(e < edges[i + 1]))) mine |= 1;
  }
  for (int i = threadIdx.x; repr && i < B; i += blockDim.x) {
    const double r = repr[i];
    if (!__builtin_isfinite(r) || (i == 0 && !(r >= 0.0)) || (i + 1 < B && !(r <= repr[i + 1]))) mine |= 2;
  }
  for (int i = threadIdx.x; plen && i < Q; i += blockDim.x)
    if (plen[i] < 0) mine |= 4;
  if (mine) atomicOr(&bad, mine);
  __syncthreads();
  if (threadIdx.x == 0) *status = bad;
}

hipError_t launch_ingest_bf16(const float* src, size_t n, uint16_t* dst, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  LaunchScope scope("ingest_bf16", stream);
  hipLaunchKernelGGL(ingest_bf16_kernel, dim3(grid_for(n / 4 + 1, 256, 8192)), dim3(256), 0, stream,
                     src, n, dst);
  return hipGetLastError();
}

namespace {
dim3 panels_grid(int rows, int d) {
  const int px = grid_for((size_t)rows * 4, 256, 4096);
  const int py = d / 32 < 65535 ? d / 32 : 65535;
  // about 8192 blocks in all
  int gx = px, gy = py;
  while ((long)gx * gy > 8192 && gx > 1) gx = (gx + 1) / 2;
  return dim3(gx, gy);
}
// Standing queue of the streaming scheduler (Sec. 3.3: the queue is
// re-ranked at every decision). Admit: new request i takes slot free[i]: its
// predicted masses, prompt length and arrival number. Slots outside
// [0, slots) are skipped.
__global__ void queue_admit_kernel(const int64_t* __restrict__ free_slots, const float* __restrict__ new_mass,
                                   const int32_t* __restrict__ new_plen, int B, long long next_request,
                                   int slots, float* __restrict__ mass, int32_t* __restrict__ plen,
                                   int64_t* __restrict__ request) {
  const int i = blockIdx.x;
  const long long s = free_slots[i];
  if (s < 0 || s >= slots) return;
  for (int b = threadIdx.x; b < B; b += blockDim.x) mass[s * B + b] = new_mass[(size_t)i * B + b];
  if (threadIdx.x == 0) {
    plen[s] = new_plen[i];
    request[s] = next_request + i;
  }
}
// Dispatch: the first `batch` slots of the order leave; their slots are
// freed for the next arrivals and their request numbers reported.
__global__ void queue_dispatch_kernel(const int32_t* __restrict__ order, int batch,
                                      const int64_t* __restrict__ request, int slots,
                                      int64_t* __restrict__ free_slots, int64_t* __restrict__ dispatched) {
  const int i = blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= batch) return;
  const int s = order[i];
  free_slots[i] = s;
  dispatched[i] = (s >= 0 && s < slots) ? request[s] : -1;
}

}  // namespace

hipError_t launch_ingest_panels(const float* src, int rows, int d, uint16_t* dst, hipStream_t stream) {
  if (rows == 0) return hipSuccess;
  LaunchScope scope("ingest_bf16", stream);
  hipLaunchKernelGGL(ingest_panels_kernel, panels_grid(rows, d), dim3(256), 0, stream, src, rows, d, dst);
  return hipGetLastError();
}

hipError_t launch_panels_from_rows(const uint16_t* src, int rows, int d, uint16_t* dst, hipStream_t stream) {
  if (rows == 0) return hipSuccess;
  LaunchScope scope("panels_from_rows", stream);
  hipLaunchKernelGGL(panels_from_rows_kernel, panels_grid(rows, d), dim3(256), 0, stream, src, rows, d, dst);
  return hipGetLastError();
}

hipError_t launch_store_insert(const float* emb, const int32_t* out_len, int n, int d, long long total,
                               int cap, uint16_t* ring_emb, int32_t* ring_len, hipStream_t stream) {
  const int first = n > cap ? n - cap : 0;     // earlier records of the batch would be evicted at once
  const size_t work = (size_t)(n - first) * (d / 8);
  if (work == 0) return hipSuccess;
  LaunchScope scope("store_insert", stream);
  hipLaunchKernelGGL(store_insert_kernel, dim3(grid_for(work, 256, 8192)), dim3(256), 0, stream, emb, out_len,
                     n, d, first, total, cap, ring_emb, ring_len);
  return hipGetLastError();
}

hipError_t launch_queue_admit(const int64_t* free_slots, int batch, const float* new_mass,
                              const int32_t* new_plen, int B, long long next_request, int slots, float* mass,
                              int32_t* plen, int64_t* request, hipStream_t stream) {
  if (batch == 0) return hipSuccess;
  LaunchScope scope("queue_admit", stream);
  hipLaunchKernelGGL(queue_admit_kernel, dim3(batch), dim3(256), 0, stream, free_slots, new_mass, new_plen, B,
                     next_request, slots, mass, plen, request);
  return hipGetLastError();
}

hipError_t launch_queue_dispatch(const int32_t* order, int batch, const int64_t* request, int slots,
                                 int64_t* free_slots, int64_t* dispatched, hipStream_t stream) {
  if (batch == 0) return hipSuccess;
  LaunchScope scope("queue_dispatch", stream);
  hipLaunchKernelGGL(queue_dispatch_kernel, dim3((batch + 255) / 256), dim3(256), 0, stream, order, batch,
                     request, slots, free_slots, dispatched);
  return hipGetLastError();
}

hipError_t launch_mix_uniform(const float* mass, int Q, int B, float weight, float* out,
                              hipStream_t stream) {
  if (Q == 0) return hipSuccess;
  LaunchScope scope("mix_uniform", stream);
  hipLaunchKernelGGL(mix_uniform_kernel, dim3(grid_for((size_t)Q, 4, 16384)), dim3(256), 0, stream, mass,
                     Q, B, weight, out);
  return hipGetLastError();
}

hipError_t launch_cost(const int32_t* prompt_len, int Q, const double* bin_repr, int B, float* cost,
                       hipStream_t stream) {
  if (Q == 0) return hipSuccess;
  LaunchScope scope("cost", stream);
  hipLaunchKernelGGL(cost_kernel, dim3(grid_for((size_t)Q * B, 256, 8192)), dim3(256), 0, stream,
                     prompt_len, Q, bin_repr, B, cost);
  return hipGetLastError();
}

hipError_t launch_check_inputs(const double* edges, int n_edges, const double* repr, int B, const int32_t* plen,
                               int Q, int32_t* status, hipStream_t stream) {
  hipLaunchKernelGGL(check_inputs_kernel, dim3(1), dim3(1024), 0, stream, edges, n_edges, repr, B, plen, Q, status);
  return hipGetLastError();
}

}  // namespace sage
