// Adapter drift: squared distances between the current adapter and stored
// versions, chunked over all (version, layer, target, factor) segments, then
// reduced in a fixed order (deterministic).  Accumulation in fp64.
#include <math.h>

#include <mutex>

#include "../../include/crf.h"
#include "kernels.hpp"

// Fixed device scratch of crf_layer_drift_noalloc (tables and partials), one
// copy per device, held until the process ends.  Host code never passes this
// name to a kernel: the device address comes from hipGetSymbolAddress.
static __device__ __align__(256) char scratch[CRF_DRIFT_NOALLOC_MAX_BYTES];

namespace crf {
namespace {

template <typename T>
CRF_DEV double tod(T x);
template <>
CRF_DEV double tod<float>(float x) { return (double)x; }
template <>
CRF_DEV double tod<bf16>(bf16 x) { return (double)bf2f(x); }

template <typename T>
__global__ __launch_bounds__(256) void drift_partials_kernel(const DriftSeg *__restrict__ segs,
                                                             const DriftChunk *__restrict__ chunks,
                                                             double *__restrict__ partials) {
  __shared__ double red[256];
  const DriftChunk ch = chunks[blockIdx.x];
  const DriftSeg sg = segs[ch.seg];
  const T *a = (const T *)sg.a + ch.start;
  const T *b = (const T *)sg.b + ch.start;
  double acc = 0.0;
  for (int64_t i = threadIdx.x; i < ch.len; i += 256) {
    const double d = tod<T>(a[i]) - tod<T>(b[i]);
    acc = fma(d, d, acc);
  }
  red[threadIdx.x] = acc;
  __syncthreads();
  for (int o = 128; o > 0; o >>= 1) {
    if ((int)threadIdx.x < o) red[threadIdx.x] += red[threadIdx.x + o];
    __syncthreads();
  }
  if (threadIdx.x == 0) partials[blockIdx.x] = red[0];
}

// Single workgroup: sq[o] = sum of its chunks (in order); then per layer l
// d_l = sqrt(sum_l' sq[anchor(l), l'])  (or sqrt(sq[anchor(l), l]) per layer).
__global__ __launch_bounds__(256) void drift_finalize_kernel(const double *__restrict__ partials,
                                                             const int *__restrict__ chunk_first,
                                                             const int *__restrict__ chunk_count, int n_versions,
                                                             int n_layers, const int *__restrict__ anchor,
                                                             const float *__restrict__ sens, int per_layer_only,
                                                             float *drift, float *risk, float *sq_out,
                                                             double *scratch) {
  const int n_out = n_versions * n_layers;
  for (int o = threadIdx.x; o < n_out; o += 256) {
    double s = 0.0;
    for (int c = 0; c < chunk_count[o]; ++c) s += partials[chunk_first[o] + c];
    scratch[o] = s;
    if (sq_out) sq_out[o] = (float)s;
  }
  __syncthreads();
  for (int l = threadIdx.x; l < n_layers; l += 256) {
    const int v = anchor[l];
    double s;
    if (per_layer_only) {
      s = scratch[v * n_layers + l];
    } else {
      s = 0.0;
      for (int k = 0; k < n_layers; ++k) s += scratch[v * n_layers + k];
    }
    const double d = sqrt(s);
    drift[l] = (float)d;
    risk[l] = (float)(d * (sens ? (double)sens[l] : 1.0));
  }
}

constexpr int MAX_DEVICES = 64;
void *g_scratch[MAX_DEVICES];
std::once_flag g_scratch_once[MAX_DEVICES];
hipError_t g_scratch_err[MAX_DEVICES];

}  // namespace

hipError_t drift_noalloc_scratch(void **out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= MAX_DEVICES) return hipErrorInvalidDevice;
  // once per device, with that device current (it is: hipGetDevice above)
  std::call_once(g_scratch_once[dev], [dev] {
    void *p = nullptr;
    g_scratch_err[dev] = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
    g_scratch[dev] = g_scratch_err[dev] == hipSuccess ? p : nullptr;
  });
  *out = g_scratch[dev];
  return g_scratch_err[dev];
}

hipError_t launch_drift_partials(hipStream_t s, const DriftSeg *segs, const DriftChunk *chunks, int n_chunks,
                                 bool f32, double *partials) {
  if (n_chunks <= 0) return hipSuccess;
  if (f32)
    hipLaunchKernelGGL(drift_partials_kernel<float>, dim3(n_chunks), dim3(256), 0, s, segs, chunks, partials);
  else
    hipLaunchKernelGGL(drift_partials_kernel<bf16>, dim3(n_chunks), dim3(256), 0, s, segs, chunks, partials);
  return hipGetLastError();
}

hipError_t launch_drift_finalize(hipStream_t s, const double *partials, const int *chunk_first,
                                 const int *chunk_count, int n_versions, int n_layers, const int *anchor,
                                 const float *sens, int per_layer_only, float *drift, float *risk, float *sq_out,
                                 double *scratch) {
  hipLaunchKernelGGL(drift_finalize_kernel, dim3(1), dim3(256), 0, s, partials, chunk_first, chunk_count,
                     n_versions, n_layers, anchor, sens, per_layer_only, drift, risk, sq_out, scratch);
  return hipGetLastError();
}

}  // namespace crf
