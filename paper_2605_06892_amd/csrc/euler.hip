// Cached Euler update (Section 2.4, Eq. 6): every token advances by the shared
// step dsig = sigma_{i+1} - sigma_i with the last velocity it produced.
//
// Two streaming kernels on one stream:
//   1. (only when fresh velocities are given) scatter: v_cache[idx[j]] = v_fresh[j]
//   2. x = fmaf(v_cache, dsig, x) over all n_tokens * channels values.
// Both are HBM-bound element streams: 16-byte vector accesses when the rows
// allow it, grid sized to a few workgroups per CU and grid-stride loops.
#include "common.h"

namespace hsa {
namespace {

constexpr int kThreads = 256;

__global__ __launch_bounds__(kThreads) void scatter_rows_f32x4(float* __restrict__ v_cache,
                                                               const float* __restrict__ v_fresh,
                                                               const int32_t* __restrict__ idx,
                                                               int n_active, long n_tokens,
                                                               int vec_per_row) {
  const long total = (long)n_active * vec_per_row;
  for (long e = blockIdx.x * (long)kThreads + threadIdx.x; e < total;
       e += (long)gridDim.x * kThreads) {
    const long j = e / vec_per_row;
    const int c = (int)(e - j * vec_per_row);
    const int t = idx[j];
    if (t < 0 || t >= n_tokens) continue;
    const float4 v = reinterpret_cast<const float4*>(v_fresh)[e];
    reinterpret_cast<float4*>(v_cache)[(long)t * vec_per_row + c] = v;
  }
}

__global__ __launch_bounds__(kThreads) void scatter_rows_f32(float* __restrict__ v_cache,
                                                             const float* __restrict__ v_fresh,
                                                             const int32_t* __restrict__ idx,
                                                             int n_active, long n_tokens,
                                                             int channels) {
  const long total = (long)n_active * channels;
  for (long e = blockIdx.x * (long)kThreads + threadIdx.x; e < total;
       e += (long)gridDim.x * kThreads) {
    const long j = e / channels;
    const int c = (int)(e - j * channels);
    const int t = idx[j];
    if (t < 0 || t >= n_tokens) continue;
    v_cache[(long)t * channels + c] = v_fresh[e];
  }
}

__global__ __launch_bounds__(kThreads) void euler_f32x4(float4* __restrict__ x,
                                                        const float4* __restrict__ v, long n4,
                                                        float dsig) {
  for (long e = blockIdx.x * (long)kThreads + threadIdx.x; e < n4;
       e += (long)gridDim.x * kThreads) {
    float4 a = x[e];
    const float4 b = v[e];
    a.x = fmaf(b.x, dsig, a.x);
    a.y = fmaf(b.y, dsig, a.y);
    a.z = fmaf(b.z, dsig, a.z);
    a.w = fmaf(b.w, dsig, a.w);
    x[e] = a;
  }
}

__global__ __launch_bounds__(kThreads) void euler_f32(float* __restrict__ x,
                                                      const float* __restrict__ v, long n,
                                                      float dsig) {
  for (long e = blockIdx.x * (long)kThreads + threadIdx.x; e < n;
       e += (long)gridDim.x * kThreads)
    x[e] = fmaf(v[e], dsig, x[e]);
}

int grid_for(long work_items) {
  // 256 CUs x 8 workgroups of 256 threads keeps every CU streaming.
  long g = (work_items + kThreads - 1) / kThreads;
  if (g > 2048) g = 2048;
  if (g < 1) g = 1;
  return (int)g;
}

}  // namespace

hipError_t launch_cached_euler(float* x, float* v_cache, const float* v_fresh,
                               const int32_t* idx, int n_active, long n_tokens, int channels,
                               float dsig, hipStream_t s) {
  const bool vec = (channels % 4) == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(v_cache) & 15) == 0 &&
                   (v_fresh == nullptr || (reinterpret_cast<uintptr_t>(v_fresh) & 15) == 0);
  if (v_fresh != nullptr && n_active > 0) {
    if (vec) {
      const int vpr = channels / 4;
      hipLaunchKernelGGL(scatter_rows_f32x4, dim3(grid_for((long)n_active * vpr)), dim3(kThreads),
                         0, s, v_cache, v_fresh, idx, n_active, n_tokens, vpr);
    } else {
      hipLaunchKernelGGL(scatter_rows_f32, dim3(grid_for((long)n_active * channels)),
                         dim3(kThreads), 0, s, v_cache, v_fresh, idx, n_active, n_tokens,
                         channels);
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  const long n = n_tokens * (long)channels;
  if (n == 0) return hipSuccess;
  if (vec) {
    hipLaunchKernelGGL(euler_f32x4, dim3(grid_for(n / 4)), dim3(kThreads), 0, s,
                       reinterpret_cast<float4*>(x), reinterpret_cast<const float4*>(v_cache),
                       n / 4, dsig);
  } else {
    hipLaunchKernelGGL(euler_f32, dim3(grid_for(n)), dim3(kThreads), 0, s, x, v_cache, n, dsig);
  }
  return hipGetLastError();
}

}  // namespace hsa
