// fp32 active-query attention (Section 2.3, step 3) for fp32 workloads: each
// active query attends to all N cached key/value rows of its head.
//
// One wave per (active row, head). Keys are taken 64 at a time, one per lane:
// the lane forms its score against the query (held in LDS), the wave reduces
// the running maximum and sum with shuffles (online softmax), and each lane
// accumulates head_dim/64 output channels by walking the 64 probabilities of
// the chunk. exp is the accurate libm expf.
#include "common.h"

namespace hsa {
namespace {

constexpr int kThreads = 256;
constexpr int kWavesPerBlock = kThreads / kWave;

template <int DH>
__global__ __launch_bounds__(kThreads) void attention_f32_kernel(
    const float* __restrict__ q, const float* __restrict__ k, const float* __restrict__ v,
    float* __restrict__ o, int n_q, int n_kv, int heads, int d, float scale,
    const float* __restrict__ k2, const float* __restrict__ v2, int n_split) {
  constexpr int R = DH / kWave;  // output channels per lane
  __shared__ float qs[kWavesPerBlock][DH];
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  const long pair = (long)blockIdx.x * kWavesPerBlock + w;
  const bool valid = pair < (long)n_q * heads;
  const int j = valid ? (int)(pair / heads) : 0;
  const int h = valid ? (int)(pair % heads) : 0;
  const long col0 = (long)h * DH;
  for (int c = lane; c < DH; c += kWave) qs[w][c] = valid ? q[(long)j * d + col0 + c] : 0.f;
  __syncthreads();
  if (!valid) return;

  float m_run = -INFINITY, l_run = 0.f;
  float acc[R];
#pragma unroll
  for (int r = 0; r < R; ++r) acc[r] = 0.f;

  for (int n0 = 0; n0 < n_kv; n0 += kWave) {
    const int n = n0 + lane;
    float s = -INFINITY;
    if (n < n_kv) {
      const float* kr = (n < n_split ? k + (long)n * d : k2 + (long)(n - n_split) * d) + col0;
      float dot = 0.f;
#pragma unroll 8
      for (int c = 0; c < DH; ++c) dot = fmaf(qs[w][c], kr[c], dot);
      s = dot * scale;
    }
    const float m_new = fmaxf(m_run, wave_max(s));
    const float alpha = expf(m_run - m_new);  // 0 on the first chunk
    const float p = (n < n_kv) ? expf(s - m_new) : 0.f;
    l_run = l_run * alpha + wave_sum(p);
#pragma unroll
    for (int r = 0; r < R; ++r) acc[r] *= alpha;
    const int cnt = min(kWave, n_kv - n0);
    for (int i = 0; i < cnt; ++i) {
      const float pi = __shfl(p, i);
      const int nv = n0 + i;
      const float* vr = (nv < n_split ? v + (long)nv * d : v2 + (long)(nv - n_split) * d) + col0;
#pragma unroll
      for (int r = 0; r < R; ++r) acc[r] = fmaf(pi, vr[lane + kWave * r], acc[r]);
    }
    m_run = m_new;
  }
  const float inv = 1.f / l_run;
#pragma unroll
  for (int r = 0; r < R; ++r) o[(long)j * d + col0 + lane + kWave * r] = acc[r] * inv;
}

}  // namespace

hipError_t launch_attention_f32(const void* q, const void* k, const void* v, void* o, int n_q,
                                int n_kv, int heads, int head_dim, float scale, hipStream_t s,
                                const void* k2, const void* v2, int n_split) {
  if (!k2 || !v2) n_split = n_kv;
  if (n_q <= 0) return hipSuccess;
  const long pairs = (long)n_q * heads;
  const dim3 grid((unsigned)((pairs + kWavesPerBlock - 1) / kWavesPerBlock));
  const int d = heads * head_dim;
  const float* qf = static_cast<const float*>(q);
  const float* kf = static_cast<const float*>(k);
  const float* vf = static_cast<const float*>(v);
  float* of = static_cast<float*>(o);
  const float* k2f = static_cast<const float*>(k2);
  const float* v2f = static_cast<const float*>(v2);
  if (head_dim == 64)
    hipLaunchKernelGGL(attention_f32_kernel<64>, grid, dim3(kThreads), 0, s, qf, kf, vf, of, n_q,
                       n_kv, heads, d, scale, k2f, v2f, n_split);
  else
    hipLaunchKernelGGL(attention_f32_kernel<128>, grid, dim3(kThreads), 0, s, qf, kf, vf, of, n_q,
                       n_kv, heads, d, scale, k2f, v2f, n_split);
  return hipGetLastError();
}

}  // namespace hsa
