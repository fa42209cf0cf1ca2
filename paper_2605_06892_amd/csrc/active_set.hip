// Active set A_i of one HSA iteration: an ordered compaction of the token
// indices whose step budget puts them on this iteration's schedule.
//
// Rule (Section 2.2): token n with budget s_n (a divisor of T, Eq. 5) is active
// at iteration i iff i mod (T / s_n) == 0. Phase-aware window (Section 2.5):
// with margin m > 0 the iterations i < m and i > T - m - 1 are outside the
// window, where every token is active -- at every such iteration (the
// paper's wording, outside period 1), or only where i mod p == 0 for an
// outside period p (p = T / s_max: every token follows the largest budget's
// schedule there, the reading under which the HSA-25 preset of Appendix C
// meets its printed runtime).
//
// The budget array is small (4 bytes per token: 131 KB at N = 32760), so one
// workgroup of 1024 threads walks it in chunks of 16384 tokens: each thread
// classifies 16 consecutive tokens, a wave prefix sum plus a 16-entry LDS scan
// gives each thread its output offset, and the thread writes its active token
// indices in order. The result is ascending by construction. Budget validity
// and activity per budget value come from a per-launch LDS table (T <= 1024),
// so the hot loop has no integer division.
#include "common.h"

namespace hsa {
namespace {

constexpr int kThreads = 1024;
constexpr int kPer = 16;
constexpr int kChunk = kThreads * kPer;
constexpr int kMaxTableT = 1024;

// 0: invalid budget, 1: valid and skipped, 2: valid and active.
__device__ __forceinline__ int classify(int s, int T, int iter, bool outside, bool outside_active) {
  if (s < 1 || s > T || (T % s) != 0) return 0;
  if (outside) return outside_active ? 2 : 1;
  return (iter % (T / s)) == 0 ? 2 : 1;
}

__global__ __launch_bounds__(kThreads) void active_set_kernel(const int32_t* __restrict__ budget,
                                                              int n, int T, int iter, int margin,
                                                              int outside_period,
                                                              int32_t* __restrict__ idx,
                                                              int32_t* __restrict__ n_active) {
  __shared__ int wave_total[kThreads / kWave];
  __shared__ unsigned char table[kMaxTableT + 1];
  __shared__ int bad_any;

  const int t = threadIdx.x;
  const int lane = t & (kWave - 1);
  const int w = t / kWave;
  const bool outside = margin > 0 && (iter < margin || iter > T - margin - 1);
  const bool outside_active = outside && (iter % outside_period) == 0;
  const bool use_table = T <= kMaxTableT;
  if (t == 0) bad_any = 0;
  if (use_table) {
    for (int s = t; s <= T; s += kThreads)
      table[s] = (unsigned char)classify(s, T, iter, outside, outside_active);
  }
  __syncthreads();

  const bool aligned = (reinterpret_cast<uintptr_t>(budget) & 15) == 0;
  int base = 0;  // active tokens before the current chunk
  int bad = 0;
  for (int c0 = 0; c0 < n; c0 += kChunk) {
    const int e0 = c0 + t * kPer;
    int b[kPer];
    if (aligned && e0 + kPer <= n) {
      const int4* p = reinterpret_cast<const int4*>(budget + e0);
#pragma unroll
      for (int r = 0; r < kPer / 4; ++r) {
        int4 v = p[r];
        b[4 * r + 0] = v.x;
        b[4 * r + 1] = v.y;
        b[4 * r + 2] = v.z;
        b[4 * r + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int r = 0; r < kPer; ++r) b[r] = (e0 + r < n) ? budget[e0 + r] : 0;
    }
    unsigned mask = 0;
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
      if (e0 + r < n) {
        const int s = b[r];
        int cls;
        if (use_table) cls = (s >= 1 && s <= T) ? table[s] : 0;
        else cls = classify(s, T, iter, outside, outside_active);
        bad |= (cls == 0);
        mask |= (cls == 2 ? 1u : 0u) << r;
      }
    }
    const int cnt = __popc(mask);
    int inc = cnt;  // inclusive prefix over the wave
#pragma unroll
    for (int o = 1; o < kWave; o <<= 1) {
      const int y = __shfl_up(inc, o);
      if (lane >= o) inc += y;
    }
    if (lane == kWave - 1) wave_total[w] = inc;
    __syncthreads();
    int before = 0, total = 0;
#pragma unroll
    for (int i = 0; i < kThreads / kWave; ++i) {
      const int v = wave_total[i];
      before += (i < w) ? v : 0;
      total += v;
    }
    int pos = base + before + inc - cnt;
    while (mask) {
      const int r = __builtin_ctz(mask);
      idx[pos++] = e0 + r;
      mask &= mask - 1;
    }
    base += total;
    __syncthreads();  // wave_total is rewritten by the next chunk
  }
  if (bad) atomicOr(&bad_any, 1);
  __syncthreads();
  if (t == 0) n_active[0] = bad_any ? -1 : base;
}

}  // namespace

hipError_t launch_active_set(const int32_t* budget, int n, int T, int iter, int margin,
                             int outside_period, int32_t* idx, int32_t* n_active, hipStream_t s) {
  hipLaunchKernelGGL(active_set_kernel, dim3(1), dim3(kThreads), 0, s, budget, n, T, iter, margin,
                     outside_period, idx, n_active);
  return hipGetLastError();
}

}  // namespace hsa
