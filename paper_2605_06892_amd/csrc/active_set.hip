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
// The budget array is small (4 bytes per token: 131 KB at N = 32760), so the
// work is latency-bound. Up to 16 workgroups of 1024 threads each take one
// contiguous range of the tokens. A workgroup first counts the active tokens
// of all ranges before its own (every workgroup reads that prefix itself:
// there is no scratch memory to pass counts between workgroups, and the
// prefix reads hit the L2), then walks its range in chunks of 16384 tokens:
// each thread classifies 16 consecutive tokens, a wave prefix sum plus a
// 16-entry LDS scan gives each thread its output offset, and the thread
// writes its active token indices in order. The result is ascending by
// construction. Budget validity and activity per budget value come from a
// per-launch LDS table (T <= 1024), so the hot loop has no integer division.
// The last workgroup has seen every token (its prefix and its own range), so
// it alone writes |A_i|, or -1 if any budget is invalid. All of a thread's
// first global loads are issued before the LDS table is built and before any
// of them is used, so the launch pays about one memory latency.
#include "common.h"

#include <algorithm>

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

// Sum of v over the workgroup (every thread gets it). Uses red[], which the
// caller must not be using; ends with a barrier.
__device__ __forceinline__ int block_sum(int v, int* red) {
  const int lane = threadIdx.x & (kWave - 1), w = threadIdx.x / kWave;
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  if (lane == 0) red[w] = v;
  __syncthreads();
  int total = 0;
#pragma unroll
  for (int i = 0; i < kThreads / kWave; ++i) total += red[i];
  __syncthreads();
  return total;
}

// Workgroup b takes tokens [b * range, min(n, (b + 1) * range)); range is a
// multiple of 4. Every global load a thread makes for the prefix count (up to
// kPrefix int4 per thread per round) and for its first chunk is issued before
// the LDS table is built, so their latencies overlap.
constexpr int kPrefix = 8;  // prefix loads per thread per round: 32768 tokens per round

__device__ __forceinline__ int4 load4(const int32_t* __restrict__ p, bool aligned) {
  if (aligned) return *reinterpret_cast<const int4*>(p);
  return make_int4(p[0], p[1], p[2], p[3]);
}

__global__ __launch_bounds__(kThreads) void active_set_kernel(const int32_t* __restrict__ budget,
                                                              int n, int range, int T, int iter,
                                                              int margin, int outside_period,
                                                              int32_t* __restrict__ idx,
                                                              int32_t* __restrict__ n_active) {
  __shared__ int wave_total[kThreads / kWave];
  __shared__ unsigned char table[kMaxTableT + 1];

  const int t = threadIdx.x;
  const int lane = t & (kWave - 1);
  const int w = t / kWave;
  const bool aligned = (reinterpret_cast<uintptr_t>(budget) & 15) == 0;
  const int r0 = (int)min((long)blockIdx.x * range, (long)n);
  const int r1 = (int)min((long)r0 + range, (long)n);

  // loads first: the first round of the prefix and the first chunk of the range
  int4 pre[kPrefix];
#pragma unroll
  for (int q = 0; q < kPrefix; ++q) {
    const int e = (q * kThreads + t) * 4;
    pre[q] = e < r0 ? load4(budget + e, aligned) : make_int4(0, 0, 0, 0);
  }
  int b[kPer];
  {
    const int e0 = r0 + t * kPer;
    if (aligned && e0 + kPer <= r1) {
      const int4* p = reinterpret_cast<const int4*>(budget + e0);
#pragma unroll
      for (int r = 0; r < kPer / 4; ++r) {
        const int4 v = p[r];
        b[4 * r + 0] = v.x;
        b[4 * r + 1] = v.y;
        b[4 * r + 2] = v.z;
        b[4 * r + 3] = v.w;
      }
    } else {
#pragma unroll
      for (int r = 0; r < kPer; ++r) b[r] = (e0 + r < r1) ? budget[e0 + r] : 0;
    }
  }

  const bool outside = margin > 0 && (iter < margin || iter > T - margin - 1);
  const bool outside_active = outside && (iter % outside_period) == 0;
  const bool use_table = T <= kMaxTableT;
  if (use_table) {
    for (int s = t; s <= T; s += kThreads)
      table[s] = (unsigned char)classify(s, T, iter, outside, outside_active);
  }
  __syncthreads();
  auto cls_of = [&](int s) {
    if (use_table) return (s >= 1 && s <= T) ? (int)table[s] : 0;
    return classify(s, T, iter, outside, outside_active);
  };

  int bad = 0;
  // active tokens before this workgroup's range
  int before_me = 0;
  if (r0 > 0) {
    int cnt = 0;
    auto count4 = [&](int4 v) {
      const int c0 = cls_of(v.x), c1 = cls_of(v.y), c2 = cls_of(v.z), c3 = cls_of(v.w);
      bad |= (c0 == 0) | (c1 == 0) | (c2 == 0) | (c3 == 0);
      cnt += (c0 == 2) + (c1 == 2) + (c2 == 2) + (c3 == 2);
    };
#pragma unroll
    for (int q = 0; q < kPrefix; ++q)
      if ((q * kThreads + t) * 4 < r0) count4(pre[q]);
    // further rounds (prefixes beyond 32768 tokens)
    for (long e = (long)(kPrefix * kThreads + t) * 4; e < r0; e += kThreads * 4)
      count4(load4(budget + e, aligned));
    before_me = block_sum(cnt, wave_total);
  }

  int base = before_me;  // active tokens before the current chunk
  for (long c0 = r0; c0 < r1; c0 += kChunk) {
    const long e0 = c0 + t * kPer;
    if (c0 != r0) {  // the first chunk was loaded above
      if (aligned && e0 + kPer <= r1) {
        const int4* p = reinterpret_cast<const int4*>(budget + e0);
#pragma unroll
        for (int r = 0; r < kPer / 4; ++r) {
          const int4 v = p[r];
          b[4 * r + 0] = v.x;
          b[4 * r + 1] = v.y;
          b[4 * r + 2] = v.z;
          b[4 * r + 3] = v.w;
        }
      } else {
#pragma unroll
        for (int r = 0; r < kPer; ++r) b[r] = (e0 + r < r1) ? budget[e0 + r] : 0;
      }
    }
    unsigned mask = 0;
#pragma unroll
    for (int r = 0; r < kPer; ++r) {
      if (e0 + r < r1) {
        const int cls = cls_of(b[r]);
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
      idx[pos++] = (int32_t)(e0 + r);
      mask &= mask - 1;
    }
    base += total;
    __syncthreads();  // wave_total is rewritten by the next chunk
  }
  if (blockIdx.x == gridDim.x - 1) {  // this workgroup has seen every token
    const int any_bad = block_sum(bad, wave_total);
    if (t == 0) n_active[0] = any_bad ? -1 : base;
  }
}

}  // namespace

hipError_t launch_active_set(const int32_t* budget, int n, int T, int iter, int margin,
                             int outside_period, int32_t* idx, int32_t* n_active, hipStream_t s) {
  // up to 16 ranges of at least 4096 tokens (a multiple of 4 each)
  constexpr int kMaxGroups = 16, kMinRange = 4096;
  int groups = (int)std::min<long>(kMaxGroups, std::max<long>(1, ((long)n + kMinRange - 1) / kMinRange));
  int range = (int)((((long)n + groups - 1) / groups + 3) / 4 * 4);
  if (range < 4) range = 4;
  groups = (int)std::max<long>(1, ((long)n + range - 1) / range);
  hipLaunchKernelGGL(active_set_kernel, dim3(groups), dim3(kThreads), 0, s, budget, n, range, T, iter,
                     margin, outside_period, idx, n_active);
  return hipGetLastError();
}

}  // namespace hsa
