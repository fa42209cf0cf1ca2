// Kernels of the multi-layer sampling loop that are not matrix products.
//
//   * gather_latent: the fp32 latent rows of the active tokens, converted to
//     the model dtype, as the compact input of the patch embedding (Section
//     2.3: only the active rows flow through the model).
//   * velocity_keys + rank_budgets: the group refresh. Group sizes are fixed
//     and membership follows a per-token velocity ranking (Section 2.2,
//     Appendix B): the key of a token is the squared L2 norm of its velocity,
//     a float64 sum of the exact squares in channel order, and its rank is
//     its position in ascending (key, token) order, keys compared as their
//     IEEE bit patterns (a total order on non-negative doubles; NaN keys are
//     made the canonical positive NaN, above every number). The n_1 lowest
//     ranks get budget s_1, the next n_2 get s_2, and so on.
//
//   * l1_rel_accumulate: strategy D (Appendix B, Eq. 7): per token, the sum
//     over the initial full-budget steps of |v_i - v_{i-1}|_1 / |v_i|_1, the
//     two L1 norms summed in float64 in channel order, one float64 division
//     per step; v_{i-1} is kept in a token-major copy.
//   * reorder_plan_kernel + permute_rows_kernel: token reordering (Section
//     2.5): non-baseline tokens first, then the baseline group, each part in
//     index order, and the row permutation that applies it to token-indexed
//     state (and inverts it at the end).
//   * row_rms_scale: 1 / sqrt(mean(h^2) + eps) of every compact hidden row, the
//     RMS normalization before each layer's Q/K/V projections and before the
//     velocity head. A per-row factor commutes with the projection, so the
//     normalized rows are never written: the GEMM epilogue scales its rows.
//
// All of them are small (N x C fp32 reads, N budgets, one read of the hidden
// state): one pass each, grid-stride loops; the ranking compares every pair of
// keys from LDS tiles, O(N^2) VALU work that runs once per refresh.
#include "common.h"

namespace hsa {
namespace {

constexpr int kThreads = 256;

int grid_for(long work) {
  long g = (work + kThreads - 1) / kThreads;
  if (g > 4096) g = 4096;
  if (g < 1) g = 1;
  return (int)g;
}

// Each thread keeps kGatherU independent 16-byte row loads in flight before
// its stores; the latent rows are streamed once (nontemporal loads).
constexpr int kGatherU = 4;

template <bool BF16>
__global__ __launch_bounds__(kThreads) void gather_latent_vec(const f32x4* __restrict__ x,
                                                              const int32_t* __restrict__ idx,
                                                              int n_active, long n_tokens, int vpr,
                                                              void* __restrict__ xa) {
  const long total = (long)n_active * vpr;
  for (long e0 = blockIdx.x * (long)(kThreads * kGatherU) + threadIdx.x; e0 < total;
       e0 += (long)gridDim.x * kThreads * kGatherU) {
    f32x4 v[kGatherU];
#pragma unroll
    for (int u = 0; u < kGatherU; ++u) {
      const long e = e0 + (long)u * kThreads;
      v[u] = (f32x4){0.f, 0.f, 0.f, 0.f};
      if (e < total) {
        const long j = e / vpr;
        const int c = (int)(e - j * vpr);
        const int t = idx[j];
        if (t >= 0 && t < n_tokens) v[u] = __builtin_nontemporal_load(x + (long)t * vpr + c);
      }
    }
#pragma unroll
    for (int u = 0; u < kGatherU; ++u) {
      const long e = e0 + (long)u * kThreads;
      if (e >= total) break;
      if constexpr (BF16)
        static_cast<bf16x4*>(xa)[e] = to_bf16x4(v[u]);
      else
        static_cast<f32x4*>(xa)[e] = v[u];
    }
  }
}

template <bool BF16>
__global__ __launch_bounds__(kThreads) void gather_latent_scalar(const float* __restrict__ x,
                                                                 const int32_t* __restrict__ idx,
                                                                 int n_active, long n_tokens,
                                                                 int channels,
                                                                 void* __restrict__ xa) {
  const long total = (long)n_active * channels;
  for (long e = blockIdx.x * (long)kThreads + threadIdx.x; e < total;
       e += (long)gridDim.x * kThreads) {
    const long j = e / channels;
    const int c = (int)(e - j * channels);
    const int t = idx[j];
    const float v = (t >= 0 && t < n_tokens) ? x[(long)t * channels + c] : 0.f;
    if constexpr (BF16)
      static_cast<bf16*>(xa)[e] = (bf16)v;
    else
      static_cast<float*>(xa)[e] = v;
  }
}

__device__ __forceinline__ double canonical_key(double acc) {
  return acc != acc ? __longlong_as_double(0x7FF8000000000000LL) : acc;
}

// bit pattern of a key, NaNs made the canonical positive NaN
__device__ __forceinline__ unsigned long long key_bits(unsigned long long k) {
  const unsigned long long e = 0x7FF0000000000000ull;
  return ((k & e) == e && (k & 0x000FFFFFFFFFFFFFull)) ? 0x7FF8000000000000ull : k;
}

__global__ __launch_bounds__(kThreads) void l1_rel_accumulate(const float* __restrict__ v,
                                                              float* __restrict__ v_prev, long n,
                                                              int channels, double* __restrict__ acc,
                                                              int first) {
  for (long t = blockIdx.x * (long)kThreads + threadIdx.x; t < n; t += (long)gridDim.x * kThreads) {
    const float* row = v + t * channels;
    float* prev = v_prev + t * channels;
    if (first) {
      acc[t] = 0.0;
    } else {
      double num = 0.0, den = 0.0;
      for (int c = 0; c < channels; ++c) {
        const double a = row[c], b = prev[c];
        num = num + fabs(a - b);
        den = den + fabs(a);
      }
      acc[t] = acc[t] + num / den;
    }
    for (int c = 0; c < channels; ++c) prev[c] = row[c];
  }
}

// one thread per token; channel order is the summation order
__global__ __launch_bounds__(kThreads) void velocity_keys_vec(const f32x4* __restrict__ v, long n,
                                                              int vpr, double* __restrict__ keys) {
  for (long t = blockIdx.x * (long)kThreads + threadIdx.x; t < n; t += (long)gridDim.x * kThreads) {
    const f32x4* row = v + t * vpr;
    double acc = 0.0;
    for (int c = 0; c < vpr; ++c) {
      const f32x4 e = row[c];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const double w = e[u];
        acc = acc + w * w;  // w * w is exact in float64
      }
    }
    keys[t] = canonical_key(acc);
  }
}

__global__ __launch_bounds__(kThreads) void velocity_keys_scalar(const float* __restrict__ v,
                                                                 long n, int channels,
                                                                 double* __restrict__ keys) {
  for (long t = blockIdx.x * (long)kThreads + threadIdx.x; t < n; t += (long)gridDim.x * kThreads) {
    const float* row = v + t * channels;
    double acc = 0.0;
    for (int c = 0; c < channels; ++c) {
      const double w = row[c];
      acc = acc + w * w;
    }
    keys[t] = canonical_key(acc);
  }
}

// 64 tokens per workgroup (one per lane); the four waves split each LDS tile
// of keys and their counts are summed at the end.
constexpr int kRankTokens = 64, kRankTile = 1024;

__global__ __launch_bounds__(kThreads) void rank_budgets(const unsigned long long* __restrict__ keys,
                                                         int n, GroupTable tab,
                                                         int32_t* __restrict__ budget) {
  __shared__ unsigned long long tile[kRankTile];
  __shared__ int partial[kThreads / kWave][kRankTokens];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int t = blockIdx.x * kRankTokens + lane;
  const unsigned long long kt = t < n ? key_bits(keys[t]) : 0ull;
  int count = 0;
  for (int m0 = 0; m0 < n; m0 += kRankTile) {
    const int cnt = min(kRankTile, n - m0);
    __syncthreads();  // the previous tile is no longer read
    for (int e = threadIdx.x; e < cnt; e += kThreads) tile[e] = key_bits(keys[m0 + e]);
    __syncthreads();
    const int lo = wave * (kRankTile / 4);
    const int hi = min(lo + kRankTile / 4, cnt);
#pragma unroll 8
    for (int e = lo; e < hi; ++e) {
      const unsigned long long km = tile[e];
      count += (km < kt) | ((km == kt) & (m0 + e < t));
    }
  }
  partial[wave][lane] = count;
  __syncthreads();
  if (wave == 0 && t < n) {
    int r = 0;
#pragma unroll
    for (int w = 0; w < kThreads / kWave; ++w) r += partial[w][lane];
    int g = 0;
    while (g + 1 < tab.n && r >= tab.end[g]) ++g;
    budget[t] = tab.budget[g];
  }
}

// Token reordering plan: one workgroup walks the budgets twice in chunks of
// 1024 x 16 tokens, a wave prefix sum per chunk giving each thread its output
// offsets; pass 0 places the non-baseline tokens (budget < T), pass 1 the
// baseline tokens (budget T) after all of them.
constexpr int kPlanThreads = 1024, kPlanPer = 16;

__global__ __launch_bounds__(kPlanThreads) void reorder_plan_kernel(const int32_t* __restrict__ budget,
                                                                    int n, int T,
                                                                    int32_t* __restrict__ perm,
                                                                    int32_t* __restrict__ n_lead) {
  __shared__ int wave_total[kPlanThreads / kWave];
  __shared__ int bad_any;
  const int t = threadIdx.x, lane = t & (kWave - 1), w = t / kWave;
  if (t == 0) bad_any = 0;
  __syncthreads();
  int bad = 0, base = 0, lead_total = 0;
  for (int pass = 0; pass < 2; ++pass) {
    base = pass == 0 ? 0 : lead_total;
    for (int c0 = 0; c0 < n; c0 += kPlanThreads * kPlanPer) {
      const int e0 = c0 + t * kPlanPer;
      unsigned mask = 0;
#pragma unroll
      for (int r = 0; r < kPlanPer; ++r) {
        if (e0 + r < n) {
          const int s = budget[e0 + r];
          const bool ok = s >= 1 && s <= T && T % s == 0;
          bad |= !ok;
          const bool pick = pass == 0 ? (ok && s < T) : (!ok || s == T);
          mask |= (pick ? 1u : 0u) << r;
        }
      }
      const int cnt = __popc(mask);
      int inc = cnt;
#pragma unroll
      for (int o = 1; o < kWave; o <<= 1) {
        const int y = __shfl_up(inc, o);
        if (lane >= o) inc += y;
      }
      if (lane == kWave - 1) wave_total[w] = inc;
      __syncthreads();
      int before = 0, total = 0;
#pragma unroll
      for (int i = 0; i < kPlanThreads / kWave; ++i) {
        const int v = wave_total[i];
        before += (i < w) ? v : 0;
        total += v;
      }
      int pos = base + before + inc - cnt;
      while (mask) {
        const int r = __builtin_ctz(mask);
        perm[pos++] = e0 + r;
        mask &= mask - 1;
      }
      base += total;
      __syncthreads();  // wave_total is rewritten by the next chunk
    }
    if (pass == 0) lead_total = base;
  }
  if (bad) atomicOr(&bad_any, 1);
  __syncthreads();
  if (t == 0) n_lead[0] = bad_any ? -1 : lead_total;
}

// dst row i <- src row perm[i] (or the inverse), 16-, 4- or 1-byte units
template <typename U>
__global__ __launch_bounds__(kThreads) void permute_rows_kernel(const U* __restrict__ src,
                                                                const int32_t* __restrict__ perm,
                                                                long n_rows, long units, bool inverse,
                                                                U* __restrict__ dst) {
  const long total = n_rows * units;
  for (long e = blockIdx.x * (long)kThreads + threadIdx.x; e < total; e += (long)gridDim.x * kThreads) {
    const long i = e / units, u = e - i * units;
    const long p = perm[i];
    if (p < 0 || p >= n_rows) continue;
    if (inverse)
      dst[p * units + u] = src[e];
    else
      dst[e] = src[p * units + u];
  }
}

// one wave per row, fp32 sum of squares
template <bool BF16>
__global__ __launch_bounds__(kThreads) void row_rms_scale(const void* __restrict__ x, int n_rows,
                                                          int d, float eps, bool vec,
                                                          float* __restrict__ scale) {
  const int lane = threadIdx.x & 63;
  const long row = (long)blockIdx.x * (kThreads / kWave) + (threadIdx.x >> 6);
  if (row >= n_rows) return;  // the whole wave leaves together
  float acc = 0.f;
  if constexpr (BF16) {
    const bf16* r = static_cast<const bf16*>(x) + row * d;
    if (vec) {
      for (int c = lane * 8; c < d; c += kWave * 8) {
        const bf16x8 v = *reinterpret_cast<const bf16x8*>(r + c);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
          const float f = (float)v[u];
          acc = fmaf(f, f, acc);
        }
      }
    } else {
      for (int c = lane; c < d; c += kWave) {
        const float f = (float)r[c];
        acc = fmaf(f, f, acc);
      }
    }
  } else {
    const float* r = static_cast<const float*>(x) + row * d;
    if (vec) {
      for (int c = lane * 4; c < d; c += kWave * 4) {
        const f32x4 v = *reinterpret_cast<const f32x4*>(r + c);
#pragma unroll
        for (int u = 0; u < 4; ++u) acc = fmaf(v[u], v[u], acc);
      }
    } else {
      for (int c = lane; c < d; c += kWave) acc = fmaf(r[c], r[c], acc);
    }
  }
  acc = wave_sum(acc);
  if (lane == 0) scale[row] = 1.0f / sqrtf(acc / (float)d + eps);
}

}  // namespace

hipError_t launch_row_rms_scale(const void* x, bool bf16_in, int n_rows, int d, float eps,
                                float* scale, hipStream_t s) {
  if (n_rows <= 0 || d <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)((n_rows + kThreads / kWave - 1) / (kThreads / kWave));
  const bool vec = (reinterpret_cast<uintptr_t>(x) & 15) == 0 && d % (bf16_in ? 8 : 4) == 0;
  if (bf16_in)
    hipLaunchKernelGGL(row_rms_scale<true>, dim3(blocks), dim3(kThreads), 0, s, x, n_rows, d, eps,
                       vec, scale);
  else
    hipLaunchKernelGGL(row_rms_scale<false>, dim3(blocks), dim3(kThreads), 0, s, x, n_rows, d,
                       eps, vec, scale);
  return hipGetLastError();
}

hipError_t launch_gather_latent(const float* x, const int32_t* idx, int n_active, long n_tokens,
                                int channels, bool out_bf16, void* xa, hipStream_t s) {
  if (n_active <= 0 || channels <= 0) return hipSuccess;
  const bool vec = channels % 4 == 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0 &&
                   (reinterpret_cast<uintptr_t>(xa) & (out_bf16 ? 7 : 15)) == 0;
  if (vec) {
    const int vpr = channels / 4;
    const dim3 grid(grid_for(((long)n_active * vpr + kGatherU - 1) / kGatherU));
    if (out_bf16)
      hipLaunchKernelGGL(gather_latent_vec<true>, grid, dim3(kThreads), 0, s,
                         reinterpret_cast<const f32x4*>(x), idx, n_active, n_tokens, vpr, xa);
    else
      hipLaunchKernelGGL(gather_latent_vec<false>, grid, dim3(kThreads), 0, s,
                         reinterpret_cast<const f32x4*>(x), idx, n_active, n_tokens, vpr, xa);
  } else {
    const dim3 grid(grid_for((long)n_active * channels));
    if (out_bf16)
      hipLaunchKernelGGL(gather_latent_scalar<true>, grid, dim3(kThreads), 0, s, x, idx, n_active,
                         n_tokens, channels, xa);
    else
      hipLaunchKernelGGL(gather_latent_scalar<false>, grid, dim3(kThreads), 0, s, x, idx,
                         n_active, n_tokens, channels, xa);
  }
  return hipGetLastError();
}

hipError_t launch_reorder_plan(const int32_t* budget, int n, int T, int32_t* perm,
                               int32_t* n_lead, hipStream_t s) {
  hipLaunchKernelGGL(reorder_plan_kernel, dim3(1), dim3(kPlanThreads), 0, s, budget, n, T, perm,
                     n_lead);
  return hipGetLastError();
}

hipError_t launch_permute_rows(const void* src, const int32_t* perm, long n_rows, long row_bytes,
                               bool inverse, void* dst, hipStream_t s) {
  if (n_rows <= 0 || row_bytes <= 0) return hipSuccess;
  const uintptr_t a = reinterpret_cast<uintptr_t>(src) | reinterpret_cast<uintptr_t>(dst);
  if (row_bytes % 16 == 0 && a % 16 == 0) {
    const long u = row_bytes / 16;
    hipLaunchKernelGGL(permute_rows_kernel<u32x4>, dim3(grid_for(n_rows * u)), dim3(kThreads), 0, s,
                       static_cast<const u32x4*>(src), perm, n_rows, u, inverse,
                       static_cast<u32x4*>(dst));
  } else if (row_bytes % 4 == 0 && a % 4 == 0) {
    const long u = row_bytes / 4;
    hipLaunchKernelGGL(permute_rows_kernel<uint32_t>, dim3(grid_for(n_rows * u)), dim3(kThreads), 0,
                       s, static_cast<const uint32_t*>(src), perm, n_rows, u, inverse,
                       static_cast<uint32_t*>(dst));
  } else {
    hipLaunchKernelGGL(permute_rows_kernel<uint8_t>, dim3(grid_for(n_rows * row_bytes)),
                       dim3(kThreads), 0, s, static_cast<const uint8_t*>(src), perm, n_rows,
                       row_bytes, inverse, static_cast<uint8_t*>(dst));
  }
  return hipGetLastError();
}

hipError_t launch_rank_budgets(const double* keys, long n_tokens, const GroupTable& tab,
                               int32_t* budget, hipStream_t s) {
  if (n_tokens <= 0) return hipSuccess;
  const unsigned blocks = (unsigned)((n_tokens + kRankTokens - 1) / kRankTokens);
  hipLaunchKernelGGL(rank_budgets, dim3(blocks), dim3(kThreads), 0, s,
                     reinterpret_cast<const unsigned long long*>(keys), (int)n_tokens, tab, budget);
  return hipGetLastError();
}

hipError_t launch_l1_rel(const float* v, float* v_prev, long n_tokens, int channels, double* acc,
                         bool first, hipStream_t s) {
  if (n_tokens <= 0) return hipSuccess;
  hipLaunchKernelGGL(l1_rel_accumulate, dim3(grid_for(n_tokens)), dim3(kThreads), 0, s, v, v_prev,
                     n_tokens, channels, acc, first ? 1 : 0);
  return hipGetLastError();
}

hipError_t launch_assign_budgets(const float* v, long n_tokens, int channels,
                                 const GroupTable& tab, double* keys, int32_t* budget,
                                 hipStream_t s) {
  if (n_tokens <= 0) return hipSuccess;
  if (channels % 4 == 0 && (reinterpret_cast<uintptr_t>(v) & 15) == 0)
    hipLaunchKernelGGL(velocity_keys_vec, dim3(grid_for(n_tokens)), dim3(kThreads), 0, s,
                       reinterpret_cast<const f32x4*>(v), n_tokens, channels / 4, keys);
  else
    hipLaunchKernelGGL(velocity_keys_scalar, dim3(grid_for(n_tokens)), dim3(kThreads), 0, s, v,
                       n_tokens, channels, keys);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  return launch_rank_budgets(keys, n_tokens, tab, budget, s);
}

}  // namespace hsa
