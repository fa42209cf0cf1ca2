// Cached Euler update (Section 2.4, Eq. 6): every token advances by the shared
// step dsig = sigma_{i+1} - sigma_i with the last velocity it produced.
//
// With fresh velocities (the active tokens' rows, compact, in the order of an
// ascending index list) the update is one pass over all tokens, as the paper
// describes it: each token reads either its fresh row or its cached row, x is
// advanced, and only fresh rows are written back to the velocity cache.
// Workgroups sweep the token tiles together. A wave-wide 64-ary search
// locates the first fresh row of a run of tiles in the index list; from there
// each tile's fresh rows are the next entries of the list (ascending), whose
// positions go into an LDS slot table of the tile (double-buffered and tagged
// with the tile number, so one barrier per tile suffices). Without fresh
// velocities it is a plain stream x = fmaf(v_cache, dsig, x).
// Both are HBM-bound element streams: 16-byte nontemporal vector accesses when
// the rows allow it, each thread keeping U independent 16-byte loads of each
// input in flight before its stores.
#include "common.h"

#include <algorithm>
#include <type_traits>

namespace hsa {
namespace {

constexpr int kThreads = 256;
constexpr int U = 4;  // 16-byte elements per thread per loop trip

// Streamed data is touched once: nontemporal loads and stores keep it from
// displacing the caches (measured 5.8 TB/s vs 5.3 TB/s for plain accesses on
// a 3 GB update).
__device__ __forceinline__ f32x4 ld(const f32x4* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st(f32x4 v, f32x4* p) { __builtin_nontemporal_store(v, p); }
__device__ __forceinline__ float ld(const float* p) { return __builtin_nontemporal_load(p); }
__device__ __forceinline__ void st(float v, float* p) { __builtin_nontemporal_store(v, p); }

// x + v dsig with one rounding per value (fmaf)
__device__ __forceinline__ f32x4 fma_step(f32x4 v, float dsig, f32x4 x) {
  return (f32x4){fmaf(v[0], dsig, x[0]), fmaf(v[1], dsig, x[1]), fmaf(v[2], dsig, x[2]),
                 fmaf(v[3], dsig, x[3])};
}
__device__ __forceinline__ float fma_step(float v, float dsig, float x) { return fmaf(v, dsig, x); }

constexpr int kTileElems = kThreads * U;  // vector elements per token tile
constexpr int kMaxTileRows = kTileElems;   // one element per row at most

// First position j in idx[0 .. n) with idx[j] >= t (idx ascending), found by
// the whole wave: every round the 64 lanes probe 64 positions that cut the
// interval into 65 parts, and the ballot of "below t" (a prefix of the lanes
// for an ascending list) gives the part that holds the answer. Six rounds
// cover 2^31 entries. Wave-uniform result; for a list that is not ascending
// the result is some position in [0, n].
__device__ __forceinline__ int wave_lower_bound(const int32_t* __restrict__ idx, int n, long t) {
  const int lane = threadIdx.x & (kWave - 1);
  int lo = 0, hi = n;
  for (int round = 0; round < 8 && lo < hi; ++round) {
    const long span = hi - lo;
    const int p = lo + (int)(span * (lane + 1) / 65);
    const bool below = p < hi && idx[p] < t;
    const int c = __popcll(__ballot(below));
    const int p_lo = c > 0 ? lo + (int)(span * c / 65) : lo - 1;   // probe of lane c-1
    const int p_hi = c < kWave ? lo + (int)(span * (c + 1) / 65) : hi;  // probe of lane c
    lo = p_lo + 1;
    hi = p_hi;
  }
  return min(max(lo, 0), n);
}

// One pass with fresh rows. Elements are VW floats (16 bytes for VW = 4); a
// row holds epr elements. Token tiles hold `rows` tokens (rows * epr <=
// kTileElems). Workgroups sweep the tiles together, in runs of `run`
// consecutive tiles: workgroup g takes tiles g*run .. g*run+run-1, then the
// run `gridDim.x` runs further on, so the tiles in flight stay within one
// window of the tensors. One search per run; inside a run the list continues
// from the previous tile's last fresh row.
template <int VW>
__global__ __launch_bounds__(kThreads) void cached_euler_fused(
    float* __restrict__ x, float* __restrict__ v_cache, const float* __restrict__ v_fresh,
    const int32_t* __restrict__ idx, int n_active, long n_tokens, int epr, int rows, long n_tiles,
    int run, float dsig) {
  typedef typename std::conditional<VW == 4, f32x4, float>::type elem;
  __shared__ int2 slot[2][kMaxTileRows];  // (tile, position in idx) of a fresh row
  const int tid = threadIdx.x;
  for (int k = tid; k < kMaxTileRows; k += kThreads) {
    slot[0][k] = make_int2(-1, 0);
    slot[1][k] = make_int2(-1, 0);
  }
  __syncthreads();
  elem* xe = reinterpret_cast<elem*>(x);
  elem* ve = reinterpret_cast<elem*>(v_cache);
  const elem* fe = reinterpret_cast<const elem*>(v_fresh);
  const long stride = (long)gridDim.x * run;  // tiles between a workgroup's runs
  int j0 = 0;
  int step = 0;  // tiles done by this workgroup: selects the slot buffer
  for (long r0 = (long)blockIdx.x * run; r0 < n_tiles; r0 += stride) {
    j0 = wave_lower_bound(idx, n_active, r0 * rows);
    const long r_end = min(n_tiles, r0 + run);
    for (long tile = r0; tile < r_end; ++tile, ++step) {
      const long t0 = tile * rows;
      const long t1 = min(n_tokens, t0 + rows);
      // Buffer step & 1 was last read two tiles ago, before the previous
      // tile's barrier. The tile's fresh rows are the next entries of the
      // ascending list; the barrier inside __syncthreads_count publishes them.
      int2* sl = slot[step & 1];
      int cnt = 0;
      for (int k0 = 0; k0 < rows; k0 += kThreads) {
        const int k = k0 + tid;
        bool in = false;
        const long j = (long)j0 + k;  // 64-bit: j0 may lie near 2^31
        if (k < rows && j < n_active) {
          const long t = idx[j];
          in = t >= t0 && t < t1;
          if (in) sl[t - t0] = make_int2((int)tile, (int)j);
        }
        cnt += __syncthreads_count(in);
      }
      const int tag = (int)tile;
      elem xv[U], vv[U];
      long dst[U];
      bool fresh[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int el = tid + u * kThreads;
        const int r = el / epr;
        const int c = el - r * epr;
        dst[u] = -1;
        fresh[u] = false;
        if (r < rows && t0 + r < t1) {
          const int2 s = sl[r];
          const long e = (t0 + r) * epr + c;
          dst[u] = e;
          fresh[u] = s.x == tag;
          xv[u] = ld(xe + e);
          // one load per element: the fresh row or the cached row
          vv[u] = ld(fresh[u] ? fe + (long)s.y * epr + c : ve + e);
        }
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (dst[u] >= 0) {
          st(fma_step(vv[u], dsig, xv[u]), xe + dst[u]);
          if (fresh[u]) st(vv[u], ve + dst[u]);
        }
      }
      j0 += cnt;
    }
  }
}

// v_cache[idx[j]] = v_fresh[j] (rows wider than a token tile)
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

__global__ __launch_bounds__(kThreads) void euler_f32x4(f32x4* __restrict__ x,
                                                        const f32x4* __restrict__ v, long n4,
                                                        float dsig) {
  for (long e0 = blockIdx.x * (long)(kThreads * U) + threadIdx.x; e0 < n4;
       e0 += (long)gridDim.x * kThreads * U) {
    f32x4 a[U], b[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const long e = e0 + (long)u * kThreads;
      if (e < n4) {
        a[u] = ld(x + e);
        b[u] = ld(v + e);
      }
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const long e = e0 + (long)u * kThreads;
      if (e < n4) {
        st(fma_step(b[u], dsig, a[u]), x + e);
      }
    }
  }
}

__global__ __launch_bounds__(kThreads) void euler_f32(float* __restrict__ x,
                                                      const float* __restrict__ v, long n,
                                                      float dsig) {
  for (long e = blockIdx.x * (long)kThreads + threadIdx.x; e < n;
       e += (long)gridDim.x * kThreads)
    x[e] = fmaf(v[e], dsig, x[e]);
}

int grid_for(long work_items, int per_thread) {
  // up to 16 workgroups of 256 threads per CU (256 CUs), grid-stride beyond that
  long g = (work_items + (long)kThreads * per_thread - 1) / ((long)kThreads * per_thread);
  if (g > 4096) g = 4096;
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
  const long n = n_tokens * (long)channels;
  if (n == 0) return hipSuccess;
  if (v_fresh != nullptr && n_active > 0) {
    const int vw = vec ? 4 : 1;
    const int epr = channels / vw;  // elements per row
    const int rows = epr >= kTileElems ? 1 : kTileElems / epr;
    if (epr > kTileElems) {
      // rows wider than a tile (more than 4096 channels): scatter, then the plain stream
      hipLaunchKernelGGL(scatter_rows_f32, dim3(grid_for((long)n_active * channels, 1)),
                         dim3(kThreads), 0, s, v_cache, v_fresh, idx, n_active, n_tokens,
                         channels);
      hipError_t e = hipGetLastError();
      if (e != hipSuccess) return e;
    } else {
      // Up to 16 workgroups per CU (two rounds of 8 resident). Runs of 4 tiles
      // per search once that many tiles still give every workgroup work; small
      // launches (latency-bound) take one tile per search. Measured at 4M x 64
      // channels: 5.59 TB/s with runs of 4, 5.38 with single tiles.
      const long n_tiles = (n_tokens + rows - 1) / rows;
      const long max_wg = (long)compute_units() * 16;
      const int run = n_tiles >= 4 * max_wg ? 4 : 1;
      const long grid = std::min<long>((n_tiles + run - 1) / run, max_wg);
      if (vec)
        hipLaunchKernelGGL(cached_euler_fused<4>, dim3((unsigned)grid), dim3(kThreads), 0, s, x,
                           v_cache, v_fresh, idx, n_active, n_tokens, epr, rows, n_tiles, run, dsig);
      else
        hipLaunchKernelGGL(cached_euler_fused<1>, dim3((unsigned)grid), dim3(kThreads), 0, s, x,
                           v_cache, v_fresh, idx, n_active, n_tokens, epr, rows, n_tiles, run, dsig);
      return hipGetLastError();
    }
  }
  if (vec) {
    hipLaunchKernelGGL(euler_f32x4, dim3(grid_for(n / 4, U)), dim3(kThreads), 0, s,
                       reinterpret_cast<f32x4*>(x), reinterpret_cast<const f32x4*>(v_cache),
                       n / 4, dsig);
  } else {
    hipLaunchKernelGGL(euler_f32, dim3(grid_for(n, 1)), dim3(kThreads), 0, s, x, v_cache, n,
                       dsig);
  }
  return hipGetLastError();
}

}  // namespace hsa
