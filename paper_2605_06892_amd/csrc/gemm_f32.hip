// Row-indexed fp32 GEMM: C[crow(m)] = A[arow(m)] B^T, the fp32 variant of the
// projections of the layer step (Section 2.3) for fp32 workloads.
//
// Plain FMA tiling: a 64 x 64 output tile per 256-thread workgroup, each
// thread accumulating a 4 x 4 block, K step 16 staged through LDS. Arbitrary
// M, Nc and K (ragged edges are masked). An optional per-row scale multiplies
// each product row, an optional tanh GELU follows, and an optional fp32
// residual, indexed like the output, is added before the store.
#include "common.h"

namespace hsa {
namespace {

constexpr int TM = 64, TN = 64, TK = 16, kThreads = 256;

__global__ __launch_bounds__(kThreads) void row_gemm_f32_kernel(RowGemm g) {
  __shared__ float As[TK][TM + 4];
  __shared__ float Bs[TK][TN + 4];

  const int tiles_m = (g.M + TM - 1) / TM;
  const int tiles_n1 = (g.Nc + TN - 1) / TN;
  const int per_out = tiles_m * tiles_n1;
  const int item = xcd_contiguous(blockIdx.x, per_out * g.n_out);
  const int z = item / per_out;
  const int rem = item - z * per_out;
  const int tm = rem % tiles_m;
  const int tn = rem / tiles_m;
  const RowGemmOut oz = row_gemm_out(g, z);

  const float* __restrict__ A = static_cast<const float*>(g.A);
  const float* __restrict__ B = static_cast<const float*>(oz.B);
  const int t = threadIdx.x;
  const int tx = t & 15, ty = t >> 4;

  // load mapping: 64 rows x 16 k per tile, 4 consecutive k per thread
  const int lrow = t >> 2;
  const int lk = (t & 3) * 4;
  const int m_load = tm * TM + lrow;
  int arow = -1;
  if (m_load < g.M) arow = g.a_rows ? g.a_rows[m_load] : m_load;
  const bool a_ok = arow >= 0 && arow < g.a_limit;
  const int n_load = tn * TN + lrow;
  const bool b_ok = n_load < g.Nc;
  const float* a_src = A + (long)(a_ok ? arow : 0) * g.lda;
  const float* b_src = B + (long)(b_ok ? n_load : 0) * g.ldb;

  float acc[4][4] = {};
  for (int k0 = 0; k0 < g.K; k0 += TK) {
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      const int k = k0 + lk + e;
      As[lk + e][lrow] = (a_ok && k < g.K) ? a_src[k] : 0.f;
      Bs[lk + e][lrow] = (b_ok && k < g.K) ? b_src[k] : 0.f;
    }
    __syncthreads();
#pragma unroll
    for (int kk = 0; kk < TK; ++kk) {
      float a[4], b[4];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        a[i] = As[kk][ty * 4 + i];
        b[i] = Bs[kk][tx * 4 + i];
      }
#pragma unroll
      for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
    }
    __syncthreads();
  }

  float* C = static_cast<float*>(oz.C);  // may alias the residual
  float* C2 = static_cast<float*>(oz.C2);
  const float* R = static_cast<const float*>(g.residual);
  const int32_t* c_rows = oz.c_rows;
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = tm * TM + ty * 4 + i;
    if (m >= g.M) continue;
    const int crow = c_rows ? c_rows[m] : m;
    if (crow < 0 || crow >= oz.c_limit) continue;
    const float rs = g.row_scale ? g.row_scale[m] : 1.f;
    float v[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[j] = g.row_scale ? acc[i][j] * rs : acc[i][j];
      if (g.gelu) v[j] = gelu_tanh(v[j]);
    }
    if (g.rope_cs && ((g.rope_outs >> z) & 1)) {  // pairs (n, n+1), (n+2, n+3) of a 4-aligned run
      const RopeRow rr = rope_row(g, m);
      const int k = ((tn * TN + tx * 4) % g.rope_dh) >> 1;
      const f32x2 r0 = rope_pair(g, rr, k, v[0], v[1]);
      const f32x2 r1 = rope_pair(g, rr, k + 1, v[2], v[3]);
      v[0] = r0[0];
      v[1] = r0[1];
      v[2] = r1[0];
      v[3] = r1[1];
    }
    float* cb = C;
    long orow = crow;
    if (C2 && crow >= oz.c_split) {  // rows past the split go to the second buffer
      cb = C2;
      orow = crow - oz.c_split;
    }
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      const int n = tn * TN + tx * 4 + j;
      if (n < g.Nc) {
        const long e = orow * g.ldc + n;
        cb[e] = R ? v[j] + R[e] : v[j];
      }
    }
  }
}

}  // namespace

hipError_t launch_row_gemm_f32(const RowGemm& g, hipStream_t s) {
  if (g.M <= 0 || g.Nc <= 0 || g.n_out <= 0) return hipSuccess;
  const long tiles = (long)((g.M + TM - 1) / TM) * ((g.Nc + TN - 1) / TN) * g.n_out;
  hipLaunchKernelGGL(row_gemm_f32_kernel, dim3((unsigned)tiles), dim3(kThreads), 0, s, g);
  return hipGetLastError();
}

}  // namespace hsa
