// Row-indexed bf16 GEMM on CDNA4 matrix cores: C[crow(m)] = A[arow(m)] B^T.
//
// This one kernel carries both dense contractions of the layer step:
//   * the fresh Q/K/V projections of the active rows (Section 2.3, step 1),
//     with the gather of x[A_i] fused into the A-tile loads and the cache
//     overwrite K_hat[A_i], V_hat[A_i] (step 2) fused into the K/V epilogues;
//   * the output projection of the active rows with the scatter back to their
//     tokens fused into the epilogue.
// The compact gathered activations are never materialized in HBM.
//
// Tiling: 128 x 128 output tile per 256-thread workgroup (4 waves in 2 x 2,
// 64 x 64 per wave = 2 x 2 tiles of v_mfma_f32_32x32x16_bf16), K step 64,
// two LDS buffers (global loads of step k+1 overlap the MFMAs of step k).
// Every tile row is a contiguous 128-byte run of a token row, so the indexed
// loads stay coalesced. The product is formed transposed (B rows drive the
// MFMA A operand), which leaves each lane holding one output row and runs of
// four consecutive columns: one row-index lookup per lane and 8-byte stores.
// Tiles are ordered in groups of 8 tile-rows and laid out contiguously per XCD
// so the A and B panels a group shares stay in that XCD's L2.
#include "common.h"

namespace hsa {
namespace {

constexpr int BM = 128, BN = 128, BK = 64, kThreads = 256;
constexpr int LS = BK + 8;  // LDS row stride in bf16 (144 bytes, 16-byte aligned)
constexpr int kGroupM = 8;

// NOUT (1 or 3) is the number of outputs sharing A; it is a template
// parameter so the Q/K/V projection and the output projection are distinct
// kernels in profiles.
template <int NOUT>
__global__ __launch_bounds__(kThreads, 2) void row_gemm_bf16_kernel(RowGemm g) {
  __shared__ __attribute__((aligned(16))) bf16 As[2][BM * LS];
  __shared__ __attribute__((aligned(16))) bf16 Bs[2][BN * LS];

  const int tiles_m = (g.M + BM - 1) / BM;
  const int tiles_n1 = (g.Nc + BN - 1) / BN;  // per output
  const int tiles_n = tiles_n1 * NOUT;        // over all outputs side by side
  const int total = tiles_m * tiles_n;
  const int item = xcd_contiguous(blockIdx.x, total);
  // grouped order: kGroupM tile-rows sweep all tile-columns together
  const int group = item / (kGroupM * tiles_n);
  const int first_m = group * kGroupM;
  const int gm = min(kGroupM, tiles_m - first_m);
  const int r = item - group * kGroupM * tiles_n;
  const int tm = first_m + r % gm;
  const int tnc = r / gm;
  const int z = tnc / tiles_n1;
  const int tn = tnc - z * tiles_n1;
  const RowGemmOut oz = row_gemm_out(g, z);

  const bf16* __restrict__ A = static_cast<const bf16*>(g.A);
  const bf16* __restrict__ B = static_cast<const bf16*>(oz.B);

  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int l32 = lane & 31, hi = lane >> 5;

  // global -> LDS mapping: 8 threads per 64-element row segment, 4 rows per thread
  const int lr = t >> 3;
  const int lc = (t & 7) * 8;
  const bf16* a_src[4];
  const bf16* b_src[4];
  bool a_ok[4], b_ok[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    const int m = tm * BM + lr + 32 * i;
    int row = -1;
    if (m < g.M) row = g.a_rows ? g.a_rows[m] : m;
    a_ok[i] = row >= 0 && row < g.a_limit;
    a_src[i] = A + (long)(a_ok[i] ? row : 0) * g.lda + lc;
    const int n = tn * BN + lr + 32 * i;
    b_ok[i] = n < g.Nc;
    b_src[i] = B + (long)(b_ok[i] ? n : 0) * g.ldb + lc;
  }

  u32x4 ra[4], rb[4];
  const u32x4 zero = {0u, 0u, 0u, 0u};
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      ra[i] = a_ok[i] ? *reinterpret_cast<const u32x4*>(a_src[i] + k0) : zero;
      rb[i] = b_ok[i] ? *reinterpret_cast<const u32x4*>(b_src[i] + k0) : zero;
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      *reinterpret_cast<u32x4*>(&As[buf][(lr + 32 * i) * LS + lc]) = ra[i];
      *reinterpret_cast<u32x4*>(&Bs[buf][(lr + 32 * i) * LS + lc]) = rb[i];
    }
  };

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j) acc[i][j] = (f32x16){};

  const int nk = g.K / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 af[2], bfr[2];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        af[i] = *reinterpret_cast<const bf16x8*>(
            &As[buf][(wm * 64 + i * 32 + l32) * LS + kk * 16 + hi * 8]);
        bfr[i] = *reinterpret_cast<const bf16x8*>(
            &Bs[buf][(wn * 64 + i * 32 + l32) * LS + kk * 16 + hi * 8]);
      }
#pragma unroll
      for (int i = 0; i < 2; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
    }
    if (kt + 1 < nk) lstore(buf ^ 1);
    __syncthreads();
  }

  // acc[i][j][e]: output row m = tile row + i*32 + l32,
  //               column n = tile col + j*32 + (e/4)*8 + hi*4 + e%4
  bf16* __restrict__ C = static_cast<bf16*>(oz.C);
  const int32_t* c_rows = oz.c_rows;
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int m = tm * BM + wm * 64 + i * 32 + l32;
    if (m >= g.M) continue;
    const int crow = c_rows ? c_rows[m] : m;
    if (crow < 0 || crow >= oz.c_limit) continue;
    bf16* dst = C + (long)crow * g.ldc;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = tn * BN + wn * 64 + j * 32 + q * 8 + hi * 4;
        if (n < g.Nc) {
          f32x4 v = {acc[i][j][4 * q + 0], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                     acc[i][j][4 * q + 3]};
          *reinterpret_cast<bf16x4*>(dst + n) = to_bf16x4(v);
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_row_gemm_bf16(const RowGemm& g, hipStream_t s) {
  if (g.M <= 0 || g.Nc <= 0 || (g.n_out != 1 && g.n_out != 3)) return hipSuccess;
  const long tiles = (long)((g.M + BM - 1) / BM) * ((g.Nc + BN - 1) / BN) * g.n_out;
  if (g.n_out == 3)
    hipLaunchKernelGGL(row_gemm_bf16_kernel<3>, dim3((unsigned)tiles), dim3(kThreads), 0, s, g);
  else
    hipLaunchKernelGGL(row_gemm_bf16_kernel<1>, dim3((unsigned)tiles), dim3(kThreads), 0, s, g);
  return hipGetLastError();
}

}  // namespace hsa
