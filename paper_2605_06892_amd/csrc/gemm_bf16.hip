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
// Tiling: BM x BN output tile per 512-thread workgroup (8 waves in a WM x WN
// grid), K step 64, v_mfma_f32_32x32x16_bf16; the fragments of the next
// 16-wide k slice are read from LDS while the MFMAs of the current one run.
// Tiles go global -> LDS directly
// (global_load_lds_dwordx4: one wave instruction fills one contiguous 1 KB
// segment = 8 tile rows of 128 bytes) into two stages, the loads of step k+1
// in flight during the MFMAs of step k, one barrier per step. The 16-byte
// chunks of tile row r sit at slot chunk ^ ((r >> 1) & 7), which keeps the
// fragment reads (16 rows, one chunk) on disjoint banks. Each stage is its own
// LDS array and the K loop is unrolled by 2, so the compiler can tell the
// asynchronous loads from reads of the other stage.
// Every tile row is a contiguous 128-byte run of a token row, so the indexed
// loads stay coalesced; rows outside the problem are read from a valid row and
// their results dropped. The product is formed transposed (B rows drive the
// MFMA A operand), which leaves each lane holding one output row and runs of
// four consecutive columns: one row-index lookup per lane and 8-byte stores.
// Tiles are ordered in groups of 8 tile-rows and laid out contiguously per XCD
// so the A and B panels a group shares stay in that XCD's L2.
#include "common.h"

#include <type_traits>

namespace hsa {
namespace {

constexpr int BK = 64, kWaves = 8, kThreads = kWaves * 64;
constexpr int kGroupM = 8;

typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void global_cvoid;

constexpr int waitcnt_vm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

__device__ __forceinline__ int swz(int r) { return (r >> 1) & 7; }

// Epilogues (after the optional per-row scale): bf16 store, bf16 store of
// (product + bf16 residual) rounded once, fp32 store, bf16 store of the tanh
// GELU of the product.
enum Epilogue { kEpiBf16 = 0, kEpiBf16Residual = 1, kEpiF32 = 2, kEpiBf16Gelu = 3 };

// NOUT (1 or 3) is the number of outputs sharing A; it is a template
// parameter so the Q/K/V projection and the output projection are distinct
// kernels in profiles.
template <int BM, int BN, int WM, int NOUT, int EPI>
__global__ __launch_bounds__(kThreads) void row_gemm_bf16_kernel(RowGemm g) {
  constexpr int WN = kWaves / WM;
  constexpr int TM = BM / WM, TN = BN / WN;  // wave tile
  constexpr int MI = TM / 32, NI = TN / 32;  // 32x32 MFMA tiles per wave
  constexpr int SEG_A = BM / 8, SEG_B = BN / 8;  // 1 KB segments per stage
  constexpr int LOADS = (SEG_A + SEG_B) / kWaves;
  static_assert(LOADS * kWaves == SEG_A + SEG_B, "stage load must split evenly over waves");
  __shared__ __attribute__((aligned(16))) bf16 A0[BM * BK], A1[BM * BK];
  __shared__ __attribute__((aligned(16))) bf16 B0[BN * BK], B1[BN * BK];
  auto abuf = [&](auto s) -> bf16* { if constexpr (decltype(s)::value == 0) return A0; else return A1; };
  auto bbuf = [&](auto s) -> bf16* { if constexpr (decltype(s)::value == 0) return B0; else return B1; };

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

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int l32 = lane & 31, hi = lane >> 5;

  // This lane's rows of the stage loads: segment s = i*8 + wave covers tile
  // rows 8s .. 8s+7 (A tile first, then B tile); the lane fetches row
  // 8s + lane/8, global chunk (lane%8) ^ swz(row) into LDS slot lane%8.
  const bf16* src[LOADS];
  int dst[LOADS];  // element offset of the segment in its tile
#pragma unroll
  for (int i = 0; i < LOADS; ++i) {
    const int s = i * kWaves + wave;
    const bool a = s < SEG_A;
    const int trow = (a ? s : s - SEG_A) * 8 + lane / 8;
    const int chunk = (lane % 8) ^ swz(trow);
    long grow;
    if (a) {
      const int m = tm * BM + trow;
      int row = (m < g.M) ? (g.a_rows ? g.a_rows[m] : m) : 0;
      if (row < 0 || row >= g.a_limit) row = 0;
      grow = (long)row * g.lda;
    } else {
      const int n = min(tn * BN + trow, g.Nc - 1);
      grow = (long)n * g.ldb;
    }
    src[i] = (a ? A : B) + grow + chunk * 8;
    dst[i] = (a ? s : s - SEG_A) * 512;
  }
  auto issue = [&](auto st, int k0) {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      // segments i*8 + wave: all of one wave's segments of load i lie in the
      // same tile when SEG_A is a multiple of 8 (always true here)
      bf16* base = (i * kWaves < SEG_A) ? abuf(st) : bbuf(st);
      __builtin_amdgcn_global_load_lds((global_cvoid*)(src[i] + k0), (lds_void*)(base + dst[i]), 16, 0, 0);
    }
  };
  static_assert(SEG_A % kWaves == 0, "A segments must fill whole load rounds");

  // fragment read offsets: row (tile-local) l32 + 32*t, chunk kk*2 + hi
  const int xr = ((hi ^ swz(l32)) * 8);  // chunk kk*2+hi ^ f = (kk*2) ^ (hi ^ f); f(r) = f(r % 16)
  f32x16 acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j) acc[i][j] = (f32x16){};

  auto compute = [&](auto st) {
    const bf16* As = abuf(st) + (wm * TM + l32) * BK;
    const bf16* Bs = bbuf(st) + (wn * TN + l32) * BK;
    bf16x8 af[2][MI], bfr[2][NI];
    auto ld = [&](int kk, int b) {
      const int off = (kk * 16) ^ xr;
#pragma unroll
      for (int i = 0; i < MI; ++i) af[b][i] = *reinterpret_cast<const bf16x8*>(As + i * 32 * BK + off);
#pragma unroll
      for (int j = 0; j < NI; ++j) bfr[b][j] = *reinterpret_cast<const bf16x8*>(Bs + j * 32 * BK + off);
    };
    ld(0, 0);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      if (kk + 1 < BK / 16) ld(kk + 1, (kk + 1) & 1);
#pragma unroll
      for (int i = 0; i < MI; ++i)
#pragma unroll
        for (int j = 0; j < NI; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[kk & 1][j], af[kk & 1][i], acc[i][j], 0, 0, 0);
      if (kk + 1 < BK / 16) {
        __builtin_amdgcn_sched_group_barrier(0x100, MI + NI, 0);
        __builtin_amdgcn_sched_group_barrier(0x008, MI * NI, 0);
      }
    }
  };

  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  const int nk = g.K / BK;
  issue(S0{}, 0);
  // step k lives in stage k % 2: wait for its loads, make them visible (and
  // free the other stage), start step k+1's loads, compute step k
  auto step = [&](auto st, auto other, int k) {
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();
    if (k + 1 < nk) issue(other, (k + 1) * BK);
    compute(st);
  };
  for (int k = 0; k < nk; k += 2) {
    step(S0{}, S1{}, k);
    if (k + 1 < nk) step(S1{}, S0{}, k + 1);
  }

  // acc[i][j][e]: output row m = tile row + i*32 + l32,
  //               column n = tile col + j*32 + (e/4)*8 + hi*4 + e%4
  const int32_t* c_rows = oz.c_rows;
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    const int m = tm * BM + wm * TM + i * 32 + l32;
    if (m >= g.M) continue;
    const int crow = c_rows ? c_rows[m] : m;
    if (crow < 0 || crow >= oz.c_limit) continue;
    void* cbase = oz.C;
    long orow = crow;
    if (oz.C2 && crow >= oz.c_split) {  // rows past the split go to the second buffer
      cbase = oz.C2;
      orow = crow - oz.c_split;
    }
    const long obase = orow * g.ldc;
    const float rs = g.row_scale ? g.row_scale[m] : 1.f;
    const bool rope = g.rope_cs && ((g.rope_outs >> z) & 1);
    RopeRow rr{0, 0, 0};
    if (rope) rr = rope_row(g, m);
#pragma unroll
    for (int j = 0; j < NI; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int n = tn * BN + wn * TN + j * 32 + q * 8 + hi * 4;
        if (n < g.Nc) {
          f32x4 v = {acc[i][j][4 * q + 0], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2],
                     acc[i][j][4 * q + 3]};
          if (g.row_scale) v *= rs;
          if (rope) {
            const int k = (n % g.rope_dh) >> 1;
            const f32x2 r0 = rope_pair(g, rr, k, v[0], v[1]);
            const f32x2 r1 = rope_pair(g, rr, k + 1, v[2], v[3]);
            v = (f32x4){r0[0], r0[1], r1[0], r1[1]};
          }
          if constexpr (EPI == kEpiF32) {
            *reinterpret_cast<f32x4*>(static_cast<float*>(cbase) + obase + n) = v;
          } else {
            if constexpr (EPI == kEpiBf16Residual) {
              const bf16x4 r =
                  *reinterpret_cast<const bf16x4*>(static_cast<const bf16*>(g.residual) + obase + n);
              v += __builtin_convertvector(r, f32x4);
            }
            if constexpr (EPI == kEpiBf16Gelu) {
#pragma unroll
              for (int u = 0; u < 4; ++u) v[u] = gelu_tanh(v[u]);
            }
            *reinterpret_cast<bf16x4*>(static_cast<bf16*>(cbase) + obase + n) = to_bf16x4(v);
          }
        }
      }
    }
  }
}

template <int BM, int BN, int WM, int NOUT, int EPI>
hipError_t launch(const RowGemm& g, hipStream_t s) {
  const long tiles = (long)((g.M + BM - 1) / BM) * ((g.Nc + BN - 1) / BN) * NOUT;
  hipLaunchKernelGGL((row_gemm_bf16_kernel<BM, BN, WM, NOUT, EPI>), dim3((unsigned)tiles),
                     dim3(kThreads), 0, s, g);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_row_gemm_bf16(const RowGemm& g, hipStream_t s) {
  if (g.M <= 0 || g.Nc <= 0 || (g.n_out != 1 && g.n_out != 3)) return hipSuccess;
  // 256 x 256 tiles (8 waves of 128 x 64) for the three-output projection and
  // for single-output products with at least two workgroups per CU of them;
  // 256 x 128 tiles (8 waves of 64 x 64) for smaller single-output products,
  // whose grid would otherwise leave CUs idle in the last round.
  if (g.n_out == 3) return launch<256, 256, 2, 3, kEpiBf16>(g, s);
  const long big = (long)((g.M + 255) / 256) * ((g.Nc + 255) / 256);
  if (g.c_f32) return launch<256, 128, 4, 1, kEpiF32>(g, s);
  if (big >= 512) {
    if (g.gelu) return launch<256, 256, 2, 1, kEpiBf16Gelu>(g, s);
    if (g.residual) return launch<256, 256, 2, 1, kEpiBf16Residual>(g, s);
    return launch<256, 256, 2, 1, kEpiBf16>(g, s);
  }
  if (g.gelu) return launch<256, 128, 4, 1, kEpiBf16Gelu>(g, s);
  if (g.residual) return launch<256, 128, 4, 1, kEpiBf16Residual>(g, s);
  return launch<256, 128, 4, 1, kEpiBf16>(g, s);
}

}  // namespace hsa
