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
// Tiling (struct Tiling): BM x BN output tile per workgroup of 8 waves in a
// WM x WN grid, K step 64, v_mfma_f32_32x32x16_bf16. Tiles go global -> LDS
// directly (buffer_load_dwordx4 ... lds through one buffer resource over A
// and one over B, or global_load_lds_dwordx4 with 64-bit lane pointers for a
// matrix of 4 GiB or more: one wave instruction fills one contiguous 1 KB
// segment = 8 tile rows of 128 bytes) into two stages, the
// loads of step k+1 in flight during the MFMAs of step k, one barrier per
// step. Within a step the fragment reads of k slice s+1 and the stage loads
// are placed one per MFMA between the MFMAs of slice s, so neither the LDS
// latency nor the load issue stalls the matrix pipe (measured: issuing them
// in bursts ahead of the MFMAs cost 5-10%), and the MFMAs of the last
// slice's fragment rows (half of them at 256 x 256 with 64-bit pointers) run
// behind the next step's barrier, where they cover that step's first reads. The 16-byte chunks of tile row r
// sit at slot chunk ^ ((r >> 1) & 7), which keeps the fragment reads (16
// rows, one chunk) on disjoint banks. Each stage is its own LDS array and the
// K loop is unrolled by the stage count, so the compiler can tell the
// asynchronous loads from reads of the other stage.
// Every tile row is a contiguous 128-byte run of a token row, so the indexed
// loads stay coalesced; rows outside the problem are read from a valid row and
// their results dropped. The product is formed transposed (B rows drive the
// MFMA A operand), which leaves each lane holding one output row and runs of
// four consecutive columns: one row-index lookup per lane and 8-byte stores.
// Tiles are ordered in groups of 8 tile-rows (4 for wide outputs) and laid
// out contiguously per XCD so the A and B panels a group shares stay in that
// XCD's L2.
#include "common.h"

#include <type_traits>

namespace hsa {
namespace {


typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void global_cvoid;

constexpr int waitcnt_vm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

// f(integral_constant<int, I>) for I = B .. E-1, unrolled at compile time
template <int B, int E, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (B < E) {
    f(std::integral_constant<int, B>{});
    static_for<B + 1, E>(f);
  }
}

// Epilogues (after the optional per-row scale): bf16 store, bf16 store of
// (product + bf16 residual) rounded once, fp32 store, bf16 store of the tanh
// GELU of the product.
enum Epilogue { kEpiBf16 = 0, kEpiBf16Residual = 1, kEpiF32 = 2, kEpiBf16Gelu = 3 };

// 16 bytes per lane from base + voff + soff, a buffer resource over the
// nbytes bytes from base, straight into LDS at dst (the wave's 1 KB segment).
// Against 64-bit lane pointers this needs no per-load address arithmetic and
// half the registers; a load past nbytes reads zeros instead of faulting.
__device__ __forceinline__ void buffer_load_lds16(const void* base, unsigned nbytes, bf16* dst, unsigned voff,
                                                  unsigned soff) {
  const auto r = __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), 0, (int)nbytes, 0x00020000);
  __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)dst, 16, voff, soff, 0, 0);
}

// One tiling of the kernel: BM x BN output tile, K step BK (32 or 64),
// STAGES LDS stages (loads run STAGES-1 steps ahead), WAVES waves in a
// WM x (WAVES/WM) grid.
template <int BM_, int BN_, int BK_, int STAGES_, int WAVES_, int WM_>
struct Tiling {
  static constexpr int BM = BM_, BN = BN_, BK = BK_, STAGES = STAGES_, WAVES = WAVES_, WM = WM_;
  static constexpr int WN = WAVES / WM, THREADS = WAVES * 64;
  static constexpr int TM = BM / WM, TN = BN / WN;  // wave tile
  static constexpr int MI = TM / 32, NI = TN / 32;  // 32x32 MFMA tiles per wave
  static constexpr int CHUNKS = BK / 8;             // 16-byte chunks per tile row
  static constexpr int SEG_ROWS = 64 / CHUNKS;      // tile rows per 1 KB wave load
  static constexpr int SEG_A = BM / SEG_ROWS, SEG_B = BN / SEG_ROWS;
  static constexpr int LOADS = (SEG_A + SEG_B) / WAVES;  // load instructions per lane per stage
  static constexpr int STAGE = (BM + BN) * BK;           // bf16 elements per stage
  static_assert(BK == 32 || BK == 64, "K step");
  static_assert(LOADS * WAVES == SEG_A + SEG_B && SEG_A % WAVES == 0, "stage load must split evenly over waves");
  static_assert(MI * 32 == TM && NI * 32 == TN, "wave tile");
  static_assert(LOADS * (STAGES - 2 > 0 ? STAGES - 2 : 0) <= 63, "vmcnt range");
  static_assert(STAGES * STAGE * 2 <= 160 * 1024, "LDS");
  // 16-byte chunk c of tile row r sits at slot c ^ swz(r): any 16 consecutive
  // rows read at one chunk (one fragment read, 256 bytes per 16 lanes) land
  // on 16 distinct 16-byte bank groups
  static __device__ __forceinline__ int swz(int r) { return (r / (16 / CHUNKS)) % CHUNKS; }
};

// Output tile (tm, tn) of output z in tiling TL, staged through the
// workgroup's LDS arrays L0..L3 (at least TL::STAGE elements each, as many as
// TL has stages). Each stage is its own array, so that the compiler can tell
// the asynchronous loads into one stage from the fragment reads of another.
// BUF: stage loads through buffer resources (A and B each below 4 GiB), else
// through 64-bit lane pointers. ROPE: the RoPE epilogue is compiled in (the
// Q/K/V projection only).
template <class TL, int EPI, bool BUF, bool ROPE, class LA, class LB, class LC, class LD>
__device__ __forceinline__ void row_gemm_tile(const RowGemm& g, int tm, int tn, int z, LA& L0, LB& L1,
                                              LC& L2, LD& L3) {
  constexpr int BM = TL::BM, BN = TL::BN, BK = TL::BK, STAGES = TL::STAGES, WN = TL::WN;
  constexpr int TM = TL::TM, TN = TL::TN, MI = TL::MI, NI = TL::NI, LOADS = TL::LOADS;
  constexpr int SEG_A = TL::SEG_A, CHUNKS = TL::CHUNKS, SEG_ROWS = TL::SEG_ROWS;
  auto stage = [&](auto s) -> bf16* {
    if constexpr (decltype(s)::value == 0) return L0;
    else if constexpr (decltype(s)::value == 1) return L1;
    else if constexpr (decltype(s)::value == 2) return L2;
    else return L3;
  };
  static_assert(STAGES >= 2 && STAGES <= 4, "stages");
  const RowGemmOut oz = row_gemm_out(g, z);

  const bf16* __restrict__ A = static_cast<const bf16*>(g.A);
  const bf16* __restrict__ B = static_cast<const bf16*>(oz.B);

  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int l32 = lane & 31, hi = lane >> 5;

  // This lane's rows of the stage loads: segment s = i*WAVES + wave covers
  // tile rows SEG_ROWS*s .. (A tile first, then B tile); the lane fetches
  // row SEG_ROWS*s + lane/CHUNKS, global chunk (lane%CHUNKS) ^ swz(row),
  // into LDS slot lane%CHUNKS.
  const bf16* src[LOADS];  // !BUF: the lane's chunk of its row in A or B
  unsigned voff[LOADS];    // BUF: the same as a byte offset from A or B
  int dst[LOADS];          // element offset of the segment in its stage
#pragma unroll
  for (int i = 0; i < LOADS; ++i) {
    const int s = i * TL::WAVES + wave;
    const bool a = s < SEG_A;
    const int trow = (a ? s : s - SEG_A) * SEG_ROWS + lane / CHUNKS;
    const int chunk = (lane % CHUNKS) ^ TL::swz(trow);
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
    if constexpr (BUF)
      voff[i] = (unsigned)((grow + chunk * 8) * 2);
    else
      src[i] = (a ? A : B) + grow + chunk * 8;
    dst[i] = s * 512;  // the B tile follows the A tile in the stage
  }
  // segment i of every wave lies in A when i * WAVES < SEG_A (SEG_A is a
  // multiple of WAVES), so the resource of a load is known at compile time
  const unsigned a_bytes = (unsigned)((long)g.a_limit * g.lda * 2), b_bytes = (unsigned)((long)g.Nc * g.ldb * 2);
  auto issue = [&](auto st, int k0) -> void {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      if constexpr (BUF) {
        if (i * TL::WAVES < SEG_A)
          buffer_load_lds16(A, a_bytes, stage(st) + dst[i], voff[i], (unsigned)(k0 * 2));
        else
          buffer_load_lds16(B, b_bytes, stage(st) + dst[i], voff[i], (unsigned)(k0 * 2));
      } else {
        __builtin_amdgcn_global_load_lds((global_cvoid*)(src[i] + k0), (lds_void*)(stage(st) + dst[i]), 16, 0, 0);
      }
    }
  };

  // fragment read offsets: row (tile-local) l32 + 32*t, chunk kk*2 + hi;
  // swz(l32 + 32 t) = swz(l32)
  const int xr = ((hi ^ TL::swz(l32)) * 8);
  f32x16 acc[MI][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i)
#pragma unroll
    for (int j = 0; j < NI; ++j) acc[i][j] = (f32x16){};

  // Fragments live in two register buffers: slice kk of a stage goes to
  // buffer kk & 1, so a stage's last slice is in buffer 1. The MFMAs of its
  // last DEF fragment rows are deferred to the start of the next stage's
  // compute, behind the barrier: they need registers only, and they keep the
  // matrix pipe busy while the next stage's first fragment reads are in
  // flight (otherwise every wave waits for them right after the barrier).
  // DEF is all rows, except at four row tiles per wave with 64-bit lane
  // pointers for the loads: there only half of them fit in 256 registers
  // (the buffer-resource loads free the registers for all of them: 1.6-2.5%
  // faster). Buffer 1 starts at zero, so the first stage's deferred MFMAs add
  // exact zeros.
  bf16x8 af[2][MI], bfr[2][NI];
#pragma unroll
  for (int i = 0; i < MI; ++i) af[1][i] = (bf16x8){};
#pragma unroll
  for (int j = 0; j < NI; ++j) bfr[1][j] = (bf16x8){};
  constexpr int DEF = (MI <= 2 || BUF) ? MI : MI / 2;
  // the MFMAs of fragment rows i0 .. i1-1 of buffer b
  auto mfmas = [&](auto bc, auto i0c, auto i1c) {
    constexpr int b = decltype(bc)::value, i0 = decltype(i0c)::value, i1 = decltype(i1c)::value;
#pragma unroll
    for (int i = i0; i < i1; ++i)
#pragma unroll
      for (int j = 0; j < NI; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[b][j], af[b][i], acc[i][j], 0, 0, 0);
  };
  auto compute = [&](auto st, auto lg) {
    constexpr int LG = decltype(lg)::value, KS = BK / 16, R = MI + NI, M = MI * NI;
    static_assert(M >= R, "one MFMA per fragment read at least");
    static_assert(KS % 2 == 0, "the last slice of a stage is in buffer 1");
    const bf16* As = stage(st) + (wm * TM + l32) * BK;
    const bf16* Bs = stage(st) + BM * BK + (wn * TN + l32) * BK;
    auto ld = [&](int kk, int b) {
      const int off = (kk * 16) ^ xr;
#pragma unroll
      for (int i = 0; i < MI; ++i) af[b][i] = *reinterpret_cast<const bf16x8*>(As + i * 32 * BK + off);
#pragma unroll
      for (int j = 0; j < NI; ++j) bfr[b][j] = *reinterpret_cast<const bf16x8*>(Bs + j * 32 * BK + off);
    };
    ld(0, 0);
    // the previous stage's deferred rows, then this stage's slices 0 .. KS-2
    // with the reads of each next slice and the stage loads between the MFMAs
    mfmas(std::integral_constant<int, 1>{}, std::integral_constant<int, MI - DEF>{},
          std::integral_constant<int, MI>{});
    __builtin_amdgcn_sched_group_barrier(0x100, R, 0);
    static_for<0, DEF * NI>([&](auto mc) {
      constexpr int m = decltype(mc)::value;
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      if constexpr (m < LG) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
    });
    static_for<0, KS - 1>([&](auto kc) {
      constexpr int kk = decltype(kc)::value;
      ld(kk + 1, (kk + 1) & 1);
      mfmas(std::integral_constant<int, kk & 1>{}, std::integral_constant<int, 0>{},
            std::integral_constant<int, MI>{});
      static_for<0, M>([&](auto mc) {
        constexpr int m = decltype(mc)::value;
        __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        if constexpr (m < R) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
        if constexpr (DEF * NI + kk * M + m < LG) __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);
      });
    });
    // slice KS-1: the rows before the deferred ones
    mfmas(std::integral_constant<int, 1>{}, std::integral_constant<int, 0>{},
          std::integral_constant<int, MI - DEF>{});
    static_for<0, (MI - DEF) * NI>([&](auto mc) { __builtin_amdgcn_sched_group_barrier(0x008, 1, 0); });
  };

  using S0 = std::integral_constant<int, 0>;
  using S1 = std::integral_constant<int, 1>;
  using S2 = std::integral_constant<int, 2 % STAGES>;
  using S3 = std::integral_constant<int, 3 % STAGES>;
  using Interleave = std::integral_constant<int, LOADS>;
  using NoLoads = std::integral_constant<int, 0>;
  const int nk = g.K / BK;
  // prologue: steps 0 .. STAGES-2 in flight
  issue(S0{}, 0);
  if constexpr (STAGES > 2) if (1 < nk) issue(S1{}, BK);
  if constexpr (STAGES > 3) if (2 < nk) issue(S2{}, 2 * BK);
  // step k lives in stage k % STAGES: wait for its loads (the loads of the
  // up to STAGES-2 later steps may stay in flight; loads complete in order),
  // make them visible to all waves (which also frees stage (k-1) % STAGES),
  // start step k+STAGES-1's loads into that stage, compute step k. In the
  // steady state (full) the loads are unconditional and share the scheduling
  // region of the MFMAs; near the end of K they are conditional.
  auto step = [&](auto st, auto nxt, int k, auto full) {
    if (STAGES > 2 && k + STAGES - 2 < nk) __builtin_amdgcn_s_waitcnt(waitcnt_vm(LOADS * (STAGES > 2 ? STAGES - 2 : 0)));
    else __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();
    if constexpr (decltype(full)::value) {
      issue(nxt, (k + STAGES - 1) * BK);
      compute(st, Interleave{});
    } else {
      if (k + STAGES - 1 < nk) issue(nxt, (k + STAGES - 1) * BK);
      compute(st, NoLoads{});
    }
  };
  // nxt = (k + STAGES - 1) % STAGES = (k - 1) % STAGES. Whole rounds of
  // STAGES steps whose loads all fall inside K run in the loop, the remaining
  // steps after it, so that the loop body has no conditional step (the
  // accumulators stay in place).
  auto round = [&](int k, int n, auto full) __attribute__((always_inline)) {
    if constexpr (STAGES == 2) {
      step(S0{}, S1{}, k, full);
      if (n > 1) step(S1{}, S0{}, k + 1, full);
    } else if constexpr (STAGES == 3) {
      step(S0{}, S2{}, k, full);
      if (n > 1) step(S1{}, S0{}, k + 1, full);
      if (n > 2) step(S2{}, S1{}, k + 2, full);
    } else {
      step(S0{}, S3{}, k, full);
      if (n > 1) step(S1{}, S0{}, k + 1, full);
      if (n > 2) step(S2{}, S1{}, k + 2, full);
      if (n > 3) step(S3{}, S2{}, k + 3, full);
    }
  };
  int k = 0;
  for (; k + 2 * STAGES - 1 <= nk; k += STAGES) round(k, STAGES, std::true_type{});
  for (; k < nk; k += STAGES) round(k, min(STAGES, nk - k), std::false_type{});
  mfmas(std::integral_constant<int, 1>{}, std::integral_constant<int, MI - DEF>{},
        std::integral_constant<int, MI>{});  // the last stage's deferred rows

  // Epilogue through LDS. acc[i][j][e] is output row (tile row + i*32 + l32),
  // column (tile col + j*32 + (e/4)*8 + hi*4 + e%4): a lane holds 4 columns
  // of one row, so direct stores would write 16-byte pieces of 32 rows per
  // instruction. Instead, for each 32-row block i, every wave writes its
  // fp32 values (row scale, RoPE and GELU applied) to its own LDS region,
  // then reads them back row-contiguous, 4 columns per lane (the residual is
  // added there, then the value rounded once), and stores runs of 4 columns
  // per lane, 128 bytes or more per row. Waves 0-3 use the first stage's
  // array, 4-7 the second; the scatter target of each row travels through
  // LDS too. Every global load of the epilogue (row indices, row scales,
  // RoPE positions and angles, residuals) precedes its first store: the
  // results of all blocks are held in registers and stored after the last
  // one. A wave waits for a load by counting its outstanding memory
  // accesses, stores included, so a load behind a store would also wait for
  // that store (measured: the output projection 2-9% faster this way).
  constexpr int TNP = TN + 4;         // padded staging row, floats
  constexpr int QPR = TN / 4;         // 4-column groups per row
  constexpr int NT = QPR / 2;         // read-back passes of the wave per block
  constexpr int REGION = 32 * TNP * 4 + MI * 32 * (8 + 4);
  static_assert(4 * REGION <= TL::STAGE * 2, "epilogue staging must fit in a stage");
  static_assert(QPR % 2 == 0, "the wave covers whole rows in each read-back pass");
  __syncthreads();  // every wave is done with the stages
  char* region = reinterpret_cast<char*>((wave < 4) ? L0 : L1) + (wave % 4) * REGION;
  float* blk = reinterpret_cast<float*>(region);
  // per block i, row r: output element offset and target (0: C, 1: C2, -1: none)
  long* row_off = reinterpret_cast<long*>(region + 32 * TNP * 4);
  int* row_buf = reinterpret_cast<int*>(region + 32 * TNP * 4 + MI * 32 * 8);
  const int32_t* c_rows = oz.c_rows;
  const bool rope = ROPE && g.rope_cs && ((g.rope_outs >> z) & 1);
  const int col0 = tn * BN + wn * TN;  // first output column of the wave tile
  const int m0 = tm * BM + wm * TM + l32;  // the lane's row in block 0
  int crow[MI];
  float rs[MI];
  RopeRow rr[MI];
  // Loads under a lane condition would each be waited for inside their
  // branch, one after the other: every load here and below reads a valid
  // address unconditionally (row M-1 for the rows past M) and its value is
  // selected afterwards.
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    const int m = m0 + i * 32;
    const int mc = min(m, g.M - 1);
    const int cr = c_rows ? c_rows[mc] : m;
    crow[i] = m < g.M ? cr : -1;
    rs[i] = g.row_scale ? g.row_scale[mc] : 1.f;
    rr[i] = RopeRow{0, 0, 0};
    if (rope) rr[i] = rope_row(g, mc);
  }
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    int buf = -1;
    long obase = 0;
    if (crow[i] >= 0 && crow[i] < oz.c_limit) {
      const bool second = oz.C2 && crow[i] >= oz.c_split;  // rows past the split go to C2
      buf = second ? 1 : 0;
      obase = (long)(second ? crow[i] - oz.c_split : crow[i]) * g.ldc;
    }
    if (hi == 0) {
      row_off[i * 32 + l32] = obase;
      row_buf[i * 32 + l32] = buf;
    }
  }
  __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");  // the row tables are visible
  typedef typename std::conditional<EPI == kEpiF32, f32x4, bf16x4>::type OutT;
  OutT ov[MI][NT];  // block i, read-back pass t: the lane's 4 output values
#pragma unroll
  for (int i = 0; i < MI; ++i) {
    if constexpr (EPI == kEpiBf16Residual) {  // the residual first takes the output's place
      __builtin_amdgcn_sched_barrier(0);  // one block's residuals at a time (registers)
      bool in[NT];
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        const int f = lane + 64 * t;
        const int r = f / QPR, cq = f - r * QPR;
        const int n = col0 + cq * 4;
        in[t] = row_buf[i * 32 + r] >= 0 && n < g.Nc;
        // element 0 of the residual exists: the launcher runs no residual
        // product without output rows
        ov[i][t] = *reinterpret_cast<const bf16x4*>(static_cast<const bf16*>(g.residual) +
                                                    (in[t] ? row_off[i * 32 + r] + n : 0));
      }
      // an empty asm that uses every value keeps the loads unconditional (the
      // compiler would otherwise move each into a branch of its own)
#pragma unroll
      for (int t = 0; t < NT; ++t) {
        asm volatile("" : "+v"(ov[i][t]));
        if (!in[t]) ov[i][t] = (bf16x4){};
      }
    }
    // the block's RoPE angles, all loaded before any is used (every index is
    // in the table, so the loads need no condition)
    f32x2 cs[NI][4][2];
    if (rope) {
#pragma unroll
      for (int j = 0; j < NI; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int k = ((col0 + j * 32 + q * 8 + hi * 4) % g.rope_dh) >> 1;
          cs[j][q][0] = rope_angle(g, rr[i], k);
          cs[j][q][1] = rope_angle(g, rr[i], k + 1);
        }
    }
#pragma unroll
    for (int j = 0; j < NI; ++j) {
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int c = j * 32 + q * 8 + hi * 4;
        f32x4 v = {acc[i][j][4 * q + 0], acc[i][j][4 * q + 1], acc[i][j][4 * q + 2], acc[i][j][4 * q + 3]};
        if (g.row_scale) v *= rs[i];
        if (rope) {
          const f32x2 r0 = rope_rotate(cs[j][q][0], v[0], v[1]);
          const f32x2 r1 = rope_rotate(cs[j][q][1], v[2], v[3]);
          v = (f32x4){r0[0], r0[1], r1[0], r1[1]};
        }
        if constexpr (EPI == kEpiBf16Gelu) {
#pragma unroll
          for (int u = 0; u < 4; ++u) v[u] = gelu_tanh(v[u]);
        }
        *reinterpret_cast<f32x4*>(blk + l32 * TNP + c) = v;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");
    // row-contiguous read-back: 4 columns per lane, QPR lanes per row
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int f = lane + 64 * t;
      const int r = f / QPR, cq = f - r * QPR;
      f32x4 v = *reinterpret_cast<const f32x4*>(blk + r * TNP + cq * 4);
      if constexpr (EPI == kEpiF32) {
        ov[i][t] = v;
      } else {
        if constexpr (EPI == kEpiBf16Residual) v += __builtin_convertvector(ov[i][t], f32x4);
        ov[i][t] = to_bf16x4(v);
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_SEQ_CST, "wavefront");  // reads done before the next block's writes
  }
  // the stores read their targets from the row tables again (a compiler-only
  // barrier): kept from the residual loads, 64-bit offsets would fill 64
  // registers and spill
  asm volatile("" ::: "memory");
#pragma unroll
  for (int i = 0; i < MI; ++i) {
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      const int f = lane + 64 * t;
      const int r = f / QPR, cq = f - r * QPR;
      const int rb = row_buf[i * 32 + r];
      const int n = col0 + cq * 4;
      if (rb < 0 || n >= g.Nc) continue;
      const long o = row_off[i * 32 + r] + n;
      *reinterpret_cast<OutT*>(static_cast<typename std::conditional<EPI == kEpiF32, float, bf16>::type*>(
          rb ? oz.C2 : oz.C) + o) = ov[i][t];
    }
  }
}

// The three tilings of 8 waves (see launch_best); a 256 x 256 tile splits
// into two 256 x 128 halves.
using TBig = Tiling<256, 256, 64, 2, 8, 2>;
using T192 = Tiling<256, 192, 64, 2, 8, 4>;
using TMid = Tiling<256, 128, 64, 2, 8, 4>;

// NOUT (1 or 3) is the number of outputs sharing A; it is a template
// parameter so the Q/K/V projection and the output projection are distinct
// kernels in profiles. Workgroup b takes tile item xcd_contiguous(b, tiles):
// tiles are ordered in groups of g.group_m tile-rows that sweep all tile-columns
// (of all outputs) together, and each XCD runs a contiguous range of items.
// With the 256 x 256 tiling, the workgroups from g.split_from on take halves:
// workgroups split_from + 2j and split_from + 2j + 1 compute the two 256 x 128
// halves of the tile workgroup split_from + j would have taken. The launcher
// sets split_from so that a last, partly filled round of big tiles becomes
// one round of halves.
template <class TL, int NOUT, int EPI, bool BUF>
__global__ __launch_bounds__(TL::THREADS) void row_gemm_bf16_kernel(RowGemm g) {
  constexpr int STAGES = TL::STAGES;
  constexpr bool kSplit = std::is_same<TL, TBig>::value;
  static_assert(!kSplit || (TMid::STAGE <= TL::STAGE && TMid::THREADS == TL::THREADS), "halves");
  __shared__ __attribute__((aligned(16))) bf16 L0[TL::STAGE];
  __shared__ __attribute__((aligned(16))) bf16 L1[TL::STAGE];
  __shared__ __attribute__((aligned(16))) bf16 L2[STAGES > 2 ? TL::STAGE : 1];
  __shared__ __attribute__((aligned(16))) bf16 L3[STAGES > 3 ? TL::STAGE : 1];

  const int tiles_m = (g.M + TL::BM - 1) / TL::BM;
  const int tiles_n1 = (g.Nc + TL::BN - 1) / TL::BN;  // per output
  const int tiles_n = tiles_n1 * NOUT;                 // over all outputs side by side
  const int total = tiles_m * tiles_n;
  int b = blockIdx.x, half = -1;
  if constexpr (kSplit) {
    if (b >= g.split_from) {
      half = (b - g.split_from) & 1;
      b = g.split_from + (b - g.split_from) / 2;
    }
  }
  const int item = xcd_contiguous(b, total);
  const int group = item / (g.group_m * tiles_n);
  const int first_m = group * g.group_m;
  const int gm = min(g.group_m, tiles_m - first_m);
  const int r = item - group * g.group_m * tiles_n;
  const int tm = first_m + r % gm;
  const int tnc = r / gm;
  const int z = tnc / tiles_n1;
  const int tn = tnc - z * tiles_n1;
  if constexpr (kSplit) {
    if (half >= 0) {
      row_gemm_tile<TMid, EPI, BUF, NOUT == 3>(g, tm, tn * 2 + half, z, L0, L1, L2, L3);
      return;
    }
  }
  row_gemm_tile<TL, EPI, BUF, NOUT == 3>(g, tm, tn, z, L0, L1, L2, L3);
}

// Rounds of a launch of `tiles` tiles on the CUs, in units of a full round
// of this tiling: with the 256 x 256 tiling, a last round at most half full
// is run as halves and costs a round of 256 x 128 tiles (kHalfRound).
constexpr double kHalfRound = 0.675;
template <class TL>
bool split_tail(long tiles) {
  const long cus = compute_units(), rem = tiles % cus;
  return std::is_same<TL, TBig>::value && tiles > cus && rem > 0 && 2 * rem <= cus;
}
template <class TL>
double rounds(long tiles) {
  const long cus = compute_units();
  return split_tail<TL>(tiles) ? (double)(tiles / cus) + kHalfRound : (double)((tiles + cus - 1) / cus);
}

template <class TL, int NOUT, int EPI>
hipError_t launch(const RowGemm& g0, hipStream_t s) {
  const long tiles = (long)((g0.M + TL::BM - 1) / TL::BM) * ((g0.Nc + TL::BN - 1) / TL::BN) * NOUT;
  RowGemm g = g0;
  // tile-row groups: 8, or 4 for outputs of 32 or more tile-columns (the FFN
  // up projection at 8960 columns: 7% faster at 32760 rows, neutral at 8190)
  g.group_m = (g0.Nc + TL::BN - 1) / TL::BN >= 32 ? 4 : 8;
  g.split_from = 0x7fffffff;
  long grid = tiles;
  if (split_tail<TL>(tiles)) {
    const long rem = tiles % compute_units();
    g.split_from = (int)(tiles - rem);
    grid = tiles + rem;
  }
  // buffer resources address 4 GiB - 1 bytes from their base (32-bit offsets)
  const long lim = 0xffffffffL;
  if ((long)g.a_limit * g.lda * 2 <= lim && (long)g.Nc * g.ldb * 2 <= lim)
    hipLaunchKernelGGL((row_gemm_bf16_kernel<TL, NOUT, EPI, true>), dim3((unsigned)grid), dim3(TL::THREADS), 0, s, g);
  else
    hipLaunchKernelGGL((row_gemm_bf16_kernel<TL, NOUT, EPI, false>), dim3((unsigned)grid), dim3(TL::THREADS), 0, s, g);
  return hipGetLastError();
}

// Three tilings of 8 waves. Per FLOP 256 x 256 (waves of 128 x 64) is the
// fastest; 256 x 192 (waves of 64 x 96) costs about 1.14x and 256 x 128
// (waves of 64 x 64) about 1.35x (measured on the stack shapes), but their
// finer grids can fill the last round of a launch better. Each launch takes
// the tiling with the least estimated time, rounds x cost per round, with
// rounds as counted by rounds() (ceil(tiles / CUs), or the split tail of
// 256 x 256) and the per-round cost relative to 256 x 256 (tile area x cost
// per FLOP): 1, 0.855, 0.675. A tiling other than 256 x 256 must win by 3%.
// The narrow fp32 velocity head always takes 256 x 128.
template <class TL>
double estimate(const RowGemm& g, double per_round) {
  const long tiles = (long)((g.M + TL::BM - 1) / TL::BM) * ((g.Nc + TL::BN - 1) / TL::BN) * g.n_out;
  return rounds<TL>(tiles) * per_round;
}

template <int NOUT, int EPI>
hipError_t launch_best(const RowGemm& g, hipStream_t s) {
  const double eb = estimate<TBig>(g, 1.0), e192 = estimate<T192>(g, 0.855),
               em = estimate<TMid>(g, kHalfRound);
  if (e192 < 0.97 * eb && e192 <= em) return launch<T192, NOUT, EPI>(g, s);
  if (em < 0.97 * eb && em < e192) return launch<TMid, NOUT, EPI>(g, s);
  return launch<TBig, NOUT, EPI>(g, s);
}

}  // namespace

hipError_t launch_row_gemm_bf16(const RowGemm& g, hipStream_t s) {
  if (g.M <= 0 || g.Nc <= 0 || (g.n_out != 1 && g.n_out != 3)) return hipSuccess;
  if (g.K % TBig::BK || g.K % T192::BK || g.K % TMid::BK) return hipErrorInvalidValue;
  if (g.rope_cs && g.rope_outs && g.n_out != 3) return hipErrorInvalidValue;  // RoPE: Q/K/V only
  if (g.residual && g.out[0].c_limit <= 0) return hipSuccess;  // no output row
  if (g.n_out == 3) return launch_best<3, kEpiBf16>(g, s);
  if (g.c_f32) return launch<TMid, 1, kEpiF32>(g, s);
  if (g.gelu) return launch_best<1, kEpiBf16Gelu>(g, s);
  if (g.residual) return launch_best<1, kEpiBf16Residual>(g, s);
  return launch_best<1, kEpiBf16>(g, s);
}

}  // namespace hsa
