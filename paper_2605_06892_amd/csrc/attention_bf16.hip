// bf16 active-query attention on CDNA4 matrix cores (Section 2.3, step 3):
// for every active row j and head h, o[j,h] = softmax(scale q[j,h] K_h^T) V_h
// over all N cached rows. Cost O(|A_i| N d) instead of O(N^2 d).
//
// Work split: one workgroup of NW waves per (head, tile of NW*32*QT active
// queries); each wave owns 32*QT queries. Workgroups of one head are placed
// contiguously on one XCD so concurrently running query tiles stream the same
// K/V rows through that XCD's L2.
//
// Per key tile of 64 cached rows (double-buffered in LDS, the next tile's
// global loads in flight during the current tile's math):
//   S^T = K Q^T - m   v_mfma_f32_32x32x16_bf16 with K rows as the A operand
//                 straight from LDS and the wave's Q fragments resident in
//                 VGPRs as the B operand. Q is pre-multiplied by
//                 scale*log2(e) and the accumulator is seeded (C operand, not
//                 written) with -m, m the wave's reference maximum in log2
//                 units, so each score leaves the MFMA ready for exp2. Each
//                 lane holds 16 scores of ONE query (column l%32) over 32
//                 keys shared with lane l^32.
//   softmax       the fast path is exp2, a running sum and the bf16 pack per
//                 score. The reference maximum m is set from the first 32
//                 keys and only raised (rescaling O and the sum) when some
//                 probability of a 32-key block exceeds 2^16, detected from
//                 the block's sum: a wave-uniform branch that is almost never
//                 taken. Probabilities therefore stay below 2^16 and the sum
//                 at or above 1.
//   O^T += V^T P^T  the probabilities, rounded to bf16, are the B operand as
//                 they sit in the S^T accumulators; the contraction slot
//                 (hi*8 + e) of each 16-key step maps to key (e/4)*8 + hi*4 +
//                 e%4. The V^T operand is read from the row-major LDS tile
//                 with ds_read_b64_tr_b16 (gfx950 LDS transpose read): in each
//                 16-lane group, lane i points at 4 consecutive channels of
//                 key row i/4, and lane L receives one channel of 4 keys. The
//                 V tile row stride is an odd multiple of 16 dwords so the
//                 eight key rows one read touches fall on disjoint banks.
//   Every lane owns one query column in both S^T and O^T, so the softmax
//   statistics never need to be broadcast across lanes.
#include "common.h"

namespace hsa {
namespace {

constexpr int BKV = 64;                 // cached rows per LDS tile
constexpr float kSlowSum = 65536.0f;    // 2^16: raise the reference maximum

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;

template <int DH, int QT, int NW>
__global__ __launch_bounds__(NW * 64) void attention_bf16_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ kc, const bf16* __restrict__ vc,
    bf16* __restrict__ o, int n_q, int n_kv, int d, float sl2e, int n_qtiles, int heads) {
  constexpr int NT = NW * 64;        // threads
  constexpr int BQ = NW * 32 * QT;   // queries per workgroup
  constexpr int KS = DH + 8;         // K tile row stride in bf16 (68 dwords for DH=128)
  constexpr int VS = DH == 128 ? 160 : 96;  // V tile row stride: 80 / 48 dwords
  constexpr int CPR = DH / 8;        // 16-byte chunks per cached row
  constexpr int LOADS = BKV * CPR / NT;
  constexpr int DT = DH / 32;        // 32-wide head-dim tiles of O^T
  constexpr int KK = DH / 16;        // k-steps of S^T
  static_assert(LOADS * NT == BKV * CPR, "tile load must split evenly");
  __shared__ __attribute__((aligned(16))) bf16 Ks[2][BKV * KS];
  __shared__ __attribute__((aligned(16))) bf16 Vs[2][BKV * VS];

  const int item = xcd_contiguous(blockIdx.x, n_qtiles * heads);
  const int h = item / n_qtiles;
  const int qt = item - h * n_qtiles;
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int l32 = lane & 31, hi = lane >> 5;
  const long col0 = (long)h * DH;

  // Q fragments, pre-scaled by scale*log2(e): lane holds
  // Q[query l32 of sub-tile tq][kk*16 + hi*8 + 0..7]
  bf16x8 qf[QT][KK];
#pragma unroll
  for (int tq = 0; tq < QT; ++tq) {
    const int qrow = qt * BQ + wave * 32 * QT + tq * 32 + l32;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      bf16x8 raw = (bf16x8){};
      if (qrow < n_q)
        raw = *reinterpret_cast<const bf16x8*>(q + (long)qrow * d + col0 + kk * 16 + hi * 8);
      f32x4 lo = {(float)raw[0] * sl2e, (float)raw[1] * sl2e, (float)raw[2] * sl2e, (float)raw[3] * sl2e};
      f32x4 up = {(float)raw[4] * sl2e, (float)raw[5] * sl2e, (float)raw[6] * sl2e, (float)raw[7] * sl2e};
      qf[tq][kk] = __builtin_shufflevector(to_bf16x4(lo), to_bf16x4(up), 0, 1, 2, 3, 4, 5, 6, 7);
    }
  }

  u32x4 rk[LOADS], rv[LOADS];
  auto gload = [&](int kv0) {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int id = t + NT * i;
      const int row = id / CPR, cc = id % CPR;
      const int n = kv0 + row;
      if (n < n_kv) {
        const long off = (long)n * d + col0 + cc * 8;
        rk[i] = *reinterpret_cast<const u32x4*>(kc + off);
        rv[i] = *reinterpret_cast<const u32x4*>(vc + off);
      } else {
        rk[i] = (u32x4){0u, 0u, 0u, 0u};
        rv[i] = (u32x4){0u, 0u, 0u, 0u};
      }
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int id = t + NT * i;
      const int row = id / CPR, cc = id % CPR;
      *reinterpret_cast<u32x4*>(&Ks[buf][row * KS + cc * 8]) = rk[i];
      *reinterpret_cast<u32x4*>(&Vs[buf][row * VS + cc * 8]) = rv[i];
    }
  };

  // transpose-read source of this lane inside a 16-key step (see header)
  const int v_lane = (hi * 4 + ((lane & 15) >> 2)) * VS + 16 * ((lane >> 4) & 1) + 4 * (lane & 3);
  const int k_lane = l32 * KS + hi * 8;

  f32x16 acc[QT][DT];
  f32x16 negm[QT];  // every element -m_ref: the seed of the score accumulators
  float m_ref[QT], l_run[QT];
#pragma unroll
  for (int tq = 0; tq < QT; ++tq) {
    m_ref[tq] = 0.f;
    l_run[tq] = 0.f;
    negm[tq] = (f32x16){};
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[tq][dt] = (f32x16){};
  }
  bool have_ref = false;  // becomes true after the first 32 keys (wave-uniform)

  const int n_tiles = (n_kv + BKV - 1) / BKV;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int it = 0; it < n_tiles; ++it) {
    const int buf = it & 1;
    const int kv0 = it * BKV;
    if (it + 1 < n_tiles) gload(kv0 + BKV);
    const bf16* Kt = Ks[buf];
    const bf16* Vt = Vs[buf];
#pragma unroll
    for (int sb = 0; sb < BKV / 32; ++sb) {
      f32x16 s[QT];
      {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Kt[sb * 32 * KS + k_lane]);
#pragma unroll
        for (int tq = 0; tq < QT; ++tq)
          s[tq] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[tq][0], negm[tq], 0, 0, 0);
      }
#pragma unroll
      for (int kk = 1; kk < KK; ++kk) {
        const bf16x8 kf = *reinterpret_cast<const bf16x8*>(&Kt[sb * 32 * KS + k_lane + kk * 16]);
#pragma unroll
        for (int tq = 0; tq < QT; ++tq)
          s[tq] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[tq][kk], s[tq], 0, 0, 0);
      }
      // s[tq][e] = scaled score of key kv0 + sb*32 + (e/4)*8 + hi*4 + e%4, minus m_ref
      if (kv0 + sb * 32 + 32 > n_kv) {
        const int key0 = kv0 + sb * 32 + hi * 4;
#pragma unroll
        for (int tq = 0; tq < QT; ++tq)
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (key0 + (e >> 2) * 8 + (e & 3) >= n_kv) s[tq][e] = -INFINITY;
      }
      bf16x8 pf[QT][2];
      float p[QT][16];
      float ls[QT];
      bool slow = !have_ref;
#pragma unroll
      for (int tq = 0; tq < QT; ++tq) {
        ls[tq] = 0.f;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          p[tq][e] = __builtin_amdgcn_exp2f(s[tq][e]);
          ls[tq] += p[tq][e];
        }
        slow |= !(ls[tq] <= kSlowSum);
      }
      if (__any(slow)) {
        // set or raise the reference maximum, rescale what was accumulated
#pragma unroll
        for (int tq = 0; tq < QT; ++tq) {
          float mx = s[tq][0];
#pragma unroll
          for (int e = 1; e < 16; ++e) mx = fmaxf(mx, s[tq][e]);
          mx = fmaxf(mx, __shfl_xor(mx, 32));            // block max relative to m_ref
          const float up = have_ref ? fmaxf(mx, 0.f) : mx;  // amount to raise m_ref by
          const float alpha = have_ref ? __builtin_amdgcn_exp2f(-up) : 0.f;
          ls[tq] = 0.f;
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            p[tq][e] = __builtin_amdgcn_exp2f(s[tq][e] - up);
            ls[tq] += p[tq][e];
          }
          l_run[tq] *= alpha;
#pragma unroll
          for (int dt = 0; dt < DT; ++dt) acc[tq][dt] *= alpha;
          m_ref[tq] += up;
#pragma unroll
          for (int e = 0; e < 16; ++e) negm[tq][e] = -m_ref[tq];
        }
        have_ref = true;
      }
#pragma unroll
      for (int tq = 0; tq < QT; ++tq) {
        l_run[tq] += ls[tq];
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          f32x4 lo = {p[tq][8 * half + 0], p[tq][8 * half + 1], p[tq][8 * half + 2], p[tq][8 * half + 3]};
          f32x4 up = {p[tq][8 * half + 4], p[tq][8 * half + 5], p[tq][8 * half + 6], p[tq][8 * half + 7]};
          pf[tq][half] = __builtin_shufflevector(to_bf16x4(lo), to_bf16x4(up), 0, 1, 2, 3, 4, 5, 6, 7);
        }
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          const bf16* vb = Vt + (sb * 32 + ks * 16) * VS + dt * 32 + v_lane;
          const bf16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vb));
          const bf16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(vb + 8 * VS));
          const bf16x8 vf = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
          for (int tq = 0; tq < QT; ++tq)
            acc[tq][dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[tq][ks], acc[tq][dt], 0, 0, 0);
        }
      }
    }
    if (it + 1 < n_tiles) lstore(buf ^ 1);
    __syncthreads();
  }

  // acc[tq][dt][e]: channel dt*32 + (e/4)*8 + hi*4 + e%4 of query l32
#pragma unroll
  for (int tq = 0; tq < QT; ++tq) {
    const float l_tot = l_run[tq] + __shfl_xor(l_run[tq], 32);
    const float inv = 1.f / l_tot;
    const int qrow = qt * BQ + wave * 32 * QT + tq * 32 + l32;
    if (qrow >= n_q) continue;
    bf16* dst = o + (long)qrow * d + col0;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 v = {acc[tq][dt][4 * g + 0] * inv, acc[tq][dt][4 * g + 1] * inv,
                   acc[tq][dt][4 * g + 2] * inv, acc[tq][dt][4 * g + 3] * inv};
        *reinterpret_cast<bf16x4*>(dst + dt * 32 + g * 8 + hi * 4) = to_bf16x4(v);
      }
    }
  }
}

template <int DH, int QT, int NW>
hipError_t launch_cfg(const void* q, const void* k, const void* v, void* o, int n_q, int n_kv,
                      int heads, float sl2e, hipStream_t s) {
  constexpr int BQ = NW * 32 * QT;
  const int n_qtiles = (n_q + BQ - 1) / BQ;
  const int d = heads * DH;
  hipLaunchKernelGGL((attention_bf16_kernel<DH, QT, NW>), dim3((unsigned)(n_qtiles * heads)),
                     dim3(NW * 64), 0, s, static_cast<const bf16*>(q),
                     static_cast<const bf16*>(k), static_cast<const bf16*>(v),
                     static_cast<bf16*>(o), n_q, n_kv, d, sl2e, n_qtiles, heads);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_bf16(const void* q, const void* k, const void* v, void* o, int n_q,
                                 int n_kv, int heads, int head_dim, float scale, hipStream_t s) {
  if (n_q <= 0) return hipSuccess;
  const float sl2e = scale * 1.4426950408889634f;
  // Workgroup shape: 8 waves x 32 queries (two waves per SIMD, so one wave's
  // softmax overlaps the other's MFMAs) whenever that still gives every CU a
  // workgroup; 4 waves x 32 queries for small problems. HSA_ATTN_CFG (1, 2, 3)
  // forces a shape for measurement sweeps.
  static const int forced = [] {
    const char* e = getenv("HSA_ATTN_CFG");
    return e ? atoi(e) : 0;
  }();
  int cfg = forced;
  if (cfg < 1 || cfg > 3) cfg = ((long)((n_q + 255) / 256) * heads >= 256) ? 3 : 1;
  if (head_dim == 64) {
    switch (cfg) {
      case 2: return launch_cfg<64, 2, 4>(q, k, v, o, n_q, n_kv, heads, sl2e, s);
      case 3: return launch_cfg<64, 1, 8>(q, k, v, o, n_q, n_kv, heads, sl2e, s);
      default: return launch_cfg<64, 1, 4>(q, k, v, o, n_q, n_kv, heads, sl2e, s);
    }
  }
  switch (cfg) {
    case 2: return launch_cfg<128, 2, 4>(q, k, v, o, n_q, n_kv, heads, sl2e, s);
    case 3: return launch_cfg<128, 1, 8>(q, k, v, o, n_q, n_kv, heads, sl2e, s);
    default: return launch_cfg<128, 1, 4>(q, k, v, o, n_q, n_kv, heads, sl2e, s);
  }
}

}  // namespace hsa
