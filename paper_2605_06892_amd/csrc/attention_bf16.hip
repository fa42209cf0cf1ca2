// bf16 active-query attention on CDNA4 matrix cores (Section 2.3, step 3):
// for every active row j and head h, o[j,h] = softmax(scale q[j,h] K_h^T) V_h
// over all N cached rows. Cost O(|A_i| N d) instead of O(N^2 d).
//
// Work split: one 256-thread workgroup (4 waves) per (head, tile of 128*QT
// active queries); each wave owns 32*QT queries. Workgroups of one head are
// placed contiguously on one XCD so concurrently running query tiles stream
// the same K/V rows through that XCD's L2.
//
// Per key tile of 64 cached rows (double-buffered in LDS, the next tile's
// global loads in flight during the current tile's math):
//   S^T = K Q^T   v_mfma_f32_32x32x16_bf16, K rows as the A operand straight
//                 from LDS, the wave's Q fragments resident in VGPRs as the B
//                 operand. Each lane then holds 16 scores of ONE query
//                 (column l%32), spread over 32 keys shared with lane l^32.
//   softmax       online, in the log2 domain with scale*log2(e) folded into
//                 one FMA per score; the row maximum needs a single cross-lane
//                 exchange (lane l <-> l^32); row sums stay per lane and are
//                 combined once at the end.
//   O^T += V^T P^T  the probabilities, rounded to bf16, are used directly as
//                 the B operand: the accumulator layout of S^T already puts 8
//                 keys of the lane's query in each half-fragment, provided the
//                 contraction slots are mapped to keys in the permuted order
//                 slot (hi*8 + e) -> key (e/4)*8 + hi*4 + e%4 (per 16 keys).
//                 The V^T operand is gathered from the row-major LDS tile in
//                 that same order (2-byte reads, bank-conflict free).
//   Because every lane owns one query column in both S^T and O^T, the
//   rescale by exp2(m_old - m_new) needs no cross-lane traffic.
#include "common.h"

namespace hsa {
namespace {

constexpr int kThreads = 256;
constexpr int BKV = 64;  // cached rows per LDS tile

template <int DH, int QT>
__global__ __launch_bounds__(kThreads) void attention_bf16_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ kc, const bf16* __restrict__ vc,
    bf16* __restrict__ o, int n_q, int n_kv, int d, float sl2e, int n_qtiles, int heads) {
  constexpr int BQ = 4 * 32 * QT;
  constexpr int KS = DH + 8;         // LDS row stride in bf16 (272 B for DH=128)
  constexpr int CPR = DH / 8;        // 16-byte chunks per cached row
  constexpr int LOADS = BKV * CPR / kThreads;
  constexpr int DT = DH / 32;        // 32-wide head-dim tiles of O^T
  constexpr int KK = DH / 16;        // k-steps of S^T
  __shared__ __attribute__((aligned(16))) bf16 Ks[2][BKV * KS];
  __shared__ __attribute__((aligned(16))) bf16 Vs[2][BKV * KS];

  const int item = xcd_contiguous(blockIdx.x, n_qtiles * heads);
  const int h = item / n_qtiles;
  const int qt = item - h * n_qtiles;
  const int t = threadIdx.x;
  const int lane = t & 63, wave = t >> 6;
  const int l32 = lane & 31, hi = lane >> 5;
  const long col0 = (long)h * DH;

  // Q fragments: lane holds Q[query l32 of sub-tile tq][kk*16 + hi*8 + 0..7]
  bf16x8 qf[QT][KK];
#pragma unroll
  for (int tq = 0; tq < QT; ++tq) {
    const int qrow = qt * BQ + wave * 32 * QT + tq * 32 + l32;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      if (qrow < n_q)
        qf[tq][kk] = *reinterpret_cast<const bf16x8*>(q + (long)qrow * d + col0 + kk * 16 + hi * 8);
      else
        qf[tq][kk] = (bf16x8){};
    }
  }

  u32x4 rk[LOADS], rv[LOADS];
  auto gload = [&](int kv0) {
#pragma unroll
    for (int i = 0; i < LOADS; ++i) {
      const int id = t + kThreads * i;
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
      const int id = t + kThreads * i;
      const int row = id / CPR, cc = id % CPR;
      *reinterpret_cast<u32x4*>(&Ks[buf][row * KS + cc * 8]) = rk[i];
      *reinterpret_cast<u32x4*>(&Vs[buf][row * KS + cc * 8]) = rv[i];
    }
  };

  f32x16 acc[QT][DT];
  float m_run[QT], l_run[QT];
#pragma unroll
  for (int tq = 0; tq < QT; ++tq) {
    m_run[tq] = -INFINITY;
    l_run[tq] = 0.f;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) acc[tq][dt] = (f32x16){};
  }

  const int n_tiles = (n_kv + BKV - 1) / BKV;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int it = 0; it < n_tiles; ++it) {
    const int buf = it & 1;
    const int kv0 = it * BKV;
    if (it + 1 < n_tiles) gload(kv0 + BKV);
    const bf16* Kt = Ks[buf];
    const unsigned short* Vt = reinterpret_cast<const unsigned short*>(Vs[buf]);
#pragma unroll
    for (int sb = 0; sb < BKV / 32; ++sb) {
      f32x16 s[QT];
#pragma unroll
      for (int tq = 0; tq < QT; ++tq) s[tq] = (f32x16){};
#pragma unroll
      for (int kk = 0; kk < KK; ++kk) {
        const bf16x8 kf =
            *reinterpret_cast<const bf16x8*>(&Kt[(sb * 32 + l32) * KS + kk * 16 + hi * 8]);
#pragma unroll
        for (int tq = 0; tq < QT; ++tq)
          s[tq] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[tq][kk], s[tq], 0, 0, 0);
      }
      // s[tq][e] is the score of key kv0 + sb*32 + (e/4)*8 + hi*4 + e%4
      const int key0 = kv0 + sb * 32 + hi * 4;
      const bool ragged = kv0 + sb * 32 + 32 > n_kv;
      bf16x8 pf[QT][2];
#pragma unroll
      for (int tq = 0; tq < QT; ++tq) {
        if (ragged) {
#pragma unroll
          for (int e = 0; e < 16; ++e)
            if (key0 + (e >> 2) * 8 + (e & 3) >= n_kv) s[tq][e] = -INFINITY;
        }
        float mx = s[tq][0];
#pragma unroll
        for (int e = 1; e < 16; ++e) mx = fmaxf(mx, s[tq][e]);
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m_run[tq], mx * sl2e);
        const float alpha = __builtin_amdgcn_exp2f(m_run[tq] - m_new);
        float p[16];
        float ls = 0.f;
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          p[e] = __builtin_amdgcn_exp2f(fmaf(s[tq][e], sl2e, -m_new));
          ls += p[e];
        }
        l_run[tq] = l_run[tq] * alpha + ls;
        m_run[tq] = m_new;
#pragma unroll
        for (int dt = 0; dt < DT; ++dt) acc[tq][dt] *= alpha;
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          f32x4 lo = {p[8 * half + 0], p[8 * half + 1], p[8 * half + 2], p[8 * half + 3]};
          f32x4 up = {p[8 * half + 4], p[8 * half + 5], p[8 * half + 6], p[8 * half + 7]};
          const bf16x4 a = to_bf16x4(lo), b = to_bf16x4(up);
          pf[tq][half] = (bf16x8){a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
        }
      }
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
        for (int ks = 0; ks < 2; ++ks) {
          // V^T operand: row dh = dt*32 + l32, slot hi*8 + e <- key sb*32 + ks*16 + (e/4)*8 + hi*4 + e%4
          const int base = (sb * 32 + ks * 16 + hi * 4) * KS + dt * 32 + l32;
          unsigned short u[8];
#pragma unroll
          for (int e = 0; e < 8; ++e) u[e] = Vt[base + ((e >> 2) * 8 + (e & 3)) * KS];
          bf16x8 vf;
#pragma unroll
          for (int e = 0; e < 8; ++e) vf[e] = __builtin_bit_cast(bf16, u[e]);
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

template <int DH, int QT>
hipError_t launch_tq(const void* q, const void* k, const void* v, void* o, int n_q, int n_kv,
                     int heads, float sl2e, hipStream_t s) {
  constexpr int BQ = 4 * 32 * QT;
  const int n_qtiles = (n_q + BQ - 1) / BQ;
  const int d = heads * DH;
  hipLaunchKernelGGL((attention_bf16_kernel<DH, QT>), dim3((unsigned)(n_qtiles * heads)),
                     dim3(kThreads), 0, s, static_cast<const bf16*>(q),
                     static_cast<const bf16*>(k), static_cast<const bf16*>(v),
                     static_cast<bf16*>(o), n_q, n_kv, d, sl2e, n_qtiles, heads);
  return hipGetLastError();
}

}  // namespace

hipError_t launch_attention_bf16(const void* q, const void* k, const void* v, void* o, int n_q,
                                 int n_kv, int heads, int head_dim, float scale, hipStream_t s) {
  if (n_q <= 0) return hipSuccess;
  const float sl2e = scale * 1.4426950408889634f;
  // Two 32-query sub-tiles per wave halve the LDS traffic per MFMA; use them
  // when that still gives every CU at least two workgroups.
  const long wgs2 = (long)((n_q + 255) / 256) * heads;
  const bool two = wgs2 >= 512;
  if (head_dim == 64)
    return two ? launch_tq<64, 2>(q, k, v, o, n_q, n_kv, heads, sl2e, s)
               : launch_tq<64, 1>(q, k, v, o, n_q, n_kv, heads, sl2e, s);
  return two ? launch_tq<128, 2>(q, k, v, o, n_q, n_kv, heads, sl2e, s)
             : launch_tq<128, 1>(q, k, v, o, n_q, n_kv, heads, sl2e, s);
}

}  // namespace hsa
