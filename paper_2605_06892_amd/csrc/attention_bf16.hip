// bf16 active-query attention on CDNA4 matrix cores (Section 2.3, step 3):
// for every active row j and head h, o[j,h] = softmax(scale q[j,h] K_h^T) V_h
// over all N cached rows. Cost O(|A_i| N d) instead of O(N^2 d).
//
// Work split: one workgroup of NW waves per (head, tile of 32*NW active
// queries); each wave owns 32 queries. Workgroups of one head are placed
// contiguously on one XCD so concurrently running query tiles stream the same
// K/V rows through that XCD's L2. A launch of few workgroups (few heads or
// few active rows, e.g. 384 for 12 heads at 25% active on 256 CUs) may also
// split the cached rows into key parts: each part's workgroup writes its
// unnormalized output with its softmax maximum and sum (fp32, caller
// workspace) and attention_combine merges the parts, rescaling each by
// 2^(m_p - max m) (the softmax of a concatenation).
//
// K/V tiles of 96 cached rows go global -> LDS directly (global_load_lds_dwordx4:
// each wave instruction fills one contiguous 1 KB segment of LDS, lane l at
// byte 16*l), three tiles deep (144 KB of LDS at 128-wide heads), issued two
// tiles ahead by one wave per SIMD, one barrier per tile (every three 32-key
// blocks).
// Rows are stored unpadded with the 16-byte chunks of each row permuted by an
// XOR with a function of the row (K: f(r) = ((r&3)<<2)|((r>>2)&3) for 128-wide
// heads; V: f(r) = (r&3)<<2), so that the K fragment reads (16 rows, one chunk)
// and the V transpose reads (4 rows, 4 chunks) both hit disjoint LDS banks.
// Rows beyond N are loaded from row N-1 and masked out of the softmax. The N
// rows may come in two segments: a cache prefix and, from row n_split on,
// fresh rows of a second buffer (the prefix-only cache of reordered tokens);
// a tile across n_split picks the segment per row.
//
// Keys are consumed in 32-row blocks. Per block:
//   S^T = K Q^T - m   v_mfma_f32_32x32x16_bf16 with K rows as the A operand
//                 from LDS and the wave's Q fragments resident in VGPRs as
//                 the B operand. Q is pre-multiplied by scale*log2(e) and the
//                 accumulator is seeded (C operand, not written) with -m, m the
//                 wave's reference maximum in log2 units, so each score leaves
//                 the MFMA ready for exp2. Each lane holds 16 scores of ONE
//                 query (column l%32) over 32 keys shared with lane l^32.
//   softmax       the fast path is exp2, a running sum and the bf16 pack per
//                 score. The reference maximum m is set from the first 32 keys
//                 and only raised (rescaling O and the sum) when some
//                 probability of a block exceeds 2^16, detected from the
//                 block's sum: a wave-uniform branch that is almost never
//                 taken. Probabilities stay below 2^16 and the sum at or
//                 above 1.
//   O^T += V^T P^T  the probabilities, rounded to bf16, are the B operand as
//                 they sit in the S^T accumulators; the contraction slot
//                 (hi*8 + e) of each 16-key step maps to key (e/4)*8 + hi*4 +
//                 e%4. The V^T operand comes from ds_read_b64_tr_b16 (gfx950
//                 LDS transpose read): in each 16-lane group, lane i points at
//                 4 consecutive channels of key row i/4, and lane L receives
//                 one channel of 4 keys.
// Software pipeline: the S^T MFMAs of block b+1 are issued next to the
// exp2/sum instructions of block b (they are independent), then the PV MFMAs
// of block b, next to the LDS reads of half the K fragments of block b+2. Every
// lane owns one query column in both S^T and O^T, so the softmax statistics
// never need to be broadcast across lanes.
#include "common.h"

#include <type_traits>

namespace hsa {
namespace {

constexpr int BKV = 96;                 // cached rows per LDS tile (three 32-key blocks)
constexpr int NBUF = 3;                 // LDS tiles in flight
constexpr float kSlowSum = 65536.0f;    // 2^16: raise the reference maximum

// Key parts of one launch (split over the cached rows, merged afterwards)
struct KvParts {
  int parts;        // 1: no split, the kernel writes o directly
  int chunk;        // cached rows per part (a multiple of BKV)
  float* o_part;    // [parts, n_q, d] unnormalized outputs
  float* ml_part;   // [parts, n_q, heads] (m, l) pairs
};

typedef __attribute__((address_space(3))) bf16x4 lds_bf16x4;
typedef __attribute__((address_space(3))) void lds_void;
typedef __attribute__((address_space(1))) const void global_cvoid;

// s_waitcnt immediate for "vector memory counter <= n", other counters free
constexpr int waitcnt_vm(int n) { return (n & 15) | (7 << 4) | (15 << 8) | ((n >> 4) << 14); }

// chunk permutation of cached row r inside a tile (see header)
template <int DH>
__device__ __forceinline__ int swz_k(int r) {
  return DH == 128 ? (((r & 3) << 2) | ((r >> 2) & 3)) : ((r >> 1) & 7);
}
template <int DH>
__device__ __forceinline__ int swz_v(int r) {
  return DH == 128 ? ((r & 3) << 2) : (((r >> 1) & 1) << 2);
}

template <int DH, int NW, bool SPLIT>
__global__ __launch_bounds__(NW * 64) void attention_bf16_kernel(
    const bf16* __restrict__ q, const bf16* __restrict__ kc, const bf16* __restrict__ vc,
    bf16* __restrict__ o, int n_q, int n_kv, int d, float sl2e, int n_qtiles,
    const bf16* __restrict__ kc2, const bf16* __restrict__ vc2, int n_split, int kv_chunk,
    int parts, float* __restrict__ o_part, float* __restrict__ ml_part) {
  constexpr int BQ = NW * 32;        // queries per workgroup
  constexpr int CPR = DH / 8;        // 16-byte chunks per cached row
  constexpr int RPS = 64 / CPR;      // rows per 1 KB LDS segment
  constexpr int SEGS = BKV / RPS;    // segments per tile
  constexpr int DT = DH / 32;        // 32-wide head-dim tiles of O^T
  constexpr int KK = DH / 16;        // k-steps of S^T
  // one array per buffer: with compile-time buffer indices the compiler can
  // tell the asynchronous tile loads from the LDS reads of other buffers
  __shared__ __attribute__((aligned(16))) bf16 K0[BKV * DH], K1[BKV * DH], K2[BKV * DH];
  __shared__ __attribute__((aligned(16))) bf16 V0[BKV * DH], V1[BKV * DH], V2[BKV * DH];
  auto kbuf = [&](auto b) -> bf16* {
    constexpr int B = decltype(b)::value;
    if constexpr (B == 0) return K0; else if constexpr (B == 1) return K1; else return K2;
  };
  auto vbuf = [&](auto b) -> bf16* {
    constexpr int B = decltype(b)::value;
    if constexpr (B == 0) return V0; else if constexpr (B == 1) return V1; else return V2;
  };

  const int heads = d / DH;
  const int item = xcd_contiguous(blockIdx.x, n_qtiles * heads * parts);
  const int hp = item / n_qtiles;  // (head, key part); the query tiles of one pair are adjacent
  const int qt = item - hp * n_qtiles;
  const int h = hp / parts;
  const int part = hp - h * parts;
  // cached rows of this part (all of them when parts == 1); kv_chunk is a
  // multiple of the tile, so tiles never straddle a part
  const int kv_begin = part * kv_chunk;
  const int kv_end = min(n_kv, kv_begin + kv_chunk);
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: scalar
  const int l32 = lane & 31, hi = lane >> 5;
  const long col0 = (long)h * DH;

  // Q fragments, pre-scaled by scale*log2(e): lane holds Q[query l32][kk*16 + hi*8 + 0..7]
  bf16x8 qf[KK];
  {
    const int qrow = qt * BQ + wave * 32 + l32;
#pragma unroll
    for (int kk = 0; kk < KK; ++kk) {
      bf16x8 raw = (bf16x8){};
      if (qrow < n_q)
        raw = *reinterpret_cast<const bf16x8*>(q + (long)qrow * d + col0 + kk * 16 + hi * 8);
      f32x4 lo = {(float)raw[0] * sl2e, (float)raw[1] * sl2e, (float)raw[2] * sl2e, (float)raw[3] * sl2e};
      f32x4 up = {(float)raw[4] * sl2e, (float)raw[5] * sl2e, (float)raw[6] * sl2e, (float)raw[7] * sl2e};
      qf[kk] = __builtin_shufflevector(to_bf16x4(lo), to_bf16x4(up), 0, 1, 2, 3, 4, 5, 6, 7);
    }
  }

  // this lane's part of a tile load: segment seg = i*NW + wave, row seg*RPS + lane/CPR,
  // LDS slot lane%CPR holding global chunk slot ^ f(row)
  const bf16* kg = kc + col0;
  const bf16* vg = vc + col0;
  const bf16* kg2 = kc2 + col0;  // rows n_split.. (unused when n_split >= n_kv)
  const bf16* vg2 = vc2 + col0;
  // Tile loads come from waves 0..3 only, one per SIMD (waves w and w+4
  // share a SIMD): a wave stalls while its global -> LDS loads issue, and the
  // other wave of its SIMD keeps the matrix pipe busy meanwhile (measured: 3%
  // faster than loads from all 8 waves). Loader wave w fetches segments
  // i*4 + w, i < LL: tile rows RPS*(i*4 + w) + lane/CPR = r0 + i*RSTEP.
  constexpr int LW = 4;                 // loader waves
  constexpr int LL = SEGS / LW;         // segment loads per loader wave per tensor
  constexpr int RSTEP = RPS * LW;       // tile rows between a loader's segments
  static_assert(LL * LW == SEGS, "loader waves must cover the tile");
  const int r0 = wave * RPS + lane / CPR;
  const int slot = lane % CPR;
  // chunk permutation of row r0 + i*RSTEP (the same for every i when RSTEP
  // is a multiple of the permutation's period, 16 rows)
  auto kch = [&](int i) { return (slot ^ swz_k<DH>(r0 + i * RSTEP)) * 8; };
  auto vch = [&](int i) { return (slot ^ swz_v<DH>(r0 + i * RSTEP)) * 8; };
  static_assert(RSTEP % 16 == 0, "one chunk permutation for all of a loader's rows");
  const long k_lane = ((long)r0 * d + kch(0)) * 2;  // bytes from the tile's first row
  const long v_lane = ((long)r0 * d + vch(0)) * 2;
  auto issue_tile = [&](auto buf, int kv0) {
    if (wave >= LW) return;
    bf16* kd = kbuf(buf) + wave * 512;
    bf16* vd = vbuf(buf) + wave * 512;
    // segment of the tile when all of its rows exist and lie on one side of
    // the split, chosen once per tile
    const bool tail = SPLIT && kv0 >= n_split;
    const bf16* kb = tail ? kg2 : kg;
    const bf16* vb = tail ? vg2 : vg;
    const long off = tail ? (long)n_split : 0;
    if (kv0 + BKV <= n_kv && (!SPLIT || tail || kv0 + BKV <= n_split)) {
      // uniform tile base (scalar) + the lane's 32-bit byte offset
      const char* ks = reinterpret_cast<const char*>(kb + (long)(kv0 - off) * d);
      const char* vs = reinterpret_cast<const char*>(vb + (long)(kv0 - off) * d);
#pragma unroll
      for (int i = 0; i < LL; ++i) {
        __builtin_amdgcn_global_load_lds((global_cvoid*)(ks + (long)i * RSTEP * d * 2 + k_lane),
                                         (lds_void*)(kd + i * LW * 512), 16, 0, 0);
        __builtin_amdgcn_global_load_lds((global_cvoid*)(vs + (long)i * RSTEP * d * 2 + v_lane),
                                         (lds_void*)(vd + i * LW * 512), 16, 0, 0);
      }
    } else {  // the last, ragged tile (rows past N are read from row N-1) or a
              // tile across the split: segment and row chosen per row
#pragma unroll
      for (int i = 0; i < LL; ++i) {
        const int n = min(kv0 + r0 + i * RSTEP, n_kv - 1);
        const bool t = SPLIT && n >= n_split;
        const long row = t ? n - n_split : n;
        __builtin_amdgcn_global_load_lds((global_cvoid*)((t ? kg2 : kg) + row * d + kch(i)),
                                         (lds_void*)(kd + i * LW * 512), 16, 0, 0);
        __builtin_amdgcn_global_load_lds((global_cvoid*)((t ? vg2 : vg) + row * d + vch(i)),
                                         (lds_void*)(vd + i * LW * 512), 16, 0, 0);
      }
    }
  };

  // LDS element offsets this lane reads, relative to a 32-key block
  int koff[KK];  // K fragment kk: row l32, chunk kk*2 + hi
#pragma unroll
  for (int kk = 0; kk < KK; ++kk) koff[kk] = l32 * DH + (((kk * 2 + hi) ^ swz_k<DH>(l32)) * 8);
  int voff[DT];  // V transpose read, head-dim tile dt: row hi*4 + k, channel dt*32 + 16g + 4(lane&3)
  {
    const int k4 = (lane & 15) >> 2, g = (lane >> 4) & 1;
    const int r = hi * 4 + k4;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
      const int col = dt * 32 + 16 * g + 4 * (lane & 3);
      voff[dt] = r * DH + (((col >> 3) ^ swz_v<DH>(r)) * 8) + (col & 7);
    }
  }

  f32x16 acc[DT];
#pragma unroll
  for (int dt = 0; dt < DT; ++dt) acc[dt] = (f32x16){};
  f32x16 negm = (f32x16){};  // every element -m_ref: the seed of the score accumulators
  float m_ref = 0.f, l_run = 0.f;
  bool have_ref = false;     // becomes true after the first 32 keys (wave-uniform)
  // K fragments 0..KP-1 of the block whose scores the next step computes,
  // read one step ahead (during the previous block's PV): the S^T MFMAs of a
  // block then start without waiting on LDS. Four, together with the V
  // fragments of head-dim tile 0 read before the softmax (below), measured
  // best: 2-3% over no read-ahead; all eight K fragments need 252 registers
  // and gain less.
  constexpr int KP = KK < 4 ? KK : 4;
  bf16x8 kpre[KP];
  auto kfrag = [&](auto buf, int kb, int kk) {
    return *reinterpret_cast<const bf16x8*>(kbuf(buf) + kb * DH + koff[kk]);
  };

  // S^T of the 32-key block starting at row kb of tile buffer buf
  auto scores = [&](auto buf, int kb, f32x16& s) {
    const bf16* base = kbuf(buf) + kb * DH;
    bf16x8 kf[KK];
#pragma unroll
    for (int kk = 0; kk < KP; ++kk) kf[kk] = kpre[kk];
#pragma unroll
    for (int kk = KP; kk < KK; ++kk) kf[kk] = *reinterpret_cast<const bf16x8*>(base + koff[kk]);
    s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[0], qf[0], negm, 0, 0, 0);
#pragma unroll
    for (int kk = 1; kk < KK; ++kk) s = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf[kk], qf[kk], s, 0, 0, 0);
  };

  // One pipeline step: issue S^T of the next block, softmax of the current
  // block (keys key0 .. key0+31, V rows vb .. vb+31 of buffer buf), PV. The
  // next block's scores are always computed from a valid LDS address so that
  // they share a scheduling region with the softmax; after the last block
  // they are unused.
  auto step = [&](f32x16& s_cur, f32x16& s_nxt, auto nbuf, int nkb, auto buf, int vb, int key0,
                  auto nnbuf, int nnkb) {
    if (key0 + 32 > kv_end) {  // ragged last block: mask the keys beyond the part
      const int kbase = key0 + hi * 4;
#pragma unroll
      for (int e = 0; e < 16; ++e)
        if (kbase + (e >> 2) * 8 + (e & 3) >= kv_end) s_cur[e] = -INFINITY;
    }
    scores(nbuf, nkb, s_nxt);
    const bf16* vbase = vbuf(buf) + vb * DH;
    constexpr int NV = 1;  // head-dim tiles whose V fragments are read before the softmax
                           // (their latency then hides behind it)
    bf16x8 vfa[NV][2];
#pragma unroll
    for (int dt = 0; dt < NV; ++dt)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const bf16* src = vbase + ks * 16 * DH + voff[dt];
        const bf16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(src));
        const bf16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(src + 8 * DH));
        vfa[dt][ks] = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
      }
    float p[16];
#pragma unroll
    for (int e = 0; e < 16; ++e) p[e] = __builtin_amdgcn_exp2f(s_cur[e]);
    float ls = ((p[0] + p[1]) + (p[2] + p[3])) + ((p[4] + p[5]) + (p[6] + p[7])) +
               (((p[8] + p[9]) + (p[10] + p[11])) + ((p[12] + p[13]) + (p[14] + p[15])));
    if (__any(!have_ref || !(ls <= kSlowSum))) {
      // set or raise the reference maximum, rescale what was accumulated
      float mx = s_cur[0];
#pragma unroll
      for (int e = 1; e < 16; ++e) mx = fmaxf(mx, s_cur[e]);
      mx = fmaxf(mx, __shfl_xor(mx, 32));               // block max relative to m_ref
      const float up = have_ref ? fmaxf(mx, 0.f) : mx;  // amount to raise m_ref by
      const float alpha = have_ref ? __builtin_amdgcn_exp2f(-up) : 0.f;
      ls = 0.f;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        p[e] = __builtin_amdgcn_exp2f(s_cur[e] - up);
        ls += p[e];
      }
      l_run *= alpha;
#pragma unroll
      for (int dt = 0; dt < DT; ++dt) acc[dt] *= alpha;
      m_ref += up;
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        negm[e] = -m_ref;
        s_nxt[e] -= up;  // the next block's scores were seeded with the old reference
      }
      have_ref = true;
    }
    l_run += ls;
    bf16x8 pf[2];
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      f32x4 lo = {p[8 * half + 0], p[8 * half + 1], p[8 * half + 2], p[8 * half + 3]};
      f32x4 up = {p[8 * half + 4], p[8 * half + 5], p[8 * half + 6], p[8 * half + 7]};
      pf[half] = __builtin_shufflevector(to_bf16x4(lo), to_bf16x4(up), 0, 1, 2, 3, 4, 5, 6, 7);
    }
#pragma unroll
    for (int kk = 0; kk < KP; ++kk) kpre[kk] = kfrag(nnbuf, nnkb, kk);
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        bf16x8 vf;
        if (dt < NV) {
          vf = vfa[dt][ks];
        } else {
          const bf16* src = vbase + ks * 16 * DH + voff[dt];
          const bf16x4 v0 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(src));
          const bf16x4 v1 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16((lds_bf16x4*)(src + 8 * DH));
          vf = __builtin_shufflevector(v0, v1, 0, 1, 2, 3, 4, 5, 6, 7);
        }
        acc[dt] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[ks], acc[dt], 0, 0, 0);
      }
    }
  };

  using B0 = std::integral_constant<int, 0>;
  using B1 = std::integral_constant<int, 1>;
  using B2 = std::integral_constant<int, 2>;
  const int n_tiles = (kv_end - kv_begin + BKV - 1) / BKV;
  issue_tile(B0{}, kv_begin);
  if (n_tiles > 1) issue_tile(B1{}, kv_begin + BKV);
  __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
  __syncthreads();
  f32x16 sa, sb;
#pragma unroll
  for (int kk = 0; kk < KP; ++kk) kpre[kk] = kfrag(B0{}, 0, kk);
  scores(B0{}, 0, sa);
#pragma unroll
  for (int kk = 0; kk < KP; ++kk) kpre[kk] = kfrag(B0{}, 32, kk);
  // tile it lives in buffer it % 3; the loop is unrolled by 3 so that every
  // buffer index is a compile-time constant
  // s0 holds the scores of the tile's block 0 on entry; the three steps
  // alternate the two score registers, so the next tile starts from s1
  auto tile = [&](auto buf, auto nxt, auto nn, int it, f32x16& s0, f32x16& s1) {
    const int kv0 = kv_begin + it * BKV;
    // block 0 of this tile; the next block is block 1 of the same tile
    step(s0, s1, buf, 32, buf, 0, kv0, buf, 64);
    // tile it+1 (issued one tile ago) has landed; after this barrier every
    // wave is done with tile it-1, whose buffer receives tile it+2
    __builtin_amdgcn_s_waitcnt(waitcnt_vm(0));
    __syncthreads();
    if (it + 2 < n_tiles) issue_tile(nn, kv0 + 2 * BKV);
    // block 1; the next block is block 2 of the same tile
    if (kv0 + 32 < kv_end) step(s1, s0, buf, 64, buf, 32, kv0 + 32, nxt, 0);
    // block 2; the next block is block 0 of tile it+1
    if (kv0 + 64 < kv_end) step(s0, s1, nxt, 0, buf, 64, kv0 + 64, nxt, 32);
  };
  for (int it = 0; it < n_tiles; it += NBUF) {
    tile(B0{}, B1{}, B2{}, it, sa, sb);
    if (it + 1 < n_tiles) tile(B1{}, B2{}, B0{}, it + 1, sb, sa);
    if (it + 2 < n_tiles) tile(B2{}, B0{}, B1{}, it + 2, sa, sb);
    const f32x16 t = sa;  // three tiles of three steps: the roles swap
    sa = sb;
    sb = t;
  }

  // acc[dt][e]: channel dt*32 + (e/4)*8 + hi*4 + e%4 of query l32
  const float l_tot = l_run + __shfl_xor(l_run, 32);
  const int qrow = qt * BQ + wave * 32 + l32;
  if (qrow >= n_q) return;
  if (parts == 1) {
    const float inv = 1.f / l_tot;
    bf16* dst = o + (long)qrow * d + col0;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int g = 0; g < 4; ++g) {
        f32x4 v = {acc[dt][4 * g + 0] * inv, acc[dt][4 * g + 1] * inv, acc[dt][4 * g + 2] * inv,
                   acc[dt][4 * g + 3] * inv};
        *reinterpret_cast<bf16x4*>(dst + dt * 32 + g * 8 + hi * 4) = to_bf16x4(v);
      }
    }
  } else {
    // this part's unnormalized output sum_n 2^(s_n - m) v_n, with m (log2
    // units) and l = sum_n 2^(s_n - m); attention_combine merges the parts
    const long prow = (long)part * n_q + qrow;
    float* dst = o_part + prow * d + col0;
#pragma unroll
    for (int dt = 0; dt < DT; ++dt) {
#pragma unroll
      for (int g = 0; g < 4; ++g)
        *reinterpret_cast<f32x4*>(dst + dt * 32 + g * 8 + hi * 4) =
            (f32x4){acc[dt][4 * g + 0], acc[dt][4 * g + 1], acc[dt][4 * g + 2], acc[dt][4 * g + 3]};
    }
    if (hi == 0)
      *reinterpret_cast<f32x2*>(ml_part + (prow * heads + h) * 2) =
          (f32x2){have_ref ? m_ref : -INFINITY, l_tot};
  }
}

// Merge of the key parts (the softmax of a concatenation): per query row and
// head, m = max_p m_p, w_p = 2^(m_p - m), o = sum_p w_p O_p / sum_p w_p l_p.
// One workgroup per query row; each thread produces 4 consecutive channels.
__global__ __launch_bounds__(256) void attention_combine_kernel(const float* __restrict__ o_part,
                                                               const float* __restrict__ ml_part,
                                                               bf16* __restrict__ o, int n_q,
                                                               int d, int head_dim, int parts) {
  const int row = blockIdx.x;
  const int heads = d / head_dim;
  for (int c = threadIdx.x * 4; c < d; c += blockDim.x * 4) {
    const int h = c / head_dim;
    float mp[kMaxKvParts], lp[kMaxKvParts];
    float m = -INFINITY;
#pragma unroll
    for (int p = 0; p < kMaxKvParts; ++p) {
      if (p < parts) {
        const f32x2 ml = *reinterpret_cast<const f32x2*>(ml_part + (((long)p * n_q + row) * heads + h) * 2);
        mp[p] = ml[0];
        lp[p] = ml[1];
        m = fmaxf(m, ml[0]);
      }
    }
    f32x4 acc = {};
    float l = 0.f;
#pragma unroll
    for (int p = 0; p < kMaxKvParts; ++p) {
      if (p < parts) {
        const float w = __builtin_amdgcn_exp2f(mp[p] - m);  // 0 for an empty part (m_p = -inf)
        l += w * lp[p];
        acc += w * *reinterpret_cast<const f32x4*>(o_part + ((long)p * n_q + row) * d + c);
      }
    }
    *reinterpret_cast<bf16x4*>(o + (long)row * d + c) = to_bf16x4(acc * (1.f / l));
  }
}

template <int DH, int NW, bool SPLIT>
hipError_t launch_split(const void* q, const void* k, const void* v, void* o, int n_q, int n_kv,
                        int heads, float sl2e, hipStream_t s, const void* k2, const void* v2,
                        int n_split, const KvParts& kp) {
  constexpr int BQ = NW * 32;
  const int n_qtiles = (n_q + BQ - 1) / BQ;
  const int d = heads * DH;
  hipLaunchKernelGGL((attention_bf16_kernel<DH, NW, SPLIT>), dim3((unsigned)(n_qtiles * heads * kp.parts)),
                     dim3(NW * 64), 0, s, static_cast<const bf16*>(q),
                     static_cast<const bf16*>(k), static_cast<const bf16*>(v),
                     static_cast<bf16*>(o), n_q, n_kv, d, sl2e, n_qtiles,
                     static_cast<const bf16*>(k2), static_cast<const bf16*>(v2), n_split, kp.chunk,
                     kp.parts, kp.o_part, kp.ml_part);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || kp.parts == 1) return e;
  hipLaunchKernelGGL(attention_combine_kernel, dim3((unsigned)n_q), dim3(256), 0, s,
                     kp.o_part, kp.ml_part, static_cast<bf16*>(o), n_q, d, DH, kp.parts);
  return hipGetLastError();
}

// keys in two segments only when the split falls inside the rows
template <int DH, int NW>
hipError_t launch_cfg(const void* q, const void* k, const void* v, void* o, int n_q, int n_kv,
                      int heads, float sl2e, hipStream_t s, const void* k2, const void* v2,
                      int n_split, const KvParts& kp) {
  if (n_split < n_kv)
    return launch_split<DH, NW, true>(q, k, v, o, n_q, n_kv, heads, sl2e, s, k2, v2, n_split, kp);
  return launch_split<DH, NW, false>(q, k, v, o, n_q, n_kv, heads, sl2e, s, k2, v2, n_split, kp);
}

// Key parts for a grid of `wgs` workgroups: the count p <= kMaxKvParts that
// minimizes the launch's rounds per unit of work, ceil(wgs p / CUs) / p, if
// that is at least 8% below a single part, each part keeps at least 8 tiles
// and the workspace holds the partial results; HSA_ATTN_KV_PARTS (1..4)
// forces a count for measurement sweeps and tests (workspace permitting).
KvParts choose_kv_parts(int wgs, int n_q, int n_kv, int heads, int head_dim, void* ws,
                        size_t ws_bytes) {
  KvParts kp{1, n_kv, nullptr, nullptr};
  if (!ws || n_kv <= 0) return kp;
  const int tiles = (n_kv + BKV - 1) / BKV;
  int p = 1;
  const char* forced = getenv("HSA_ATTN_KV_PARTS");
  const int f = forced ? atoi(forced) : 0;
  if (f >= 1 && f <= kMaxKvParts) {
    p = f;
  } else {
    const int cus = compute_units();
    const double one = (double)((wgs + cus - 1) / cus);
    double best = one;
    for (int c = 2; c <= kMaxKvParts; ++c) {
      if (tiles < 8 * c) break;
      const double r = (double)(((long)wgs * c + cus - 1) / cus) / c;
      if (r < best * 0.999) { best = r; p = c; }
    }
    if (best > 0.92 * one) p = 1;
  }
  p = std::min(p, tiles);
  if (p <= 1) return kp;
  const int chunk = (tiles + p - 1) / p * BKV;  // every part but the last gets `chunk` rows
  p = (n_kv + chunk - 1) / chunk;               // and none is empty
  if (p <= 1 || attention_parts_bytes(p, n_q, heads, head_dim) > ws_bytes) return kp;
  kp.parts = p;
  kp.chunk = chunk;
  kp.o_part = static_cast<float*>(ws);
  kp.ml_part = kp.o_part + (size_t)p * n_q * heads * head_dim;
  return kp;
}

}  // namespace

size_t attention_parts_bytes(int parts, int n_q, int heads, int head_dim) {
  return (size_t)parts * n_q * heads * (head_dim + 2) * sizeof(float);
}

hipError_t launch_attention_bf16(const void* q, const void* k, const void* v, void* o, int n_q,
                                 int n_kv, int heads, int head_dim, float scale, hipStream_t s,
                                 const void* k2, const void* v2, int n_split, void* ws,
                                 size_t ws_bytes) {
  if (n_q <= 0) return hipSuccess;
  if (!k2 || !v2) {
    k2 = k;  // any valid pointer: never read
    v2 = v;
    n_split = n_kv;
  }
  const float sl2e = scale * 1.4426950408889634f;
  // Workgroup shape: 8 waves (two per SIMD, 256 queries). Measured, 4 waves
  // (one per SIMD, 128 queries) is slower even where 8-wave workgroups leave
  // CUs idle (12 heads at 16% active: 640 against 1130 TFLOP/s); key parts
  // fill such grids instead. HSA_ATTN_WAVES=4 forces the 4-wave shape for
  // measurement sweeps and tests.
  const char* forced = getenv("HSA_ATTN_WAVES");
  const int nw = (forced && atoi(forced) == 4) ? 4 : 8;
  const int wgs = (n_q + nw * 32 - 1) / (nw * 32) * heads;
  const KvParts kp = choose_kv_parts(wgs, n_q, n_kv, heads, head_dim, ws, ws_bytes);
  if (head_dim == 64)
    return nw == 8 ? launch_cfg<64, 8>(q, k, v, o, n_q, n_kv, heads, sl2e, s, k2, v2, n_split, kp)
                   : launch_cfg<64, 4>(q, k, v, o, n_q, n_kv, heads, sl2e, s, k2, v2, n_split, kp);
  return nw == 8 ? launch_cfg<128, 8>(q, k, v, o, n_q, n_kv, heads, sl2e, s, k2, v2, n_split, kp)
                 : launch_cfg<128, 4>(q, k, v, o, n_q, n_kv, heads, sl2e, s, k2, v2, n_split, kp);
}

}  // namespace hsa
