// Internal helpers shared by the HIP translation units of the HSA step library.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace hsa {

typedef __bf16 bf16;
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));  // 16 raw bytes
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kWave = 64;
constexpr int kXcds = 8;  // MI355X: 8 XCDs, workgroups dispatched round-robin over them

// Map a linear workgroup id to a work item so that the items given to one XCD
// are contiguous: workgroup L runs on XCD L % 8, and the i-th workgroup an XCD
// receives gets item (first item of that XCD) + i. Bijective on [0, total).
__device__ __forceinline__ int xcd_contiguous(int L, int total) {
  const int xcd = L % kXcds;
  const int slot = L / kXcds;
  const int base = total / kXcds;
  const int rem = total % kXcds;
  return xcd * base + (xcd < rem ? xcd : rem) + slot;
}

// Compute units of the current device (queried once; 256 if the query fails).
inline int compute_units() {
  static int cus = 0;
  if (!cus) {
    int dev = 0, n = 0;
    cus = (hipGetDevice(&dev) == hipSuccess &&
           hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0)
              ? n
              : 256;
  }
  return cus;
}

// Round fp32 to bf16, nearest-even (v_cvt_pk_bf16_f32 on gfx950).
__device__ __forceinline__ bf16x4 to_bf16x4(f32x4 v) { return __builtin_convertvector(v, bf16x4); }

// 0.5 x (1 + tanh(y)), y = sqrt(2/pi) (x + 0.044715 x^3), evaluated as
// x / (1 + exp(-2y)) (the same function: 0.5 (1 + tanh(y)) is the logistic
// function of 2y), with the hardware exp2 and reciprocal.
__device__ __forceinline__ float gelu_tanh(float x) {
  const float k0 = 0.7978845608028654f;  // sqrt(2/pi)
  const float y = k0 * fmaf(0.044715f * x, x * x, x);
  const float t = __builtin_amdgcn_exp2f(-2.8853900817779268f * y);  // exp(-2y)
  return x * __builtin_amdgcn_rcpf(1.f + t);
}

__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v = fmaxf(v, __shfl_xor(v, o));
  return v;
}

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
  return v;
}

}  // namespace hsa

// Launchers (host side, one per translation unit). Each returns the HIP error
// of the launch.
namespace hsa {

hipError_t launch_active_set(const int32_t* budget, int n, int T, int iter, int margin,
                             int outside_period, int32_t* idx, int32_t* n_active, hipStream_t s);

// C[crow(m)][n] = sum_k A[arow(m)][k] * B_z[n][k] for up to three (B, C, c_rows)
// outputs sharing A. a_rows / c_rows may be null (identity); rows whose index is
// outside [0, a_limit) / [0, c_limit) are skipped. Row m of the product may be
// scaled by row_scale[m] (an RMS normalization of A's rows folded into the
// product), then optionally passed through the tanh GELU (the FFN's first
// product). Single-output products may add a residual R indexed like C
// (R[crow(m)][n], same leading dimension; R may be C itself) before the one
// rounding, and a bf16 product may store fp32.
struct RowGemmOut {
  const void* B;
  void* C;
  const int32_t* c_rows;
  int c_limit;
  void* C2;     // if set: rows crow >= c_split go to C2 row crow - c_split
  int c_split;
};
struct RowGemm {
  const void* A;
  const int32_t* a_rows;
  int a_limit;
  int M, Nc, K;  // rows of the product, output columns, reduction length
  long lda, ldb, ldc;
  RowGemmOut out[3];
  int n_out;
  const void* residual;    // n_out == 1 only; in the output's dtype
  int c_f32;               // bf16 inputs, fp32 output (no residual)
  const float* row_scale;  // null, or one factor per product row m < M
  int gelu;                // apply the tanh GELU after the row scale (no residual)
  // Rotary embedding of the outputs z with bit z of rope_outs set: row m is
  // token rope_tok[m] at grid position p = rope_pos[token] (the token itself
  // if null; outside [0, F*H*W) reads as 0; both are read for every m < M,
  // stored or not), coordinates (p / (H*W),
  // (p / W) % H, p % W). Channel pair k of a head of rope_dh channels lies in
  // the temporal band (k < nt), the row band (k < nt + nh) or the column
  // band; its (cos, sin) is rope_cs[r * rope_dh/2 + k] with r the frame,
  // F + row or F + H + column. Applied after the row scale, before rounding.
  const f32x2* rope_cs;
  const int32_t* rope_tok;
  const int32_t* rope_pos;
  int rope_outs, rope_dh, rope_nt, rope_nh, rope_f, rope_h, rope_w;
  // set by the bf16 launcher: workgroups from this index on take halves of
  // the remaining 256x256 tiles (see gemm_bf16.hip)
  int split_from;
  int group_m;  // set by the bf16 launcher: tile-rows per group of the tile order
};

// Grid coordinates of row m's token for the rotary embedding of g.
struct RopeRow {
  int f, y, x;
};
__device__ __forceinline__ RopeRow rope_row(const RowGemm& g, int m) {
  const int tok = g.rope_tok[m];
  const int hw = g.rope_h * g.rope_w;
  int p = g.rope_pos ? g.rope_pos[tok] : tok;
  if (p < 0 || p >= g.rope_f * hw) p = 0;
  return {p / hw, (p / g.rope_w) % g.rope_h, p % g.rope_w};
}

// (cos, sin) of head-local channel pair k (0 <= k < rope_dh/2) of a row at
// grid coordinates r; always an entry of the table.
__device__ __forceinline__ f32x2 rope_angle(const RowGemm& g, const RopeRow& r, int k) {
  const int row = k < g.rope_nt ? r.f
                  : (k < g.rope_nt + g.rope_nh ? g.rope_f + r.y : g.rope_f + g.rope_h + r.x);
  return g.rope_cs[row * (g.rope_dh >> 1) + k];
}
// The channel pair (a, b) rotated by the angle with (cos, sin) = cs.
__device__ __forceinline__ f32x2 rope_rotate(f32x2 cs, float a, float b) {
  return (f32x2){a * cs[0] - b * cs[1], a * cs[1] + b * cs[0]};
}
// The channel pair (a, b) at head-local pair index k, rotated.
__device__ __forceinline__ f32x2 rope_pair(const RowGemm& g, const RopeRow& r, int k, float a,
                                           float b) {
  return rope_rotate(rope_angle(g, r, k), a, b);
}
hipError_t launch_row_gemm_bf16(const RowGemm& g, hipStream_t s);

// Output z of a RowGemm, selected field by field so that a kernel never
// indexes its by-value argument dynamically (which would copy it to scratch).
__device__ __forceinline__ RowGemmOut row_gemm_out(const RowGemm& g, int z) {
  RowGemmOut o;
  o.B = z == 0 ? g.out[0].B : (z == 1 ? g.out[1].B : g.out[2].B);
  o.C = z == 0 ? g.out[0].C : (z == 1 ? g.out[1].C : g.out[2].C);
  o.c_rows = z == 0 ? g.out[0].c_rows : (z == 1 ? g.out[1].c_rows : g.out[2].c_rows);
  o.c_limit = z == 0 ? g.out[0].c_limit : (z == 1 ? g.out[1].c_limit : g.out[2].c_limit);
  o.C2 = z == 0 ? g.out[0].C2 : (z == 1 ? g.out[1].C2 : g.out[2].C2);
  o.c_split = z == 0 ? g.out[0].c_split : (z == 1 ? g.out[1].c_split : g.out[2].c_split);
  return o;
}
hipError_t launch_row_gemm_f32(const RowGemm& g, hipStream_t s);

// Keys/values: rows n < n_split come from (k, v), rows n_split .. n_kv-1 from
// (k2, v2) at row n - n_split (a cache prefix followed by fresh rows); any
// n_split.
// bf16 attention. With a workspace of at least attention_parts_bytes(p, ...)
// bytes the launch may split the cached rows into p <= kMaxKvParts parts
// (when that fills the CUs better) and merge them in a second kernel.
constexpr int kMaxKvParts = 4;
size_t attention_parts_bytes(int parts, int n_q, int heads, int head_dim);
hipError_t launch_attention_bf16(const void* q, const void* k, const void* v, void* o, int n_q,
                                 int n_kv, int heads, int head_dim, float scale, hipStream_t s,
                                 const void* k2 = nullptr, const void* v2 = nullptr,
                                 int n_split = 0x7fffffff, void* ws = nullptr,
                                 size_t ws_bytes = 0);
hipError_t launch_attention_f32(const void* q, const void* k, const void* v, void* o, int n_q,
                                int n_kv, int heads, int head_dim, float scale, hipStream_t s,
                                const void* k2 = nullptr, const void* v2 = nullptr,
                                int n_split = 0x7fffffff);

hipError_t launch_cached_euler(float* x, float* v_cache, const float* v_fresh,
                               const int32_t* idx, int n_active, long n_tokens, int channels,
                               float dsig, hipStream_t s);

}  // namespace hsa

// Multi-layer sampling loop (stack.hip).
namespace hsa {

// xa[j][c] = x[idx[j]][c] in the model dtype (bf16 rounded to nearest even,
// or fp32); rows whose index is outside [0, n_tokens) are written as zeros.
hipError_t launch_gather_latent(const float* x, const int32_t* idx, int n_active, long n_tokens,
                                int channels, bool out_bf16, void* xa, hipStream_t s);

// scale[m] = 1 / sqrt(mean_k x[m][k]^2 + eps) for m < n_rows (fp32 sums).
hipError_t launch_row_rms_scale(const void* x, bool bf16_in, int n_rows, int d, float eps,
                                float* scale, hipStream_t s);

// Token reordering: perm = tokens with budget < T, then those with budget T
// (each part in index order); n_lead = number of the former, or -1 if a
// budget is invalid (1 <= s <= T, T % s == 0).
hipError_t launch_reorder_plan(const int32_t* budget, int n, int T, int32_t* perm,
                               int32_t* n_lead, hipStream_t s);

// dst[i] = src[perm[i]] (inverse: dst[perm[i]] = src[i]) for rows of row_bytes;
// indices outside [0, n_rows) skip the row.
hipError_t launch_permute_rows(const void* src, const int32_t* perm, long n_rows, long row_bytes,
                               bool inverse, void* dst, hipStream_t s);

// Budget groups in ascending budget order: group k holds the tokens of rank
// end[k-1] .. end[k]-1 (end[-1] = 0) and gets step budget budget[k].
constexpr int kMaxGroups = 16;
struct GroupTable {
  int n;
  int32_t budget[kMaxGroups];
  int64_t end[kMaxGroups];
};

// budget[t] from the rank of (keys[t], t), keys compared as bit patterns.
hipError_t launch_rank_budgets(const double* keys, long n_tokens, const GroupTable& tab,
                               int32_t* budget, hipStream_t s);

// Strategy D: acc[t] += |v[t] - v_prev[t]|_1 / |v[t]|_1 (acc[t] = 0 when
// first), then v_prev[t] = v[t].
hipError_t launch_l1_rel(const float* v, float* v_prev, long n_tokens, int channels, double* acc,
                         bool first, hipStream_t s);

// Group refresh: keys[t] = squared L2 norm of v[t] (float64, channel order),
// then budget[t] from the rank of (keys[t], t).
hipError_t launch_assign_budgets(const float* v, long n_tokens, int channels,
                                 const GroupTable& tab, double* keys, int32_t* budget,
                                 hipStream_t s);

}  // namespace hsa
