// C ABI entry points of the multi-layer sampling loop: host-side argument
// checks, then kernel launches on the caller's stream. The contract of every
// call is stated with its declaration in include/hsa_step.h.
#include <math.h>

#include <vector>

#include "api_util.h"

using namespace hsa_api;

namespace {

// Layers of one stack (the host arrays hold 4 and 2 pointers per layer).
constexpr int kMaxLayers = 1 << 16;

struct Span {
  const void* p;
  size_t n;
};

bool any_overlap(const std::vector<Span>& a) {
  for (size_t i = 0; i < a.size(); ++i)
    for (size_t j = i + 1; j < a.size(); ++j)
      if (overlaps(a[i].p, a[i].n, a[j].p, a[j].n)) return true;
  return false;
}

bool any_overlap(const std::vector<Span>& a, const std::vector<Span>& b) {
  for (const Span& x : a)
    for (const Span& y : b)
      if (overlaps(x.p, x.n, y.p, y.n)) return true;
  return false;
}

// Group table checks (strictly ascending divisors of T, sizes summing to N).
int make_group_table(int32_t T, const int32_t* gb, const int64_t* gs, int32_t n_groups,
                     int64_t n_tokens, hsa::GroupTable* tab) {
  if (n_groups < 1 || n_groups > hsa::kMaxGroups || !gb || !gs) return HSA_STEP_ERR_BUDGET;
  if (T < 1) return HSA_STEP_ERR_BUDGET;
  int64_t total = 0;
  for (int k = 0; k < n_groups; ++k) {
    if (gb[k] < 1 || gb[k] > T || T % gb[k] != 0) return HSA_STEP_ERR_BUDGET;
    if (k > 0 && gb[k] <= gb[k - 1]) return HSA_STEP_ERR_BUDGET;
    if (gs[k] < 0 || gs[k] > n_tokens) return HSA_STEP_ERR_BUDGET;
    total += gs[k];
    tab->budget[k] = gb[k];
    tab->end[k] = total;
  }
  if (total != n_tokens) return HSA_STEP_ERR_BUDGET;
  tab->n = n_groups;
  return HSA_STEP_OK;
}

int64_t refresh_period(int32_t T, const int32_t* gb, int32_t n_groups) {
  int64_t p = 1;
  for (int k = 0; k < n_groups; ++k) {
    int64_t q = T / gb[k], a = p, b = q;
    while (b) {
      const int64_t r = a % b;
      a = b;
      b = r;
    }
    p = p / a * q;
  }
  return p;
}

constexpr float kRmsEps = 1e-6f;

RowGemm compact_gemm(const void* x, int n_rows, int d_in, const void* w, int d_out,
                     const float* row_scale, const void* residual, bool f32_out, void* y) {
  RowGemm g{};
  g.A = x;
  g.a_rows = nullptr;
  g.a_limit = n_rows;
  g.M = n_rows;
  g.Nc = d_out;
  g.K = d_in;
  g.lda = d_in;
  g.ldb = d_in;
  g.ldc = d_out;
  g.out[0] = {w, y, nullptr, n_rows};
  g.n_out = 1;
  g.residual = residual;
  g.c_f32 = f32_out ? 1 : 0;
  g.row_scale = row_scale;
  return g;
}

hipError_t launch_gemm(int dtype, const RowGemm& g, hipStream_t s) {
  return dtype == HSA_STEP_BF16 ? hsa::launch_row_gemm_bf16(g, s) : hsa::launch_row_gemm_f32(g, s);
}

}  // namespace

HSA_API int hsa_gather_rows(int dtype, const float* x, const int32_t* idx, int32_t n_active,
                            int64_t n_tokens, int32_t channels, void* xa, hipStream_t stream) {
  const size_t es = elem_size(dtype);
  if (!es) return HSA_STEP_ERR_DTYPE;
  if (n_active < 0 || n_tokens < 0 || n_tokens > kMaxRows || channels < 0)
    return HSA_STEP_ERR_SHAPE;
  if (!fits(n_tokens, channels, 4)) return HSA_STEP_ERR_SHAPE;
  if (n_active == 0 || channels == 0) return HSA_STEP_OK;
  if (!x || !idx || !xa) return HSA_STEP_ERR_NULL;
  if (!aligned(x, 4) || !aligned(idx, 4) || !aligned(xa, es)) return HSA_STEP_ERR_SHAPE;
  const size_t xab = (size_t)n_active * channels * es;
  if (overlaps(xa, xab, x, (size_t)n_tokens * channels * 4) ||
      overlaps(xa, xab, idx, (size_t)n_active * 4))
    return HSA_STEP_ERR_ALIAS;
  return launch_status(hsa::launch_gather_latent(x, idx, n_active, n_tokens, channels,
                                                 dtype == HSA_STEP_BF16, xa, stream));
}

HSA_API int hsa_row_rms_scale(int dtype, const void* x, int32_t n_rows, int32_t d, float eps,
                              float* scale, hipStream_t stream) {
  const size_t es = elem_size(dtype);
  if (!es) return HSA_STEP_ERR_DTYPE;
  if (n_rows < 0 || d <= 0 || !(eps >= 0.f) || !isfinite(eps)) return HSA_STEP_ERR_SHAPE;
  if (!fits(n_rows, d, es)) return HSA_STEP_ERR_SHAPE;
  if (n_rows == 0) return HSA_STEP_OK;
  if (!x || !scale) return HSA_STEP_ERR_NULL;
  if (!aligned(x, es) || !aligned(scale, 4)) return HSA_STEP_ERR_SHAPE;
  if (overlaps(scale, (size_t)n_rows * 4, x, (size_t)n_rows * d * es)) return HSA_STEP_ERR_ALIAS;
  return launch_status(
      hsa::launch_row_rms_scale(x, dtype == HSA_STEP_BF16, n_rows, d, eps, scale, stream));
}

HSA_API int hsa_linear(int dtype, const void* x, int32_t n_rows, int32_t d_in, const void* w,
                       int32_t d_out, const float* row_scale, const void* residual, int32_t gelu,
                       int out_dtype, void* y, hipStream_t stream) {
  const size_t es = elem_size(dtype), oes = elem_size(out_dtype);
  if (!es || !oes) return HSA_STEP_ERR_DTYPE;
  if (out_dtype != dtype && !(dtype == HSA_STEP_BF16 && out_dtype == HSA_STEP_F32))
    return HSA_STEP_ERR_DTYPE;
  const bool f32_out = dtype == HSA_STEP_BF16 && out_dtype == HSA_STEP_F32;
  if (n_rows < 0 || d_in <= 0 || d_out <= 0) return HSA_STEP_ERR_SHAPE;
  if (!fits(n_rows, d_in, 4) || !fits(n_rows, d_out, 4) || !fits(d_out, d_in, 4)) return HSA_STEP_ERR_SHAPE;
  if ((f32_out || gelu) && residual) return HSA_STEP_ERR_SHAPE;
  if (f32_out && gelu) return HSA_STEP_ERR_SHAPE;
  if (dtype == HSA_STEP_BF16 && (d_in % 64 != 0 || d_out % 4 != 0)) return HSA_STEP_ERR_SHAPE;
  if (n_rows == 0) return HSA_STEP_OK;
  if (!x || !w || !y) return HSA_STEP_ERR_NULL;
  const size_t align = dtype == HSA_STEP_BF16 ? 16 : 4;
  if (!aligned(x, align) || !aligned(w, align) || !aligned(y, align) ||
      (residual && !aligned(residual, align)) || (row_scale && !aligned(row_scale, 4)))
    return HSA_STEP_ERR_SHAPE;
  const size_t yb = (size_t)n_rows * d_out * oes;
  if (overlaps(y, yb, x, (size_t)n_rows * d_in * es) ||
      overlaps(y, yb, w, (size_t)d_out * d_in * es) || overlaps(y, yb, row_scale, (size_t)n_rows * 4))
    return HSA_STEP_ERR_ALIAS;
  if (residual && residual != y && overlaps(y, yb, residual, yb)) return HSA_STEP_ERR_ALIAS;
  RowGemm g = compact_gemm(x, n_rows, d_in, w, d_out, row_scale, residual, f32_out, y);
  g.gelu = gelu ? 1 : 0;
  return launch_status(launch_gemm(dtype, g, stream));
}

HSA_API size_t hsa_assign_budgets_workspace_bytes(int64_t n_tokens) {
  return n_tokens > 0 ? (size_t)n_tokens * 8 : 0;
}

HSA_API int hsa_assign_budgets(const float* v, int64_t n_tokens, int32_t channels, int32_t T,
                               const int32_t* group_budget, const int64_t* group_size,
                               int32_t n_groups, int32_t* budget, void* workspace,
                               size_t workspace_bytes, hipStream_t stream) {
  if (n_tokens < 0 || n_tokens > kMaxRows || channels < 0) return HSA_STEP_ERR_SHAPE;
  if (!fits(n_tokens, channels, 4)) return HSA_STEP_ERR_SHAPE;
  hsa::GroupTable tab{};
  const int st = make_group_table(T, group_budget, group_size, n_groups, n_tokens, &tab);
  if (st != HSA_STEP_OK) return st;
  if (n_tokens == 0) return HSA_STEP_OK;
  if (!v || !budget) return HSA_STEP_ERR_NULL;
  const size_t need = hsa_assign_budgets_workspace_bytes(n_tokens);
  if (!workspace || workspace_bytes < need) return HSA_STEP_ERR_WORKSPACE;
  if (!aligned(v, 4) || !aligned(budget, 4) || !aligned(workspace, 8)) return HSA_STEP_ERR_SHAPE;
  const size_t vb = (size_t)n_tokens * channels * 4, bb = (size_t)n_tokens * 4;
  if (overlaps(budget, bb, v, vb) || overlaps(workspace, need, v, vb) ||
      overlaps(workspace, need, budget, bb))
    return HSA_STEP_ERR_ALIAS;
  return launch_status(hsa::launch_assign_budgets(v, n_tokens, channels, tab,
                                                  static_cast<double*>(workspace), budget, stream));
}

HSA_API size_t hsa_rope_table_floats(int32_t head_dim, int32_t grid_f, int32_t grid_h,
                                     int32_t grid_w) {
  if (head_dim < 6 || head_dim % 2 || grid_f < 1 || grid_h < 1 || grid_w < 1) return 0;
  const int64_t rows = (int64_t)grid_f + grid_h + grid_w;
  if (!fits(rows, head_dim, 4)) return 0;
  return (size_t)rows * head_dim;
}

HSA_API int hsa_rope_table(float theta, int32_t head_dim, int32_t grid_f, int32_t grid_h,
                           int32_t grid_w, float* table_host) {
  if (!hsa_rope_table_floats(head_dim, grid_f, grid_h, grid_w) || !(theta > 1.f) ||
      !isfinite(theta))
    return HSA_STEP_ERR_SHAPE;
  if (!table_host) return HSA_STEP_ERR_NULL;
  const int half = head_dim / 2, sp = head_dim / 6;
  const int band_pairs[3] = {(head_dim - 4 * sp) / 2, sp, sp};
  const int band_rows[3] = {grid_f, grid_h, grid_w};
  int row0 = 0, pair0 = 0;
  for (int b = 0; b < 3; ++b) {
    for (int c = 0; c < band_rows[b]; ++c) {
      float* row = table_host + (size_t)(row0 + c) * head_dim;
      for (int k = 0; k < half; ++k) {
        const int j = k - pair0;
        double cs = 0.0, sn = 0.0;
        if (j >= 0 && j < band_pairs[b]) {
          const double ang = c * pow((double)theta, -2.0 * j / (2.0 * band_pairs[b]));
          cs = cos(ang);
          sn = sin(ang);
        }
        row[2 * k] = (float)cs;
        row[2 * k + 1] = (float)sn;
      }
    }
    row0 += band_rows[b];
    pair0 += band_pairs[b];
  }
  return HSA_STEP_OK;
}

HSA_API int hsa_reorder_plan(const int32_t* budget, int64_t n_tokens, int32_t T, int32_t* perm,
                             int32_t* n_lead_dev, int32_t* n_lead_host, hipStream_t stream) {
  if (n_tokens < 0 || n_tokens > kMaxRows) return HSA_STEP_ERR_SHAPE;
  if (T < 1) return HSA_STEP_ERR_BUDGET;
  if (!n_lead_dev || (n_tokens > 0 && (!budget || !perm))) return HSA_STEP_ERR_NULL;
  if (!aligned(budget, 4) || !aligned(perm, 4) || !aligned(n_lead_dev, 4)) return HSA_STEP_ERR_SHAPE;
  const size_t nb = (size_t)n_tokens * 4;
  if (overlaps(perm, nb, budget, nb) || overlaps(n_lead_dev, 4, budget, nb) ||
      overlaps(n_lead_dev, 4, perm, nb))
    return HSA_STEP_ERR_ALIAS;
  if (hsa::launch_reorder_plan(budget, (int)n_tokens, T, perm, n_lead_dev, stream) != hipSuccess)
    return HSA_STEP_ERR_LAUNCH;
  if (n_lead_host) {
    int32_t v = 0;
    if (hipMemcpyAsync(&v, n_lead_dev, 4, hipMemcpyDeviceToHost, stream) != hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess)
      return HSA_STEP_ERR_LAUNCH;
    *n_lead_host = v;
    if (v < 0) return HSA_STEP_ERR_BUDGET;
  }
  return HSA_STEP_OK;
}

HSA_API int hsa_permute_rows(const void* src, const int32_t* perm, int64_t n_rows, int64_t row_bytes,
                             int32_t inverse, void* dst, hipStream_t stream) {
  if (n_rows < 0 || n_rows > kMaxRows || row_bytes < 0) return HSA_STEP_ERR_SHAPE;
  if (!fits(n_rows, row_bytes)) return HSA_STEP_ERR_SHAPE;
  if (n_rows == 0 || row_bytes == 0) return HSA_STEP_OK;
  if (!src || !perm || !dst) return HSA_STEP_ERR_NULL;
  if (!aligned(perm, 4)) return HSA_STEP_ERR_SHAPE;
  const size_t b = (size_t)n_rows * row_bytes;
  if (overlaps(src, b, dst, b) || overlaps(perm, (size_t)n_rows * 4, dst, b))
    return HSA_STEP_ERR_ALIAS;
  return launch_status(hsa::launch_permute_rows(src, perm, n_rows, row_bytes, inverse != 0, dst,
                                                stream));
}

HSA_API int hsa_l1_rel_accumulate(const float* v, float* v_prev, int64_t n_tokens,
                                  int32_t channels, double* acc, int32_t first,
                                  hipStream_t stream) {
  if (n_tokens < 0 || n_tokens > kMaxRows || channels < 0) return HSA_STEP_ERR_SHAPE;
  if (!fits(n_tokens, channels, 4)) return HSA_STEP_ERR_SHAPE;
  if (n_tokens == 0) return HSA_STEP_OK;
  if (!v || !v_prev || !acc) return HSA_STEP_ERR_NULL;
  if (!aligned(v, 4) || !aligned(v_prev, 4) || !aligned(acc, 8)) return HSA_STEP_ERR_SHAPE;
  const size_t vb = (size_t)n_tokens * channels * 4, ab = (size_t)n_tokens * 8;
  if (overlaps(v_prev, vb, v, vb) || overlaps(acc, ab, v, vb) || overlaps(acc, ab, v_prev, vb))
    return HSA_STEP_ERR_ALIAS;
  return launch_status(hsa::launch_l1_rel(v, v_prev, n_tokens, channels, acc, first != 0, stream));
}

HSA_API int hsa_assign_budgets_by_key(const double* keys, int64_t n_tokens, int32_t T,
                                      const int32_t* group_budget, const int64_t* group_size,
                                      int32_t n_groups, int32_t* budget, hipStream_t stream) {
  if (n_tokens < 0 || n_tokens > kMaxRows) return HSA_STEP_ERR_SHAPE;
  hsa::GroupTable tab{};
  const int st = make_group_table(T, group_budget, group_size, n_groups, n_tokens, &tab);
  if (st != HSA_STEP_OK) return st;
  if (n_tokens == 0) return HSA_STEP_OK;
  if (!keys || !budget) return HSA_STEP_ERR_NULL;
  if (!aligned(keys, 8) || !aligned(budget, 4)) return HSA_STEP_ERR_SHAPE;
  if (overlaps(budget, (size_t)n_tokens * 4, keys, (size_t)n_tokens * 8)) return HSA_STEP_ERR_ALIAS;
  return launch_status(hsa::launch_rank_budgets(keys, n_tokens, tab, budget, stream));
}

HSA_API int hsa_stack_iteration(const hsa_stack* s, int32_t T, int32_t iter, int32_t margin,
                                int32_t outside_period, float sigma_i, float sigma_next,
                                const int32_t* group_budget, const int64_t* group_size,
                                int32_t n_groups, int32_t selection, int32_t* n_active_host,
                                int32_t* refreshed_host, hipStream_t stream) {
  if (!s) return HSA_STEP_ERR_NULL;
  const size_t es = elem_size(s->dtype);
  if (!es) return HSA_STEP_ERR_DTYPE;
  const int64_t N = s->n_tokens;
  const int L = s->n_layers, C = s->channels, dh = s->head_dim;
  const int F = s->ffn_dim, Lc = s->ctx_len;
  if (N < 1 || N > kMaxRows || L < 0 || L > kMaxLayers || s->heads <= 0 || (dh != 64 && dh != 128) ||
      C <= 0 || s->reserved != 0 || s->reserved2 != 0 || (int64_t)s->heads * dh > INT32_MAX / 4 ||
      F < 0 || Lc < 0 || Lc > kMaxRows)
    return HSA_STEP_ERR_SHAPE;
  {
    const int64_t dd = (int64_t)s->heads * dh;
    if (!fits(N, dd, 4) || !fits(N, C, 4) || !fits(N, F, 4) || !fits(dd, dd, 4) || !fits(F, dd, 4) ||
        !fits(Lc, dd, 4) || !fits(C, dd, 4))
      return HSA_STEP_ERR_SHAPE;
  }
  const bool rope = s->rope_cs != nullptr;
  const bool prefix = s->prefix_cache != 0;
  if (s->reserved3 != 0 || (s->prefix_cache != 0 && s->prefix_cache != 1)) return HSA_STEP_ERR_SHAPE;
  if (prefix && (s->n_cached < 0 || s->n_cached > N || (s->n_cached % 64 != 0 && s->n_cached != N)))
    return HSA_STEP_ERR_SHAPE;
  if (prefix && n_groups != 0) return HSA_STEP_ERR_BUDGET;
  const int64_t n_rows_cache = prefix ? s->n_cached : N;  // rows of each layer's cache
  const int64_t n_tail = N - n_rows_cache;
  if (rope && (s->grid_f < 1 || s->grid_h < 1 || s->grid_w < 1 ||
               (int64_t)s->grid_f * s->grid_h * s->grid_w < N ||
               (int64_t)s->grid_f * s->grid_h * s->grid_w > kMaxRows))
    return HSA_STEP_ERR_SHAPE;
  const int d = s->heads * dh;
  if (s->dtype == HSA_STEP_BF16 && (C % 64 != 0 || F % 64 != 0)) return HSA_STEP_ERR_SHAPE;
  if (T < 1 || iter < 0 || iter >= T || margin < 0 || margin > T / 2) return HSA_STEP_ERR_BUDGET;
  if (outside_period < 1 || T % outside_period != 0) return HSA_STEP_ERR_BUDGET;
  if (selection != HSA_SELECT_VELOCITY_NORM && selection != HSA_SELECT_L1_REL)
    return HSA_STEP_ERR_BUDGET;
  const bool l1rel = n_groups != 0 && selection == HSA_SELECT_L1_REL;
  if (l1rel && (margin < 2 || outside_period != 1)) return HSA_STEP_ERR_BUDGET;
  hsa::GroupTable tab{};
  if (n_groups != 0) {
    if (n_groups < 0) return HSA_STEP_ERR_BUDGET;
    const int st = make_group_table(T, group_budget, group_size, n_groups, N, &tab);
    if (st != HSA_STEP_OK) return st;
  }
  if (!s->w_embed || !s->w_head || !s->x || !s->v_hat || !s->budget || !s->idx || !s->n_active ||
      !s->xa || !s->h || !s->q || !s->o || !s->v_fresh || !s->row_scale ||
      (n_groups && !s->keys) || (l1rel && !s->v_prev) || (F > 0 && !s->f) ||
      (n_tail > 0 && (!s->k_tail || !s->v_tail)))
    return HSA_STEP_ERR_NULL;
  if (L > 0 && (!s->w_layers || !s->caches || (Lc > 0 && !s->w_cross) || (F > 0 && !s->w_ffn)))
    return HSA_STEP_ERR_NULL;
  for (int i = 0; i < 4 * L; ++i)
    if (!s->w_layers[i] || (Lc > 0 && !s->w_cross[i])) return HSA_STEP_ERR_NULL;
  for (int i = 0; i < 2 * L; ++i)
    if (!s->caches[i] || (F > 0 && !s->w_ffn[i])) return HSA_STEP_ERR_NULL;

  const size_t row_d = (size_t)d * es, row_c = (size_t)C * es;
  std::vector<Span> written = {
      {s->x, (size_t)N * C * 4},   {s->v_hat, (size_t)N * C * 4}, {s->budget, (size_t)N * 4},
      {s->idx, (size_t)N * 4},     {s->n_active, 4},              {s->xa, (size_t)N * row_c},
      {s->h, (size_t)N * row_d},   {s->q, (size_t)N * row_d},     {s->o, (size_t)N * row_d},
      {s->v_fresh, (size_t)N * C * 4}, {s->row_scale, (size_t)N * 4}};
  if (n_groups) written.push_back({s->keys, (size_t)N * 8});
  if (l1rel) written.push_back({s->v_prev, (size_t)N * C * 4});
  if (F > 0) written.push_back({s->f, (size_t)N * F * es});
  if (n_tail > 0) {
    written.push_back({s->k_tail, (size_t)n_tail * row_d});
    written.push_back({s->v_tail, (size_t)n_tail * row_d});
  }
  if (s->attn_parts_bytes < 0 || (s->attn_parts_bytes > 0 && !s->attn_parts)) return HSA_STEP_ERR_SHAPE;
  const bool parts = s->attn_parts && s->attn_parts_bytes > 0 && s->dtype == HSA_STEP_BF16;
  if (parts) written.push_back({s->attn_parts, (size_t)s->attn_parts_bytes});
  for (int i = 0; i < 2 * L; ++i) written.push_back({s->caches[i], (size_t)n_rows_cache * row_d});
  std::vector<Span> weights = {{s->w_embed, (size_t)d * row_c}, {s->w_head, (size_t)C * row_d}};
  for (int i = 0; i < 4 * L; ++i) weights.push_back({s->w_layers[i], (size_t)d * row_d});
  for (int l = 0; l < L && Lc > 0; ++l) {
    const void* const* wc = s->w_cross + 4 * l;
    weights.push_back({wc[0], (size_t)d * row_d});
    weights.push_back({wc[1], (size_t)d * row_d});
    weights.push_back({wc[2], (size_t)Lc * row_d});
    weights.push_back({wc[3], (size_t)Lc * row_d});
  }
  for (int i = 0; i < 2 * L && F > 0; ++i) weights.push_back({s->w_ffn[i], (size_t)F * row_d});
  if (rope) {
    weights.push_back({s->rope_cs, hsa_rope_table_floats(dh, s->grid_f, s->grid_h, s->grid_w) * 4});
    if (s->pos) weights.push_back({s->pos, (size_t)N * 4});
  }
  for (const Span& b : written)
    if (!aligned(b.p, 16)) return HSA_STEP_ERR_SHAPE;
  for (const Span& b : weights) {
    const bool table = rope && (b.p == s->rope_cs || b.p == s->pos);
    if (!aligned(b.p, table ? 8 : 16)) return HSA_STEP_ERR_SHAPE;
  }
  if (any_overlap(written) || any_overlap(written, weights)) return HSA_STEP_ERR_ALIAS;

  // 1. active set and its size on the host
  if (hsa::launch_active_set(s->budget, (int)N, T, iter, margin, outside_period, s->idx,
                             s->n_active, stream) != hipSuccess)
    return HSA_STEP_ERR_LAUNCH;
  int32_t n = 0;
  if (hipMemcpyAsync(&n, s->n_active, 4, hipMemcpyDeviceToHost, stream) != hipSuccess ||
      hipStreamSynchronize(stream) != hipSuccess)
    return HSA_STEP_ERR_LAUNCH;
  if (n < 0 || n > N) return HSA_STEP_ERR_BUDGET;
  if (n_tail > 0) {  // the baseline suffix must be active: the last n_tail entries of idx are it
    if (n < n_tail) return HSA_STEP_ERR_BUDGET;
    int32_t first = -1;
    if (hipMemcpy(&first, s->idx + (n - n_tail), 4, hipMemcpyDeviceToHost) != hipSuccess)
      return HSA_STEP_ERR_LAUNCH;
    if (first != n_rows_cache) return HSA_STEP_ERR_BUDGET;
  }
  if (n_active_host) *n_active_host = n;
  if (refreshed_host) *refreshed_host = 0;
  // a refresh iteration (step 4) needs a fresh velocity for every token: refuse
  // it before anything that changes the caller's state is enqueued
  const bool refresh_now = n_groups && !l1rel && iter % refresh_period(T, group_budget, n_groups) == 0;
  const bool l1_now = l1rel && iter < margin;
  if ((refresh_now || l1_now) && n != N) return HSA_STEP_ERR_BUDGET;

  // 2. the stack on the active rows
  const int dt = s->dtype;
  const bool bf = dt == HSA_STEP_BF16;
  const float scale = 1.0f / sqrtf((float)dh);
  auto ok = [](hipError_t e) { return e == hipSuccess; };
  auto rms = [&]() { return ok(hsa::launch_row_rms_scale(s->h, bf, n, d, kRmsEps, s->row_scale, stream)); };
  auto attend = [&](const void* q, const void* k, const void* v, int n_kv, const void* k2 = nullptr,
                    const void* v2 = nullptr, int n_split = 0x7fffffff) {
    return ok(bf ? hsa::launch_attention_bf16(q, k, v, s->o, n, n_kv, s->heads, dh, scale, stream,
                                              k2, v2, n_split, parts ? s->attn_parts : nullptr,
                                              parts ? (size_t)s->attn_parts_bytes : 0)
                 : hsa::launch_attention_f32(q, k, v, s->o, n, n_kv, s->heads, dh, scale, stream, k2,
                                             v2, n_split));
  };
  auto gemm = [&](const RowGemm& g) { return ok(launch_gemm(dt, g, stream)); };
  if (n > 0) {
    if (!ok(hsa::launch_gather_latent(s->x, s->idx, n, N, C, bf, s->xa, stream)) ||
        !gemm(compact_gemm(s->xa, n, C, s->w_embed, d, nullptr, nullptr, false, s->h)))
      return HSA_STEP_ERR_LAUNCH;
    for (int l = 0; l < L; ++l) {
      const void* const* w = s->w_layers + 4 * l;
      void* kc = s->caches[2 * l];
      void* vc = s->caches[2 * l + 1];
      // self-attention: Q/K/V of rms(h) with the cache overwrite, all N cached rows
      RowGemm g{};
      g.A = s->h;
      g.a_rows = nullptr;
      g.a_limit = n;
      g.M = n;
      g.Nc = d;
      g.K = d;
      g.lda = g.ldb = g.ldc = d;
      g.out[0] = {w[0], s->q, nullptr, n};
      g.out[1] = {w[1], kc, s->idx, (int)N};
      g.out[2] = {w[2], vc, s->idx, (int)N};
      if (n_tail > 0) {  // baseline rows: fresh keys and values only
        g.out[1].C2 = s->k_tail;
        g.out[1].c_split = (int)n_rows_cache;
        g.out[2].C2 = s->v_tail;
        g.out[2].c_split = (int)n_rows_cache;
      }
      g.n_out = 3;
      g.row_scale = s->row_scale;
      if (rope) {
        g.rope_cs = reinterpret_cast<const hsa::f32x2*>(s->rope_cs);
        g.rope_tok = s->idx;
        g.rope_pos = s->pos;
        g.rope_outs = 3;  // Q and K
        g.rope_dh = dh;
        g.rope_nt = (dh - 4 * (dh / 6)) / 2;
        g.rope_nh = dh / 6;
        g.rope_f = s->grid_f;
        g.rope_h = s->grid_h;
        g.rope_w = s->grid_w;
      }
      const bool split = n_tail > 0;
      if (!rms() || !gemm(g) ||
          !attend(s->q, kc, vc, (int)N, split ? s->k_tail : nullptr, split ? s->v_tail : nullptr,
                  split ? (int)n_rows_cache : 0x7fffffff) ||
          !gemm(compact_gemm(s->o, n, d, w[3], d, nullptr, s->h, false, s->h)))
        return HSA_STEP_ERR_LAUNCH;
      if (Lc > 0) {  // cross-attention of the active rows to the context
        const void* const* wc = s->w_cross + 4 * l;
        if (!rms() || !gemm(compact_gemm(s->h, n, d, wc[0], d, s->row_scale, nullptr, false, s->q)) ||
            !attend(s->q, wc[2], wc[3], Lc) ||
            !gemm(compact_gemm(s->o, n, d, wc[1], d, nullptr, s->h, false, s->h)))
          return HSA_STEP_ERR_LAUNCH;
      }
      if (F > 0) {  // feed-forward network of the active rows
        const void* const* wf = s->w_ffn + 2 * l;
        RowGemm up = compact_gemm(s->h, n, d, wf[0], F, s->row_scale, nullptr, false, s->f);
        up.gelu = 1;
        if (!rms() || !gemm(up) ||
            !gemm(compact_gemm(s->f, n, F, wf[1], d, nullptr, s->h, false, s->h)))
          return HSA_STEP_ERR_LAUNCH;
      }
    }
    if (!rms() ||
        !gemm(compact_gemm(s->h, n, d, s->w_head, C, s->row_scale, nullptr, bf, s->v_fresh)))
      return HSA_STEP_ERR_LAUNCH;
  }

  // 3. velocity cache refresh of the active rows, Euler step of every token
  const float dsig = sigma_next - sigma_i;  // fp32 difference
  if (!ok(hsa::launch_cached_euler(s->x, s->v_hat, n > 0 ? s->v_fresh : nullptr, s->idx, n, N, C,
                                   dsig, stream)))
    return HSA_STEP_ERR_LAUNCH;

  // 4. group membership
  double* keys = static_cast<double*>(s->keys);
  if (refresh_now) {
    if (!ok(hsa::launch_assign_budgets(s->v_hat, N, C, tab, keys, s->budget, stream)))
      return HSA_STEP_ERR_LAUNCH;
    if (refreshed_host) *refreshed_host = 1;
  }
  if (l1_now) {
    if (!ok(hsa::launch_l1_rel(s->v_hat, s->v_prev, N, C, keys, iter == 0, stream)))
      return HSA_STEP_ERR_LAUNCH;
    if (iter == margin - 1) {
      if (!ok(hsa::launch_rank_budgets(keys, N, tab, s->budget, stream))) return HSA_STEP_ERR_LAUNCH;
      if (refreshed_host) *refreshed_host = 1;
    }
  }
  return HSA_STEP_OK;
}
