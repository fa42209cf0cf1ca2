// C ABI entry points of the HSA step library: host-side argument checks, then
// kernel launches on the caller's stream. See include/hsa_step.h for the
// contract of every call.
#include <math.h>

#include "api_util.h"

using namespace hsa_api;

HSA_API const char* hsa_step_status_string(int status) {
  switch (status) {
    case HSA_STEP_OK: return "ok";
    case HSA_STEP_ERR_NULL: return "required pointer is NULL";
    case HSA_STEP_ERR_SHAPE: return "sizes negative, inconsistent or unsupported";
    case HSA_STEP_ERR_BUDGET: return "schedule out of range or a budget does not divide T";
    case HSA_STEP_ERR_DTYPE: return "unknown dtype";
    case HSA_STEP_ERR_ALIAS: return "output overlaps a buffer it must not overlap";
    case HSA_STEP_ERR_WORKSPACE: return "workspace missing or too small";
    case HSA_STEP_ERR_LAUNCH: return "HIP launch or synchronization error";
    default: return "unknown status";
  }
}

HSA_API int32_t hsa_window_margin(int32_t center_percent, int32_t T) {
  if (center_percent < 0 || center_percent > 100 || T < 1) return -1;
  return (int32_t)(((int64_t)(100 - center_percent) * T) / 200);
}

HSA_API int hsa_build_active_set_window(const int32_t* budget, int64_t n_tokens, int32_t T,
                                        int32_t iter, int32_t margin, int32_t outside_period,
                                        int32_t* idx, int32_t* n_active_dev,
                                        int32_t* n_active_host, hipStream_t stream) {
  if (n_tokens < 0 || n_tokens > kMaxRows) return HSA_STEP_ERR_SHAPE;
  if (T < 1 || iter < 0 || iter >= T || margin < 0 || margin > T / 2) return HSA_STEP_ERR_BUDGET;
  if (outside_period < 1 || T % outside_period != 0) return HSA_STEP_ERR_BUDGET;
  if (!n_active_dev || (n_tokens > 0 && (!budget || !idx))) return HSA_STEP_ERR_NULL;
  const size_t nb = (size_t)n_tokens * 4;
  if (overlaps(idx, nb, budget, nb) || overlaps(n_active_dev, 4, budget, nb) ||
      overlaps(n_active_dev, 4, idx, nb))
    return HSA_STEP_ERR_ALIAS;
  hipError_t e = hsa::launch_active_set(budget, (int)n_tokens, T, iter, margin, outside_period, idx,
                                        n_active_dev, stream);
  if (e != hipSuccess) return HSA_STEP_ERR_LAUNCH;
  if (n_active_host) {
    // straight into the caller's int: a direct DMA when it is pinned host memory
    if (hipMemcpyAsync(n_active_host, n_active_dev, sizeof(int32_t), hipMemcpyDeviceToHost, stream) !=
            hipSuccess ||
        hipStreamSynchronize(stream) != hipSuccess)
      return HSA_STEP_ERR_LAUNCH;
    if (*n_active_host < 0) return HSA_STEP_ERR_BUDGET;
  }
  return HSA_STEP_OK;
}

HSA_API int hsa_build_active_set(const int32_t* budget, int64_t n_tokens, int32_t T, int32_t iter,
                                 int32_t margin, int32_t* idx, int32_t* n_active_dev,
                                 int32_t* n_active_host, hipStream_t stream) {
  return hsa_build_active_set_window(budget, n_tokens, T, iter, margin, 1, idx, n_active_dev,
                                     n_active_host, stream);
}

HSA_API int hsa_qkv_scatter(int dtype, const void* x, int32_t x_compact, const int32_t* idx,
                            int32_t n_active, int64_t n_tokens, int32_t d, const void* wq,
                            const void* wk, const void* wv, void* q_out, void* k_cache,
                            void* v_cache, hipStream_t stream) {
  const size_t es = elem_size(dtype);
  if (!es) return HSA_STEP_ERR_DTYPE;
  if (d <= 0 || n_active < 0 || n_tokens < 0 || n_tokens > kMaxRows || n_active > n_tokens)
    return HSA_STEP_ERR_SHAPE;
  if (dtype == HSA_STEP_BF16 && d % 64 != 0) return HSA_STEP_ERR_SHAPE;
  if (!fits(n_tokens, d, es) || !fits(d, d, es)) return HSA_STEP_ERR_SHAPE;
  if (n_active == 0) return HSA_STEP_OK;
  if (!x || !idx || !wq || !wk || !wv || !q_out || !k_cache || !v_cache) return HSA_STEP_ERR_NULL;
  const size_t align = dtype == HSA_STEP_BF16 ? 16 : 4;
  const void* ptrs[] = {x, wq, wk, wv, q_out, k_cache, v_cache};
  for (const void* p : ptrs)
    if (!aligned(p, align)) return HSA_STEP_ERR_SHAPE;
  if (!aligned(idx, 4)) return HSA_STEP_ERR_SHAPE;
  const size_t row = (size_t)d * es;
  const size_t xb = row * (size_t)(x_compact ? n_active : n_tokens);
  const size_t wb = row * (size_t)d;
  const size_t qb = row * (size_t)n_active;
  const size_t cb = row * (size_t)n_tokens;
  const size_t ib = (size_t)n_active * 4;
  const void* ins[] = {x, wq, wk, wv, idx};
  const size_t inb[] = {xb, wb, wb, wb, ib};
  void* outs[] = {q_out, k_cache, v_cache};
  const size_t outb[] = {qb, cb, cb};
  for (int o = 0; o < 3; ++o) {
    for (int i = 0; i < 5; ++i)
      if (overlaps(outs[o], outb[o], ins[i], inb[i])) return HSA_STEP_ERR_ALIAS;
    for (int p = o + 1; p < 3; ++p)
      if (overlaps(outs[o], outb[o], outs[p], outb[p])) return HSA_STEP_ERR_ALIAS;
  }
  RowGemm g{};
  g.A = x;
  g.a_rows = x_compact ? nullptr : idx;
  g.a_limit = x_compact ? n_active : (int)n_tokens;
  g.M = n_active;
  g.Nc = d;
  g.K = d;
  g.lda = g.ldb = g.ldc = d;
  g.out[0] = {wq, q_out, nullptr, n_active};
  g.out[1] = {wk, k_cache, idx, (int)n_tokens};
  g.out[2] = {wv, v_cache, idx, (int)n_tokens};
  g.n_out = 3;
  return launch_status(dtype == HSA_STEP_BF16 ? hsa::launch_row_gemm_bf16(g, stream)
                                              : hsa::launch_row_gemm_f32(g, stream));
}

namespace {

// hsa_attention_core with an optional workspace for key parts (bf16 only)
int attention_core(int dtype, const void* q, const void* k_cache, const void* v_cache,
                   int32_t n_active, int64_t n_tokens, int32_t heads, int32_t head_dim,
                   float scale, void* o, void* parts_ws, size_t parts_bytes, hipStream_t stream) {
  const size_t es = elem_size(dtype);
  if (!es) return HSA_STEP_ERR_DTYPE;
  if (heads <= 0 || (head_dim != 64 && head_dim != 128) || n_active < 0 || n_tokens < 0 ||
      n_tokens > kMaxRows || (n_active > 0 && n_tokens < 1) || !(scale > 0.f) || !isfinite(scale))
    return HSA_STEP_ERR_SHAPE;
  if ((int64_t)heads * head_dim > INT32_MAX) return HSA_STEP_ERR_SHAPE;
  if (!fits(n_tokens, (int64_t)heads * head_dim, es)) return HSA_STEP_ERR_SHAPE;
  if (n_active == 0) return HSA_STEP_OK;
  if (!q || !k_cache || !v_cache || !o) return HSA_STEP_ERR_NULL;
  const size_t align = dtype == HSA_STEP_BF16 ? 16 : 4;
  if (!aligned(q, align) || !aligned(k_cache, align) || !aligned(v_cache, align) ||
      !aligned(o, align))
    return HSA_STEP_ERR_SHAPE;
  const size_t row = (size_t)heads * head_dim * es;
  const size_t ab = row * (size_t)n_active, cb = row * (size_t)n_tokens;
  if (overlaps(o, ab, q, ab) || overlaps(o, ab, k_cache, cb) || overlaps(o, ab, v_cache, cb))
    return HSA_STEP_ERR_ALIAS;
  if (parts_ws && (overlaps(parts_ws, parts_bytes, q, ab) || overlaps(parts_ws, parts_bytes, o, ab) ||
                   overlaps(parts_ws, parts_bytes, k_cache, cb) ||
                   overlaps(parts_ws, parts_bytes, v_cache, cb)))
    return HSA_STEP_ERR_ALIAS;
  if (parts_ws && !aligned(parts_ws, 16)) return HSA_STEP_ERR_SHAPE;
  hipError_t e = dtype == HSA_STEP_BF16
                     ? hsa::launch_attention_bf16(q, k_cache, v_cache, o, n_active, (int)n_tokens,
                                                  heads, head_dim, scale, stream, nullptr, nullptr,
                                                  0x7fffffff, parts_ws, parts_bytes)
                     : hsa::launch_attention_f32(q, k_cache, v_cache, o, n_active, (int)n_tokens,
                                                 heads, head_dim, scale, stream);
  return launch_status(e);
}

size_t round_up_256(size_t b) { return (b + 255) / 256 * 256; }

}  // namespace

HSA_API int hsa_attention_core(int dtype, const void* q, const void* k_cache, const void* v_cache,
                               int32_t n_active, int64_t n_tokens, int32_t heads,
                               int32_t head_dim, float scale, void* o, hipStream_t stream) {
  return attention_core(dtype, q, k_cache, v_cache, n_active, n_tokens, heads, head_dim, scale, o,
                        nullptr, 0, stream);
}

HSA_API int hsa_attention_core_parts(int dtype, const void* q, const void* k_cache,
                                     const void* v_cache, int32_t n_active, int64_t n_tokens,
                                     int32_t heads, int32_t head_dim, float scale, void* o,
                                     void* parts, size_t parts_bytes, hipStream_t stream) {
  return attention_core(dtype, q, k_cache, v_cache, n_active, n_tokens, heads, head_dim, scale, o,
                        parts_bytes > 0 ? parts : nullptr, parts ? parts_bytes : 0, stream);
}

HSA_API int hsa_out_scatter(int dtype, const void* o, const int32_t* idx, int32_t n_active,
                            int64_t n_tokens, int32_t d, const void* wo, void* out,
                            hipStream_t stream) {
  const size_t es = elem_size(dtype);
  if (!es) return HSA_STEP_ERR_DTYPE;
  if (d <= 0 || n_active < 0 || n_tokens < 0 || n_tokens > kMaxRows || n_active > n_tokens)
    return HSA_STEP_ERR_SHAPE;
  if (dtype == HSA_STEP_BF16 && d % 64 != 0) return HSA_STEP_ERR_SHAPE;
  if (!fits(n_tokens, d, es) || !fits(d, d, es)) return HSA_STEP_ERR_SHAPE;
  if (n_active == 0) return HSA_STEP_OK;
  if (!o || !idx || !wo || !out) return HSA_STEP_ERR_NULL;
  const size_t align = dtype == HSA_STEP_BF16 ? 16 : 4;
  if (!aligned(o, align) || !aligned(wo, align) || !aligned(out, align) || !aligned(idx, 4))
    return HSA_STEP_ERR_SHAPE;
  const size_t row = (size_t)d * es;
  const size_t outb = row * (size_t)n_tokens;
  if (overlaps(out, outb, o, row * (size_t)n_active) || overlaps(out, outb, wo, row * (size_t)d) ||
      overlaps(out, outb, idx, (size_t)n_active * 4))
    return HSA_STEP_ERR_ALIAS;
  RowGemm g{};
  g.A = o;
  g.a_rows = nullptr;
  g.a_limit = n_active;
  g.M = n_active;
  g.Nc = d;
  g.K = d;
  g.lda = g.ldb = g.ldc = d;
  g.out[0] = {wo, out, idx, (int)n_tokens};
  g.n_out = 1;
  return launch_status(dtype == HSA_STEP_BF16 ? hsa::launch_row_gemm_bf16(g, stream)
                                              : hsa::launch_row_gemm_f32(g, stream));
}

HSA_API size_t hsa_attention_workspace_bytes(int dtype, int32_t n_active, int32_t d) {
  const size_t es = elem_size(dtype);
  if (!es || n_active < 0 || d < 0) return 0;
  return es * (size_t)n_active * (size_t)d;
}

HSA_API size_t hsa_attention_parts_workspace_bytes(int dtype, int32_t n_active, int32_t heads,
                                                   int32_t head_dim) {
  if (heads < 0 || head_dim < 0 || (int64_t)heads * head_dim > INT32_MAX) return 0;
  const size_t base = hsa_attention_workspace_bytes(dtype, n_active, heads * head_dim);
  if (dtype != HSA_STEP_BF16 || base == 0) return base;
  return round_up_256(base) + hsa::attention_parts_bytes(hsa::kMaxKvParts, n_active, heads, head_dim);
}

HSA_API int hsa_active_attention(int dtype, const void* q, const void* k_cache,
                                 const void* v_cache, const int32_t* idx, int32_t n_active,
                                 int64_t n_tokens, int32_t heads, int32_t head_dim, float scale,
                                 const void* wo, void* out, void* workspace,
                                 size_t workspace_bytes, hipStream_t stream) {
  const size_t es = elem_size(dtype);
  if (!es) return HSA_STEP_ERR_DTYPE;
  if (heads <= 0 || head_dim <= 0 || (int64_t)heads * head_dim > INT32_MAX)
    return HSA_STEP_ERR_SHAPE;
  const int32_t d = heads * head_dim;
  if (n_active < 0 || n_tokens < 0 || n_active > n_tokens) return HSA_STEP_ERR_SHAPE;
  if (!fits(n_tokens, d, es) || !fits(d, d, es)) return HSA_STEP_ERR_SHAPE;
  if (n_active == 0) return HSA_STEP_OK;
  const size_t need = hsa_attention_workspace_bytes(dtype, n_active, d);
  if (!workspace || workspace_bytes < need) return HSA_STEP_ERR_WORKSPACE;
  // bytes past the compact O (from a 256-byte boundary) hold key parts
  void* parts_ws = nullptr;
  size_t parts_bytes = 0;
  if (dtype == HSA_STEP_BF16 && workspace_bytes > round_up_256(need)) {
    parts_ws = static_cast<char*>(workspace) + round_up_256(need);
    parts_bytes = workspace_bytes - round_up_256(need);
  }
  if (!out) return HSA_STEP_ERR_NULL;
  const size_t row = (size_t)d * es;
  const size_t outb = row * (size_t)n_tokens;
  if (overlaps(out, outb, workspace, need) || overlaps(out, outb, q, row * (size_t)n_active) ||
      overlaps(out, outb, k_cache, outb) || overlaps(out, outb, v_cache, outb) ||
      overlaps(workspace, need, q, row * (size_t)n_active) ||
      overlaps(workspace, need, k_cache, outb) || overlaps(workspace, need, v_cache, outb) ||
      overlaps(workspace, need, wo, row * (size_t)d) ||
      overlaps(workspace, need, idx, (size_t)n_active * 4))
    return HSA_STEP_ERR_ALIAS;
  // validate the second half before enqueueing the first
  if (!idx || !wo) return HSA_STEP_ERR_NULL;
  if (dtype == HSA_STEP_BF16 && d % 64 != 0) return HSA_STEP_ERR_SHAPE;
  const size_t align = dtype == HSA_STEP_BF16 ? 16 : 4;
  if (!aligned(workspace, align) || !aligned(wo, align) || !aligned(out, align) ||
      !aligned(idx, 4))
    return HSA_STEP_ERR_SHAPE;
  if (overlaps(out, outb, wo, row * (size_t)d) || overlaps(out, outb, idx, (size_t)n_active * 4))
    return HSA_STEP_ERR_ALIAS;
  if (parts_ws && (overlaps(out, outb, parts_ws, parts_bytes) ||
                   overlaps(wo, row * (size_t)d, parts_ws, parts_bytes) ||
                   overlaps(idx, (size_t)n_active * 4, parts_ws, parts_bytes)))
    return HSA_STEP_ERR_ALIAS;
  int st = attention_core(dtype, q, k_cache, v_cache, n_active, n_tokens, heads, head_dim, scale,
                          workspace, parts_ws, parts_bytes, stream);
  if (st != HSA_STEP_OK) return st;
  return hsa_out_scatter(dtype, workspace, idx, n_active, n_tokens, d, wo, out, stream);
}

HSA_API int hsa_cached_euler(float* x, float* v_cache, const float* v_fresh, const int32_t* idx,
                             int32_t n_active, int64_t n_tokens, int32_t channels, float sigma_i,
                             float sigma_next, hipStream_t stream) {
  if (n_tokens < 0 || n_tokens > kMaxRows || channels < 0) return HSA_STEP_ERR_SHAPE;
  if (!fits(n_tokens, channels, 4)) return HSA_STEP_ERR_SHAPE;
  if (v_fresh && (n_active < 0 || n_active > n_tokens)) return HSA_STEP_ERR_SHAPE;
  const size_t nb = (size_t)n_tokens * (size_t)channels * 4;
  if (nb == 0) return HSA_STEP_OK;
  if (!x || !v_cache) return HSA_STEP_ERR_NULL;
  if (v_fresh && n_active > 0 && !idx) return HSA_STEP_ERR_NULL;
  if (!aligned(x, 4) || !aligned(v_cache, 4) || (v_fresh && !aligned(v_fresh, 4)) ||
      (idx && !aligned(idx, 4)))
    return HSA_STEP_ERR_SHAPE;
  const size_t fb = v_fresh ? (size_t)n_active * (size_t)channels * 4 : 0;
  if (overlaps(x, nb, v_cache, nb) || overlaps(x, nb, v_fresh, fb) ||
      overlaps(v_cache, nb, v_fresh, fb) ||
      (v_fresh && (overlaps(x, nb, idx, (size_t)n_active * 4) ||
                   overlaps(v_cache, nb, idx, (size_t)n_active * 4))))
    return HSA_STEP_ERR_ALIAS;
  const float dsig = sigma_next - sigma_i;  // fp32 difference
  return launch_status(hsa::launch_cached_euler(x, v_cache, v_fresh, idx, v_fresh ? n_active : 0,
                                                n_tokens, channels, dsig, stream));
}
