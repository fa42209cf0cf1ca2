/*
 * hsa_step.h -- C ABI of the HSA active-token layer step for AMD MI355X (gfx950).
 *
 * Heterogeneous Step Allocation (HSA) gives every token n of an N-token latent
 * sequence its own step budget s_n, a divisor of the total step count T. At
 * iteration i only the active set A_i takes a model step; every other token
 * keeps its cached key/value rows and its cached velocity. This library
 * implements the per-layer hot path of one iteration on one GPU:
 *
 *   hsa_build_active_set   A_i from the budgets            (Section 2.2, Eq. 5 rule;
 *                                                           Section 2.5 window)
 *   hsa_qkv_scatter        fresh Q/K/V of A_i, K/V cache    (Section 2.3, steps 1-2)
 *                          rows A_i overwritten
 *   hsa_active_attention   active queries against all N     (Section 2.3, step 3 and
 *                          cached rows, output projection,   the paragraph after it)
 *                          result scattered to rows A_i
 *   hsa_cached_euler       x <- x + v_hat (sigma_{i+1} -     (Section 2.4, Eq. 6)
 *                          sigma_i) over all N tokens
 *
 * Conventions (all entry points):
 *   - Pointers are device pointers unless the name ends in _host.
 *   - Matrices are row-major. A token-indexed tensor has one row per token.
 *     Caches and outputs are [n_tokens, d] with d = heads * head_dim; head h
 *     occupies columns [h*head_dim, (h+1)*head_dim).
 *   - Weights have the [d_out, d_in] orientation: y = x W^T (the layout of a
 *     torch.nn.Linear weight). No biases.
 *   - dtype: HSA_STEP_F32 (everything fp32) or HSA_STEP_BF16 (activations,
 *     weights and caches bf16; products accumulated in fp32; results rounded
 *     to bf16 to nearest-even).
 *   - The caller owns every buffer. The library allocates no device memory,
 *     keeps no state between calls and never synchronizes the stream, except
 *     where an entry point says so. Work is enqueued on `stream` (0 = the
 *     null stream) in call order; calls on one stream see each other's
 *     results.
 *   - Every entry point returns an hsa_step_status. Arguments are checked on
 *     the host before anything is enqueued; on an error nothing is enqueued.
 *     HSA_STEP_ERR_LAUNCH reports a HIP error from enqueueing (or from the
 *     one synchronizing call).
 *   - Index lists hold int32 token indices. An index list produced by
 *     hsa_build_active_set is ascending and duplicate-free; the other entry
 *     points require duplicate-free indices in [0, n_tokens). Kernels never
 *     access memory outside the buffers for an out-of-range index: such a row
 *     is skipped (its result is unspecified), it does not fault.
 */
#ifndef HSA_STEP_H
#define HSA_STEP_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum hsa_step_status {
  HSA_STEP_OK = 0,
  HSA_STEP_ERR_NULL = 1,      /* a required pointer is NULL */
  HSA_STEP_ERR_SHAPE = 2,     /* sizes negative, inconsistent or unsupported */
  HSA_STEP_ERR_BUDGET = 3,    /* T, iteration or margin out of range, or a budget that
                                 does not divide T (reported by hsa_build_active_set) */
  HSA_STEP_ERR_DTYPE = 4,     /* unknown dtype */
  HSA_STEP_ERR_ALIAS = 5,     /* an output overlaps a buffer it must not overlap */
  HSA_STEP_ERR_WORKSPACE = 6, /* workspace missing or too small */
  HSA_STEP_ERR_LAUNCH = 7     /* HIP error while enqueueing or synchronizing */
} hsa_step_status;

typedef enum hsa_step_dtype { HSA_STEP_F32 = 0, HSA_STEP_BF16 = 1 } hsa_step_dtype;

/* Human-readable name of a status code (static string, never NULL). */
const char* hsa_step_status_string(int status);

/*
 * Active set A_i (Section 2.2: token n is active at iteration i iff
 * i mod (T / s_n) == 0; Section 2.5: with margin m > 0 every token is active
 * for i < m and for i > T - m - 1).
 *
 *   budget[n_tokens]   int32 step budgets s_n; each must satisfy 1 <= s_n <= T
 *                      and T % s_n == 0 (Eq. 5). Checked on the device.
 *   T, iter            1 <= T; 0 <= iter < T.
 *   margin             0 <= margin <= T/2; 0 disables the window.
 *   idx                int32 output, capacity n_tokens; receives A_i in
 *                      ascending order in idx[0 .. n_active).
 *   n_active_dev       int32 output (one element): |A_i|, or -1 if some budget
 *                      is invalid (then idx is unspecified).
 *   n_active_host      optional host int32*: if not NULL the call copies
 *                      n_active_dev to it and synchronizes the stream (the one
 *                      per-iteration host read-back), and returns
 *                      HSA_STEP_ERR_BUDGET if a budget was invalid.
 *   n_tokens           0 <= n_tokens < 2^31.
 */
int hsa_build_active_set(const int32_t* budget, int64_t n_tokens, int32_t T, int32_t iter,
                         int32_t margin, int32_t* idx, int32_t* n_active_dev,
                         int32_t* n_active_host, hipStream_t stream);

/*
 * Fresh Q/K/V for the active rows and the KV-cache overwrite (Section 2.3,
 * steps 1 and 2). For j < n_active, with token t = idx[j]:
 *   input row  r_j = x[t]  (x_compact == 0, x is [n_tokens, d])
 *              r_j = x[j]  (x_compact != 0, x is [n_active, d], the compact
 *                           hidden state of a deeper layer)
 *   q_out[j]   = r_j Wq^T             (compact, [n_active, d])
 *   k_cache[t] = r_j Wk^T,  v_cache[t] = r_j Wv^T
 * Cache rows of tokens not in idx are not written (bit-for-bit unchanged).
 *   wq, wk, wv      [d, d] each.
 *   d               d > 0; for HSA_STEP_BF16, d % 64 == 0.
 * q_out must not overlap x, the weights or the caches; the caches must not
 * overlap x, the weights or each other (HSA_STEP_ERR_ALIAS).
 */
int hsa_qkv_scatter(int dtype, const void* x, int32_t x_compact, const int32_t* idx,
                    int32_t n_active, int64_t n_tokens, int32_t d, const void* wq,
                    const void* wk, const void* wv, void* q_out, void* k_cache, void* v_cache,
                    hipStream_t stream);

/*
 * Attention of the active queries against the full cache (Section 2.3,
 * step 3), without the output projection. Per head h and active row j:
 *   o[j, h] = softmax_n( scale * <q[j, h], k_cache[n, h]> ) v_cache[n, h],
 * the softmax running over all n < n_tokens (no mask).
 *   q, o            [n_active, d] compact; k_cache, v_cache [n_tokens, d].
 *   d = heads * head_dim; head_dim in {64, 128}; n_tokens >= 1 if n_active > 0.
 *   scale           softmax scale (1/sqrt(head_dim) for standard attention).
 * o must not overlap q or the caches.
 */
int hsa_attention_core(int dtype, const void* q, const void* k_cache, const void* v_cache,
                       int32_t n_active, int64_t n_tokens, int32_t heads, int32_t head_dim,
                       float scale, void* o, hipStream_t stream);

/*
 * Output projection of the active rows, scattered back to their tokens
 * (Section 2.3: everything after self-attention acts on A_i only):
 *   out[idx[j]] = o[j] Wo^T for j < n_active; other rows of out untouched.
 *   o [n_active, d], wo [d, d], out [n_tokens, d]. d % 64 == 0 for bf16.
 * out must not overlap o or wo.
 */
int hsa_out_scatter(int dtype, const void* o, const int32_t* idx, int32_t n_active,
                    int64_t n_tokens, int32_t d, const void* wo, void* out, hipStream_t stream);

/* Workspace bytes hsa_active_attention needs: one compact [n_active, d]
 * tensor of the dtype. 0 for an unknown dtype or negative sizes. */
size_t hsa_attention_workspace_bytes(int dtype, int32_t n_active, int32_t d);

/*
 * Active-query attention followed by the output projection and the scatter
 * of the result (Section 2.3, step 3 and the paragraph after it): for each
 * active row j, out[idx[j]] = (attention of q[j] over all n_tokens cached
 * rows, per head) Wo^T. Equivalent to hsa_attention_core into `workspace`
 * followed by hsa_out_scatter. Rows of out not in idx are untouched.
 *   workspace       device buffer of at least
 *                   hsa_attention_workspace_bytes(dtype, n_active, d) bytes,
 *                   owned by the caller; its contents are overwritten.
 * out must not overlap q, the caches, wo or the workspace.
 */
int hsa_active_attention(int dtype, const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* idx, int32_t n_active, int64_t n_tokens, int32_t heads,
                         int32_t head_dim, float scale, const void* wo, void* out,
                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/*
 * Cached Euler update (Section 2.4, Eq. 6), fp32, for all n_tokens tokens:
 *   if v_fresh != NULL: v_cache[idx[j]] = v_fresh[j] for j < n_active
 *                       (active tokens take their fresh velocity);
 *   then x[n, c] = fmaf(v_cache[n, c], sigma_next - sigma_i, x[n, c]) for every
 *   n < n_tokens, c < channels, the difference taken in fp32.
 *   x, v_cache      [n_tokens, channels] fp32; v_fresh [n_active, channels].
 * With v_fresh == NULL, idx and n_active are ignored (the velocity cache is
 * already current, e.g. it was the scatter target of hsa_out_scatter).
 * x must not overlap v_cache or v_fresh; v_fresh must not overlap v_cache.
 */
int hsa_cached_euler(float* x, float* v_cache, const float* v_fresh, const int32_t* idx,
                     int32_t n_active, int64_t n_tokens, int32_t channels, float sigma_i,
                     float sigma_next, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HSA_STEP_H */
