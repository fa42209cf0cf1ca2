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

/* How a multi-layer loop sets group membership (Appendix B). */
typedef enum hsa_step_selection {
  HSA_SELECT_VELOCITY_NORM = 0, /* refresh from squared velocity norms where every schedule fires */
  HSA_SELECT_L1_REL = 1         /* strategy D: summed L1_rel (Eq. 7) over the initial full steps */
} hsa_step_selection;

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
 *                      HSA_STEP_ERR_BUDGET if a budget was invalid. Pinned
 *                      host memory (hipHostMalloc) makes the copy a direct
 *                      DMA; pageable memory works too.
 *   n_tokens           0 <= n_tokens < 2^31.
 */
int hsa_build_active_set(const int32_t* budget, int64_t n_tokens, int32_t T, int32_t iter,
                         int32_t margin, int32_t* idx, int32_t* n_active_dev,
                         int32_t* n_active_host, hipStream_t stream);

/*
 * Margin m of a phase-aware caching window over the centre k% of a T-step
 * trajectory (Section 2.5: m = floor((1 - k) T / 2)), in exact integer
 * arithmetic: m = ((100 - center_percent) * T) div 200. (Evaluated in
 * floating point, (1 - 0.8) * 40 / 2 falls just below 4 and floors to 3;
 * the printed HSA-50 runtime of Appendix C, 50%, needs m = 4: 49.6% of the
 * token-steps, against 47.5% with m = 3.) Host-only; enqueues nothing.
 *   center_percent   0 <= k <= 100 (100: no window, m = 0)
 *   T                T >= 1
 * Returns m (0 <= m <= T/2), or -1 for arguments out of range.
 */
int32_t hsa_window_margin(int32_t center_percent, int32_t T);

/*
 * The same with a choice of what happens outside the window (Section 2.5
 * says every token is active there; read literally, the HSA-25 preset of
 * Appendix C then takes 34.8% of the token-steps instead of its printed 25%).
 * Outside the window (margin > 0 and i < m or i > T - m - 1) every token is
 * active iff iter % outside_period == 0, and none is otherwise:
 *   outside_period 1          the literal rule (= hsa_build_active_set);
 *   outside_period T / s_max  every token follows the largest budget's
 *                             schedule there (24.8% for HSA-25).
 * outside_period must divide T (else HSA_STEP_ERR_BUDGET). Other arguments
 * as for hsa_build_active_set.
 */
int hsa_build_active_set_window(const int32_t* budget, int64_t n_tokens, int32_t T, int32_t iter,
                                int32_t margin, int32_t outside_period, int32_t* idx,
                                int32_t* n_active_dev, int32_t* n_active_host,
                                hipStream_t stream);

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
 * hsa_attention_core with a caller scratch for key parts (bf16): a launch of
 * few workgroups may split the cached rows into up to 4 parts and merge them
 * (the exact softmax of the concatenation; only the rounding order differs).
 *   parts           device scratch, 16-byte aligned, or NULL (no split);
 *                   its contents are overwritten
 *   parts_bytes     its size; with hsa_attention_parts_workspace_bytes(dtype,
 *                   n_active, heads, head_dim) - hsa_attention_workspace_bytes(
 *                   dtype, n_active, d) bytes every split fits
 * parts must not overlap q, o or the caches. Ignored for HSA_STEP_F32.
 */
int hsa_attention_core_parts(int dtype, const void* q, const void* k_cache, const void* v_cache,
                             int32_t n_active, int64_t n_tokens, int32_t heads, int32_t head_dim,
                             float scale, void* o, void* parts, size_t parts_bytes,
                             hipStream_t stream);

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

/* Workspace bytes with which hsa_active_attention may also split the cached
 * rows of a bf16 launch into up to 4 key parts: the compact tensor, rounded
 * up to 256 bytes, then 4 x n_active x heads x (head_dim + 2) fp32 values
 * (each part's unnormalized output and its softmax maximum and sum). The
 * library splits only when that fills the compute units better (a grid of
 * few workgroups: few heads or few active rows) and merges the parts in a
 * second kernel, an exact rearrangement of the softmax sum. For HSA_STEP_F32
 * this equals hsa_attention_workspace_bytes. 0 for invalid sizes. */
size_t hsa_attention_parts_workspace_bytes(int dtype, int32_t n_active, int32_t heads,
                                           int32_t head_dim);

/*
 * Active-query attention followed by the output projection and the scatter
 * of the result (Section 2.3, step 3 and the paragraph after it): for each
 * active row j, out[idx[j]] = (attention of q[j] over all n_tokens cached
 * rows, per head) Wo^T. Equivalent to hsa_attention_core into `workspace`
 * followed by hsa_out_scatter. Rows of out not in idx are untouched.
 *   workspace       device buffer of at least
 *                   hsa_attention_workspace_bytes(dtype, n_active, d) bytes,
 *                   owned by the caller; its contents are overwritten. For
 *                   bf16, the bytes past the compact tensor (from the next
 *                   256-byte boundary) may hold key parts; with
 *                   hsa_attention_parts_workspace_bytes bytes every split the
 *                   library chooses fits, with fewer it may split less.
 * out must not overlap q, the caches, wo or the workspace.
 */
int hsa_active_attention(int dtype, const void* q, const void* k_cache, const void* v_cache,
                         const int32_t* idx, int32_t n_active, int64_t n_tokens, int32_t heads,
                         int32_t head_dim, float scale, const void* wo, void* out,
                         void* workspace, size_t workspace_bytes, hipStream_t stream);

/* Size of the fixed device scratch of hsa_active_attention_noalloc: 96 MiB. */
#define HSA_STEP_NOALLOC_SCRATCH_BYTES (96u << 20)

/*
 * hsa_active_attention without a workspace argument, for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc). Same arguments, results and checks as
 * hsa_active_attention, with the workspace taken from a fixed array of
 * HSA_STEP_NOALLOC_SCRATCH_BYTES bytes in this library's device code: each
 * GPU the library runs on holds its own array until the process ends. The
 * call allocates nothing (no hipMalloc, no allocating library call). Its
 * first call on a device looks up the array's address there (the device the
 * stream belongs to must be current).
 *   Limit: hsa_attention_workspace_bytes(dtype, n_active, heads * head_dim)
 *   must not exceed HSA_STEP_NOALLOC_SCRATCH_BYTES (bf16 at d = 5120: up to
 *   9830 active rows; at d = 1536: up to 32768), else HSA_STEP_ERR_WORKSPACE
 *   and nothing is enqueued. Bytes past the compact output may hold key parts
 *   as for hsa_active_attention.
 *   Every call on one GPU shares that GPU's array: calls that may overlap in
 *   time on one GPU (different streams, different host threads without
 *   ordering) race and give unspecified results. Calls on one stream are
 *   ordered and safe. Nothing in the array needs to start at zero.
 * HSA_STEP_ERR_LAUNCH if the array's address cannot be found on the current
 * device.
 */
int hsa_active_attention_noalloc(int dtype, const void* q, const void* k_cache,
                                 const void* v_cache, const int32_t* idx, int32_t n_active,
                                 int64_t n_tokens, int32_t heads, int32_t head_dim, float scale,
                                 const void* wo, void* out, hipStream_t stream);

/*
 * Cached Euler update (Section 2.4, Eq. 6), fp32, for all n_tokens tokens:
 *   if v_fresh != NULL: v_cache[idx[j]] = v_fresh[j] for j < n_active
 *                       (active tokens take their fresh velocity);
 *   then x[n, c] = fmaf(v_cache[n, c], sigma_next - sigma_i, x[n, c]) for every
 *   n < n_tokens, c < channels, the difference taken in fp32.
 * One pass over the tokens (one kernel): every token reads its fresh row or
 * its cached row, x is advanced, and only fresh rows are written to v_cache.
 *   x, v_cache      [n_tokens, channels] fp32; v_fresh [n_active, channels].
 *   idx             int32 [n_active], strictly ascending, in [0, n_tokens)
 *                   (as hsa_build_active_set produces it). For another order
 *                   the result is unspecified (no access outside the buffers).
 * With v_fresh == NULL, idx and n_active are ignored (the velocity cache is
 * already current, e.g. it was the scatter target of hsa_out_scatter).
 * x must not overlap v_cache or v_fresh; v_fresh must not overlap v_cache.
 */
int hsa_cached_euler(float* x, float* v_cache, const float* v_fresh, const int32_t* idx,
                     int32_t n_active, int64_t n_tokens, int32_t channels, float sigma_i,
                     float sigma_next, hipStream_t stream);

/* ------------------------------------------------------------------------
 * Multi-layer sampling loop.
 *
 * A stack of self-attention layers driven by the HSA schedule (Sections
 * 2.2-2.4): the active tokens' latent rows are embedded, every layer
 * recomputes Q/K/V for those rows only, overwrites their rows of its own
 * cache and attends to all N cached rows, and the hidden state of the active
 * tokens stays compact (one row per active token) from the embedding to the
 * velocity head. A stack layer is h <- h + Attn(rms(h)) Wo^T with
 * rms(h) = h / sqrt(mean(h^2) + 1e-6) per row feeding Q/K/V; a final rms()
 * precedes the head. The patch embedding maps the C latent values of a token
 * to d, the velocity head maps d back to C (fp32). Weights are [d_out, d_in],
 * no biases.
 * ------------------------------------------------------------------------ */

/*
 * Active rows of the fp32 latent in the model dtype (the embedding input):
 *   xa[j][c] = dtype(x[idx[j]][c]) for j < n_active, c < channels,
 * bf16 rounded to nearest even. Rows whose index lies outside [0, n_tokens)
 * are written as zeros.
 *   x    [n_tokens, channels] fp32     xa   [n_active, channels] dtype
 * xa must not overlap x or idx.
 */
int hsa_gather_rows(int dtype, const float* x, const int32_t* idx, int32_t n_active,
                    int64_t n_tokens, int32_t channels, void* xa, hipStream_t stream);

/*
 * Per-row RMS factor of compact rows (the normalization before a layer's
 * Q/K/V projections and before the velocity head):
 *   scale[m] = 1 / sqrt(mean over k < d of x[m][k]^2 + eps),  m < n_rows,
 * squares summed in fp32. x [n_rows, d] dtype; scale [n_rows] fp32, which
 * must not overlap x. eps >= 0 and finite.
 */
int hsa_row_rms_scale(int dtype, const void* x, int32_t n_rows, int32_t d, float eps,
                      float* scale, hipStream_t stream);

/*
 * Compact row map of the stack (the embedding, the residual output
 * projection of a layer, the FFN, the velocity head; Section 2.3: after
 * attention every per-token computation runs on the active rows only):
 *   y[m] = act(s[m] (x[m] W^T)) (+ residual[m]),  m < n_rows,
 * with s = row_scale (1 if NULL) and act the tanh GELU 0.5 z (1 + tanh(
 * sqrt(2/pi) (z + 0.044715 z^3))) if gelu != 0, else the identity;
 * accumulated in fp32 and rounded once to out_dtype. With row_scale from
 * hsa_row_rms_scale(x) the product is rms(x) W^T.
 *   x          [n_rows, d_in] dtype     w  [d_out, d_in] dtype
 *   row_scale  NULL or [n_rows] fp32
 *   residual   NULL or [n_rows, d_out] out_dtype; it may be y itself (in-place
 *              h += ...), but must not overlap y otherwise
 *   y          [n_rows, d_out] out_dtype
 * out_dtype is dtype, or HSA_STEP_F32 with dtype HSA_STEP_BF16 (then no
 * residual and no GELU); GELU takes no residual. bf16 inputs need
 * d_in % 64 == 0, d_out % 4 == 0 and 16-byte aligned pointers. y must not
 * overlap x, w or row_scale.
 */
int hsa_linear(int dtype, const void* x, int32_t n_rows, int32_t d_in, const void* w,
               int32_t d_out, const float* row_scale, const void* residual, int32_t gelu,
               int out_dtype, void* y, hipStream_t stream);

/* Bytes of device workspace hsa_assign_budgets needs: 8 * n_tokens. */
size_t hsa_assign_budgets_workspace_bytes(int64_t n_tokens);

/*
 * Group refresh from velocity norms (Section 2.2 and Appendix B: group
 * sizes are fixed, membership follows a per-token velocity statistic,
 * smaller values to lower budgets). For every token t:
 *   key[t]  = sum over c = 0, 1, ..., channels-1 of v[t][c]^2 in float64
 *             (exact squares, added in channel order);
 *   rank[t] = number of tokens u with key[u] < key[t], or key[u] == key[t]
 *             and u < t (keys compared as IEEE bit patterns, NaN keys as one
 *             canonical positive NaN above every number);
 *   budget[t] = group_budget[k] for the group k with
 *               sum_{j<k} group_size[j] <= rank[t] < sum_{j<=k} group_size[j].
 *   v             [n_tokens, channels] fp32 velocities
 *   group_budget  HOST array, n_groups budgets, strictly ascending, each a
 *                 divisor of T (Eq. 5)
 *   group_size    HOST array, n_groups sizes >= 0 summing to n_tokens
 *   n_groups      1 .. 16
 *   budget        [n_tokens] int32, overwritten
 *   workspace     device buffer of hsa_assign_budgets_workspace_bytes
 * Group-table errors return HSA_STEP_ERR_BUDGET before any launch.
 */
int hsa_assign_budgets(const float* v, int64_t n_tokens, int32_t channels, int32_t T,
                       const int32_t* group_budget, const int64_t* group_size, int32_t n_groups,
                       int32_t* budget, void* workspace, size_t workspace_bytes,
                       hipStream_t stream);

/*
 * Rotary-embedding table for the stack (Section 2.3: the positional
 * frequencies are subsampled to the active set, i.e. every active row is
 * rotated by its own token's grid position). A head of head_dim channels is
 * cut into a temporal band of head_dim - 4 floor(head_dim/6) channels and
 * two spatial bands of 2 floor(head_dim/6) channels; pair j of a band of b
 * channels at coordinate c turns by c * theta^(-2j/b). The HOST table has
 * (grid_f + grid_h + grid_w) rows of head_dim/2 (cos, sin) float pairs: row
 * c holds frame c, row grid_f + c grid row c, row grid_f + grid_h + c grid
 * column c; entries of pairs outside the row's band are 0. Computed in double
 * precision, stored in float. hsa_rope_table_floats gives the float count
 * (0 for invalid sizes).
 */
size_t hsa_rope_table_floats(int32_t head_dim, int32_t grid_f, int32_t grid_h, int32_t grid_w);
int hsa_rope_table(float theta, int32_t head_dim, int32_t grid_f, int32_t grid_h, int32_t grid_w,
                   float* table_host);

/*
 * Token reordering (Section 2.5): perm receives the tokens with budget < T
 * followed by those with budget T (the baseline group, active at every
 * iteration), each part in index order; *n_lead = the count of the former,
 * i.e. the cache rows a reordered stack needs. Invalid budgets give
 * n_lead = -1 (and HSA_STEP_ERR_BUDGET with n_lead_host). perm and n_lead_dev
 * are device int32 ([n_tokens], [1]); n_lead_host, if not NULL, is filled
 * after one stream synchronization.
 */
int hsa_reorder_plan(const int32_t* budget, int64_t n_tokens, int32_t T, int32_t* perm,
                     int32_t* n_lead_dev, int32_t* n_lead_host, hipStream_t stream);

/*
 * Row permutation of token-indexed state: dst[i] = src[perm[i]] for
 * i < n_rows, or with inverse != 0, dst[perm[i]] = src[i] (undoing the
 * reordering before the latent leaves the sampler). Rows are row_bytes wide;
 * perm entries outside [0, n_rows) skip their row. src and dst must not
 * overlap.
 */
int hsa_permute_rows(const void* src, const int32_t* perm, int64_t n_rows, int64_t row_bytes,
                     int32_t inverse, void* dst, hipStream_t stream);

/*
 * Strategy D accumulation (Appendix B, Eq. 7), for every token t:
 *   first != 0:  acc[t] = 0;
 *   first == 0:  acc[t] += (sum_c |v[t][c] - v_prev[t][c]|) / (sum_c |v[t][c]|),
 *                both sums in float64 in channel order, one float64 division
 *                (0/0 gives NaN, x/0 infinity);
 *   then v_prev[t] = v[t].
 *   v, v_prev  [n_tokens, channels] fp32     acc  [n_tokens] float64
 * v_prev and acc must not overlap v or each other.
 */
int hsa_l1_rel_accumulate(const float* v, float* v_prev, int64_t n_tokens, int32_t channels,
                          double* acc, int32_t first, hipStream_t stream);

/*
 * Group assignment from given per-token keys (float64), with the rank,
 * key order and group table of hsa_assign_budgets (which uses the squared
 * velocity norms as keys). keys must not overlap budget.
 */
int hsa_assign_budgets_by_key(const double* keys, int64_t n_tokens, int32_t T,
                              const int32_t* group_budget, const int64_t* group_size,
                              int32_t n_groups, int32_t* budget, hipStream_t stream);

/*
 * Device state and caller-owned scratch of one stack. Every pointer except
 * the two host arrays is a device pointer, 16-byte aligned. d = heads *
 * head_dim, N = n_tokens, C = channels, es = 2 (bf16) or 4 (fp32).
 */
typedef struct hsa_stack {
  int32_t dtype;      /* HSA_STEP_BF16 or HSA_STEP_F32: weights, caches, hidden state */
  int32_t n_layers;   /* >= 0 */
  int32_t heads;
  int32_t head_dim;   /* 64 or 128 */
  int32_t channels;   /* C; bf16 stacks need C % 64 == 0 */
  int32_t reserved;   /* 0 */
  int64_t n_tokens;   /* N >= 1 */
  const void* w_embed;            /* [d, C] */
  const void* w_head;             /* [C, d] */
  const void* const* w_layers;    /* HOST array of 4 * n_layers pointers: Wq, Wk, Wv, Wo of
                                     layer 0, then of layer 1, ...; each [d, d] */
  void* const* caches;            /* HOST array of 2 * n_layers pointers: K_hat, V_hat of
                                     layer 0, then of layer 1, ...; each [N, d] */
  float* x;                       /* [N, C] latent, advanced in place */
  float* v_hat;                   /* [N, C] velocity cache */
  int32_t* budget;                /* [N] step budgets, rewritten at refresh iterations */
  int32_t* idx;                   /* scratch [N] int32: the active set */
  int32_t* n_active;              /* scratch [1] int32 */
  void* xa;                       /* scratch [N, C] dtype */
  void* h;                        /* scratch [N, d] dtype: compact hidden state */
  void* q;                        /* scratch [N, d] dtype */
  void* o;                        /* scratch [N, d] dtype */
  float* v_fresh;                 /* scratch [N, C] fp32 */
  void* keys;                     /* scratch 8 * N bytes (used by refresh iterations) */
  float* row_scale;               /* scratch [N] fp32: per-row RMS factors */
  /* full blocks (Section 2.3: cross-attention and FFN of the active rows) */
  int32_t ffn_dim;                /* 0: no FFN sub-layer; else the hidden width (bf16: % 64 == 0) */
  int32_t ctx_len;                /* 0: no cross-attention; else the context rows */
  const void* const* w_cross;     /* HOST array of 4 * n_layers pointers when ctx_len > 0:
                                     Wq_c, Wo_c ([d, d]), then the context keys K_c = ctx Wk_c^T
                                     and values V_c = ctx Wv_c^T ([ctx_len, d], computed once by
                                     the caller, e.g. with hsa_linear) of layer 0, then layer 1... */
  const void* const* w_ffn;       /* HOST array of 2 * n_layers pointers when ffn_dim > 0:
                                     W1 [ffn_dim, d], W2 [d, ffn_dim] of each layer */
  void* f;                        /* scratch [N, ffn_dim] dtype when ffn_dim > 0 */
  float* v_prev;                  /* scratch [N, C] fp32 (HSA_SELECT_L1_REL) */
  /* rotary embedding of Q and K (NULL rope_cs: none) */
  const float* rope_cs;           /* device copy of the hsa_rope_table of (head_dim, grid) */
  const int32_t* pos;             /* [N] grid position of every token (NULL: the token index) */
  int32_t grid_f, grid_h, grid_w; /* latent grid in tokens; grid_f * grid_h * grid_w >= N */
  int32_t reserved2;              /* 0 */
  /* prefix-only KV cache of reordered tokens (Section 2.5) */
  int32_t prefix_cache;           /* 1: tokens n_cached .. N-1 are the baseline group (budget T,
                                     active at every iteration, as after hsa_reorder_plan and
                                     hsa_permute_rows); each layer's K_hat/V_hat then has only
                                     n_cached rows and the baseline rows' fresh keys and values
                                     live in k_tail/v_tail. Needs n_groups == 0 (fixed groups). */
  int32_t reserved3;              /* 0 */
  int64_t n_cached;               /* prefix_cache only: a multiple of 64, or N, at least the
                                     number of non-baseline tokens (baseline tokens in the
                                     prefix are cached and rewritten at every iteration) */
  void* k_tail;                   /* scratch [N - n_cached, d] dtype shared by the layers */
  void* v_tail;
  /* optional scratch for key parts of the bf16 attention launches (NULL: no split); with
     hsa_attention_parts_workspace_bytes(dtype, N, heads, head_dim) bytes every split fits */
  void* attn_parts;
  int64_t attn_parts_bytes;
} hsa_stack;

/*
 * One iteration i of the multi-layer HSA sampler (Sections 2.2-2.4):
 *   1. A_i from the budgets (and the margin and outside period of Section
 *      2.5), as hsa_build_active_set_window; |A_i| is copied to the host (one
 *      stream synchronization per iteration);
 *   2. h = embed(dtype(x[A_i])); for each layer: Q/K/V of rms(h) (Q and K
 *      rotated by their tokens' grid positions when rope_cs is set), cache rows
 *      A_i overwritten, attention of the |A_i| queries against all N cached
 *      rows (scale 1/sqrt(head_dim)), h <- h + O Wo^T; with ctx_len > 0
 *      h <- h + CrossAttn(rms(h) Wq_c^T, K_c, V_c) Wo_c^T; with ffn_dim > 0
 *      h <- h + gelu(rms(h) W1^T) W2^T; then v_fresh = rms(h) W_head^T;
 *   3. v_hat[A_i] = v_fresh, then x <- x + v_hat (sigma_next - sigma_i) for
 *      all tokens (Eq. 6, as hsa_cached_euler);
 *   4. group membership, if n_groups > 0:
 *      HSA_SELECT_VELOCITY_NORM: if i is a multiple of P = lcm over the group
 *        budgets of T / s_k (the iterations where every group's schedule
 *        fires), the budgets are reassigned from v_hat as hsa_assign_budgets.
 *        A refresh iteration where not every token is active (the budgets in
 *        force did not come from the group table) returns HSA_STEP_ERR_BUDGET
 *        right after step 1: x, v_hat, the budgets and the caches are left
 *        unchanged (only the idx and n_active scratch are written).
 *      HSA_SELECT_L1_REL (strategy D; needs margin >= 2 and outside_period
 *        1; an iteration i < margin where not every token is active returns
 *        HSA_STEP_ERR_BUDGET right after step 1, as above): at iterations
 *        i < margin (every token active) the fresh
 *        velocities feed hsa_l1_rel_accumulate into the keys scratch (first
 *        at i = 0; the keys buffer carries the sums from one call to the
 *        next), and at i = margin - 1 the budgets are assigned from the sums
 *        as hsa_assign_budgets_by_key.
 *      New budgets hold from iteration i + 1.
 * Iteration 0 activates every token whatever the budgets are, which fills
 * every cache and the velocity cache; later iterations read cache rows
 * written earlier. n_groups == 0 and every budget T is the dense loop.
 * With prefix_cache, an iteration whose active set does not contain every
 * token from n_cached on returns HSA_STEP_ERR_BUDGET before the stack runs.
 *   n_active_host   if not NULL: |A_i|
 *   refreshed_host  if not NULL: 1 if the budgets were reassigned, else 0
 * Writable buffers must not overlap each other or any weight.
 */
int hsa_stack_iteration(const hsa_stack* stack, int32_t T, int32_t iter, int32_t margin,
                        int32_t outside_period, float sigma_i, float sigma_next,
                        const int32_t* group_budget, const int64_t* group_size, int32_t n_groups,
                        int32_t selection, int32_t* n_active_host, int32_t* refreshed_host,
                        hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* HSA_STEP_H */
