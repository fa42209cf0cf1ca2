// Host-side argument checks of the C ABI under AddressSanitizer and
// UndefinedBehaviorSanitizer (built by tests/test_sanitize.py with the
// library's host code instrumented). Every call below must be refused on the
// host with its documented status before anything is enqueued; pointers are
// fake device addresses that are never dereferenced. No GPU is needed. The
// size arguments include the extremes of their types, where a product of
// sizes in a check could overflow.
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include "hsa_step.h"

static int failures = 0;
static void expect(int got, int want, const char* what, int line) {
  if (got != want) {
    fprintf(stderr, "line %d: %s returned %d, expected %d\n", line, what, got, want);
    ++failures;
  }
}
#define EXPECT(call, want) expect((call), (want), #call, __LINE__)

static void* P(uintptr_t a) { return reinterpret_cast<void*>(a); }

int main() {
  const uintptr_t A = 0x7F0000000000, B = 0x7F1000000000, C = 0x7F2000000000, D = 0x7F3000000000,
                  E = 0x7F4000000000, G = 0x7F5000000000, W = 0x7F6000000000;
  const int OK = HSA_STEP_OK, NUL = HSA_STEP_ERR_NULL, SHAPE = HSA_STEP_ERR_SHAPE,
            BUDGET = HSA_STEP_ERR_BUDGET, DTYPE = HSA_STEP_ERR_DTYPE, ALIAS = HSA_STEP_ERR_ALIAS,
            WS = HSA_STEP_ERR_WORKSPACE;
  const int BF = HSA_STEP_BF16, F32 = HSA_STEP_F32;
  const int64_t I64MAX = INT64_MAX;
  const int32_t I32MAX = INT32_MAX;

  for (int s = -1; s < 10; ++s)
    if (!hsa_step_status_string(s)) ++failures;

  // pure host helpers
  EXPECT(hsa_window_margin(80, 40), 4);
  EXPECT(hsa_window_margin(0, I32MAX), I32MAX / 2);
  EXPECT(hsa_window_margin(-5, 40), -1);
  EXPECT((int)hsa_attention_workspace_bytes(BF, -1, 256), 0);
  EXPECT(hsa_attention_parts_workspace_bytes(BF, I32MAX, I32MAX, I32MAX) == 0, 1);
  EXPECT(hsa_assign_budgets_workspace_bytes(-1) == 0, 1);
  EXPECT(hsa_rope_table_floats(128, -1, 30, 52) == 0, 1);
  float table[(3 + 4 + 5) * 32 * 2];
  EXPECT(hsa_rope_table(10000.f, 64, 3, 4, 5, table), OK);
  EXPECT(hsa_rope_table(10000.f, 64, 3, 4, 5, nullptr), NUL);

  // active set
  EXPECT(hsa_build_active_set(P(A) ? (const int32_t*)P(A) : nullptr, 100, 0, 0, 0, (int32_t*)P(B),
                              (int32_t*)P(C), nullptr, nullptr), BUDGET);
  EXPECT(hsa_build_active_set((const int32_t*)P(A), -1, 40, 0, 0, (int32_t*)P(B), (int32_t*)P(C), nullptr, nullptr), SHAPE);
  EXPECT(hsa_build_active_set((const int32_t*)P(A), I64MAX, 40, 0, 0, (int32_t*)P(B), (int32_t*)P(C), nullptr, nullptr), SHAPE);
  EXPECT(hsa_build_active_set((const int32_t*)P(A), 100, 40, 0, 0, (int32_t*)P(A + 8), (int32_t*)P(C), nullptr, nullptr), ALIAS);
  EXPECT(hsa_build_active_set_window((const int32_t*)P(A), 100, 40, 0, 4, 3, (int32_t*)P(B), (int32_t*)P(C), nullptr, nullptr), BUDGET);
  EXPECT(hsa_build_active_set_window((const int32_t*)P(A), 100, I32MAX, I32MAX - 1, I32MAX / 2, I32MAX,
                                     (int32_t*)P(A + 8), (int32_t*)P(C), nullptr, nullptr), ALIAS);

  // Q/K/V scatter
  EXPECT(hsa_qkv_scatter(5, P(A), 0, (const int32_t*)P(B), 10, 100, 256, P(C), P(D), P(E), P(G), P(W), P(W + 51200), nullptr), DTYPE);
  EXPECT(hsa_qkv_scatter(BF, P(A), 0, (const int32_t*)P(B), 10, 100, I32MAX, P(C), P(D), P(E), P(G), P(W), P(W + 51200), nullptr), SHAPE);
  EXPECT(hsa_qkv_scatter(BF, P(A), 0, (const int32_t*)P(B), 10, I64MAX, 256, P(C), P(D), P(E), P(G), P(W), P(W + 51200), nullptr), SHAPE);
  EXPECT(hsa_qkv_scatter(BF, P(A), 0, (const int32_t*)P(B), 10, 100, 256, P(C), P(D), P(E), P(A), P(W), P(W + 51200), nullptr), ALIAS);
  EXPECT(hsa_qkv_scatter(BF, nullptr, 0, (const int32_t*)P(B), 10, 100, 256, P(C), P(D), P(E), P(G), P(W), P(W + 51200), nullptr), NUL);
  // beyond the largest tensor the library accepts (2^48 bytes); the size products would wrap 64 bits
  EXPECT(hsa_qkv_scatter(BF, P(A), 0, (const int32_t*)P(B), I32MAX, I32MAX, (I32MAX / 64) * 64, P(C), P(D), P(E),
                         P(A), P(W), P(W + 51200), nullptr), SHAPE);
  // a large legal shape (2^31 rows of 64 bf16: 2^38 bytes): the alias checks still see the overlap
  EXPECT(hsa_qkv_scatter(BF, P(A), 0, (const int32_t*)P(B), I32MAX, I32MAX, 64, P(C), P(D), P(E),
                         P(A + (1ull << 37)), P(W), P(W + 51200), nullptr), ALIAS);

  // attention
  EXPECT(hsa_attention_core(9, P(A), P(B), P(C), 10, 100, 4, 64, 0.125f, P(D), nullptr), DTYPE);
  EXPECT(hsa_attention_core(BF, P(A), P(B), P(C), 10, 100, 4, 96, 0.125f, P(D), nullptr), SHAPE);
  EXPECT(hsa_attention_core(BF, P(A), P(B), P(C), 10, 100, I32MAX, 128, 0.125f, P(D), nullptr), SHAPE);
  EXPECT(hsa_attention_core(BF, P(A), P(B), P(C), 10, 100, 4, 64, NAN, P(D), nullptr), SHAPE);
  EXPECT(hsa_attention_core(BF, P(A), P(B), P(C), 10, 100, 4, 64, 0.125f, P(A), nullptr), ALIAS);
  EXPECT(hsa_attention_core_parts(BF, P(A), P(B), P(C), 10, 100, 4, 64, 0.125f, P(D), P(A + 4096), 1 << 20, nullptr), ALIAS);
  EXPECT(hsa_attention_core_parts(BF, P(A), P(B), P(C), 10, 100, 4, 64, 0.125f, P(D), P(W + 4), 1 << 20, nullptr), SHAPE);
  const size_t need = hsa_attention_workspace_bytes(BF, 10, 256);
  EXPECT(hsa_active_attention(BF, P(A), P(B), P(C), (const int32_t*)P(D), 10, 100, 4, 64, 0.125f, P(E), P(G), nullptr, need, nullptr), WS);
  EXPECT(hsa_active_attention(BF, P(A), P(B), P(C), (const int32_t*)P(D), 10, 100, 4, 64, 0.125f, P(E), P(G), P(G), need, nullptr), ALIAS);
  EXPECT(hsa_active_attention(BF, P(A), P(B), P(C), (const int32_t*)P(D), 10, 100, I32MAX, I32MAX, 0.125f, P(E), P(G), P(W), need, nullptr), SHAPE);
  EXPECT(hsa_active_attention_noalloc(BF, P(A), P(B), P(C), (const int32_t*)P(D), 9831, 32760, 40, 128, 0.088f, P(E), P(G), nullptr), WS);
  EXPECT(hsa_active_attention_noalloc(BF, P(A), P(B), P(C), (const int32_t*)P(D), I32MAX, I64MAX, 40, 128, 0.088f, P(E), P(G), nullptr), WS);
  EXPECT(hsa_out_scatter(BF, P(A), (const int32_t*)P(B), 10, 100, 256, P(C), P(A), nullptr), ALIAS);
  EXPECT(hsa_out_scatter(BF, P(A), (const int32_t*)P(B), 10, 100, 100, P(C), P(D), nullptr), SHAPE);

  // cached Euler
  EXPECT(hsa_cached_euler((float*)P(A), (float*)P(B), nullptr, nullptr, 0, -1, 16, 1.f, 0.9f, nullptr), SHAPE);
  EXPECT(hsa_cached_euler((float*)P(A), (float*)P(B), (const float*)P(C), nullptr, 10, 100, 16, 1.f, 0.9f, nullptr), NUL);
  EXPECT(hsa_cached_euler((float*)P(A), (float*)P(A + 64), nullptr, nullptr, 0, 100, 16, 1.f, 0.9f, nullptr), ALIAS);
  EXPECT(hsa_cached_euler((float*)P(A), (float*)P(B), nullptr, nullptr, 0, I32MAX, I32MAX, 1.f, 0.9f, nullptr), SHAPE);
  EXPECT(hsa_cached_euler((float*)P(A), (float*)P(B), nullptr, nullptr, 0, 100, -1, 1.f, 0.9f, nullptr), SHAPE);
  EXPECT(hsa_cached_euler(nullptr, nullptr, nullptr, nullptr, 0, 0, 16, 1.f, 0.9f, nullptr), OK);

  // multi-layer helpers
  EXPECT(hsa_gather_rows(3, (const float*)P(A), (const int32_t*)P(B), 10, 100, 16, P(C), nullptr), DTYPE);
  EXPECT(hsa_gather_rows(BF, (const float*)P(A), (const int32_t*)P(B), 10, 100, 16, P(A + 64), nullptr), ALIAS);
  EXPECT(hsa_gather_rows(BF, (const float*)P(A), (const int32_t*)P(B), I32MAX, I64MAX, I32MAX, P(C), nullptr), SHAPE);
  EXPECT(hsa_row_rms_scale(BF, P(A), 10, 64, -1.f, (float*)P(B), nullptr), SHAPE);
  EXPECT(hsa_row_rms_scale(BF, P(A), I32MAX, I32MAX, 1e-6f, (float*)P(A + 64), nullptr), SHAPE);
  EXPECT(hsa_row_rms_scale(BF, P(A), I32MAX, 64, 1e-6f, (float*)P(A + (1ull << 37)), nullptr), ALIAS);
  EXPECT(hsa_linear(F32, P(A), 10, 64, P(B), 64, nullptr, nullptr, 0, BF, P(C), nullptr), DTYPE);
  EXPECT(hsa_linear(BF, P(A), 10, 64, P(B), 64, nullptr, nullptr, 0, BF, P(A + 64), nullptr), ALIAS);
  EXPECT(hsa_linear(BF, P(A), I32MAX, (I32MAX / 64) * 64, P(B), (I32MAX / 4) * 4, nullptr, nullptr, 0, BF,
                    P(A + 64), nullptr), SHAPE);
  EXPECT(hsa_linear(BF, P(A), I32MAX, 64, P(B), 64, nullptr, nullptr, 0, BF, P(A + (1ull << 37)), nullptr), ALIAS);
  EXPECT(hsa_cached_euler((float*)P(A), (float*)P(A + (1ull << 38)), nullptr, nullptr, 0, I32MAX, 64, 1.f, 0.9f,
                          nullptr), ALIAS);
  const int32_t gb_bad[2] = {40, 10}, gb[2] = {10, 40};
  const int64_t gs[2] = {50, 50}, gs_bad[2] = {I64MAX, 1};
  const size_t ws = hsa_assign_budgets_workspace_bytes(100);
  EXPECT(hsa_assign_budgets((const float*)P(A), 100, 16, 40, gb_bad, gs, 2, (int32_t*)P(B), P(C), ws, nullptr), BUDGET);
  EXPECT(hsa_assign_budgets((const float*)P(A), 100, 16, 40, gb, gs_bad, 2, (int32_t*)P(B), P(C), ws, nullptr), BUDGET);
  EXPECT(hsa_assign_budgets((const float*)P(A), 100, 16, 40, gb, gs, 17, (int32_t*)P(B), P(C), ws, nullptr), BUDGET);
  EXPECT(hsa_assign_budgets((const float*)P(A), 100, 16, 40, gb, gs, 2, (int32_t*)P(B), P(C), ws - 8, nullptr), WS);
  EXPECT(hsa_assign_budgets_by_key((const double*)P(A), 100, 40, gb, gs_bad, 2, (int32_t*)P(B), nullptr), BUDGET);
  EXPECT(hsa_l1_rel_accumulate((const float*)P(A), (float*)P(A + 64), 100, 16, (double*)P(C), 0, nullptr), ALIAS);
  EXPECT(hsa_l1_rel_accumulate((const float*)P(A), (float*)P(B), I64MAX, I32MAX, (double*)P(C), 0, nullptr), SHAPE);
  EXPECT(hsa_reorder_plan((const int32_t*)P(A), 100, 40, (int32_t*)P(A + 8), (int32_t*)P(C), nullptr, nullptr), ALIAS);
  EXPECT(hsa_permute_rows(P(A), (const int32_t*)P(B), 10, 64, 0, P(A + 32), nullptr), ALIAS);
  EXPECT(hsa_permute_rows(P(A), (const int32_t*)P(B), I32MAX, I64MAX, 0, P(C), nullptr), SHAPE);

  // stack: a host array of layer weights with a missing entry, then overlapping caches
  hsa_stack s;
  memset(&s, 0, sizeof(s));
  const void* wl[8];
  void* cl[4];
  for (int i = 0; i < 8; ++i) wl[i] = P(0x7D0000000000 + (uintptr_t)i * (1ull << 32));
  for (int i = 0; i < 4; ++i) cl[i] = P(0x7C0000000000 + (uintptr_t)i * (1ull << 32));
  uintptr_t next = 0x7E0000000000;
  auto take = [&]() { next += 1ull << 32; return P(next); };
  s.dtype = BF; s.n_layers = 2; s.heads = 12; s.head_dim = 128; s.channels = 64; s.n_tokens = 1000;
  s.w_embed = take(); s.w_head = take(); s.w_layers = wl; s.caches = cl;
  s.x = (float*)take(); s.v_hat = (float*)take(); s.budget = (int32_t*)take(); s.idx = (int32_t*)take();
  s.n_active = (int32_t*)take(); s.xa = take(); s.h = take(); s.q = take(); s.o = take();
  s.v_fresh = (float*)take(); s.keys = take(); s.row_scale = (float*)take();
  const int32_t sgb[2] = {20, 40};
  const int64_t sgs[2] = {500, 500};
  EXPECT(hsa_stack_iteration(nullptr, 40, 0, 0, 1, 1.f, .975f, nullptr, nullptr, 0, 0, nullptr, nullptr, nullptr), NUL);
  wl[5] = nullptr;
  EXPECT(hsa_stack_iteration(&s, 40, 1, 0, 1, 1.f, .975f, sgb, sgs, 2, 0, nullptr, nullptr, nullptr), NUL);
  wl[5] = P(0x7D0000000000 + 5ull * (1ull << 32));
  cl[3] = (char*)cl[2] + 64;
  EXPECT(hsa_stack_iteration(&s, 40, 1, 0, 1, 1.f, .975f, sgb, sgs, 2, 0, nullptr, nullptr, nullptr), ALIAS);
  cl[3] = P(0x7C0000000000 + 3ull * (1ull << 32));
  EXPECT(hsa_stack_iteration(&s, 40, 1, 0, 1, 1.f, .975f, sgb, sgs, 17, 0, nullptr, nullptr, nullptr), BUDGET);
  s.n_tokens = I64MAX;
  EXPECT(hsa_stack_iteration(&s, 40, 1, 0, 1, 1.f, .975f, sgb, sgs, 2, 0, nullptr, nullptr, nullptr), SHAPE);
  s.n_tokens = 1000;
  s.n_layers = I32MAX;
  EXPECT(hsa_stack_iteration(&s, 40, 1, 0, 1, 1.f, .975f, sgb, sgs, 2, 0, nullptr, nullptr, nullptr), SHAPE);

  if (failures) {
    fprintf(stderr, "%d failures\n", failures);
    return 1;
  }
  printf("abi error paths ok\n");
  return 0;
}
