// Host-side argument checks shared by the C ABI translation units.
#pragma once

#include <stddef.h>
#include <stdint.h>

#include "../../include/hsa_step.h"
#include "common.h"

#define HSA_API extern "C" __attribute__((visibility("default")))

namespace hsa_api {

using hsa::RowGemm;

inline size_t elem_size(int dtype) { return dtype == HSA_STEP_BF16 ? 2 : (dtype == HSA_STEP_F32 ? 4 : 0); }

inline bool overlaps(const void* a, size_t na, const void* b, size_t nb) {
  if (!a || !b || na == 0 || nb == 0) return false;
  const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
  return x < y + nb && y < x + na;
}

inline bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

inline int launch_status(hipError_t e) { return e == hipSuccess ? HSA_STEP_OK : HSA_STEP_ERR_LAUNCH; }

constexpr int64_t kMaxRows = INT32_MAX;

// Largest tensor the entry points accept, in bytes: far above any device's
// memory (MI355X: 288 GB < 2^39), and low enough that no size product in the
// checks can overflow.
constexpr int64_t kMaxBytes = int64_t(1) << 48;

// True if a * b * c (all non-negative) is at most kMaxBytes; the product is
// formed in 128 bits, so it cannot wrap.
inline bool fits(int64_t a, int64_t b, int64_t c = 1) {
  if (a < 0 || b < 0 || c < 0) return false;
  return (__int128)a * b * c <= (__int128)kMaxBytes;
}

}  // namespace hsa_api
