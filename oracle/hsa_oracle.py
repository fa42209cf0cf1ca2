"""Plain CPU oracle for the HSA active-token layer step.

TEST INFRASTRUCTURE ONLY. This module is imported by the tests, by the
package smoke check and by the benchmark's CPU-baseline leg, never by the
product path. It shares no code with the HIP library: the only thing both
sides consume is the seeded input arrays from `synth`.

Everything is NumPy in float64. Values that the method materializes in a
storage dtype (Q, K, V, the cache rows, the attention output O, the projected
output Y) are rounded once from the exact float64 result to that dtype: bf16
(round to nearest, ties to even, written out below) or fp32.

What it follows, by section of the paper:
  * Section 2.2, Eqs. 3-5 and the modular rule after Eq. 5 -- the step-budget
    partition, the average step count s_bar and the active set
    A_i = union of the groups G_k with i mod (T / s_k) == 0.
  * Section 2.5, "Phase-aware caching window" -- margin m: iterations i < m
    and i > T - m - 1 treat every token as active.
  * Section 2.3, steps 1-3 -- fresh Q/K/V for the active rows only, overwrite
    of the cache rows A_i (other rows unchanged), attention of the active
    queries against all N cached keys; the output projection and everything
    after it act on the active rows only.
  * Section 2.4, Eq. 6 and the paragraph after it -- cached Euler update of
    every token with the shared step sigma_{i+1} - sigma_i, using the last
    velocity a token produced.
  * Section 2.1, Eq. 2 -- the uniform flow-matching Euler step (what Eq. 6
    reduces to when every token is active).

Readings where the paper is silent (recorded with the design notes):
  * softmax scale 1/sqrt(d_h), passed explicitly;
  * weights have the [d_out, d_in] orientation (y = x W^T), no biases;
  * the single block is QKV -> attention -> output projection, and its
    output is the token velocity;
  * the Euler step difference is taken in fp32 (both sides receive the same
    fp32 sigmas); the update is formed in float64 and rounded once to fp32.
"""

from __future__ import annotations

import math

import numpy as np

# ---------------------------------------------------------------------------
# Rounding to storage dtypes
# ---------------------------------------------------------------------------

_BF16_MAX = (2.0 - 2.0 ** -7) * 2.0 ** 127
_BF16_MIN_EXP = -133  # spacing of bf16 subnormals: 2**-133


def round_bf16(a) -> np.ndarray:
    """Round float64 values to the nearest bf16 value (ties to even), returned
    as float64. bf16 keeps 8 significant bits and fp32's exponent range."""
    a = np.asarray(a, dtype=np.float64)
    out = a.copy()
    fin = np.isfinite(a)
    v = a[fin]
    _, e = np.frexp(v)  # v = m * 2**e with 0.5 <= |m| < 1
    q = np.maximum(e - 8, _BF16_MIN_EXP)  # exponent of one unit in the last place
    r = np.ldexp(np.rint(np.ldexp(v, -q)), q)  # np.rint: half to even
    big = np.abs(r) > _BF16_MAX
    r[big] = np.copysign(np.inf, v[big])
    out[fin] = r
    return out


def round_f32(a) -> np.ndarray:
    """Round float64 values to fp32 (IEEE nearest-even), returned as float64."""
    return np.asarray(a, dtype=np.float64).astype(np.float32).astype(np.float64)


def round_to(a, dtype: str) -> np.ndarray:
    if dtype == "bf16":
        return round_bf16(a)
    if dtype == "f32":
        return round_f32(a)
    raise ValueError(f"unknown dtype {dtype!r}")


# ---------------------------------------------------------------------------
# Schedule: Section 2.2 (Eqs. 3-5) and the phase-aware window of Section 2.5
# ---------------------------------------------------------------------------


def check_budgets(budget, T: int) -> np.ndarray:
    """Budgets must be positive divisors of T (Eq. 5)."""
    b = np.asarray(budget, dtype=np.int64)
    if T <= 0:
        raise ValueError("T must be positive")
    if b.size and (b.min() < 1 or b.max() > T or np.any(T % b != 0)):
        raise ValueError("every budget s must satisfy 1 <= s <= T and s | T")
    return b


def active_set(budget, T: int, i: int, margin: int = 0, outside_period: int = 1) -> np.ndarray:
    """A_i: ascending indices n with i mod (T / s_n) == 0 (Section 2.2).

    With a phase-aware margin m > 0 (Section 2.5) the iterations i < m and
    i > T - m - 1 lie outside the caching window. The paper's rule activates
    every token there (outside_period 1). The other reading, under which the
    HSA-25 preset of Appendix C meets its printed runtime, has every token
    follow the largest budget's schedule outside the window: all tokens are
    active iff i mod outside_period == 0, with outside_period = T / s_max.
    """
    b = check_budgets(budget, T)
    if not 0 <= i < T:
        raise ValueError("iteration out of range")
    if not 0 <= margin <= T // 2:
        raise ValueError("margin out of range")
    if outside_period < 1 or T % outside_period:
        raise ValueError("outside_period must divide T")
    if margin > 0 and (i < margin or i > T - margin - 1):
        if i % outside_period == 0:
            return np.arange(b.size, dtype=np.int64)
        return np.zeros(0, dtype=np.int64)
    period = T // b
    return np.flatnonzero(i % period == 0).astype(np.int64)


def mean_steps(budget) -> float:
    """s_bar = sum_k |G_k|/N * s_k (Eq. 4), i.e. the mean per-token budget."""
    b = np.asarray(budget, dtype=np.float64)
    return float(b.sum() / b.size)


def window_margin(center_percent: int, T: int) -> int:
    """m = floor((1 - k) T / 2) for a caching window over the centre k% of the
    trajectory (Section 2.5), evaluated in exact integer arithmetic."""
    if not 0 <= center_percent <= 100:
        raise ValueError("window percent out of range")
    return ((100 - center_percent) * T) // 200


# ---------------------------------------------------------------------------
# One layer step: Section 2.3
# ---------------------------------------------------------------------------


def project(rows, w, dtype: str) -> np.ndarray:
    """rows W^T in float64, rounded once to the storage dtype."""
    return round_to(np.asarray(rows, np.float64) @ np.asarray(w, np.float64).T, dtype)


def attention(q, k_cache, v_cache, heads: int, dh: int, scale: float, block: int = 512) -> np.ndarray:
    """Per head h: softmax(scale * Q_h K_h^T) V_h over all cached rows, float64,
    unrounded. q is [M, heads*dh]; k_cache / v_cache are [N, heads*dh]."""
    q = np.asarray(q, np.float64)
    k = np.asarray(k_cache, np.float64)
    v = np.asarray(v_cache, np.float64)
    M = q.shape[0]
    out = np.empty((M, heads * dh), dtype=np.float64)
    for h in range(heads):
        cols = slice(h * dh, (h + 1) * dh)
        kh = np.ascontiguousarray(k[:, cols])
        vh = np.ascontiguousarray(v[:, cols])
        for r0 in range(0, M, block):
            s = scale * (q[r0:r0 + block, cols] @ kh.T)
            s -= s.max(axis=1, keepdims=True)
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            out[r0:r0 + block, cols] = p @ vh
    return out


def qkv_cache_update(x, idx, wq, wk, wv, k_cache, v_cache, dtype: str, x_compact: bool = False) -> dict:
    """Section 2.3 steps 1-2: fresh Q/K/V for the active rows, then overwrite
    the cache rows A_i. Returns Q (compact, one row per active token) and new
    copies of both caches; rows outside A_i are the old rows, untouched."""
    idx = np.asarray(idx, dtype=np.int64)
    xa = np.asarray(x, np.float64) if x_compact else np.asarray(x, np.float64)[idx]
    q = project(xa, wq, dtype)
    k = project(xa, wk, dtype)
    v = project(xa, wv, dtype)
    k_new = np.array(k_cache, dtype=np.float64, copy=True)
    v_new = np.array(v_cache, dtype=np.float64, copy=True)
    k_new[idx] = k
    v_new[idx] = v
    return {"q": q, "k": k, "v": v, "k_cache": k_new, "v_cache": v_new}


def attention_output(q, k_cache, v_cache, wo, heads: int, dh: int, scale: float, dtype: str) -> dict:
    """Section 2.3 step 3 followed by the output projection, on active rows:
    O = round(attention), Y = round(O Wo^T)."""
    o = round_to(attention(q, k_cache, v_cache, heads, dh, scale), dtype)
    y = project(o, wo, dtype)
    return {"o": o, "y": y}


def layer_step(x, idx, w: dict, k_cache, v_cache, out, heads: int, dh: int, scale: float,
               dtype: str, x_compact: bool = False) -> dict:
    """One HSA layer step over the active set idx: Q/K/V of the active rows,
    cache overwrite, attention against all N cached rows, output projection,
    scatter of the result into out[idx] (other rows of out unchanged)."""
    idx = np.asarray(idx, dtype=np.int64)
    r = qkv_cache_update(x, idx, w["wq"], w["wk"], w["wv"], k_cache, v_cache, dtype, x_compact)
    a = attention_output(r["q"], r["k_cache"], r["v_cache"], w["wo"], heads, dh, scale, dtype)
    out_new = np.array(out, dtype=np.float64, copy=True)
    out_new[idx] = a["y"]
    r.update(a)
    r["out"] = out_new
    return r


# ---------------------------------------------------------------------------
# Cached Euler update: Section 2.4, Eq. 6
# ---------------------------------------------------------------------------


def euler_delta(sigma_i, sigma_next) -> float:
    """The shared step sigma_{i+1} - sigma_i, taken in fp32 on fp32 inputs."""
    return float(np.float32(np.float64(np.float32(sigma_next)) - np.float64(np.float32(sigma_i))))


def cached_euler(x, v_cache, v_fresh, idx, sigma_i, sigma_next) -> tuple:
    """Eq. 6 for every token. If v_fresh is given, the velocity cache rows idx
    are first replaced by it (active tokens use their fresh velocity, skipped
    tokens keep the cached one); then x <- x + v_hat * (sigma_{i+1} - sigma_i)
    over all rows, rounded once to fp32. Returns (x_new, v_cache_new)."""
    v = np.array(v_cache, dtype=np.float64, copy=True)
    if v_fresh is not None:
        v[np.asarray(idx, dtype=np.int64)] = np.asarray(v_fresh, np.float64)
    dsig = euler_delta(sigma_i, sigma_next)
    x_new = round_f32(np.asarray(x, np.float64) + v * dsig)
    return x_new, v


# ---------------------------------------------------------------------------
# Multi-iteration trajectory of one block (Sections 2.2-2.4 together)
# ---------------------------------------------------------------------------


def trajectory(x0, budget, T: int, sigmas, w: dict, heads: int, dh: int, dtype: str = "f32",
               margin: int = 0, iterations=None) -> list:
    """Run iterations i = 0..T-1 of the single-block HSA sampler.

    At every iteration: A_i from the budgets, the layer step on A_i (its
    output rows refresh the velocity cache v_hat[A_i]), then the cached Euler
    update of all tokens. The caches start empty; iteration 0 activates every
    token (0 mod p == 0), which fills them. Returns one record per iteration
    with the state after it.
    """
    x = np.asarray(x0, np.float64)
    N, d = x.shape
    scale = 1.0 / math.sqrt(dh)
    k_cache = np.zeros((N, d))
    v_cache = np.zeros((N, d))
    v_hat = np.zeros((N, d))
    records = []
    n_iter = T if iterations is None else iterations
    for i in range(n_iter):
        idx = active_set(budget, T, i, margin)
        r = layer_step(x, idx, w, k_cache, v_cache, v_hat, heads, dh, scale, dtype)
        k_cache, v_cache, v_hat = r["k_cache"], r["v_cache"], r["out"]
        x_in = x
        x, _ = cached_euler(x, v_hat, None, idx, sigmas[i], sigmas[i + 1])
        records.append({"i": i, "idx": idx, "x_in": x_in, "q": r["q"], "k_cache": k_cache,
                        "v_cache": v_cache, "o": r["o"], "y": r["y"], "v_hat": v_hat, "x": x})
    return records
