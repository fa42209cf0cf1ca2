"""Plain CPU oracle for the multi-layer HSA sampling loop.

TEST INFRASTRUCTURE ONLY, like the rest of this package: imported by the
tests, the package smoke check and the benchmark's CPU-baseline leg, never by
the product path, and sharing no code with the HIP library.

It extends the single-block oracle to a stack of L self-attention layers
driven by the HSA schedule, float64 throughout with one rounding to the
storage dtype wherever a value is materialized.

What it follows, by section of the paper:
  * Section 2.3 -- every self-attention layer l keeps its own cache
    K_hat^(l), V_hat^(l) over all N tokens, written at the first iteration;
    at iteration i only the rows A_i are recomputed and overwritten, every
    active query attends to all N cached rows, and everything after
    attention runs on the active rows only. The hidden state of the active
    tokens therefore stays compact (one row per active token) from the patch
    embedding through the last layer to the velocity head.
  * Section 2.4, Eq. 6 -- the velocity head's output refreshes v_hat[A_i];
    then every token takes the Euler step with its cached velocity.
  * Section 2.2 and Appendix B -- group sizes |G_k| are fixed; membership is
    set by ranking tokens on a per-token velocity statistic, smaller values
    to lower budgets.

Readings where the paper is silent:
  * A stack layer is the pre-norm self-attention sub-layer with its
    residual, h <- h + Attn_l(rms(h)) W_o^T, where rms(h) = h / sqrt(mean(h^2)
    + eps) per row (eps = 1e-6, no learned scale) feeds the Q/K/V
    projections; no modulation. The residual stream
    is stored in the model dtype, rounded once per layer (the product and
    the add are formed exactly, then rounded). The normalized rows are not
    stored: each projection of rms(h) is formed exactly and rounded once.
    A final rms() precedes the velocity head. (Without the norms a random
    stack's residual stream grows from layer to layer and the sampled
    latent diverges within a few iterations.)
  * Full blocks (Section 2.3: cross-attention and the feed-forward network
    also run on the active rows only) add two pre-norm residual sub-layers
    after self-attention: h <- h + CrossAttn(rms(h), ctx) W_oc^T, with keys
    and values ctx W_kc^T, ctx W_vc^T of a fixed context of ctx_len rows (a
    stand-in for the text embedding, in the model width, no mask); and
    h <- h + gelu(rms(h) W_1^T) W_2^T with the tanh form of GELU. Every
    materialized value (the context keys and values, the cross-attention
    output, the FFN hidden activation) is rounded once to the model dtype.
  * Patch embedding: a linear map of the C values of a patch token (16
    latent channels times a 1x2x2 patch = 64) to d, no bias; the fp32
    latent rows are rounded once to the model dtype first. Velocity head: a
    linear map d -> C with an fp32 output. No timestep conditioning.
  * RoPE subsampling (Section 2.3: the positional frequencies are subsampled
    to the active set): with rotary embeddings on, Q and K of the active
    rows are rotated by the positions of their own tokens in the latent
    grid, never by their place in the compact active sequence. The paper
    does not spell out the embedding; the reading is 3D rotary embedding
    over (frame, row, column): the head dimension is cut into a temporal
    band of dh - 4 floor(dh/6) channels and two spatial bands of
    2 floor(dh/6) channels each; inside a band of b channels, the pair
    (2j, 2j+1) at coordinate c turns by the angle c * theta^(-2j/b)
    (theta = 10000). V is not rotated, nor is cross-attention.
  * Strategy D (Appendix B, Eq. 7) is taken as: over the initial full-budget
    steps -- the iterations 0 .. m-1 before the caching window, where every
    token is active -- the per-token L1_rel between consecutive fresh
    velocities is summed (float64, channel-order sums, one division per
    step), and after step m-1 tokens are ranked by the sum (the mean ranks
    the same) with the same key order and group filling as below.
  * Group refresh: at the iterations i with i mod P == 0, P = lcm over the
    budgets of T/s_k -- the iterations at which every group's schedule fires,
    so every token has just produced a fresh velocity -- tokens are ranked
    by the squared L2 norm of their velocity, ascending, and the fixed group
    sizes are filled in ascending budget order. The key is the float64 sum
    of the squared fp32 components, added in channel order (each square is
    exact in float64); keys compare as their IEEE bit patterns (a total
    order on non-negative values) and ties go to the lower token index. The
    new budgets hold from iteration i + 1.
"""

from __future__ import annotations

import math

import numpy as np

from .hsa_oracle import active_set, attention, cached_euler, check_budgets, qkv_cache_update, round_to


# ---------------------------------------------------------------------------
# Compact per-row maps (patch embedding, residual output projection, head)
# ---------------------------------------------------------------------------


def gather_latent(x, idx, dtype: str) -> np.ndarray:
    """Rows idx of the fp32 latent, rounded once to the model dtype."""
    return round_to(np.asarray(x, np.float64)[np.asarray(idx, np.int64)], dtype)


RMS_EPS = 1e-6


ROPE_THETA = 10000.0


def rope_bands(dh: int) -> tuple:
    """Channel pairs of the temporal, row and column bands of one head."""
    sp = dh // 6
    return ((dh - 4 * sp) // 2, sp, sp)


def rope_angles(positions, grid, dh: int, theta: float = ROPE_THETA) -> np.ndarray:
    """Rotation angle of every channel pair of a head for tokens at the given
    linear grid positions (frame-major, then row, then column): [M, dh/2]."""
    F, H, W = grid
    p = np.asarray(positions, np.int64)
    coords = (p // (H * W), (p // W) % H, p % W)
    cols = []
    for n_pairs, c in zip(rope_bands(dh), coords):
        j = np.arange(n_pairs, dtype=np.float64)
        cols.append(c[:, None].astype(np.float64) * theta ** (-2.0 * j / (2 * n_pairs)))
    return np.concatenate(cols, axis=1)


def apply_rope(x, angles, heads: int, dh: int) -> np.ndarray:
    """Rotate the channel pairs (2k, 2k+1) of every head of the rows of x by
    angles[:, k], float64, unrounded."""
    x = np.asarray(x, np.float64).reshape(x.shape[0], heads, dh // 2, 2)
    c = np.cos(angles)[:, None, :]
    s = np.sin(angles)[:, None, :]
    a, b = x[..., 0], x[..., 1]
    return np.stack([a * c - b * s, a * s + b * c], axis=-1).reshape(x.shape[0], heads * dh)


def gelu_tanh(x) -> np.ndarray:
    """0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3))), float64."""
    x = np.asarray(x, np.float64)
    return 0.5 * x * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (x + 0.044715 * x ** 3)))


def rms_normalize(h, eps: float = RMS_EPS) -> np.ndarray:
    """h / sqrt(mean over the row of h^2 + eps), float64, unrounded."""
    h = np.asarray(h, np.float64)
    return h / np.sqrt(np.mean(h * h, axis=1, keepdims=True) + eps)


def linear(a, w, dtype: str, residual=None) -> np.ndarray:
    """a W^T (+ residual) formed in float64, rounded once to dtype. w is
    [d_out, d_in]."""
    acc = np.asarray(a, np.float64) @ np.asarray(w, np.float64).T
    if residual is not None:
        acc = acc + np.asarray(residual, np.float64)
    return round_to(acc, dtype)


# ---------------------------------------------------------------------------
# Group refresh from velocity norms
# ---------------------------------------------------------------------------


def velocity_keys(v) -> np.ndarray:
    """Per-token squared L2 norm of the fp32 velocity rows: float64, summed
    over channels in channel order."""
    v = np.asarray(v, np.float64)
    acc = np.zeros(v.shape[0], dtype=np.float64)
    for c in range(v.shape[1]):
        acc = acc + v[:, c] * v[:, c]
    return acc


def token_ranks(keys) -> np.ndarray:
    """rank[n] = number of tokens before n in ascending (key, index) order;
    keys compare by their float64 bit patterns."""
    k = np.array(keys, dtype=np.float64)
    k[np.isnan(k)] = np.nan  # one canonical positive NaN, above every number
    k = k.view(np.uint64)
    order = np.lexsort((np.arange(k.size), k))  # key first, then token index
    rank = np.empty(k.size, dtype=np.int64)
    rank[order] = np.arange(k.size)
    return rank


def check_group_sizes(group_sizes, N: int, T: int | None = None) -> tuple:
    """((s_k, n_k), ...) in strictly ascending budget order, sizes summing to N."""
    gs = tuple((int(s), int(n)) for s, n in group_sizes)
    if not gs:
        raise ValueError("no groups")
    if any(b[0] <= a[0] for a, b in zip(gs, gs[1:])):
        raise ValueError("budgets must be strictly ascending")
    if any(n < 0 for _, n in gs) or sum(n for _, n in gs) != N:
        raise ValueError("group sizes must be non-negative and sum to N")
    if T is not None and any(s < 1 or s > T or T % s for s, _ in gs):
        raise ValueError("every budget must divide T")
    return gs


def assign_by_key(keys, group_sizes) -> np.ndarray:
    """Budgets from per-token keys: the n_1 lowest-ranked tokens get s_1,
    the next n_2 get s_2, and so on (int32[N])."""
    keys = np.asarray(keys, np.float64)
    gs = check_group_sizes(group_sizes, keys.shape[0])
    rank = token_ranks(keys)
    bounds = np.cumsum([n for _, n in gs])
    g = np.searchsorted(bounds, rank, side="right")
    return np.array([s for s, _ in gs], dtype=np.int32)[g]


def assign_groups(v, group_sizes) -> np.ndarray:
    """Budgets from the velocity rows, ranked by squared L2 norm."""
    return assign_by_key(velocity_keys(v), group_sizes)


def l1_rel(v, v_prev) -> np.ndarray:
    """Per-token L1 relative change of the velocity (Appendix B, Eq. 7):
    sum_c |v - v_prev| / sum_c |v|, both sums in float64 in channel order over
    the fp32 values, then one float64 division."""
    v = np.asarray(v, np.float64)
    vp = np.asarray(v_prev, np.float64)
    num = np.zeros(v.shape[0])
    den = np.zeros(v.shape[0])
    for c in range(v.shape[1]):
        num = num + np.abs(v[:, c] - vp[:, c])
        den = den + np.abs(v[:, c])
    with np.errstate(divide="ignore", invalid="ignore"):
        return num / den


SELECT_NORM = "norm"      # refresh from velocity norms where every schedule fires
SELECT_L1REL = "l1rel"    # strategy D: mean L1_rel over the initial full-budget steps


def boundary_gaps(keys, group_sizes) -> np.ndarray:
    """Relative gap between the last key of each group and the first key of
    the next one in ranked order (how far a group decision is from a tie)."""
    k = np.sort(np.asarray(keys, np.float64))
    gaps = []
    edge = 0
    for _, n in list(group_sizes)[:-1]:
        edge += n
        if 0 < edge < k.size:
            gaps.append((k[edge] - k[edge - 1]) / max(k[edge], np.finfo(np.float64).tiny))
    return np.array(gaps)


def reorder_plan(budget, T: int) -> tuple:
    """Token reordering (Section 2.5): every non-baseline token (budget < T)
    first, then the baseline group (budget T), each part in its old order.
    Returns (perm, n_cached): new position i holds old token perm[i], and only
    the first n_cached positions need cache rows (the baseline group is
    active at every iteration, so its keys and values are always fresh)."""
    b = check_budgets(budget, T)
    lead = np.flatnonzero(b < T)
    perm = np.concatenate([lead, np.flatnonzero(b == T)]).astype(np.int64)
    return perm, int(lead.size)


def refresh_period(T: int, budgets) -> int:
    """P = lcm of T/s_k: every group's schedule fires at the multiples of P."""
    p = 1
    for s in budgets:
        p = p * (T // int(s)) // math.gcd(p, T // int(s))
    return p


# ---------------------------------------------------------------------------
# Stack forward on the active rows, one iteration, a trajectory
# ---------------------------------------------------------------------------


def stack_forward(xa, idx, weights: dict, caches, heads: int, dh: int, dtype: str, rope=None) -> dict:
    """Embedding, L pre-norm layers (self-attention, and for full blocks
    cross-attention and FFN), final norm and velocity head for the active
    rows.

    xa: [|A|, C] model-dtype latent rows of the tokens idx. caches: one
    (K_hat, V_hat) pair of [N, d] arrays per layer. Returns the fp32-valued
    fresh velocities [|A|, C], new copies of the caches (rows outside idx
    untouched) and the compact hidden state entering each layer and leaving
    the last one. rope: None, or {"grid": (F, H, W), "pos": original grid
    position of every token (None: the token index), "theta": ...}; Q and K
    of the active rows are then rotated by the positions of their tokens.
    """
    scale = 1.0 / math.sqrt(dh)
    idx = np.asarray(idx, np.int64)
    angles = None
    if rope is not None:
        pos = idx if rope.get("pos") is None else np.asarray(rope["pos"], np.int64)[idx]
        angles = rope_angles(pos, rope["grid"], dh, rope.get("theta", ROPE_THETA))
    h = linear(xa, weights["w_embed"], dtype)
    hidden = [h]
    new_caches = []
    for lw, (k_hat, v_hat) in zip(weights["layers"], caches):
        hn = rms_normalize(h)
        if angles is None:
            r = qkv_cache_update(hn, idx, lw["wq"], lw["wk"], lw["wv"], k_hat, v_hat, dtype, x_compact=True)
        else:
            prod = lambda w: hn @ np.asarray(w, np.float64).T  # noqa: E731
            k = round_to(apply_rope(prod(lw["wk"]), angles, heads, dh), dtype)
            r = {"q": round_to(apply_rope(prod(lw["wq"]), angles, heads, dh), dtype),
                 "k_cache": np.array(k_hat, dtype=np.float64, copy=True),
                 "v_cache": np.array(v_hat, dtype=np.float64, copy=True)}
            r["k_cache"][idx] = k
            r["v_cache"][idx] = round_to(prod(lw["wv"]), dtype)
        o = round_to(attention(r["q"], r["k_cache"], r["v_cache"], heads, dh, scale), dtype)
        h = linear(o, lw["wo"], dtype, residual=h)
        if "wq_c" in lw:  # cross-attention of the active rows to the fixed context
            kc = linear(weights["ctx"], lw["wk_c"], dtype)
            vc = linear(weights["ctx"], lw["wv_c"], dtype)
            qc = linear(rms_normalize(h), lw["wq_c"], dtype)
            oc = round_to(attention(qc, kc, vc, heads, dh, scale), dtype)
            h = linear(oc, lw["wo_c"], dtype, residual=h)
        if "w1" in lw:  # feed-forward network of the active rows
            f = round_to(gelu_tanh(rms_normalize(h) @ np.asarray(lw["w1"], np.float64).T), dtype)
            h = linear(f, lw["w2"], dtype, residual=h)
        hidden.append(h)
        new_caches.append((r["k_cache"], r["v_cache"]))
    v = linear(rms_normalize(h), weights["w_head"], "f32")
    return {"v_fresh": v, "caches": new_caches, "hidden": hidden}


def initial_state(x0, n_layers: int, d: int, T: int) -> dict:
    """Latent x0 (fp32 values), empty caches and velocity cache, every budget
    T (iteration 0 activates every token whatever the budgets are)."""
    x = np.asarray(x0, np.float64)
    N, C = x.shape
    return {"x": x, "v_hat": np.zeros((N, C)), "budget": np.full(N, T, dtype=np.int32),
            "caches": [(np.zeros((N, d)), np.zeros((N, d))) for _ in range(n_layers)],
            "v_prev": np.zeros((N, C)), "l1": np.zeros(N)}


def stack_iteration(state: dict, weights: dict, i: int, T: int, sigmas, heads: int, dh: int,
                    dtype: str, group_sizes=None, margin: int = 0, outside_period: int = 1,
                    selection: str = SELECT_NORM, rope=None) -> dict:
    """One iteration of the multi-layer HSA sampler (rope as for
    stack_forward).

    A_i from the budgets in force (and the window); the stack on the active
    rows (embedding of the gathered latent, each layer's cache overwrite and
    attention, the residual output projection, cross-attention and FFN for
    full blocks, the velocity head); v_hat[A_i] refreshed and every token
    advanced by Eq. 6. Group membership (group_sizes given):
      SELECT_NORM   at refresh iterations (i mod P == 0) the budgets are
                    reassigned from the squared norms of v_hat;
      SELECT_L1REL  strategy D of Appendix B: over the initial full-budget
                    steps 0 .. m-1 (the window margin m >= 2, every token
                    active) the L1_rel of Eq. 7 between consecutive fresh
                    velocities is summed per token (i = 1 .. m-1; the sum
                    ranks like the mean), and at i = m - 1 tokens are
                    assigned by its ranking, smallest change to the smallest
                    budget.
    Returns the new state plus the active set, the fresh velocities and the
    hidden states.
    """
    x = state["x"]
    N = x.shape[0]
    idx = active_set(state["budget"], T, i, margin, outside_period)
    xa = gather_latent(x, idx, dtype)
    f = stack_forward(xa, idx, weights, state["caches"], heads, dh, dtype, rope)
    x_new, v_hat = cached_euler(x, state["v_hat"], f["v_fresh"], idx, sigmas[i], sigmas[i + 1])
    budget = state["budget"]
    v_prev, l1 = state.get("v_prev"), state.get("l1")
    refreshed = False
    if group_sizes is not None:
        gs = check_group_sizes(group_sizes, N, T)
        if selection == SELECT_NORM:
            if i % refresh_period(T, [s for s, _ in gs]) == 0:
                if idx.size != N:
                    raise ValueError("a refresh iteration must have every token active")
                budget = assign_groups(v_hat, gs)
                refreshed = True
        elif selection == SELECT_L1REL:
            if margin < 2 or outside_period != 1:
                raise ValueError("strategy D needs a window margin >= 2 with every token active outside it")
            if i < margin:
                l1 = np.zeros(N) if i == 0 else l1 + l1_rel(v_hat, v_prev)
                v_prev = v_hat
                if i == margin - 1:
                    budget = assign_by_key(l1, gs)
                    refreshed = True
        else:
            raise ValueError(f"unknown selection {selection!r}")
    return {"i": i, "idx": idx, "x": x_new, "v_hat": v_hat, "caches": f["caches"], "budget": budget,
            "refreshed": refreshed, "v_fresh": f["v_fresh"], "hidden": f["hidden"], "v_prev": v_prev,
            "l1": l1}


def stack_trajectory(x0, weights: dict, T: int, sigmas, heads: int, dh: int, dtype: str,
                     group_sizes=None, margin: int = 0, iterations=None, state=None,
                     outside_period: int = 1, selection: str = SELECT_NORM, rope=None) -> list:
    """Iterations 0..T-1 (or the first `iterations`) of the multi-layer
    sampler from initial_state (or the given state). With group_sizes None
    and every budget T this is the dense flow-matching loop. Returns one
    record per iteration."""
    d = heads * dh
    if state is None:
        state = initial_state(x0, len(weights["layers"]), d, T)
    records = []
    for i in range(T if iterations is None else iterations):
        r = stack_iteration(state, weights, i, T, sigmas, heads, dh, dtype, group_sizes, margin,
                            outside_period, selection, rope)
        records.append(r)
        state = {"x": r["x"], "v_hat": r["v_hat"], "budget": r["budget"], "caches": r["caches"],
                 "v_prev": r["v_prev"], "l1": r["l1"]}
    return records
