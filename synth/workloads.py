"""Workload shapes and seeded input draws for the HSA active-token layer step.

Token counts follow the video-DiT patchify rule of the paper's preliminaries
(Section 2.1): a VAE latent of F x H_l x W_l patchified with [1, 2, 2] gives
N = F * (H_l/2) * (W_l/2) tokens. The grids below are already in token units
(F x H_l/2 x W_l/2), e.g. 21 x 30 x 52 = 32760 tokens for Wan-2 at 480p and
21 x 45 x 80 = 75600 at 720p.

Nothing here implements the method: the active-set rule, the projections,
attention and the cached Euler update live in the oracle and in the HIP
library, separately. This module only draws random inputs, in a fixed order
from a seeded generator, and assigns per-token step budgets (an input of the
method, Section 2.2, Eq. 3) by ranking a seeded per-token norm.

bf16 inputs are represented on the host as float32 arrays whose values are
exactly representable in bf16 (rounded to nearest-even by torch's own
conversion); `bf16_tensor` turns them into torch bf16 tensors losslessly.
"""

from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np
import torch


@dataclass(frozen=True)
class Workload:
    """One synthetic single-block workload.

    groups: ((budget s_k, token fraction), ...) of the step-budget partition
    (Section 2.2, Eq. 3); every budget divides T (Eq. 5).
    C: channels of the Euler state. None means the block output itself is the
    velocity (the Euler state is the block input, C = d).
    iters: iterations at which the workload is measured or checked.
    layers: self-attention layers of a stack workload (embedding C -> d,
    `layers` layers, velocity head d -> C); 1 for the single-block workloads.
    ffn, ctx: for full blocks, the FFN hidden width and the context length of
    the cross-attention (0: no such sub-layer).
    """

    name: str
    grid: tuple
    d: int
    heads: int
    dh: int
    dtype: str
    T: int
    groups: tuple
    iters: tuple = ()
    C: int | None = None
    layers: int = 1
    ffn: int = 0
    ctx: int = 0
    notes: str = field(default="", compare=False)

    @property
    def N(self) -> int:
        return int(np.prod(self.grid))

    @property
    def euler_channels(self) -> int:
        return self.d if self.C is None else self.C


WORKLOADS = {
    # Tiny fp32 self-attention block; full 8-iteration trajectory.
    "tiny_f32": Workload(
        "tiny_f32", (4, 16, 16), 256, 4, 64, "f32", 8,
        ((8, 1 / 3), (4, 1 / 3), (2, 1 / 3)), iters=tuple(range(8)),
        notes="N=1024, d=256, 4x64 heads, fp32; budgets {8,4,2} by velocity-norm thirds",
    ),
    # Wan-2.1-1.3B-shaped block: d=1536, 12 heads x 128.
    "wan1.3b": Workload(
        "wan1.3b", (21, 30, 52), 1536, 12, 128, "bf16", 40,
        ((40, 0.25), (20, 0.25), (10, 0.25), (5, 0.25)), iters=(2,),
        notes="N=32760, d=1536, 12x128, bf16; iteration 2 has 50% of tokens active",
    ),
    # Wan-2.1-14B-shaped block: d=5120, 40 heads x 128.
    "wan14b": Workload(
        "wan14b", (21, 30, 52), 5120, 40, 128, "bf16", 40,
        ((40, 0.25), (20, 0.25), (10, 0.25), (5, 0.25)), iters=(1, 2, 8),
        notes="N=32760, d=5120, 40x128, bf16; iterations 1/2/8 have 25/50/100% active",
    ),
    # 720p-shaped long sequence with a 16-channel fp32 Euler state.
    "wan14b_720p": Workload(
        "wan14b_720p", (21, 45, 80), 5120, 40, 128, "bf16", 40,
        ((40, 0.25), (10, 0.25), (5, 0.5)), iters=(1,), C=16,
        notes="N=75600, d=5120, 40x128, bf16; iteration 1 has 25% active; Euler over N x 16 fp32",
    ),
    # Stacks for the multi-layer sampling loop: latent of C = 64 values per
    # patch token (16 channels x a 1x2x2 patch), embedding C -> d, `layers`
    # self-attention layers with residual, velocity head d -> C.
    "tiny_stack_f32": Workload(
        "tiny_stack_f32", (3, 10, 10), 128, 2, 64, "f32", 8,
        ((8, 1 / 3), (4, 1 / 3), (2, 1 / 3)), iters=tuple(range(8)), C=16, layers=3,
        notes="N=300, d=128, 2x64, fp32, C=16, 3 layers; T=8, budgets {8,4,2} in thirds",
    ),
    "small_stack_bf16": Workload(
        "small_stack_bf16", (2, 20, 25), 256, 2, 128, "bf16", 8,
        ((8, 0.25), (4, 0.25), (2, 0.5)), iters=(0, 1, 2), C=64, layers=4,
        notes="N=1000, d=256, 2x128, bf16, C=64, 4 layers; T=8, budgets {8:25%, 4:25%, 2:50%}",
    ),
    "tiny_block_f32": Workload(
        "tiny_block_f32", (3, 10, 10), 128, 2, 64, "f32", 8,
        ((8, 1 / 3), (4, 1 / 3), (2, 1 / 3)), iters=tuple(range(8)), C=16, layers=2, ffn=256, ctx=40,
        notes="N=300, d=128, 2x64, fp32, C=16, 2 full blocks (FFN 256, context 40); T=8, budgets {8,4,2}",
    ),
    "small_block_bf16": Workload(
        "small_block_bf16", (2, 20, 25), 256, 2, 128, "bf16", 8,
        ((8, 0.25), (4, 0.25), (2, 0.5)), iters=(0, 1, 2), C=64, layers=3, ffn=512, ctx=77,
        notes="N=1000, d=256, 2x128, bf16, C=64, 3 full blocks (FFN 512, context 77)",
    ),
    "wan1.3b_blocks": Workload(
        "wan1.3b_blocks", (21, 30, 52), 1536, 12, 128, "bf16", 40,
        ((40, 0.25), (20, 0.25), (10, 0.25), (5, 0.25)), iters=tuple(range(40)), C=64, layers=30, ffn=8960,
        ctx=512,
        notes="N=32760, d=1536, 12x128, bf16, C=64, 30 full blocks (FFN 8960, context 512); T=40, quarters",
    ),
    "wan1.3b_stack": Workload(
        "wan1.3b_stack", (21, 30, 52), 1536, 12, 128, "bf16", 40,
        ((40, 0.25), (20, 0.25), (10, 0.25), (5, 0.25)), iters=tuple(range(40)), C=64, layers=30,
        notes="N=32760, d=1536, 12x128, bf16, C=64, 30 layers; T=40, budgets {40,20,10,5} in quarters",
    ),
}


# Budget presets of the paper's Appendix C (runtimes also in Table 1): token
# percentages per step budget, the centred caching window (percent of the
# trajectory) and the token allocation strategy, with T = 40.
PRESETS = {
    "HSA-75A": {"T": 40, "groups": ((40, 0.25), (20, 0.25), (10, 0.50)), "window": 50, "strategy": "D",
                "printed_runtime": 0.75},
    "HSA-75B": {"T": 40, "groups": ((40, 0.33), (10, 0.67)), "window": 50, "strategy": "D",
                "printed_runtime": 0.75},
    "HSA-50": {"T": 40, "groups": ((40, 0.16), (10, 0.84)), "window": 80, "strategy": "D",
               "printed_runtime": 0.50},
    "HSA-25": {"T": 40, "groups": ((20, 0.16), (5, 0.84)), "window": 80, "strategy": "R",
               "printed_runtime": 0.25},
}


def to_bf16_values(a: np.ndarray) -> np.ndarray:
    """Round a float32 array to bf16 (torch's nearest-even conversion) and return
    the rounded values as float32."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32))
    return t.to(torch.bfloat16).to(torch.float32).numpy()


def bf16_tensor(a: np.ndarray) -> torch.Tensor:
    """torch bf16 tensor holding the values of a bf16-valued float32 array."""
    t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
    back = t.to(torch.float32).numpy()
    if not np.array_equal(back, a, equal_nan=True):
        raise ValueError("array is not bf16-valued")
    return t


def _normal(rng: np.random.Generator, shape, scale: float = 1.0) -> np.ndarray:
    z = rng.standard_normal(shape, dtype=np.float32)
    if scale != 1.0:
        z *= np.float32(scale)
    return z


def draw_block(wl: Workload, seed: int = 0, n_tokens: int | None = None) -> dict:
    """Draw the block inputs in the fixed order x, Wq, Wk, Wv, Wo, v_group.

    x ~ N(0, 1) of shape [N, d]; W ~ N(0, 1/d) of shape [d, d] in the
    [d_out, d_in] orientation (y = x W^T); v_group ~ N(0, 1) of shape [N, C],
    whose per-token norms rank tokens into budget groups.
    All arrays are float32; for bf16 workloads they are bf16-valued.
    """
    N = wl.N if n_tokens is None else int(n_tokens)
    d = wl.d
    rng = np.random.default_rng(seed)
    x = _normal(rng, (N, d))
    ws = [_normal(rng, (d, d), 1.0 / math.sqrt(d)) for _ in range(4)]
    v_group = _normal(rng, (N, wl.euler_channels))
    if wl.dtype == "bf16":
        x = to_bf16_values(x)
        ws = [to_bf16_values(w) for w in ws]
    wq, wk, wv, wo = ws
    return {"x": x, "wq": wq, "wk": wk, "wv": wv, "wo": wo, "v_group": v_group}


def assign_budgets(v_group: np.ndarray, groups, layout: str = "scattered", frame_tokens: int = 0,
                   seed: int | None = None) -> np.ndarray:
    """Per-token step budgets (int32[N]) for a budget partition.

    Group sizes: floor(N * fraction) for every budget except the largest, which
    takes the remaining tokens.
    layout "scattered": tokens ranked by the L2 norm of their v_group row
    (stable ascending sort, ties to the lower index); the lowest-norm block
    gets the smallest budget and the highest-norm block the largest.
    layout "contiguous": consecutive index ranges in ascending budget order,
    the largest budget last (the reordered sequence of Section 2.5).
    layout "random": a seeded random permutation of the tokens (strategy R of
    Appendix B), seeded from `seed`, or from the v_group values if None.
    layout "uniform": strategy U of Appendix B, every group spread over the
    whole sequence: tokens ordered by frac(n * golden ratio), a low-discrepancy
    order, and cut into consecutive blocks.
    layout "first_frame": strategy F of Appendix B: the first frame_tokens
    tokens (the first latent frame in row-major patch order) go to the
    largest budget, the rest are placed at random (seeded as "random").
    """
    N = v_group.shape[0]
    order_groups = group_sizes(N, groups)
    if layout == "scattered":
        norms = np.sqrt(np.sum(v_group.astype(np.float64) ** 2, axis=1))
        rank = np.argsort(norms, kind="stable")
    elif layout == "contiguous":
        rank = np.arange(N)
    elif layout in ("random", "first_frame"):
        if seed is None:
            seed = int(np.frombuffer(np.ascontiguousarray(v_group[:1], np.float32).tobytes(), np.uint32)[0])
        rank = np.random.default_rng(seed).permutation(N)
        if layout == "first_frame":
            if not 0 <= frame_tokens <= order_groups[-1][1]:
                raise ValueError("the first frame must fit in the largest-budget group")
            # frame tokens last in the order, so they fall in the largest-budget block
            rest = rank[rank >= frame_tokens]
            rank = np.concatenate([rest, np.arange(frame_tokens)])
    elif layout == "uniform":
        golden = (math.sqrt(5.0) - 1.0) / 2.0
        rank = np.argsort(np.mod(np.arange(N, dtype=np.float64) * golden, 1.0), kind="stable")
    else:
        raise ValueError(f"unknown layout {layout!r}")
    budget = np.empty(N, dtype=np.int32)
    start = 0
    for s, n in order_groups:
        budget[rank[start:start + n]] = s
        start += n
    return budget


def random_budgets(N: int, groups, seed: int) -> np.ndarray:
    """Strategy R for N tokens: a seeded random permutation cut into groups."""
    return assign_budgets(np.zeros((N, 1), np.float32), groups, "random", seed=seed)


def group_sizes(N: int, groups) -> tuple:
    """((s_k, |G_k|), ...) in ascending budget order for N tokens: floor(N *
    fraction) for every budget except the largest, which takes the rest."""
    order_groups = sorted(groups, key=lambda g: g[0])
    sizes = [int(math.floor(N * f)) for _, f in order_groups[:-1]]
    sizes.append(N - sum(sizes))
    if min(sizes) < 0:
        raise ValueError("group fractions exceed 1")
    return tuple((int(s), n) for (s, _), n in zip(order_groups, sizes))


def draw_stack(wl: Workload, seed: int = 0, n_tokens: int | None = None, layers: int | None = None):
    """Initial latent and random-init weights of a stack workload, drawn in the
    fixed order x0, W_embed, then Wq, Wk, Wv, Wo of each layer, then W_head.

    x0 ~ N(0, 1) fp32 [N, C] (the latent at sigma = 1); W_embed ~ N(0, 1/C)
    [d, C]; layer weights ~ N(0, 1/d) [d, d]; W_head ~ N(0, 1/d) [C, d]; all
    [d_out, d_in]. Weights are bf16-valued for bf16 workloads. Full-block
    workloads then draw, from a second stream, the context ctx ~ N(0, 1)
    [ctx_len, d] and per layer Wq_c, Wk_c, Wv_c, Wo_c ~ N(0, 1/d) [d, d],
    W_1 ~ N(0, 1/d) [ffn, d] and W_2 ~ N(0, 1/ffn) [d, ffn].
    """
    N = wl.N if n_tokens is None else int(n_tokens)
    L = wl.layers if layers is None else int(layers)
    d, C = wl.d, wl.euler_channels
    rng = np.random.default_rng([seed, 0x57AC])
    cast = to_bf16_values if wl.dtype == "bf16" else (lambda a: a)
    x0 = _normal(rng, (N, C))
    w_embed = cast(_normal(rng, (d, C), 1.0 / math.sqrt(C)))
    layer_ws = []
    for _ in range(L):
        ws = [cast(_normal(rng, (d, d), 1.0 / math.sqrt(d))) for _ in range(4)]
        layer_ws.append(dict(zip(("wq", "wk", "wv", "wo"), ws)))
    w_head = cast(_normal(rng, (C, d), 1.0 / math.sqrt(d)))
    out = {"x0": x0, "w_embed": w_embed, "layers": layer_ws, "w_head": w_head}
    if wl.ctx or wl.ffn:
        # full blocks: a second stream, so the self-attention draws above do not change
        rng2 = np.random.default_rng([seed, 0xB10C])
        if wl.ctx:
            out["ctx"] = cast(_normal(rng2, (wl.ctx, d)))
        for lw in layer_ws:
            if wl.ctx:
                for k in ("wq_c", "wk_c", "wv_c", "wo_c"):
                    lw[k] = cast(_normal(rng2, (d, d), 1.0 / math.sqrt(d)))
            if wl.ffn:
                lw["w1"] = cast(_normal(rng2, (wl.ffn, d), 1.0 / math.sqrt(d)))
                lw["w2"] = cast(_normal(rng2, (d, wl.ffn), 1.0 / math.sqrt(wl.ffn)))
    return out


def draw_stack_state(wl: Workload, seed: int, n_tokens: int | None = None, layers: int | None = None):
    """A mid-trajectory state of a stack workload: latent x and velocity cache
    [N, C] fp32 ~ N(0, 1) and one (K_hat, V_hat) pair [N, d] ~ N(0, 1) per
    layer (model dtype values), standing in for what earlier iterations left."""
    N = wl.N if n_tokens is None else int(n_tokens)
    L = wl.layers if layers is None else int(layers)
    rng = np.random.default_rng([seed, 0x5747])
    cast = to_bf16_values if wl.dtype == "bf16" else (lambda a: a)
    x = _normal(rng, (N, wl.euler_channels))
    v_hat = _normal(rng, (N, wl.euler_channels))
    caches = [(cast(_normal(rng, (N, wl.d))), cast(_normal(rng, (N, wl.d)))) for _ in range(L)]
    return {"x": x, "v_hat": v_hat, "caches": caches}


def linear_sigmas(T: int) -> np.ndarray:
    """Noise levels sigma_j = (T - j) / T for j = 0..T (1 down to 0), float32."""
    return (np.arange(T, -1, -1, dtype=np.float64) / T).astype(np.float32)


def draw_cache(N: int, d: int, seed: int, dtype: str = "bf16") -> tuple:
    """Synthetic per-layer cache contents (K_hat, V_hat), each [N, d] ~ N(0, 1).

    Stands in for the rows a dense step at an earlier iteration left in the
    cache: with x ~ N(0,1) and W ~ N(0, 1/d), projected rows are ~ N(0, 1) too.
    """
    rng = np.random.default_rng([seed, 0xCACE])
    k = _normal(rng, (N, d))
    v = _normal(rng, (N, d))
    if dtype == "bf16":
        k, v = to_bf16_values(k), to_bf16_values(v)
    return k, v


def draw_euler_state(N: int, C: int, n_fresh: int, seed: int) -> dict:
    """fp32 latent x [N, C], velocity cache [N, C] and fresh velocities
    [n_fresh, C], all ~ N(0, 1)."""
    rng = np.random.default_rng([seed, 0xE01E])
    return {
        "x": _normal(rng, (N, C)),
        "v_cache": _normal(rng, (N, C)),
        "v_fresh": _normal(rng, (n_fresh, C)),
    }
