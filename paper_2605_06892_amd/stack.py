"""Device buffers and the iteration loop of a multi-layer HSA sampler.

The stack (patch embedding, pre-norm self-attention layers with residual and
per-layer caches, final norm and velocity head) and one whole iteration of
the sampler run inside the HIP library (hsa_stack_iteration); this module only
allocates the device tensors with torch, fills the struct the library reads
and calls it once per iteration (Sections 2.2-2.4).
"""

from __future__ import annotations

from dataclasses import dataclass, field

import torch

from . import hsa_step as H


@dataclass
class StackBuffers:
    """Weights, state and scratch of one stack of L layers over N tokens."""

    x: torch.Tensor          # [N, C] fp32 latent
    v_hat: torch.Tensor      # [N, C] fp32 velocity cache
    budget: torch.Tensor     # int32 [N]
    w_embed: torch.Tensor    # [d, C]
    w_head: torch.Tensor     # [C, d]
    layers: list             # per layer (wq, wk, wv, wo), each [d, d]
    caches: list             # per layer (k_hat, v_hat), each [N, d]
    idx: torch.Tensor        # int32 [N]
    n_active: torch.Tensor   # int32 [1]
    xa: torch.Tensor         # [N, C] model dtype
    h: torch.Tensor          # [N, d]
    q: torch.Tensor          # [N, d]
    o: torch.Tensor          # [N, d]
    v_fresh: torch.Tensor    # [N, C] fp32
    keys: torch.Tensor       # float64 [N]
    row_scale: torch.Tensor  # fp32 [N]
    v_prev: torch.Tensor     # [N, C] fp32 (strategy D)
    heads: int
    head_dim: int
    cross: list | None = None   # per layer (wq_c, wo_c, k_c, v_c); k_c, v_c [ctx, d]
    ffn: list | None = None     # per layer (w1 [F, d], w2 [d, F])
    f: torch.Tensor | None = None  # [N, F]
    rope_cs: torch.Tensor | None = None  # rotary (cos, sin) table on the device
    pos: torch.Tensor | None = None      # int32 [N] grid position of every token
    grid: tuple = (0, 0, 0)
    n_cached: int | None = None          # prefix-only cache: rows per layer cache
    k_tail: torch.Tensor | None = None   # [N - n_cached, d] fresh baseline keys
    v_tail: torch.Tensor | None = None
    attn_parts: torch.Tensor | None = None  # uint8 scratch: key parts of the attention launches
    _handle: H.HsaStack | None = field(default=None, repr=False)

    @property
    def N(self) -> int:
        return self.x.shape[0]

    @property
    def C(self) -> int:
        return self.x.shape[1]

    @property
    def d(self) -> int:
        return self.heads * self.head_dim

    @classmethod
    def allocate(cls, N: int, C: int, n_layers: int, heads: int, head_dim: int, dtype: torch.dtype,
                 device="cuda", ffn: int = 0, ctx: int = 0, n_cached: int | None = None,
                 kv_parts: bool = True) -> "StackBuffers":
        """Tensors for N tokens, C latent values per token, n_layers layers of
        width heads * head_dim; ffn > 0 / ctx > 0 add the FFN and
        cross-attention sub-layers of full blocks; n_cached (prefix-only
        cache of reordered tokens, Section 2.5) sizes each layer's cache to
        the non-baseline prefix; kv_parts adds the scratch with which bf16
        attention launches of few workgroups split their cached rows."""
        d = heads * head_dim
        e = lambda *s, dt=dtype: torch.empty(*s, dtype=dt, device=device)  # noqa: E731
        f32 = torch.float32
        rows = N if n_cached is None else n_cached
        parts = None
        if kv_parts and dtype == torch.bfloat16:
            nb = H.hsa_attention_parts_workspace_bytes(dtype, N, heads, head_dim) - \
                H.hsa_attention_workspace_bytes(dtype, N, d)
            parts = torch.empty(max(nb, 1), dtype=torch.uint8, device=device)
        tail = None if n_cached is None else N - n_cached
        return cls(x=e(N, C, dt=f32), v_hat=e(N, C, dt=f32), budget=e(N, dt=torch.int32),
                   w_embed=e(d, C), w_head=e(C, d),
                   layers=[tuple(e(d, d) for _ in range(4)) for _ in range(n_layers)],
                   caches=[(e(max(rows, 1), d), e(max(rows, 1), d)) for _ in range(n_layers)],
                   n_cached=n_cached, k_tail=None if tail is None else e(max(tail, 1), d),
                   v_tail=None if tail is None else e(max(tail, 1), d),
                   idx=e(N, dt=torch.int32), n_active=e(1, dt=torch.int32), xa=e(N, C), h=e(N, d), q=e(N, d),
                   o=e(N, d), v_fresh=e(N, C, dt=f32), keys=e(N, dt=torch.float64), row_scale=e(N, dt=f32),
                   v_prev=e(N, C, dt=f32), heads=heads, head_dim=head_dim,
                   cross=[(e(d, d), e(d, d), e(ctx, d), e(ctx, d)) for _ in range(n_layers)] if ctx else None,
                   ffn=[(e(ffn, d), e(d, ffn)) for _ in range(n_layers)] if ffn else None,
                   f=e(N, ffn) if ffn else None, attn_parts=parts)

    def enable_rope(self, grid, theta: float = 10000.0, pos: torch.Tensor | None = None) -> None:
        """Rotate Q and K by the tokens' positions in the latent grid (F, H, W)
        (Section 2.3: the positional frequencies follow the active set). pos:
        the grid position of every token, identity if None."""
        self.rope_cs = H.hsa_rope_table(theta, self.head_dim, grid).to(self.x.device)
        self.pos = pos
        self.grid = tuple(int(g) for g in grid)
        self._handle = None

    def set_context(self, ctx: torch.Tensor, wk_c, wv_c) -> None:
        """K_c = ctx Wk_c^T and V_c = ctx Wv_c^T of every layer, computed once
        per sample on the device (hsa_linear)."""
        for (_, _, kc, vc), wk, wv in zip(self.cross, wk_c, wv_c):
            H.hsa_linear(ctx, ctx.shape[0], wk, kc)
            H.hsa_linear(ctx, ctx.shape[0], wv, vc)

    def handle(self) -> H.HsaStack:
        """The struct hsa_stack describing these tensors (built once)."""
        if self._handle is None:
            self._handle = H.make_stack(x=self.x, v_hat=self.v_hat, budget=self.budget, w_embed=self.w_embed,
                                        w_head=self.w_head, layers=self.layers, caches=self.caches, idx=self.idx,
                                        n_active=self.n_active, xa=self.xa, h=self.h, q=self.q, o=self.o,
                                        v_fresh=self.v_fresh, keys=self.keys, row_scale=self.row_scale,
                                        heads=self.heads, head_dim=self.head_dim, cross=self.cross,
                                        ffn=self.ffn, f=self.f, v_prev=self.v_prev, rope_cs=self.rope_cs,
                                        pos=self.pos, grid=self.grid, n_cached=self.n_cached,
                                        k_tail=self.k_tail, v_tail=self.v_tail, attn_parts=self.attn_parts)
        return self._handle


def reorder(b: StackBuffers, T: int) -> torch.Tensor:
    """Token reordering before the loop (Section 2.5): non-baseline tokens
    first, the budget-T group last. Permutes the latent, the velocity cache,
    the budgets and the grid positions (created if absent) on the device and
    returns the permutation (new position i holds old token perm[i])."""
    perm = torch.empty(b.N, dtype=torch.int32, device=b.x.device)
    n_lead = torch.empty(1, dtype=torch.int32, device=b.x.device)
    lead = H.hsa_reorder_plan(b.budget, T, perm, n_lead)
    if b.n_cached is not None and lead > b.n_cached:
        raise ValueError(f"{lead} non-baseline tokens but caches sized for {b.n_cached}")
    if b.pos is None:
        b.pos = torch.arange(b.N, dtype=torch.int32, device=b.x.device)
    for t in (b.x, b.v_hat, b.budget, b.pos):
        tmp = torch.empty_like(t)
        H.hsa_permute_rows(t, perm, tmp)
        t.copy_(tmp)
    b._handle = None
    return perm


def prefix_rows(n_lead: int, N: int) -> int:
    """Cache rows of the prefix-only cache for n_lead non-baseline tokens: the
    next multiple of 64, the granularity the stack accepts (at most N)."""
    return min(N, -(-n_lead // 64) * 64)


def restore_order(b: StackBuffers, perm: torch.Tensor) -> torch.Tensor:
    """The latent in the original token order (the reordering inverted)."""
    out = torch.empty_like(b.x)
    H.hsa_permute_rows(b.x, perm, out, inverse=True)
    return out


def iteration(b: StackBuffers, T: int, i: int, sigmas, group_sizes=None, margin: int = 0,
              outside_period: int = 1, selection: int = H.SELECT_VELOCITY_NORM, stream=None) -> tuple:
    """Iteration i of the sampler; returns (|A_i|, refreshed)."""
    return H.hsa_stack_iteration(b.handle(), T, i, margin, float(sigmas[i]), float(sigmas[i + 1]), group_sizes,
                                 stream, outside_period, selection)


def run(b: StackBuffers, T: int, sigmas, group_sizes=None, margin: int = 0, iterations=None,
        start: int = 0, outside_period: int = 1, selection: int = H.SELECT_VELOCITY_NORM,
        stream=None) -> list:
    """Iterations start .. start+iterations-1 (default: the whole trajectory);
    returns the (|A_i|, refreshed) of each."""
    stop = T if iterations is None else start + iterations
    return [iteration(b, T, i, sigmas, group_sizes, margin, outside_period, selection, stream)
            for i in range(start, stop)]
