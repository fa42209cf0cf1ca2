"""One HSA iteration of a single DiT self-attention block on device buffers.

Strings the C ABI calls together in stream order (Section 2.3, then 2.4):

    hsa_build_active_set   A_i from the per-token budgets
    hsa_qkv_scatter        Q of A_i, K_hat/V_hat rows A_i overwritten
    hsa_attention_core     active queries against all N cached rows (key parts
                           with the split variant when few workgroups would run)
    hsa_out_scatter        output projection, scattered to rows A_i
    hsa_cached_euler       all tokens advanced by the shared sigma step

Buffers are allocated once with torch (device memory only) and owned by the
caller; nothing here computes.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

import torch

from . import hsa_step as H


@dataclass
class BlockBuffers:
    """Device state of one single-block workload with N tokens of width d."""

    x: torch.Tensor          # [N, d] block input
    wq: torch.Tensor         # [d, d] each, [d_out, d_in]
    wk: torch.Tensor
    wv: torch.Tensor
    wo: torch.Tensor
    k_cache: torch.Tensor    # [N, d]
    v_cache: torch.Tensor    # [N, d]
    out: torch.Tensor        # [N, d] per-token block output
    q: torch.Tensor          # [N, d] capacity for the compact queries
    o: torch.Tensor          # [N, d] capacity for the compact attention output
    budget: torch.Tensor     # int32 [N]
    idx: torch.Tensor        # int32 [N]
    n_active: torch.Tensor   # int32 [1]
    heads: int
    head_dim: int
    parts: torch.Tensor | None = None  # uint8 scratch: key parts of the attention launches
    n_active_host: torch.Tensor | None = None  # pinned int32 [1]: the read-back of |A_i|

    @property
    def N(self) -> int:
        return self.k_cache.shape[0]

    @property
    def d(self) -> int:
        return self.k_cache.shape[1]

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    @classmethod
    def allocate(cls, N: int, d: int, heads: int, head_dim: int, dtype: torch.dtype,
                 device="cuda", kv_parts: bool = True) -> "BlockBuffers":
        """kv_parts adds the scratch with which bf16 attention launches of
        few workgroups split their cached rows."""
        e = lambda *s, dt=dtype: torch.empty(*s, dtype=dt, device=device)  # noqa: E731
        parts = None
        if kv_parts and dtype == torch.bfloat16:
            nb = H.hsa_attention_parts_workspace_bytes(dtype, N, heads, head_dim) - \
                H.hsa_attention_workspace_bytes(dtype, N, d)
            parts = torch.empty(max(nb, 1), dtype=torch.uint8, device=device)
        return cls(x=e(N, d), wq=e(d, d), wk=e(d, d), wv=e(d, d), wo=e(d, d),
                   k_cache=e(N, d), v_cache=e(N, d), out=e(N, d), q=e(N, d), o=e(N, d),
                   budget=e(N, dt=torch.int32), idx=e(N, dt=torch.int32),
                   n_active=e(1, dt=torch.int32), heads=heads, head_dim=head_dim, parts=parts,
                   n_active_host=torch.empty(1, dtype=torch.int32, pin_memory=torch.device(device).type == "cuda"))


def active_set(b: BlockBuffers, T: int, iteration: int, margin: int = 0, outside_period: int = 1) -> int:
    """A_i into b.idx; returns |A_i| (one stream synchronization)."""
    return H.hsa_build_active_set(b.budget, T, iteration, margin, b.idx, b.n_active,
                                  outside_period=outside_period, host_buf=b.n_active_host)


def qkv(b: BlockBuffers, n_active: int, x_compact: bool = False) -> None:
    H.hsa_qkv_scatter(b.x, b.idx, n_active, b.wq, b.wk, b.wv, b.q, b.k_cache, b.v_cache, x_compact)


def attention(b: BlockBuffers, n_active: int) -> None:
    H.hsa_attention_core(b.q, b.k_cache, b.v_cache, n_active, b.heads, b.head_dim, b.scale, b.o, parts=b.parts)


def out_projection(b: BlockBuffers, n_active: int) -> None:
    H.hsa_out_scatter(b.o, b.idx, n_active, b.wo, b.out)


def layer_step(b: BlockBuffers, n_active: int, x_compact: bool = False) -> None:
    """Q/K/V + cache overwrite, attention, output projection + scatter."""
    qkv(b, n_active, x_compact)
    attention(b, n_active)
    out_projection(b, n_active)


def block_trajectory_step(b: BlockBuffers, T: int, iteration: int, sigmas, margin: int = 0) -> int:
    """One iteration of the single-block sampler whose state is the block
    input itself: A_i, the layer step (its output rows are the fresh
    velocities, so b.out is the velocity cache), then the cached Euler update
    of every token. fp32 only (the Euler state is fp32)."""
    n = active_set(b, T, iteration, margin)
    layer_step(b, n)
    H.hsa_cached_euler(b.x, b.out, None, None, 0, float(sigmas[iteration]), float(sigmas[iteration + 1]))
    return n
