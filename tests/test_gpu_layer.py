"""GPU parity of whole HSA iterations against the CPU oracle.

* The tiny fp32 workload (N=1024, d=256, 4 heads x 64, T=8, budgets {8,4,2})
  runs its full 8-iteration trajectory on the GPU; every iteration's active
  set must match bit for bit and the latents, velocity cache and KV caches
  must stay within 1e-4 of the oracle.
* The Wan-shaped bf16 workloads run one iteration at full size in the launch
  configuration the benchmark times. The oracle computes the fresh K/V rows
  of every active token (the full cache is needed by any query) but only a
  seeded sample of 512 active query rows through attention and the output
  projection; skipped cache and output rows are compared bit for bit in full.
  The Wan-14B block is run at 25%, 50% and 100% active, in the scattered and
  contiguous budget layouts. At 100% (iteration 8, where every budget's
  schedule fires) the HSA step is the dense step (Section 2.3): the index list
  is the identity, every output row is written and finite, and the sampled
  rows match the oracle's dense step.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import DEV, TOL, Guarded, host, host_bits, i32, rel_inf, to_dev

pytest.importorskip("paper_2605_06892_amd.hsa_step")
from paper_2605_06892_amd import layer as L  # noqa: E402

pytestmark = pytest.mark.gpu


def test_tiny_f32_trajectory():
    wl = synth.WORKLOADS["tiny_f32"]
    blk = synth.draw_block(wl, 0)
    budget = synth.assign_budgets(blk["v_group"], wl.groups)
    s = synth.linear_sigmas(wl.T)
    w = {k: blk[k] for k in ("wq", "wk", "wv", "wo")}
    recs = oracle.trajectory(blk["x"], budget, wl.T, s, w, wl.heads, wl.dh, "f32")

    b = L.BlockBuffers.allocate(wl.N, wl.d, wl.heads, wl.dh, torch.float32)
    b.x.copy_(to_dev(blk["x"], "f32"))
    for k in ("wq", "wk", "wv", "wo"):
        getattr(b, k).copy_(to_dev(blk[k], "f32"))
    b.budget.copy_(i32(budget))
    for t in (b.k_cache, b.v_cache, b.out):
        t.zero_()
    for r in recs:
        n = L.block_trajectory_step(b, wl.T, r["i"], s)
        assert n == r["idx"].size
        np.testing.assert_array_equal(b.idx[:n].cpu().numpy(), r["idx"])
        assert rel_inf(host(b.q[:n]), r["q"]) <= TOL["f32"]
        assert rel_inf(host(b.k_cache), r["k_cache"]) <= TOL["f32"]
        assert rel_inf(host(b.v_cache), r["v_cache"]) <= TOL["f32"]
        assert rel_inf(host(b.o[:n]), r["o"]) <= TOL["f32"]
        assert rel_inf(host(b.out), r["v_hat"]) <= TOL["f32"]
        assert rel_inf(host(b.x), r["x"]) <= TOL["f32"], r["i"]


FULL = [
    ("wan1.3b", 2, "scattered"),
    ("wan14b", 1, "scattered"),
    ("wan14b", 1, "contiguous"),
    ("wan14b", 2, "scattered"),
    ("wan14b", 2, "contiguous"),
    ("wan14b", 8, "scattered"),       # every token active: the dense step, 5120 attention workgroups
    ("wan14b_720p", 1, "scattered"),  # N = 75600, 18900 active rows
]
SAMPLED_ROWS = 512


@pytest.mark.parametrize("name,it,layout", FULL, ids=lambda v: str(v))
def test_full_shape_iteration(name, it, layout):
    wl = synth.WORKLOADS[name]
    N, d = wl.N, wl.d
    blk = synth.draw_block(wl, 0)
    budget = synth.assign_budgets(blk["v_group"], wl.groups, layout)
    k0, v0 = synth.draw_cache(N, d, seed=1, dtype="bf16")
    out0 = synth.draw_cache(N, d, seed=2, dtype="bf16")[0]
    idx_ref = oracle.active_set(budget, wl.T, it)

    b = L.BlockBuffers.allocate(N, d, wl.heads, wl.dh, torch.bfloat16)
    # every buffer the step writes sits between red zones
    guards = {k: Guarded(tuple(getattr(b, k).shape), getattr(b, k).dtype, seed=i)
              for i, k in enumerate(("k_cache", "v_cache", "out", "q", "o", "idx", "n_active"))}
    for k, gz in guards.items():
        setattr(b, k, gz.t)
    b.x.copy_(to_dev(blk["x"], "bf16"))
    for k in ("wq", "wk", "wv", "wo"):
        getattr(b, k).copy_(to_dev(blk[k], "bf16"))
    b.budget.copy_(i32(budget))
    b.k_cache.copy_(to_dev(k0, "bf16"))
    b.v_cache.copy_(to_dev(v0, "bf16"))
    b.out.copy_(to_dev(out0, "bf16"))
    n = L.active_set(b, wl.T, it)
    assert n == idx_ref.size
    np.testing.assert_array_equal(b.idx[:n].cpu().numpy(), idx_ref)
    print(f"full-shape iteration {name} i={it} {layout}: |A|={n} of N={N}", flush=True)
    L.layer_step(b, n)
    torch.cuda.synchronize()
    for k, gz in guards.items():
        gz.check(k)
    if n == N:
        # all active: the identity index list, every output row written (none keeps its old
        # value) and finite
        np.testing.assert_array_equal(idx_ref, np.arange(N))
        assert bool(torch.isfinite(b.out).all()) and bool(torch.isfinite(b.o[:n]).all())
        changed = (b.out.view(torch.int16) != to_dev(out0, "bf16").view(torch.int16)).any(dim=1)
        assert int(changed.sum()) == N

    # skipped rows: bit for bit untouched
    skipped = np.setdiff1d(np.arange(N), idx_ref)
    for t, ref in ((b.k_cache, k0), (b.v_cache, v0), (b.out, out0)):
        np.testing.assert_array_equal(host_bits(t)[skipped], host_bits(to_dev(ref[skipped], "bf16")))

    # oracle: fresh K/V for every active row, the rest of the cache from the prefill
    xa = blk["x"][idx_ref]
    k_new = oracle.project(xa, blk["wk"], "bf16")
    v_new = oracle.project(xa, blk["wv"], "bf16")
    assert rel_inf(host(b.k_cache[torch.from_numpy(idx_ref).to(DEV)]), k_new) <= 1e-2
    assert rel_inf(host(b.v_cache[torch.from_numpy(idx_ref).to(DEV)]), v_new) <= 1e-2
    k_full = k0.astype(np.float64)
    v_full = v0.astype(np.float64)
    k_full[idx_ref] = k_new
    v_full[idx_ref] = v_new
    del k_new, v_new

    # sampled active query rows through attention and the output projection
    rng = np.random.default_rng(it)
    js = np.sort(rng.choice(n, size=min(n, SAMPLED_ROWS), replace=False))
    q_s = oracle.project(xa[js], blk["wq"], "bf16")
    assert rel_inf(host(b.q[torch.from_numpy(js).to(DEV)]), q_s) <= 1e-2
    r = oracle.attention_output(q_s, k_full, v_full, blk["wo"], wl.heads, wl.dh, 1 / math.sqrt(wl.dh), "bf16")
    o_gpu = host(b.o[torch.from_numpy(js).to(DEV)])
    assert rel_inf(o_gpu, r["o"]) <= TOL["bf16"]
    out_gpu = host(b.out[torch.from_numpy(idx_ref[js]).to(DEV)])
    assert rel_inf(out_gpu, r["y"]) <= TOL["bf16"]
