"""GPU parity of the multi-layer sampling loop against the CPU oracle.

* hsa_gather_rows, hsa_linear and hsa_assign_budgets on their own: the gather
  and the group assignment bit for bit, the linear maps within the fp32 /
  bf16 tolerances.
* The tiny fp32 stack (N=300, d=128, 3 layers, T=8, budgets {8,4,2}) runs its
  whole trajectory with group refresh at iterations 0 and 4: active sets and
  refreshed budgets bit for bit, latent, velocity cache and every layer's
  caches within 1e-4.
* The small bf16 stack (N=1000, d=256, 4 layers) runs single iterations from
  a synthetic mid-trajectory state, partial and refreshing.
* The Wan-1.3B-shaped 30-layer stack (N=32760, d=1536) runs two iterations in
  the configuration the benchmark times; checked by properties that hold at
  any size and by the oracle on a sample of layer-0 cache rows.
"""

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import DEV, TOL, host, host_bits, i32, rel_inf, to_dev, torch_dtype

pytest.importorskip("paper_2605_06892_amd.hsa_step")
from paper_2605_06892_amd import hsa_step as H  # noqa: E402
from paper_2605_06892_amd import stack as S  # noqa: E402

pytestmark = pytest.mark.gpu


# ---------------------------------------------------------------------------
# Building blocks
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("dtype,N,C,n_act", [("bf16", 1000, 64, 377), ("f32", 300, 16, 300),
                                             ("f32", 257, 7, 100), ("bf16", 64, 6, 5)])
def test_gather_rows(dtype, N, C, n_act):
    rng = np.random.default_rng(N + C)
    x = (rng.standard_normal((N, C)) * 3).astype(np.float32)
    idx = np.sort(rng.choice(N, n_act, replace=False)).astype(np.int32)
    idx_dev = idx.copy()
    idx_dev[::17] = -1  # out-of-range rows are written as zeros
    xa = torch.full((N, C), 7.0, dtype=torch_dtype(dtype), device=DEV)
    H.hsa_gather_rows(to_dev(x, "f32"), i32(idx_dev), n_act, xa)
    want = oracle.gather_latent(x, idx, dtype)
    want[::17] = 0.0
    np.testing.assert_array_equal(host(xa[:n_act]), want)
    np.testing.assert_array_equal(host(xa[n_act:]), 7.0)  # rows past n_active untouched


@pytest.mark.parametrize("dtype,n,d", [("bf16", 1000, 256), ("bf16", 777, 1536), ("bf16", 5, 200),
                                       ("f32", 300, 128), ("f32", 33, 18)])
def test_row_rms_scale(dtype, n, d):
    rng = np.random.default_rng(n + d)
    cast = synth.to_bf16_values if dtype == "bf16" else (lambda a: a)
    x = cast((rng.standard_normal((n, d)) * rng.uniform(0.01, 30, size=(n, 1))).astype(np.float32))
    x[0] = 0.0  # an all-zero row: 1 / sqrt(eps)
    s = torch.zeros(n + 3, device=DEV)
    H.hsa_row_rms_scale(to_dev(x, dtype), n, s)
    want = 1.0 / np.sqrt(np.mean(x.astype(np.float64) ** 2, axis=1) + oracle.RMS_EPS)
    np.testing.assert_allclose(host(s[:n]), want, rtol=2e-6)
    assert np.all(host(s[n:]) == 0.0)


@pytest.mark.parametrize("dtype,n,d_in,d_out,mode", [
    ("bf16", 1000, 64, 256, "plain"),      # embedding
    ("bf16", 777, 1536, 1536, "residual"),  # residual output projection
    ("bf16", 300, 256, 64, "f32out"),       # velocity head
    ("bf16", 33, 1536, 64, "f32out"),
    ("bf16", 700, 256, 768, "normed"),      # Q/K/V projection of rms(h)
    ("bf16", 300, 1536, 64, "normed_f32out"),  # head of rms(h)
    ("f32", 300, 16, 128, "plain"),
    ("f32", 301, 128, 128, "residual"),
    ("f32", 300, 128, 16, "plain"),
    ("f32", 300, 128, 48, "normed"),
    ("bf16", 500, 256, 512, "normed_gelu"),  # FFN up-projection of rms(h)
    ("bf16", 64, 1536, 8960, "normed_gelu"),
    ("f32", 300, 128, 256, "normed_gelu"),
])
def test_linear(dtype, n, d_in, d_out, mode):
    rng = np.random.default_rng(n + d_in + d_out)
    cast = synth.to_bf16_values if dtype == "bf16" else (lambda a: a)
    x = cast((rng.standard_normal((n, d_in)) * rng.uniform(0.1, 10, size=(n, 1))).astype(np.float32))
    w = cast((rng.standard_normal((d_out, d_in)) / np.sqrt(d_in)).astype(np.float32))
    out_dt = "f32" if mode.endswith("f32out") else dtype
    if mode == "residual":
        r = cast(rng.standard_normal((n, d_out)).astype(np.float32))
        y = to_dev(r, dtype)
        H.hsa_linear(to_dev(x, dtype), n, to_dev(w, dtype), y, residual=y)  # in place
        want = oracle.linear(x, w, dtype, residual=r)
    elif mode.startswith("normed"):
        xd = to_dev(x, dtype)
        s = torch.empty(n, device=DEV)
        H.hsa_row_rms_scale(xd, n, s)
        y = torch.zeros((n, d_out), dtype=torch_dtype(out_dt), device=DEV)
        gelu = mode.endswith("gelu")
        H.hsa_linear(xd, n, to_dev(w, dtype), y, row_scale=s, gelu=gelu)
        if gelu:
            want = oracle.round_to(oracle.gelu_tanh(oracle.rms_normalize(x) @ w.astype(np.float64).T), out_dt)
        else:
            want = oracle.linear(oracle.rms_normalize(x), w, out_dt)
    else:
        y = torch.zeros((n, d_out), dtype=torch_dtype(out_dt), device=DEV)
        H.hsa_linear(to_dev(x, dtype), n, to_dev(w, dtype), y)
        want = oracle.linear(x, w, out_dt)
    assert rel_inf(host(y), want) <= TOL[out_dt] / (10 if out_dt == "f32" and dtype == "bf16" else 1)
    if dtype == "bf16" and out_dt == "bf16":
        # single rounding of an fp32 accumulation: at most one bf16 ulp off
        got = host(y)
        assert np.all(np.abs(got - want) <= np.abs(want) * 2.0 ** -7 + 1e-4 * np.abs(want).max())


@pytest.mark.parametrize("n,d_in,d_out,mode", [
    (4059, 192, 8256, "plain"),     # 256 x 192 tiles (16 x 43): 3 K steps (odd), ragged rows and columns
    (4059, 448, 8256, "residual"),  # 7 K steps
    (2049, 320, 16384, "gelu"),     # 256 x 256 tiles (9 x 64 = 576): 5 K steps; the last 64 tiles
                                    # (the 9th tile-row) run as 256 x 128 halves
    (2049, 320, 16320, "residual"), # idem, the last column tile 192 wide: its second half is ragged
    (2049, 320, 16256, "plain"),    # idem, 128 wide: its second half lies past the columns
    (700, 64, 768, "plain"),        # 256 x 128 tiles (a grid of few tiles): 1 K step (no steady-state loop)
    (700, 192, 768, "residual"),    # 3 K steps: one steady-state round then the tail
    (513, 640, 1000, "gelu"),       # 10 K steps, ragged columns
])
def test_linear_k_steps(n, d_in, d_out, mode):
    """The bf16 product over K step counts that exercise the steady-state
    loop (loads interleaved with the MFMAs) and its tail, on all three
    tilings, and a last round of 256 x 256 tiles run as 256 x 128 halves."""
    rng = np.random.default_rng(n * 7 + d_in)
    x = synth.to_bf16_values(rng.standard_normal((n, d_in)).astype(np.float32))
    w = synth.to_bf16_values((rng.standard_normal((d_out, d_in)) / np.sqrt(d_in)).astype(np.float32))
    xd, wd = to_dev(x, "bf16"), to_dev(w, "bf16")
    if mode == "residual":
        r = synth.to_bf16_values(rng.standard_normal((n, d_out)).astype(np.float32))
        y = to_dev(r, "bf16")
        H.hsa_linear(xd, n, wd, y, residual=y)
        want = oracle.linear(x, w, "bf16", residual=r)
    else:
        y = torch.zeros((n, d_out), dtype=torch.bfloat16, device=DEV)
        H.hsa_linear(xd, n, wd, y, gelu=(mode == "gelu"))
        prod = x.astype(np.float64) @ w.astype(np.float64).T
        want = oracle.round_to(oracle.gelu_tanh(prod), "bf16") if mode == "gelu" else oracle.linear(x, w, "bf16")
    got = host(y)
    assert np.all(np.abs(got - want) <= np.abs(want) * 2.0 ** -7 + 1e-4 * np.abs(want).max())


@pytest.mark.parametrize("N,C,case", [(3000, 64, "normal"), (1000, 16, "normal"), (23, 5, "ties"),
                                      (32760, 64, "normal"), (700, 64, "nan")])
def test_assign_budgets(N, C, case):
    rng = np.random.default_rng(N + C)
    if case == "ties":
        v = rng.integers(-3, 4, size=(N, C)).astype(np.float32)
        v[4] = v[9] = v[17]
        v[11] = 0.0
        sizes = ((2, 6), (5, 7), (10, 10))
        T = 10
    else:
        v = rng.standard_normal((N, C)).astype(np.float32)
        if case == "nan":
            v[[3, 50, 51], 5] = np.nan
        sizes = synth.group_sizes(N, ((40, .25), (20, .25), (10, .25), (5, .25)))
        T = 40
    budget = torch.full((N,), -5, dtype=torch.int32, device=DEV)
    ws = torch.empty(H.hsa_assign_budgets_workspace_bytes(N), dtype=torch.uint8, device=DEV)
    H.hsa_assign_budgets(to_dev(v, "f32"), T, sizes, budget, ws)
    np.testing.assert_array_equal(budget.cpu().numpy(), oracle.assign_groups(v, sizes))
    # the keys left in the workspace are the oracle's, bit for bit
    keys = ws.view(torch.float64).cpu().numpy()
    np.testing.assert_array_equal(keys.view(np.uint64),
                                  np.where(np.isnan(oracle.velocity_keys(v)), np.nan,
                                           oracle.velocity_keys(v)).view(np.uint64))


def test_l1_rel_accumulate_and_assign_by_key():
    rng = np.random.default_rng(77)
    N, C = 5000, 64
    vs = [rng.standard_normal((N, C)).astype(np.float32) for _ in range(3)]
    vs[1][7] = 0.0                      # x / 0 -> inf
    vs[1][8] = vs[0][8] = 0.0           # 0 / 0 -> NaN
    acc = torch.full((N,), 5.0, dtype=torch.float64, device=DEV)
    v_prev = torch.zeros((N, C), device=DEV)
    for i, v in enumerate(vs):
        H.hsa_l1_rel_accumulate(to_dev(v, "f32"), v_prev, acc, first=(i == 0))
    want = oracle.l1_rel(vs[1], vs[0]) + oracle.l1_rel(vs[2], vs[1])
    got = acc.cpu().numpy()
    np.testing.assert_array_equal(np.isnan(got), np.isnan(want))
    fin = ~np.isnan(want)
    np.testing.assert_array_equal(got[fin].view(np.uint64), want[fin].view(np.uint64))  # bit for bit
    np.testing.assert_array_equal(host(v_prev), vs[2])
    sizes = synth.group_sizes(N, ((40, .25), (20, .25), (10, .25), (5, .25)))
    budget = torch.zeros(N, dtype=torch.int32, device=DEV)
    H.hsa_assign_budgets_by_key(acc, 40, sizes, budget)
    np.testing.assert_array_equal(budget.cpu().numpy(), oracle.assign_by_key(want, sizes))


def test_assign_budgets_rejects_bad_groups():
    v = torch.zeros((8, 4), device=DEV)
    b = torch.zeros(8, dtype=torch.int32, device=DEV)
    ws = torch.empty(64, dtype=torch.uint8, device=DEV)
    for sizes in (((4, 4), (2, 4)), ((2, 4), (4, 3)), ((3, 4), (8, 4))):
        with pytest.raises(H.HsaStepError) as e:
            H.hsa_assign_budgets(v, 8, sizes, b, ws)
        assert e.value.name == "HSA_STEP_ERR_BUDGET"
    with pytest.raises(H.HsaStepError) as e:
        H.hsa_assign_budgets(v, 8, ((2, 4), (4, 4)), b, ws[:32])
    assert e.value.name == "HSA_STEP_ERR_WORKSPACE"


# ---------------------------------------------------------------------------
# Whole iterations
# ---------------------------------------------------------------------------


def _upload(wl, wts, N, L, state=None, rope_pos=None):
    b = S.StackBuffers.allocate(N, wl.euler_channels, L, wl.heads, wl.dh, torch_dtype(wl.dtype),
                                ffn=wl.ffn, ctx=wl.ctx)
    if rope_pos is not None:
        b.enable_rope(wl.grid, pos=i32(rope_pos))
    b.w_embed.copy_(to_dev(wts["w_embed"], wl.dtype))
    b.w_head.copy_(to_dev(wts["w_head"], wl.dtype))
    for dst, lw in zip(b.layers, wts["layers"]):
        for t, k in zip(dst, ("wq", "wk", "wv", "wo")):
            t.copy_(to_dev(lw[k], wl.dtype))
    if wl.ctx:
        for dst, lw in zip(b.cross, wts["layers"]):
            dst[0].copy_(to_dev(lw["wq_c"], wl.dtype))
            dst[1].copy_(to_dev(lw["wo_c"], wl.dtype))
        b.set_context(to_dev(wts["ctx"], wl.dtype), [to_dev(lw["wk_c"], wl.dtype) for lw in wts["layers"]],
                      [to_dev(lw["wv_c"], wl.dtype) for lw in wts["layers"]])
    if wl.ffn:
        for dst, lw in zip(b.ffn, wts["layers"]):
            dst[0].copy_(to_dev(lw["w1"], wl.dtype))
            dst[1].copy_(to_dev(lw["w2"], wl.dtype))
    if state is None:
        b.x.copy_(to_dev(wts["x0"], "f32"))
        b.v_hat.zero_()
        b.budget.fill_(wl.T)
        for k, v in b.caches:
            k.zero_()
            v.zero_()
    else:
        b.x.copy_(to_dev(state["x"], "f32"))
        b.v_hat.copy_(to_dev(state["v_hat"], "f32"))
        b.budget.copy_(i32(state["budget"]))
        for (k, v), (kh, vh) in zip(b.caches, state["caches"]):
            k.copy_(to_dev(kh, wl.dtype))
            v.copy_(to_dev(vh, wl.dtype))
    return b


@pytest.mark.parametrize("name,margin,selection,rope", [
    ("tiny_stack_f32", 0, "norm", False), ("tiny_block_f32", 0, "norm", False),
    ("tiny_stack_f32", 2, "l1rel", False), ("tiny_block_f32", 3, "l1rel", False),
    ("tiny_stack_f32", 0, "norm", True), ("tiny_block_f32", 2, "l1rel", True)])
def test_tiny_f32_stack_trajectory(name, margin, selection, rope):
    wl = synth.WORKLOADS[name]
    wts = synth.draw_stack(wl, seed=0)
    sizes = synth.group_sizes(wl.N, wl.groups)
    sig = synth.linear_sigmas(wl.T)
    pos = np.random.default_rng(9).permutation(wl.N).astype(np.int32) if rope else None
    recs = oracle.stack_trajectory(wts["x0"], wts, wl.T, sig, wl.heads, wl.dh, "f32", group_sizes=sizes,
                                   margin=margin, selection=selection,
                                   rope={"grid": wl.grid, "pos": pos} if rope else None)
    sel = H.SELECT_L1_REL if selection == "l1rel" else H.SELECT_VELOCITY_NORM
    b = _upload(wl, wts, wl.N, wl.layers, rope_pos=pos)
    for r in recs:
        keys = r["l1"] if selection == "l1rel" else oracle.velocity_keys(r["v_hat"])
        n, refreshed = S.iteration(b, wl.T, r["i"], sig, sizes, margin=margin, selection=sel)
        assert (n, refreshed) == (r["idx"].size, r["refreshed"])
        np.testing.assert_array_equal(b.idx[:n].cpu().numpy(), r["idx"])
        if refreshed:  # the ranking decisions are far from ties for this seed
            assert oracle.boundary_gaps(keys, sizes).min() > TOL["f32"]
        np.testing.assert_array_equal(b.budget.cpu().numpy(), r["budget"])
        assert rel_inf(host(b.v_fresh[:n]), r["v_fresh"]) <= TOL["f32"], r["i"]
        assert rel_inf(host(b.v_hat), r["v_hat"]) <= TOL["f32"], r["i"]
        assert rel_inf(host(b.x), r["x"]) <= TOL["f32"], r["i"]
        assert rel_inf(host(b.h[:n]), r["hidden"][-1]) <= TOL["f32"], r["i"]
        for (k, v), (kr, vr) in zip(b.caches, r["caches"]):
            assert rel_inf(host(k), kr) <= TOL["f32"], r["i"]
            assert rel_inf(host(v), vr) <= TOL["f32"], r["i"]


def _state_for(wl, seed, N, L):
    st = synth.draw_stack_state(wl, seed, n_tokens=N, layers=L)
    st["budget"] = synth.assign_budgets(st["v_hat"], wl.groups)
    return st


@pytest.mark.parametrize("name,rope", [("small_stack_bf16", False), ("small_block_bf16", False),
                                       ("small_block_bf16", True)])
@pytest.mark.parametrize("iteration", [1, 2, 0])  # 25% active, 50% active, all active + refresh
def test_small_bf16_stack_iteration(iteration, name, rope):
    wl = synth.WORKLOADS[name]
    N, L = wl.N, wl.layers
    wts = synth.draw_stack(wl, seed=31)
    st = _state_for(wl, 32, N, L)
    sizes = synth.group_sizes(N, wl.groups)
    sig = synth.linear_sigmas(wl.T)
    state = {"x": st["x"].astype(np.float64), "v_hat": st["v_hat"].astype(np.float64),
             "budget": st["budget"],
             "caches": [(k.astype(np.float64), v.astype(np.float64)) for k, v in st["caches"]]}
    pos = np.random.default_rng(10).permutation(N).astype(np.int32) if rope else None
    r = oracle.stack_iteration(state, wts, iteration, wl.T, sig, wl.heads, wl.dh, "bf16", sizes,
                               rope={"grid": wl.grid, "pos": pos} if rope else None)
    b = _upload(wl, wts, N, L, st, rope_pos=pos)
    caches_before = [(host_bits(k), host_bits(v)) for k, v in b.caches]
    n, refreshed = S.iteration(b, wl.T, iteration, sig, sizes)
    assert (n, refreshed) == (r["idx"].size, r["refreshed"])
    np.testing.assert_array_equal(b.idx[:n].cpu().numpy(), r["idx"])
    skipped = np.setdiff1d(np.arange(N), r["idx"])
    assert rel_inf(host(b.v_fresh[:n]), r["v_fresh"]) <= TOL["bf16"]
    assert rel_inf(host(b.h[:n]), r["hidden"][-1]) <= TOL["bf16"]
    # the Euler update moves x by v_hat * dsig: compare the update itself
    dx = host(b.x) - st["x"].astype(np.float64)
    assert rel_inf(dx, r["x"] - st["x"]) <= TOL["bf16"]
    np.testing.assert_array_equal(host_bits(b.v_hat)[skipped], host_bits(to_dev(st["v_hat"], "f32"))[skipped])
    for (k, v), (kr, vr), (k0, v0) in zip(b.caches, r["caches"], caches_before):
        assert rel_inf(host(k), kr) <= TOL["bf16"]
        assert rel_inf(host(v), vr) <= TOL["bf16"]
        np.testing.assert_array_equal(host_bits(k)[skipped], k0[skipped])  # untouched rows
        np.testing.assert_array_equal(host_bits(v)[skipped], v0[skipped])
    got = b.budget.cpu().numpy()
    if refreshed:
        # group sizes are exact; a token may only change group across a
        # boundary it is within the velocity tolerance of
        assert [int(np.sum(got == s)) for s, _ in sizes] == [c for _, c in sizes]
        keys = oracle.velocity_keys(r["v_hat"])
        ks = np.sort(keys)
        edges = np.cumsum([c for _, c in sizes])[:-1]
        bkeys = ks[edges]
        for t in np.flatnonzero(got != r["budget"]):
            assert np.min(np.abs(keys[t] - bkeys) / bkeys) < 4 * TOL["bf16"]
        assert np.mean(got != r["budget"]) < 0.02
    else:
        np.testing.assert_array_equal(got, st["budget"])


def test_wan13b_stack_iterations():
    """Two iterations of the 30-layer Wan-1.3B-shaped stack at full size: the
    all-active first iteration (which fills every cache and refreshes the
    groups) and the 25%-active second one."""
    wl = synth.WORKLOADS["wan1.3b_stack"]
    N, L, C, d = wl.N, wl.layers, wl.euler_channels, wl.d
    wts = synth.draw_stack(wl, seed=0)
    sizes = synth.group_sizes(N, wl.groups)
    sig = synth.linear_sigmas(wl.T)
    b = _upload(wl, wts, N, L)

    n, refreshed = S.iteration(b, wl.T, 0, sig, sizes)
    assert (n, refreshed) == (N, True)
    np.testing.assert_array_equal(b.idx.cpu().numpy(), np.arange(N))
    v0 = b.v_hat.cpu().numpy()
    assert np.all(np.isfinite(v0))
    # refreshed budgets are exactly the ranking of the velocity cache
    budget1 = b.budget.cpu().numpy()
    np.testing.assert_array_equal(budget1, oracle.assign_groups(v0, sizes))
    # Euler from x0 with the fresh velocities: one fp32 rounding of x + v dsig
    dsig = oracle.euler_delta(sig[0], sig[1])
    want = oracle.round_f32(wts["x0"].astype(np.float64) + v0.astype(np.float64) * dsig)
    x1 = b.x.cpu().numpy()
    assert np.max(np.abs(x1 - want) / np.maximum(np.abs(want), 1e-30)) <= 2.0 ** -23
    # sampled layer-0 cache rows against the oracle
    rng = np.random.default_rng(5)
    rows = np.sort(rng.choice(N, 256, replace=False))
    h0 = oracle.rms_normalize(oracle.linear(oracle.gather_latent(wts["x0"], rows, "bf16"), wts["w_embed"], "bf16"))
    k0 = oracle.linear(h0, wts["layers"][0]["wk"], "bf16")
    v0c = oracle.linear(h0, wts["layers"][0]["wv"], "bf16")
    assert rel_inf(host(b.caches[0][0][rows]), k0) <= TOL["bf16"]
    assert rel_inf(host(b.caches[0][1][rows]), v0c) <= TOL["bf16"]

    caches_before = [(k.clone(), v.clone()) for k, v in b.caches]
    vhat_before = b.v_hat.clone()
    n, refreshed = S.iteration(b, wl.T, 1, sig, sizes)
    idx = oracle.active_set(budget1, wl.T, 1)
    assert (n, refreshed) == (idx.size, False) and n == sizes[-1][1]
    np.testing.assert_array_equal(b.idx[:n].cpu().numpy(), idx)
    skipped = torch.from_numpy(np.setdiff1d(np.arange(N), idx)).to(DEV)
    act = torch.from_numpy(idx).to(DEV)
    for (k, v), (k0_, v0_) in zip(b.caches, caches_before):
        assert torch.equal(k[skipped], k0_[skipped]) and torch.equal(v[skipped], v0_[skipped])
        assert not torch.equal(k[act], k0_[act])
    assert torch.equal(b.v_hat[skipped], vhat_before[skipped])
    assert torch.equal(b.v_hat[act], b.v_fresh[:n])
    assert torch.isfinite(b.v_fresh[:n]).all()
    np.testing.assert_array_equal(b.budget.cpu().numpy(), budget1)


def test_wan13b_full_blocks_iterations():
    """Two full blocks (self-attention, cross-attention to a 512-row context,
    FFN 8960) at the Wan-1.3B shape, all-active then 25%-active: skipped rows
    of both layers' caches untouched, sampled layer-0 cache rows against the
    oracle, fresh velocities finite, budgets from the velocity ranking."""
    wl = synth.WORKLOADS["wan1.3b_blocks"]
    N, L = wl.N, 2
    wts = synth.draw_stack(wl, seed=1, layers=L)
    sizes = synth.group_sizes(N, wl.groups)
    sig = synth.linear_sigmas(wl.T)
    b = _upload(wl, wts, N, L)
    n, refreshed = S.iteration(b, wl.T, 0, sig, sizes)
    assert (n, refreshed) == (N, True)
    v0 = b.v_hat.cpu().numpy()
    assert np.all(np.isfinite(v0))
    budget1 = b.budget.cpu().numpy()
    np.testing.assert_array_equal(budget1, oracle.assign_groups(v0, sizes))
    rows = np.sort(np.random.default_rng(6).choice(N, 128, replace=False))
    h0 = oracle.rms_normalize(oracle.linear(oracle.gather_latent(wts["x0"], rows, "bf16"), wts["w_embed"], "bf16"))
    assert rel_inf(host(b.caches[0][0][rows]), oracle.linear(h0, wts["layers"][0]["wk"], "bf16")) <= TOL["bf16"]
    assert rel_inf(host(b.caches[0][1][rows]), oracle.linear(h0, wts["layers"][0]["wv"], "bf16")) <= TOL["bf16"]
    before = [(k.clone(), v.clone()) for k, v in b.caches]
    n, refreshed = S.iteration(b, wl.T, 1, sig, sizes)
    idx = oracle.active_set(budget1, wl.T, 1)
    assert (n, refreshed) == (idx.size, False)
    np.testing.assert_array_equal(b.idx[:n].cpu().numpy(), idx)
    skipped = torch.from_numpy(np.setdiff1d(np.arange(N), idx)).to(DEV)
    for (k, v), (k0, v0_) in zip(b.caches, before):
        assert torch.equal(k[skipped], k0[skipped]) and torch.equal(v[skipped], v0_[skipped])
    assert torch.isfinite(b.v_fresh[:n]).all()


# ---------------------------------------------------------------------------
# Token reordering and the prefix-only cache (Section 2.5)
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("N,bad", [(1000, False), (75600, False), (37, False), (5000, True)])
def test_reorder_plan(N, bad):
    rng = np.random.default_rng(N)
    b = rng.choice(np.array([40, 20, 10, 5]), size=N).astype(np.int32)
    if bad:
        b[77] = 3
    perm = torch.full((N,), -1, dtype=torch.int32, device=DEV)
    n_lead = torch.zeros(1, dtype=torch.int32, device=DEV)
    if bad:
        with pytest.raises(H.HsaStepError) as e:
            H.hsa_reorder_plan(i32(b), 40, perm, n_lead)
        assert e.value.name == "HSA_STEP_ERR_BUDGET"
        assert sorted(perm.cpu().numpy().tolist()) == list(range(N))  # still a permutation
        return
    lead = H.hsa_reorder_plan(i32(b), 40, perm, n_lead)
    want, want_lead = oracle.reorder_plan(b, 40)
    assert lead == want_lead
    np.testing.assert_array_equal(perm.cpu().numpy(), want)


@pytest.mark.parametrize("shape,dtype", [((1000, 64), torch.float32), ((777, 3), torch.float32),
                                          ((500,), torch.int32), ((300, 5), torch.bfloat16),
                                          ((32760, 1536), torch.bfloat16)])
def test_permute_rows(shape, dtype):
    n = shape[0]
    src = torch.randn(*shape, device=DEV).to(dtype) if dtype != torch.int32 else \
        torch.randint(-99, 99, shape, dtype=torch.int32, device=DEV)
    perm_np = np.random.default_rng(n).permutation(n).astype(np.int32)
    perm = i32(perm_np)
    dst = torch.empty_like(src)
    H.hsa_permute_rows(src, perm, dst)
    assert torch.equal(dst, src[torch.from_numpy(perm_np).long().to(DEV)])
    back = torch.empty_like(src)
    H.hsa_permute_rows(dst, perm, back, inverse=True)
    assert torch.equal(back, src)


def test_tiny_prefix_cache_trajectory():
    """Reordered tokens with the prefix-only cache and RoPE by original grid
    positions: the GPU trajectory matches the oracle's reordered trajectory,
    and the restored latent matches the oracle's unreordered one."""
    wl = synth.WORKLOADS["tiny_block_f32"]
    wts = synth.draw_stack(wl, seed=61)
    budget = synth.assign_budgets(np.zeros((wl.N, 1), np.float32), wl.groups, "first_frame",
                                  frame_tokens=wl.grid[1] * wl.grid[2], seed=62)
    sig = synth.linear_sigmas(wl.T)
    perm_o, n_lead = oracle.reorder_plan(budget, wl.T)
    n_cached = S.prefix_rows(n_lead, wl.N)
    st1 = oracle.initial_state(wts["x0"][perm_o], wl.layers, wl.d, wl.T)
    st1["budget"] = budget[perm_o]
    recs = oracle.stack_trajectory(None, wts, wl.T, sig, wl.heads, wl.dh, "f32", state=st1,
                                   rope={"grid": wl.grid, "pos": perm_o})
    b = S.StackBuffers.allocate(wl.N, wl.euler_channels, wl.layers, wl.heads, wl.dh, torch.float32,
                                ffn=wl.ffn, ctx=wl.ctx, n_cached=n_cached)
    src = _upload(wl, wts, wl.N, wl.layers)  # weights and context, full-cache layout
    for name in ("w_embed", "w_head"):
        getattr(b, name).copy_(getattr(src, name))
    for dst, s_ in zip(b.layers + b.cross + b.ffn, src.layers + src.cross + src.ffn):
        for a, c in zip(dst, s_):
            a.copy_(c)
    b.x.copy_(to_dev(wts["x0"], "f32"))
    b.v_hat.zero_()
    b.budget.copy_(i32(budget))
    b.enable_rope(wl.grid)
    perm = S.reorder(b, wl.T)
    np.testing.assert_array_equal(perm.cpu().numpy(), perm_o)
    for r in recs:
        n, _ = S.iteration(b, wl.T, r["i"], sig)
        assert n == r["idx"].size
        np.testing.assert_array_equal(b.idx[:n].cpu().numpy(), r["idx"])
        assert rel_inf(host(b.x), r["x"]) <= TOL["f32"], r["i"]
        for (k, v), (kr, vr) in zip(b.caches, r["caches"]):
            assert rel_inf(host(k[:n_cached]), kr[:n_cached]) <= TOL["f32"], r["i"]
            assert rel_inf(host(v[:n_cached]), vr[:n_cached]) <= TOL["f32"], r["i"]
    st0 = oracle.initial_state(wts["x0"], wl.layers, wl.d, wl.T)
    st0["budget"] = budget
    base = oracle.stack_trajectory(None, wts, wl.T, sig, wl.heads, wl.dh, "f32", state=st0,
                                   rope={"grid": wl.grid, "pos": None})
    assert rel_inf(host(S.restore_order(b, perm)), base[-1]["x"]) <= TOL["f32"]


@pytest.mark.parametrize("kv_parts,extra", [(None, 0), ("4", 0), (None, 64), ("4", 64)])
def test_prefix_cache_equals_full_cache_bitwise(kv_parts, extra, monkeypatch):
    """At the Wan-1.3B shape (3 layers, RoPE, HSA-75A groups with a 25%
    baseline group reordered to the end) the prefix-only cache changes only
    where the baseline rows' keys live: latents, velocities and the cached
    prefix rows are bit-identical to the full-cache run. The 25%-active
    iteration splits its attention keys (2 parts by the launcher's choice,
    or 4 forced), so parts that span the cache prefix and the fresh tail
    are covered too. The smallest prefix is 24576 rows, a whole number of
    96-row key tiles; with 64 more cached rows (baseline tokens kept in the
    prefix) one key tile spans the prefix and the fresh tail."""
    if kv_parts:
        monkeypatch.setenv("HSA_ATTN_KV_PARTS", kv_parts)
    wl = synth.WORKLOADS["wan1.3b_stack"]
    N, L = wl.N, 3
    wts = synth.draw_stack(wl, seed=7, layers=L)
    groups = synth.PRESETS["HSA-75A"]["groups"]
    budget = synth.random_budgets(N, groups, seed=8)
    sig = synth.linear_sigmas(wl.T)
    runs = []
    for n_cached in (None, S.prefix_rows(int(np.sum(budget < wl.T)), N) + extra):
        b = S.StackBuffers.allocate(N, wl.euler_channels, L, wl.heads, wl.dh, torch.bfloat16, n_cached=n_cached)
        src = _upload(wl, wts, N, L) if not runs else runs[0][0]
        if runs:
            for name in ("w_embed", "w_head"):
                getattr(b, name).copy_(getattr(src, name))
            for dst, s_ in zip(b.layers, src.layers):
                for a, c in zip(dst, s_):
                    a.copy_(c)
        else:
            b = src
        b.x.copy_(to_dev(wts["x0"], "f32"))
        b.v_hat.zero_()
        b.budget.copy_(i32(budget))
        b.pos = None
        b.enable_rope(wl.grid)
        S.reorder(b, wl.T)
        for i in range(3):  # 100%, then the 40+20 groups, then 40 only
            S.iteration(b, wl.T, i, sig)
        runs.append((b, n_cached))
    (full, _), (pre, n_cached) = runs
    assert torch.equal(full.x, pre.x) and torch.equal(full.v_hat, pre.v_hat)
    for (k0, v0), (k1, v1) in zip(full.caches, pre.caches):
        assert torch.equal(k0[:n_cached], k1) and torch.equal(v0[:n_cached], v1)
    assert torch.equal(full.caches[-1][0][n_cached:], pre.k_tail)  # the last layer's fresh baseline keys


def test_refused_refresh_leaves_state_unchanged():
    # a refresh iteration (every group's schedule fires, i = 4 for T = 8 and budgets {8, 4, 2}) where
    # the budgets in force leave a token inactive is refused before anything changes the caller's state
    wl = synth.WORKLOADS["tiny_stack_f32"]
    N, L = wl.N, wl.layers
    wts = synth.draw_stack(wl, seed=5)
    st = _state_for(wl, 6, N, L)
    st["budget"] = np.full(N, 4, np.int32)  # active at even iterations
    st["budget"][17] = 1                    # active at i = 0 only
    b = _upload(wl, wts, N, L, state=st)
    sizes = synth.group_sizes(N, wl.groups)
    sig = synth.linear_sigmas(wl.T)
    before = [t.clone() for t in (b.x, b.v_hat, b.budget)] + [t.clone() for kv in b.caches for t in kv]
    with pytest.raises(H.HsaStepError) as e:
        S.iteration(b, wl.T, 4, sig, sizes)
    assert e.value.name == "HSA_STEP_ERR_BUDGET"
    torch.cuda.synchronize()
    after = [b.x, b.v_hat, b.budget] + [t for kv in b.caches for t in kv]
    for x0, x1 in zip(before, after):
        assert torch.equal(x0, x1)
    # the same state at a non-refresh iteration runs
    n, refreshed = S.iteration(b, wl.T, 2, sig, sizes)
    assert n == N - 1 and not refreshed
