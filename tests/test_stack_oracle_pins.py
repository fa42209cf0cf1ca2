"""Pins of the multi-layer sampling-loop oracle.

Each test checks oracle/stack_oracle.py against something other than itself:
torch's linear map and scaled-dot-product attention (an independent
implementation of one stack iteration), numpy's L2 norm for the velocity
ranking, exact integer arithmetic and brute force for the group assignment,
closed forms of the linear model that remains when attention contributes
nothing, and invariants the paper states (skipped cache rows untouched,
telescoping of the cached Euler step).
"""

import math

import numpy as np
import pytest
import torch
import torch.nn.functional as F

import oracle
import synth


# ---------------------------------------------------------------------------
# Compact linear maps
# ---------------------------------------------------------------------------


def test_linear_matches_torch_linear_with_residual():
    rng = np.random.default_rng(3)
    a = rng.standard_normal((37, 48)).astype(np.float32)
    w = rng.standard_normal((21, 48)).astype(np.float32)
    r = rng.standard_normal((37, 21)).astype(np.float32)
    t = F.linear(torch.from_numpy(a).double(), torch.from_numpy(w).double()) + torch.from_numpy(r).double()
    np.testing.assert_allclose(oracle.linear(a, w, "f32", residual=r), t.float().double().numpy(),
                               rtol=2e-7, atol=0)
    tb = F.linear(torch.from_numpy(a).double(), torch.from_numpy(w).double())
    np.testing.assert_array_equal(oracle.linear(a, w, "bf16"), oracle.round_bf16(tb.numpy()))


def test_linear_rounds_once():
    # exact value 1 + 2^-8 + 2^-40: nearest bf16 is 1 + 2^-7; going through
    # fp32 first would land on the tie 1 + 2^-8 and then on 1.0
    a = np.array([[1.0, 2.0 ** -8, 2.0 ** -40]])
    w = np.ones((1, 3))
    assert oracle.linear(a, w, "bf16")[0, 0] == 1 + 2.0 ** -7
    # the residual is part of the one rounding as well
    assert oracle.linear(a[:, :2], w[:, :2], "bf16", residual=np.array([[2.0 ** -40]]))[0, 0] == 1 + 2.0 ** -7


def test_gather_latent_rounds_selected_rows():
    x = np.array([[1.0, 1 + 2.0 ** -8], [3.0, 1 + 3 * 2.0 ** -8], [5.0, 7.0]], np.float32)
    got = oracle.gather_latent(x, [2, 1], "bf16")
    ref = torch.from_numpy(x[[2, 1]]).to(torch.bfloat16).double().numpy()
    np.testing.assert_array_equal(got, ref)


# ---------------------------------------------------------------------------
# Group refresh
# ---------------------------------------------------------------------------


def test_velocity_ranking_is_l2_norm_ranking():
    rng = np.random.default_rng(5)
    v = rng.standard_normal((3000, 64)).astype(np.float32)
    keys = oracle.velocity_keys(v)
    norms = np.linalg.norm(v.astype(np.float64), axis=1)
    s = np.sort(norms)
    assert np.min(np.diff(s) / s[1:]) > 1e-12  # no near ties: the rankings must agree
    ref_rank = np.empty(v.shape[0], np.int64)
    ref_rank[np.argsort(norms, kind="stable")] = np.arange(v.shape[0])
    np.testing.assert_array_equal(oracle.token_ranks(keys), ref_rank)
    # each key is within a few ulp of the correctly rounded sum of squares
    exact = np.array([math.fsum(float(c) ** 2 for c in row) for row in v.astype(np.float64)])
    np.testing.assert_allclose(keys, exact, rtol=64 * 2.0 ** -53, atol=0)


def test_assign_groups_brute_force_with_ties():
    rng = np.random.default_rng(7)
    v = rng.integers(-3, 4, size=(23, 5)).astype(np.float32)
    v[4] = v[9] = v[17]  # equal norms in three tokens
    v[11] = 0.0
    v[20] = -v[2]
    sizes = ((2, 6), (5, 7), (10, 10))
    got = oracle.assign_groups(v, sizes)
    # integer components: the squared norms are exact small integers
    sq = [int(sum(int(c) ** 2 for c in row)) for row in v]
    want = []
    for n in range(len(sq)):
        rank = sum(1 for m in range(len(sq)) if sq[m] < sq[n] or (sq[m] == sq[n] and m < n))
        want.append(2 if rank < 6 else (5 if rank < 13 else 10))
    np.testing.assert_array_equal(got, want)
    assert [int(np.sum(got == s)) for s, _ in sizes] == [6, 7, 10]


def test_assign_groups_equivariant_and_monotone():
    rng = np.random.default_rng(8)
    v = rng.standard_normal((500, 16)).astype(np.float32)
    sizes = synth.group_sizes(500, ((40, 0.25), (20, 0.25), (10, 0.25), (5, 0.25)))
    b = oracle.assign_groups(v, sizes)
    perm = rng.permutation(500)
    np.testing.assert_array_equal(oracle.assign_groups(v[perm], sizes), b[perm])
    norms = np.linalg.norm(v.astype(np.float64), axis=1)
    order = np.argsort(norms)
    assert np.all(np.diff(b[order]) >= 0)  # larger velocity norm, never a smaller budget


def test_group_sizes_follow_fraction_rule():
    assert synth.group_sizes(1024, ((8, 1 / 3), (4, 1 / 3), (2, 1 / 3))) == ((2, 341), (4, 341), (8, 342))
    assert synth.group_sizes(32760, ((40, .25), (20, .25), (10, .25), (5, .25))) == (
        (5, 8190), (10, 8190), (20, 8190), (40, 8190))
    with pytest.raises(ValueError):
        oracle.check_group_sizes(((4, 3), (2, 3)), 6)
    with pytest.raises(ValueError):
        oracle.check_group_sizes(((2, 3), (4, 2)), 6)
    with pytest.raises(ValueError):
        oracle.check_group_sizes(((3, 3), (8, 3)), 6, T=8)


@pytest.mark.parametrize("T,budgets", [(40, (40, 20, 10, 5)), (40, (40, 20, 8)), (8, (8, 4, 2)),
                                       (12, (12, 4, 3)), (40, (20, 5))])
def test_refresh_period_is_where_every_group_fires(T, budgets):
    b = np.array(budgets)
    full = [i for i in range(T) if oracle.active_set(b, T, i).size == b.size]
    P = oracle.refresh_period(T, budgets)
    assert full == list(range(0, T, P))


# ---------------------------------------------------------------------------
# One stack iteration against an independent torch implementation
# ---------------------------------------------------------------------------


def _torch_iteration(x, v_hat, caches, wts, idx, heads, dh, dsig, dtype="f32", rotate=None):
    """Stack iteration written with torch's float64 linear, RMS norm and
    scaled-dot-product attention; each stored value is rounded to the model
    dtype (bf16 rounding by the separately pinned round_bf16), the velocity
    and the latent to fp32."""
    f32 = lambda t: t.float().double()  # noqa: E731
    D = lambda a: torch.from_numpy(np.asarray(a, np.float64))  # noqa: E731
    rnd = f32 if dtype == "f32" else (lambda t: D(oracle.round_bf16(t.numpy())))  # noqa: E731
    ti = torch.from_numpy(np.asarray(idx, np.int64))
    norm = lambda t: F.rms_norm(t, (t.shape[1],), eps=1e-6)  # noqa: E731
    h = rnd(F.linear(rnd(D(x)[ti]), D(wts["w_embed"])))
    new_caches = []
    for lw, (kc, vc) in zip(wts["layers"], caches):
        hn = norm(h)
        rot = rotate or (lambda t: t)
        q = rnd(rot(F.linear(hn, D(lw["wq"]))))
        K, V = D(kc).clone(), D(vc).clone()
        K[ti] = rnd(rot(F.linear(hn, D(lw["wk"]))))
        V[ti] = rnd(F.linear(hn, D(lw["wv"])))
        split = lambda t: t.view(t.shape[0], heads, dh).transpose(0, 1)  # noqa: E731
        o = F.scaled_dot_product_attention(split(q), split(K), split(V))
        o = rnd(o.transpose(0, 1).reshape(q.shape[0], heads * dh))
        h = rnd(F.linear(o, D(lw["wo"])) + h)
        if "wq_c" in lw:
            ctx = D(wts["ctx"])
            kc, vc = rnd(F.linear(ctx, D(lw["wk_c"]))), rnd(F.linear(ctx, D(lw["wv_c"])))
            qc = rnd(F.linear(norm(h), D(lw["wq_c"])))
            oc = F.scaled_dot_product_attention(split(qc), split(kc), split(vc))
            oc = rnd(oc.transpose(0, 1).reshape(qc.shape[0], heads * dh))
            h = rnd(F.linear(oc, D(lw["wo_c"])) + h)
        if "w1" in lw:
            f = rnd(F.gelu(F.linear(norm(h), D(lw["w1"])), approximate="tanh"))
            h = rnd(F.linear(f, D(lw["w2"])) + h)
        new_caches.append((K.numpy(), V.numpy()))
    v = f32(F.linear(norm(h), D(wts["w_head"])))
    vh = D(v_hat).clone()
    vh[ti] = v
    x_new = f32(D(x) + vh * dsig)
    return x_new.numpy(), vh.numpy(), v.numpy(), new_caches


@pytest.mark.parametrize("name", ["tiny_stack_f32", "tiny_block_f32"])
@pytest.mark.parametrize("iteration", [1, 2, 4])  # 33%, 67% and 100% of the tokens active
def test_stack_iteration_matches_torch(iteration, name):
    wl = synth.WORKLOADS[name]
    wts = synth.draw_stack(wl, seed=11)
    st = synth.draw_stack_state(wl, seed=12)
    budget = synth.assign_budgets(st["v_hat"], wl.groups)
    state = {"x": st["x"].astype(np.float64), "v_hat": st["v_hat"].astype(np.float64), "budget": budget,
             "caches": [(k.astype(np.float64), v.astype(np.float64)) for k, v in st["caches"]]}
    sig = synth.linear_sigmas(wl.T)
    r = oracle.stack_iteration(state, wts, iteration, wl.T, sig, wl.heads, wl.dh, "f32")
    idx = oracle.active_set(budget, wl.T, iteration)
    assert (idx.size == wl.N) == (iteration == 4) and idx.size > 0
    dsig = oracle.euler_delta(sig[iteration], sig[iteration + 1])
    x, vh, v, caches = _torch_iteration(st["x"], st["v_hat"], st["caches"], wts, idx, wl.heads, wl.dh, dsig)
    tol = dict(rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(r["v_fresh"], v, **tol)
    np.testing.assert_allclose(r["v_hat"], vh, **tol)
    np.testing.assert_allclose(r["x"], x, **tol)
    for (k, vv), (kt, vt) in zip(r["caches"], caches):
        np.testing.assert_allclose(k, kt, **tol)
        np.testing.assert_allclose(vv, vt, **tol)


@pytest.mark.parametrize("name", ["small_stack_bf16", "small_block_bf16"])
@pytest.mark.parametrize("iteration", [1, 2])
def test_bf16_stack_iteration_matches_torch(iteration, name):
    """Same check with bf16 storage: the two sides round at the same points,
    so all but a few values (where float64 summation order decides a bf16
    rounding) agree to float64 precision."""
    wl = synth.WORKLOADS[name]
    wts = synth.draw_stack(wl, seed=21, n_tokens=384, layers=2)
    st = synth.draw_stack_state(wl, seed=22, n_tokens=384, layers=2)
    budget = synth.assign_budgets(st["v_hat"], wl.groups)
    state = {"x": st["x"].astype(np.float64), "v_hat": st["v_hat"].astype(np.float64), "budget": budget,
             "caches": [(k.astype(np.float64), v.astype(np.float64)) for k, v in st["caches"]]}
    sig = synth.linear_sigmas(wl.T)
    r = oracle.stack_iteration(state, wts, iteration, wl.T, sig, wl.heads, wl.dh, "bf16")
    idx = oracle.active_set(budget, wl.T, iteration)
    dsig = oracle.euler_delta(sig[iteration], sig[iteration + 1])
    x, vh, v, caches = _torch_iteration(st["x"], st["v_hat"], st["caches"], wts, idx, wl.heads, wl.dh, dsig,
                                        "bf16")
    pairs = [(r["v_fresh"], v), (r["x"], x)] + [(a, b) for ra, rb in zip(r["caches"], caches)
                                                 for a, b in zip(ra, rb)]
    for a, b in pairs:
        scale = np.abs(b).max()
        assert np.abs(a - b).max() <= 2e-2 * scale
        assert np.mean(np.abs(a - b) > 1e-9 * scale) < 0.01


# ---------------------------------------------------------------------------
# Trajectory invariants
# ---------------------------------------------------------------------------


@pytest.fixture(scope="module")
def tiny_traj():
    wl = synth.WORKLOADS["tiny_stack_f32"]
    wts = synth.draw_stack(wl, seed=0)
    sizes = synth.group_sizes(wl.N, wl.groups)
    recs = oracle.stack_trajectory(wts["x0"], wts, wl.T, synth.linear_sigmas(wl.T), wl.heads, wl.dh,
                                   "f32", group_sizes=sizes)
    return wl, wts, sizes, recs


def test_stack_trajectory_schedule_and_refresh(tiny_traj):
    wl, _, sizes, recs = tiny_traj
    P = oracle.refresh_period(wl.T, [s for s, _ in sizes])
    budget = np.full(wl.N, wl.T)
    for r in recs:
        np.testing.assert_array_equal(r["idx"], oracle.active_set(budget, wl.T, r["i"]))
        assert r["refreshed"] == (r["i"] % P == 0)
        if r["refreshed"]:
            assert r["idx"].size == wl.N
            b = r["budget"]
            assert [int(np.sum(b == s)) for s, _ in sizes] == [n for _, n in sizes]
            norms = np.linalg.norm(r["v_hat"], axis=1)
            assert np.all(np.diff(b[np.argsort(norms)]) >= 0)
            assert oracle.boundary_gaps(oracle.velocity_keys(r["v_hat"]), sizes).min() > 1e-6
        budget = r["budget"]


def test_stack_trajectory_skipped_rows_untouched(tiny_traj):
    _, _, _, recs = tiny_traj
    for prev, r in zip(recs, recs[1:]):
        skipped = np.setdiff1d(np.arange(prev["x"].shape[0]), r["idx"])
        assert skipped.size > 0 or r["idx"].size == prev["x"].shape[0]
        for (k0, v0), (k1, v1) in zip(prev["caches"], r["caches"]):
            np.testing.assert_array_equal(k1[skipped], k0[skipped])
            np.testing.assert_array_equal(v1[skipped], v0[skipped])
        np.testing.assert_array_equal(r["v_hat"][skipped], prev["v_hat"][skipped])


def test_stack_trajectory_telescopes(tiny_traj):
    """Between two consecutive active iterations i < j of a token its velocity
    is held, so x_j - x_i = v_hat_i (sigma_j - sigma_i) up to fp32 rounding of
    the j - i cached steps (Section 2.4)."""
    wl, wts, _, recs = tiny_traj
    sig = synth.linear_sigmas(wl.T).astype(np.float64)
    xs = [r["x"] for r in recs]  # state after iteration i = x at sigma_{i+1}
    act = np.zeros((len(recs), wl.N), bool)
    for r in recs:
        act[r["i"], r["idx"]] = True
    for n in range(wl.N):
        its = list(np.flatnonzero(act[:, n])) + [len(recs)]
        for i, j in zip(its, its[1:]):
            x_i = recs[i - 1]["x"][n] if i > 0 else wts["x0"][n].astype(np.float64)
            pred = x_i + recs[i]["v_hat"][n] * (sig[j] - sig[i])
            np.testing.assert_allclose(xs[j - 1][n], pred, rtol=0, atol=(j - i) * 4e-7 * (1 + np.abs(pred)).max())


def test_stack_trajectory_permutation_equivariant(tiny_traj):
    wl, wts, sizes, recs = tiny_traj
    perm = np.random.default_rng(2).permutation(wl.N)
    wp = dict(wts)
    wp["x0"] = wts["x0"][perm]
    rp = oracle.stack_trajectory(wp["x0"], wp, wl.T, synth.linear_sigmas(wl.T), wl.heads, wl.dh, "f32",
                                 group_sizes=sizes)
    for a, b in zip(recs, rp):  # token n of the permuted run is token perm[n]
        np.testing.assert_array_equal(np.sort(perm[b["idx"]]), a["idx"])
        np.testing.assert_array_equal(b["budget"], a["budget"][perm])
        np.testing.assert_allclose(b["x"], a["x"][perm], rtol=1e-5, atol=1e-6)


def _zero_attention_weights(wts):
    w = dict(wts)
    w["layers"] = [dict(lw, wo=np.zeros_like(lw["wo"])) for lw in wts["layers"]]
    return w


def _token_velocity(wts):
    """With W_o = 0 every layer leaves the residual stream unchanged and the
    tokens decouple: each token's velocity is f(x) = rms(x W_embed^T) W_head^T
    (fp32 rounding of the stored values), written here with torch."""
    We = torch.from_numpy(wts["w_embed"].astype(np.float64))
    Wh = torch.from_numpy(wts["w_head"].astype(np.float64))

    def f(x):
        h = F.linear(torch.from_numpy(np.asarray(x, np.float64)), We).float().double()
        return F.linear(F.rms_norm(h, (h.shape[1],), eps=1e-6), Wh).float().double().numpy()
    return f


def test_dense_loop_zero_attention_is_per_token_euler():
    """With W_o = 0 the dense loop (every budget T) is Eq. 2 applied to each
    token on its own: x_{i+1} = x_i + f(x_i) (sigma_{i+1} - sigma_i)."""
    wl = synth.WORKLOADS["tiny_stack_f32"]
    wts = _zero_attention_weights(synth.draw_stack(wl, seed=4))
    sig = synth.linear_sigmas(wl.T)
    recs = oracle.stack_trajectory(wts["x0"], wts, wl.T, sig, wl.heads, wl.dh, "f32")
    assert all(r["idx"].size == wl.N for r in recs)
    f = _token_velocity(wts)
    x = wts["x0"].astype(np.float64)
    for i in range(wl.T):
        x = (x + f(x) * (float(sig[i + 1]) - float(sig[i]))).astype(np.float32).astype(np.float64)
        np.testing.assert_allclose(recs[i]["x"], x, rtol=0, atol=1e-5 * np.abs(x).max())


def test_hsa_loop_zero_attention_telescopes_per_token():
    """Same decoupled model under the HSA schedule with group refresh: a token
    with budget s advances over each of its periods p = T/s by the telescoped
    step x <- x + f(x) (sigma_{i+p} - sigma_i) (Section 2.4), and at the
    refresh iterations the budgets follow the velocity-norm ranking of f(x)."""
    wl = synth.WORKLOADS["tiny_stack_f32"]
    wts = _zero_attention_weights(synth.draw_stack(wl, seed=6))
    sig = synth.linear_sigmas(wl.T).astype(np.float64)
    sizes = synth.group_sizes(wl.N, wl.groups)
    recs = oracle.stack_trajectory(wts["x0"], wts, wl.T, synth.linear_sigmas(wl.T), wl.heads, wl.dh, "f32",
                                   group_sizes=sizes)
    f = _token_velocity(wts)
    P = oracle.refresh_period(wl.T, [s for s, _ in sizes])
    x = wts["x0"].astype(np.float64)
    for i0 in range(0, wl.T, P):
        v = f(x)  # every token is active at i0
        norms = np.linalg.norm(v, axis=1)
        s_sorted = np.sort(norms)
        budget = np.empty(wl.N, np.int64)
        order = np.argsort(norms, kind="stable")
        start = 0
        for s, n in sizes:
            budget[order[start:start + n]] = s
            if 0 < start + n < wl.N:
                assert (s_sorted[start + n] - s_sorted[start + n - 1]) / s_sorted[start + n] > 1e-5
            start += n
        np.testing.assert_array_equal(recs[i0]["budget"], budget)
        for n in range(wl.N):
            p = wl.T // budget[n]
            for i in range(i0, i0 + P, p):
                vn = v[n] if i == i0 else f(x[n:n + 1])[0]
                x[n] = x[n] + vn * (sig[i + p] - sig[i])
        np.testing.assert_allclose(recs[i0 + P - 1]["x"], x, rtol=0, atol=2e-5 * np.abs(x).max())


def test_gelu_tanh_matches_torch():
    x = np.linspace(-12, 12, 20001)
    t = F.gelu(torch.from_numpy(x), approximate="tanh").numpy()
    np.testing.assert_allclose(oracle.gelu_tanh(x), t, rtol=1e-14, atol=1e-15)


def test_rms_normalize_matches_torch():
    rng = np.random.default_rng(9)
    h = rng.standard_normal((50, 96)) * rng.uniform(0.01, 100, size=(50, 1))
    t = F.rms_norm(torch.from_numpy(h), (96,), eps=1e-6).numpy()
    np.testing.assert_allclose(oracle.rms_normalize(h), t, rtol=1e-13, atol=0)
    np.testing.assert_allclose(np.mean(oracle.rms_normalize(h) ** 2, axis=1), 1.0, rtol=1e-4)


# ---------------------------------------------------------------------------
# Strategy D: L1 relative change of the velocity (Appendix B, Eq. 7)
# ---------------------------------------------------------------------------


def test_l1_rel_exact_on_integers_and_matches_numpy():
    from fractions import Fraction
    rng = np.random.default_rng(12)
    v = rng.integers(-9, 10, size=(40, 7)).astype(np.float32)
    vp = rng.integers(-9, 10, size=(40, 7)).astype(np.float32)
    v[3] = 0.0  # zero velocity: 0/0 or x/0
    got = oracle.l1_rel(v, vp)
    for n in range(40):
        num = sum(abs(int(a) - int(b)) for a, b in zip(v[n], vp[n]))
        den = sum(abs(int(a)) for a in v[n])
        if den == 0:
            assert np.isnan(got[n]) if num == 0 else np.isinf(got[n])
        else:
            assert got[n] == float(Fraction(num, den))  # one correctly rounded division
    a = rng.standard_normal((500, 64)).astype(np.float32)
    b = rng.standard_normal((500, 64)).astype(np.float32)
    ref = np.linalg.norm(a.astype(np.float64) - b, 1, axis=1) / np.linalg.norm(a.astype(np.float64), 1, axis=1)
    np.testing.assert_allclose(oracle.l1_rel(a, b), ref, rtol=1e-14)


@pytest.mark.parametrize("margin", [2, 3])
def test_strategy_d_ranks_mean_l1_rel_of_initial_steps(margin):
    wl = synth.WORKLOADS["tiny_stack_f32"]
    wts = synth.draw_stack(wl, seed=3)
    sizes = synth.group_sizes(wl.N, wl.groups)
    recs = oracle.stack_trajectory(wts["x0"], wts, wl.T, synth.linear_sigmas(wl.T), wl.heads, wl.dh, "f32",
                                   group_sizes=sizes, margin=margin, selection=oracle.SELECT_L1REL)
    vs = [r["v_fresh"] for r in recs[:margin]]
    assert all(r["idx"].size == wl.N for r in recs[:margin])
    mean = np.mean([np.linalg.norm(vs[i] - vs[i - 1], 1, axis=1) / np.linalg.norm(vs[i], 1, axis=1)
                    for i in range(1, margin)], axis=0)
    order = np.argsort(mean, kind="stable")
    want = np.empty(wl.N, np.int32)
    start = 0
    for s, n in sizes:
        want[order[start:start + n]] = s
        start += n
    b = recs[margin - 1]["budget"]
    assert [r["refreshed"] for r in recs] == [i == margin - 1 for i in range(wl.T)]
    np.testing.assert_array_equal(b, want)
    assert oracle.boundary_gaps(recs[margin - 1]["l1"], sizes).min() > 1e-6
    assert np.all(np.diff(b[np.argsort(mean)]) >= 0)  # larger change, never a smaller budget
    for r in recs[margin:]:
        np.testing.assert_array_equal(r["budget"], b)
        np.testing.assert_array_equal(r["idx"], oracle.active_set(b, wl.T, r["i"], margin))


def test_strategy_d_needs_initial_full_steps():
    wl = synth.WORKLOADS["tiny_stack_f32"]
    wts = synth.draw_stack(wl, seed=3)
    sizes = synth.group_sizes(wl.N, wl.groups)
    for margin, period in ((1, 1), (0, 1), (2, 2)):
        with pytest.raises(ValueError):
            oracle.stack_trajectory(wts["x0"], wts, wl.T, synth.linear_sigmas(wl.T), wl.heads, wl.dh, "f32",
                                    group_sizes=sizes, margin=margin, outside_period=period,
                                    selection=oracle.SELECT_L1REL, iterations=1)


# ---------------------------------------------------------------------------
# RoPE subsampling (Section 2.3)
# ---------------------------------------------------------------------------


def test_rope_bands():
    assert oracle.rope_bands(128) == (22, 21, 21)
    assert oracle.rope_bands(64) == (12, 10, 10)
    assert sum(oracle.rope_bands(128)) * 2 == 128


def test_apply_rope_matches_complex_rotation():
    rng = np.random.default_rng(31)
    grid, heads, dh = (5, 6, 7), 3, 64
    pos = rng.integers(0, 5 * 6 * 7, size=50)
    x = rng.standard_normal((50, heads * dh))
    ang = oracle.rope_angles(pos, grid, dh)
    # the angle of pair j of a band: coordinate * theta^(-2j/band_width), from the grid coordinates
    f, y, w = pos // 42, (pos // 7) % 6, pos % 7
    nt, nh, nw = oracle.rope_bands(dh)
    np.testing.assert_allclose(ang[:, 3], f * 10000.0 ** (-6.0 / (2 * nt)), rtol=1e-15)
    np.testing.assert_allclose(ang[:, nt + 2], y * 10000.0 ** (-4.0 / (2 * nh)), rtol=1e-15)
    np.testing.assert_allclose(ang[:, nt + nh + 5], w * 10000.0 ** (-10.0 / (2 * nw)), rtol=1e-15)
    z = torch.view_as_complex(torch.from_numpy(x).reshape(50, heads, dh // 2, 2).contiguous())
    rot = torch.polar(torch.ones_like(torch.from_numpy(ang)), torch.from_numpy(ang))[:, None, :]
    ref = torch.view_as_real(z * rot).reshape(50, heads * dh).numpy()
    np.testing.assert_allclose(oracle.apply_rope(x, ang, heads, dh), ref, rtol=1e-13, atol=1e-14)
    np.testing.assert_array_equal(oracle.apply_rope(x, np.zeros_like(ang), heads, dh), x)  # position 0


def test_rope_scores_depend_on_relative_position():
    """After the rotation the score of a query and a key depends only on their
    offset along each axis: shifting both by the same grid offset leaves it."""
    rng = np.random.default_rng(32)
    grid, dh = (6, 8, 9), 128
    q = rng.standard_normal((1, dh))
    k = rng.standard_normal((1, dh))
    lin = lambda f, y, x: np.array([(f * 8 + y) * 9 + x])  # noqa: E731
    score = lambda pq, pk: float((oracle.apply_rope(q, oracle.rope_angles(pq, grid, dh), 1, dh)  # noqa: E731
                                  @ oracle.apply_rope(k, oracle.rope_angles(pk, grid, dh), 1, dh).T)[0, 0])
    s0 = score(lin(1, 2, 3), lin(0, 5, 1))
    assert score(lin(4, 3, 7), lin(3, 6, 5)) == pytest.approx(s0, rel=1e-12)
    assert score(lin(1, 2, 3), lin(0, 5, 2)) != pytest.approx(s0, rel=1e-6)


@pytest.mark.parametrize("name", ["tiny_stack_f32", "tiny_block_f32"])
def test_rope_iteration_uses_token_positions(name):
    """With RoPE the HSA iteration on a partial active set equals the torch
    reference in which every Q/K row is rotated by its token's grid position
    (the subsampled positional frequencies), not by its place among the
    active rows."""
    wl = synth.WORKLOADS[name]
    wts = synth.draw_stack(wl, seed=41)
    st = synth.draw_stack_state(wl, seed=42)
    budget = synth.assign_budgets(st["v_hat"], wl.groups)
    pos = np.random.default_rng(43).permutation(wl.N)  # tokens in a shuffled sequence order
    rope = {"grid": wl.grid, "pos": pos}
    state = {"x": st["x"].astype(np.float64), "v_hat": st["v_hat"].astype(np.float64), "budget": budget,
             "caches": [(k.astype(np.float64), v.astype(np.float64)) for k, v in st["caches"]]}
    sig = synth.linear_sigmas(wl.T)
    r = oracle.stack_iteration(state, wts, 1, wl.T, sig, wl.heads, wl.dh, "f32", rope=rope)
    idx = oracle.active_set(budget, wl.T, 1)
    ang = torch.from_numpy(oracle.rope_angles(pos[idx], wl.grid, wl.dh))
    rot = lambda t: torch.view_as_real(  # noqa: E731
        torch.view_as_complex(t.reshape(t.shape[0], wl.heads, wl.dh // 2, 2).contiguous())
        * torch.polar(torch.ones_like(ang), ang)[:, None, :]).reshape(t.shape[0], -1)
    x, vh, v, caches = _torch_iteration(st["x"], st["v_hat"], st["caches"], wts, idx, wl.heads, wl.dh,
                                        oracle.euler_delta(sig[1], sig[2]), rotate=rot)
    tol = dict(rtol=1e-5, atol=1e-6)
    np.testing.assert_allclose(r["v_fresh"], v, **tol)
    np.testing.assert_allclose(r["x"], x, **tol)
    for (k, vv), (kt, vt) in zip(r["caches"], caches):
        np.testing.assert_allclose(k, kt, **tol)
        np.testing.assert_allclose(vv, vt, **tol)
    # rotating by the compact row number instead is a different result
    r2 = oracle.stack_iteration(state, wts, 1, wl.T, sig, wl.heads, wl.dh, "f32",
                                rope={"grid": wl.grid, "pos": np.arange(wl.N)})
    assert np.abs(r2["v_fresh"] - r["v_fresh"]).max() > 1e-4


# ---------------------------------------------------------------------------
# Token reordering (Section 2.5)
# ---------------------------------------------------------------------------


def test_reorder_plan_partition():
    b = np.array([40, 10, 40, 5, 20, 40, 10])
    perm, n_cached = oracle.reorder_plan(b, 40)
    np.testing.assert_array_equal(perm, [1, 3, 4, 6, 0, 2, 5])
    assert n_cached == 4
    assert np.all(b[perm[:n_cached]] < 40) and np.all(b[perm[n_cached:]] == 40)
    _, n0 = oracle.reorder_plan(np.array([20, 5, 20]), 40)  # no baseline group: everything is cached
    assert n0 == 3


def test_reordered_trajectory_is_the_permuted_trajectory():
    """Reordering the tokens once before the loop, with their grid positions
    carried along for RoPE, changes nothing but the order: the reordered
    trajectory is the original one permuted, and the baseline tokens are
    active at every iteration."""
    wl = synth.WORKLOADS["tiny_block_f32"]
    wts = synth.draw_stack(wl, seed=51)
    budget = synth.assign_budgets(np.zeros((wl.N, 1), np.float32), wl.groups, "first_frame",
                                  frame_tokens=wl.grid[1] * wl.grid[2], seed=52)
    sig = synth.linear_sigmas(wl.T)
    st0 = oracle.initial_state(wts["x0"], wl.layers, wl.d, wl.T)
    st0["budget"] = budget
    base = oracle.stack_trajectory(None, wts, wl.T, sig, wl.heads, wl.dh, "f32", state=st0,
                                   rope={"grid": wl.grid, "pos": None})
    perm, n_cached = oracle.reorder_plan(budget, wl.T)
    st1 = oracle.initial_state(wts["x0"][perm], wl.layers, wl.d, wl.T)
    st1["budget"] = budget[perm]
    reo = oracle.stack_trajectory(None, wts, wl.T, sig, wl.heads, wl.dh, "f32", state=st1,
                                  rope={"grid": wl.grid, "pos": perm})
    for a, b in zip(base, reo):
        np.testing.assert_array_equal(np.sort(perm[b["idx"]]), a["idx"])
        assert np.all(np.isin(np.arange(n_cached, wl.N), b["idx"]))  # the baseline suffix is always active
        np.testing.assert_allclose(b["x"], a["x"][perm], rtol=1e-6, atol=1e-7)
        for (k0, _), (k1, _) in zip(a["caches"], b["caches"]):
            np.testing.assert_allclose(k1, k0[perm], rtol=1e-6, atol=1e-7)
