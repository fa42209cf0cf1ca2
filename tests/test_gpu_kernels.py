"""GPU parity of each C ABI call against the CPU oracle, on seeded inputs.

Bars: bit-exact for the active set and for gather/scatter (rows copied, rows
left alone); fp32 projections and attention within 1e-4, bf16 within 2e-2
(infinity-norm relative error max|gpu - oracle| / max|oracle|); the fp32
cached Euler update within 1e-6.
"""

import math

import numpy as np
import pytest
import torch

import oracle
import synth
from gpu_util import DEV, TOL, Guarded, host, host_bits, i32, rel_inf, to_dev, torch_dtype

H = pytest.importorskip("paper_2605_06892_amd.hsa_step")

pytestmark = pytest.mark.gpu


def _budgets(N, budgets, seed):
    return np.random.default_rng(seed).choice(np.asarray(budgets, np.int32), size=N)


# ---------------------------------------------------------------------------
# active set
# ---------------------------------------------------------------------------

AS_CASES = [
    # N, T, budgets, iterations, margin
    (0, 40, (40, 20, 10, 5), (0, 1), 0),
    (1, 40, (40, 20, 10, 5), (0, 1, 2), 0),
    (17, 8, (8, 4, 2), range(8), 0),
    (1024, 8, (8, 4, 2), range(8), 0),
    (16384, 40, (40, 20, 10, 5), (0, 1, 2, 4, 8, 39), 0),
    (16385, 40, (40, 20, 10, 5), (1, 2), 0),
    (32760, 40, (40, 20, 10, 5), range(40), 0),
    (75600, 40, (40, 10, 5), (0, 1, 2, 5, 10), 0),
    (32760, 40, (40, 20, 10, 5), (0, 3, 4, 5, 35, 36, 39), 4),
    (5000, 2000, (2000, 1000, 400, 1), (0, 1, 5, 1000, 1999), 0),   # T beyond the LDS table
    (3001, 12, (12, 6, 4, 3, 2, 1), range(12), 0),
    (300001, 40, (40, 20, 10, 5), (0, 1, 2, 3), 0),  # 16 ranges of several 16384-token chunks each
    (4097, 40, (40, 20, 10, 5), (1, 2), 0),          # two ranges, the second of one token
    (10, 1, (1,), (0,), 0),                           # T = 1: one iteration, every token active
    (2000, 1024, (1024, 512, 1), (0, 1, 2, 512, 1023), 0),       # the largest T of the LDS table
    (2000, 1025, (1025, 205, 41, 5, 1), (0, 5, 41, 205, 1024), 0),  # the smallest T past it
]


@pytest.mark.parametrize("case", AS_CASES, ids=lambda c: f"N{c[0]}_T{c[1]}_m{c[4]}")
def test_active_set_bit_exact(case):
    N, T, budgets, its, margin = case
    b = _budgets(N, budgets, N + T)
    budget = i32(b)
    gi, gc = Guarded((max(N, 1),), torch.int32, 3), Guarded((1,), torch.int32, 4)
    idx, cnt = gi.t, gc.t
    idx.fill_(-7)
    cnt.zero_()
    for i in its:
        n = H.hsa_build_active_set(budget, T, i, margin, idx, cnt)
        ref = oracle.active_set(b, T, i, margin)
        assert n == ref.size
        assert int(cnt.item()) == n
        np.testing.assert_array_equal(idx[:n].cpu().numpy(), ref)
        gi.check("idx")
        gc.check("n_active")


@pytest.mark.parametrize("N,T,budgets,margin,period", [(32760, 40, (20, 5), 4, 2), (5000, 40, (40, 10, 5), 10, 1),
                                                       (20001, 40, (20, 10), 5, 4), (3000, 2000, (1000, 10), 100, 2)])
def test_active_set_outside_period(N, T, budgets, margin, period):
    b = _budgets(N, budgets, N + T)
    idx = torch.full((N,), -7, dtype=torch.int32, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int32, device=DEV)
    its = sorted(set(list(range(0, margin + 2)) + list(range(T - margin - 2, T))))
    for i in its:
        n = H.hsa_build_active_set(i32(b), T, i, margin, idx, cnt, outside_period=period)
        ref = oracle.active_set(b, T, i, margin, period)
        assert n == ref.size, i
        np.testing.assert_array_equal(idx[:n].cpu().numpy(), ref)
    with pytest.raises(H.HsaStepError) as ei:
        H.hsa_build_active_set(i32(b), T, 0, margin, idx, cnt, outside_period=3)
    assert ei.value.name == "HSA_STEP_ERR_BUDGET"


def test_active_set_unaligned_budget_pointer():
    N, T = 4099, 40
    b = _budgets(N + 1, (40, 20, 10, 5), 3)
    full = i32(b)
    view = full[1:]  # 4-byte offset: not 16-byte aligned
    idx = torch.empty(N, dtype=torch.int32, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int32, device=DEV)
    for i in (0, 1, 2, 4):
        n = H.hsa_build_active_set(view, T, i, 0, idx, cnt)
        np.testing.assert_array_equal(idx[:n].cpu().numpy(), oracle.active_set(b[1:], T, i))


@pytest.mark.parametrize("bad", [3, 0, 41, -5])
def test_active_set_rejects_non_divisor_budget(bad):
    b = _budgets(2000, (40, 20, 10, 5), 1)
    b[1234] = bad
    with pytest.raises(ValueError):
        oracle.active_set(b, 40, 1)
    idx = torch.empty(2000, dtype=torch.int32, device=DEV)
    cnt = torch.zeros(1, dtype=torch.int32, device=DEV)
    with pytest.raises(H.HsaStepError) as ei:
        H.hsa_build_active_set(i32(b), 40, 1, 0, idx, cnt)
    assert ei.value.name == "HSA_STEP_ERR_BUDGET"
    assert int(cnt.item()) == -1


# ---------------------------------------------------------------------------
# cached Euler update
# ---------------------------------------------------------------------------


@pytest.mark.parametrize("N,C,fresh", [(1, 16, True), (1000, 16, True), (75600, 16, True),
                                       (75600, 64, False), (999, 3, True), (1024, 256, False),
                                       (32760, 16, True)])
def test_cached_euler(N, C, fresh):
    T = 40
    b = _budgets(N, (40, 10, 5), N)
    i = 1
    idx_np = oracle.active_set(b, T, i)
    st = synth.draw_euler_state(N, C, idx_np.size, seed=N + C)
    s = synth.linear_sigmas(T)
    x = to_dev(st["x"], "f32")
    vc = to_dev(st["v_cache"], "f32")
    vf = to_dev(st["v_fresh"], "f32") if fresh else None
    idx = i32(idx_np)
    H.hsa_cached_euler(x, vc, vf, idx if fresh else None, idx_np.size if fresh else 0, float(s[i]),
                       float(s[i + 1]))
    x_ref, v_ref = oracle.cached_euler(st["x"], st["v_cache"], st["v_fresh"] if fresh else None, idx_np,
                                       s[i], s[i + 1])
    np.testing.assert_array_equal(host(vc), v_ref)  # rows copied or untouched, bit for bit
    assert rel_inf(host(x), x_ref) <= 1e-6
    # fmaf is a single rounding; the oracle rounds once from float64
    assert np.mean(host(x) == x_ref) > 0.9999


def _euler_patterns(N):
    rng = np.random.default_rng(N)
    return {
        "all": np.arange(N),
        "first": np.array([0]),
        "last": np.array([N - 1]),
        "run": np.arange(N // 3, min(N, N // 3 + 700)),  # crosses token-tile boundaries
        "every_other": np.arange(1, N, 2),
        "random": np.sort(rng.choice(N, size=max(1, N // 5), replace=False)),
    }


@pytest.mark.parametrize("N,C", [(3000, 16), (1100, 7), (300, 4096), (200, 4100), (5000, 1)])
def test_cached_euler_index_patterns(N, C):
    # one pass over the tokens: fresh rows taken from v_fresh through the ascending
    # index list, cached rows otherwise; x within one rounding of the oracle
    s = synth.linear_sigmas(40)
    for name, idx_np in _euler_patterns(N).items():
        st = synth.draw_euler_state(N, C, idx_np.size, seed=N * 7 + C)
        gx, gv = Guarded((N, C), torch.float32, 1), Guarded((N, C), torch.float32, 2)
        x, vc = gx.t, gv.t
        x.copy_(to_dev(st["x"], "f32"))
        vc.copy_(to_dev(st["v_cache"], "f32"))
        H.hsa_cached_euler(x, vc, to_dev(st["v_fresh"], "f32"), i32(idx_np), idx_np.size, float(s[3]),
                           float(s[4]))
        gx.check("x")
        gv.check("v_cache")
        x_ref, v_ref = oracle.cached_euler(st["x"], st["v_cache"], st["v_fresh"], idx_np, s[3], s[4])
        np.testing.assert_array_equal(host(vc), v_ref, err_msg=name)
        assert rel_inf(host(x), x_ref) <= 1e-6, name
        assert np.mean(host(x) == x_ref) > 0.9999, name


@pytest.mark.parametrize("pattern", ["random", "run"])
def test_cached_euler_runs_of_tiles(pattern):
    # enough token tiles (16 rows of 256 channels each, 18751 tiles) that the launch takes runs of
    # 4 consecutive tiles per search
    N, C = 300001, 256
    idx_np = _euler_patterns(N)[pattern]
    st = synth.draw_euler_state(N, C, idx_np.size, seed=77)
    s = synth.linear_sigmas(40)
    gx, gv = Guarded((N, C), torch.float32, 5), Guarded((N, C), torch.float32, 6)
    x, vc = gx.t, gv.t
    x.copy_(to_dev(st["x"], "f32"))
    vc.copy_(to_dev(st["v_cache"], "f32"))
    H.hsa_cached_euler(x, vc, to_dev(st["v_fresh"], "f32"), i32(idx_np), idx_np.size, float(s[5]), float(s[6]))
    gx.check("x")
    gv.check("v_cache")
    x_ref, v_ref = oracle.cached_euler(st["x"], st["v_cache"], st["v_fresh"], idx_np, s[5], s[6])
    np.testing.assert_array_equal(host(vc), v_ref)
    assert rel_inf(host(x), x_ref) <= 1e-6
    assert np.mean(host(x) == x_ref) > 0.9999


def test_cached_euler_fp32_step_difference():
    # the shared step is sigma_next - sigma_i taken in fp32
    x = torch.zeros(4, 4, device=DEV)
    v = torch.ones(4, 4, device=DEV)
    H.hsa_cached_euler(x, v, None, None, 0, 0.7, 0.3)
    assert np.all(host(x) == np.float32(np.float32(0.3) - np.float32(0.7)))


# ---------------------------------------------------------------------------
# Q/K/V projection + cache overwrite
# ---------------------------------------------------------------------------


def _block(N, d, dtype, seed):
    wl = synth.Workload("t", (N,), d, 1, d, dtype, 8, ((8, 1.0),))
    return synth.draw_block(wl, seed)


@pytest.mark.parametrize("dtype,N,d,frac,compact", [
    ("bf16", 1000, 256, 0.3, False),
    ("bf16", 1000, 256, 0.3, True),
    ("bf16", 3000, 320, 0.5, False),   # 320 = 2.5 column tiles of 128
    ("bf16", 10000, 1536, 0.8, False),  # ~8000 rows x 3 x 1536: the 256 x 192 tiling
    ("bf16", 200, 64, 1.0, False),
    ("f32", 1024, 256, 0.33, False),
    ("f32", 333, 100, 0.5, True),
])
def test_qkv_scatter(dtype, N, d, frac, compact):
    blk = _block(N, d, dtype, seed=N + d)
    rng = np.random.default_rng(N)
    idx_np = np.flatnonzero(rng.random(N) < frac)
    nA = idx_np.size
    k0, v0 = synth.draw_cache(N, d, seed=7, dtype=dtype)
    x_in = blk["x"][idx_np] if compact else blk["x"]
    tdt = torch_dtype(dtype)
    x = to_dev(x_in, dtype)
    w = {k: to_dev(blk[k], dtype) for k in ("wq", "wk", "wv")}
    kc, vc = to_dev(k0, dtype), to_dev(v0, dtype)
    q = torch.full((nA, d), 3.0, dtype=tdt, device=DEV)
    H.hsa_qkv_scatter(x, i32(idx_np), nA, w["wq"], w["wk"], w["wv"], q, kc, vc, x_compact=compact)
    ref = oracle.qkv_cache_update(x_in, idx_np, blk["wq"], blk["wk"], blk["wv"], k0, v0, dtype, x_compact=compact)
    skipped = np.setdiff1d(np.arange(N), idx_np)
    np.testing.assert_array_equal(host_bits(kc)[skipped], host_bits(to_dev(k0, dtype))[skipped])
    np.testing.assert_array_equal(host_bits(vc)[skipped], host_bits(to_dev(v0, dtype))[skipped])
    tol = 1e-2 if dtype == "bf16" else 1e-5
    assert rel_inf(host(q), ref["q"]) <= tol
    assert rel_inf(host(kc)[idx_np], ref["k"]) <= tol
    assert rel_inf(host(vc)[idx_np], ref["v"]) <= tol


def test_qkv_scatter_beyond_4gib():
    """x, K_hat and V_hat of more than 4 GiB each (N = 2^20 + 64 rows of 2048
    bf16): byte offsets pass 32 bits, so the GEMM launcher takes its 64-bit
    lane-pointer load path instead of the buffer resources. The active rows
    include the last 64 rows of x (offsets past 2^32); only active rows of x
    are ever read, so only they hold drawn values."""
    nA, d = 8190, 2048
    N = (1 << 20) + 64
    assert N * d * 2 > 0xFFFFFFFF
    blk = _block(nA, d, "bf16", seed=4242)  # the active rows of x and the weights
    rng = np.random.default_rng(4242)
    idx_np = np.sort(np.concatenate([rng.choice(N - 64, nA - 64, replace=False), np.arange(N - 64, N)]))
    ii = torch.from_numpy(idx_np).to(DEV)
    x = torch.zeros(N, d, dtype=torch.bfloat16, device=DEV)
    x[ii] = to_dev(blk["x"], "bf16")
    w = {k: to_dev(blk[k], "bf16") for k in ("wq", "wk", "wv")}
    kc = torch.zeros(N, d, dtype=torch.bfloat16, device=DEV)
    vc = torch.zeros(N, d, dtype=torch.bfloat16, device=DEV)
    q = torch.full((nA, d), 3.0, dtype=torch.bfloat16, device=DEV)
    H.hsa_qkv_scatter(x, i32(idx_np), nA, w["wq"], w["wk"], w["wv"], q, kc, vc)
    torch.cuda.synchronize()
    assert rel_inf(host(q), oracle.project(blk["x"], blk["wq"], "bf16")) <= 1e-2
    assert rel_inf(host(kc[ii]), oracle.project(blk["x"], blk["wk"], "bf16")) <= 1e-2
    assert rel_inf(host(vc[ii]), oracle.project(blk["x"], blk["wv"], "bf16")) <= 1e-2
    # rows outside A keep their (zero) contents: the tail region and a sample
    skip = np.setdiff1d(np.concatenate([np.arange(N - 4096, N), rng.choice(N, 4096, replace=False)]), idx_np)
    si = torch.from_numpy(skip).to(DEV)
    assert int(torch.count_nonzero(kc[si])) == 0 and int(torch.count_nonzero(vc[si])) == 0
    del x, kc, vc
    torch.cuda.empty_cache()


@pytest.mark.parametrize("N,d", [(5000, 512), (777, 128)])
def test_identity_weights_gather_scatter_bit_exact(N, d):
    """Wq = Wk = Wv = I: the product is exact, so Q == x[A], K_hat[A] == V_hat[A]
    == x[A] bit for bit and every other cache row is untouched."""
    blk = _block(N, d, "bf16", seed=N)
    idx_np = np.flatnonzero(np.random.default_rng(d).random(N) < 0.4)
    eye = to_dev(np.eye(d, dtype=np.float32), "bf16")
    x = to_dev(blk["x"], "bf16")
    k0, v0 = synth.draw_cache(N, d, seed=1, dtype="bf16")
    kc, vc = to_dev(k0, "bf16"), to_dev(v0, "bf16")
    q = torch.empty(idx_np.size, d, dtype=torch.bfloat16, device=DEV)
    H.hsa_qkv_scatter(x, i32(idx_np), idx_np.size, eye, eye, eye, q, kc, vc)
    xb = host_bits(x)
    np.testing.assert_array_equal(host_bits(q), xb[idx_np])
    np.testing.assert_array_equal(host_bits(kc)[idx_np], xb[idx_np])
    np.testing.assert_array_equal(host_bits(vc)[idx_np], xb[idx_np])
    skipped = np.setdiff1d(np.arange(N), idx_np)
    np.testing.assert_array_equal(host_bits(kc)[skipped], host_bits(to_dev(k0, "bf16"))[skipped])


def test_zero_active_rows_is_a_no_op():
    N, d = 100, 128
    kc = torch.randn(N, d, device=DEV).to(torch.bfloat16)
    before = kc.clone()
    w = torch.randn(d, d, device=DEV).to(torch.bfloat16)
    x = torch.randn(N, d, device=DEV).to(torch.bfloat16)
    q = torch.empty(1, d, dtype=torch.bfloat16, device=DEV)
    idx = torch.zeros(1, dtype=torch.int32, device=DEV)
    vc = kc.clone()
    H.hsa_qkv_scatter(x, idx, 0, w, w, w, q, kc, vc)
    H.hsa_out_scatter(q, idx, 0, w, kc)
    torch.cuda.synchronize()
    assert torch.equal(kc, before)


# ---------------------------------------------------------------------------
# attention
# ---------------------------------------------------------------------------

ATTN_CASES = [
    # dtype, N keys, active queries, heads, head_dim
    ("bf16", 1000, 300, 2, 128),
    ("bf16", 1000, 300, 4, 64),
    ("bf16", 77, 5, 1, 128),
    ("bf16", 1, 1, 1, 64),
    ("bf16", 64, 128, 2, 128),
    ("bf16", 4109, 4096, 32, 128),   # two 32-query sub-tiles per wave
    ("bf16", 2000, 2048, 64, 64),    # idem, head_dim 64
    # key counts around the 96-row key tile and the 3-tile loop unroll: one block, one tile,
    # one tile + 1 row, two blocks of a second tile, three tiles, three tiles + 1 row, a
    # ragged 31-row last block
    ("bf16", 32, 7, 1, 128),
    ("bf16", 96, 40, 1, 128),
    ("bf16", 97, 40, 1, 64),
    ("bf16", 160, 9, 1, 128),
    ("bf16", 288, 70, 2, 128),
    ("bf16", 289, 70, 2, 64),
    ("bf16", 319, 33, 1, 128),
    ("f32", 1024, 342, 4, 64),
    ("f32", 100, 17, 2, 128),
    ("f32", 1, 3, 1, 64),
]


@pytest.mark.parametrize("case", ATTN_CASES, ids=lambda c: "_".join(map(str, c)))
def test_attention_core(case):
    dtype, N, nA, heads, dh = case
    d = heads * dh
    rng = np.random.default_rng(N + nA)
    q_np, k_np, v_np = (rng.standard_normal((r, d)).astype(np.float32) for r in (nA, N, N))
    if dtype == "bf16":
        q_np, k_np, v_np = (synth.to_bf16_values(a) for a in (q_np, k_np, v_np))
    scale = 1.0 / math.sqrt(dh)
    o = torch.full((nA, d), 5.0, dtype=torch_dtype(dtype), device=DEV)
    H.hsa_attention_core(to_dev(q_np, dtype), to_dev(k_np, dtype), to_dev(v_np, dtype), nA, heads, dh, scale, o)
    ref = oracle.round_to(oracle.attention(q_np, k_np, v_np, heads, dh, scale), dtype)
    err = rel_inf(host(o), ref)
    assert err <= TOL[dtype], err
    assert np.all(np.isfinite(host(o)))


def test_attention_softmax_is_shift_safe():
    """Large scores (|s| ~ 1e3) must not overflow the online softmax."""
    N, nA, heads, dh = 500, 130, 1, 128
    rng = np.random.default_rng(2)
    q_np = synth.to_bf16_values(rng.standard_normal((nA, dh)).astype(np.float32) * 8)
    k_np = synth.to_bf16_values(rng.standard_normal((N, dh)).astype(np.float32) * 8)
    v_np = synth.to_bf16_values(rng.standard_normal((N, dh)).astype(np.float32))
    o = torch.empty(nA, dh, dtype=torch.bfloat16, device=DEV)
    H.hsa_attention_core(to_dev(q_np, "bf16"), to_dev(k_np, "bf16"), to_dev(v_np, "bf16"), nA, heads, dh, 1.0, o)
    ref = oracle.round_to(oracle.attention(q_np, k_np, v_np, heads, dh, 1.0), "bf16")
    assert rel_inf(host(o), ref) <= TOL["bf16"]


@pytest.mark.parametrize("dtype,N,nA,d", [("bf16", 2000, 700, 256), ("bf16", 300, 300, 192),
                                          ("f32", 1024, 342, 256)])
def test_out_scatter(dtype, N, nA, d):
    rng = np.random.default_rng(nA)
    o_np = rng.standard_normal((nA, d)).astype(np.float32) * 0.1
    wo_np = (rng.standard_normal((d, d)) / math.sqrt(d)).astype(np.float32)
    out0 = rng.standard_normal((N, d)).astype(np.float32)
    if dtype == "bf16":
        o_np, wo_np, out0 = (synth.to_bf16_values(a) for a in (o_np, wo_np, out0))
    idx_np = np.sort(rng.choice(N, nA, replace=False))
    out = to_dev(out0, dtype)
    H.hsa_out_scatter(to_dev(o_np, dtype), i32(idx_np), nA, to_dev(wo_np, dtype), out)
    y = oracle.project(o_np, wo_np, dtype)
    skipped = np.setdiff1d(np.arange(N), idx_np)
    np.testing.assert_array_equal(host_bits(out)[skipped], host_bits(to_dev(out0, dtype))[skipped])
    assert rel_inf(host(out)[idx_np], y) <= (1e-2 if dtype == "bf16" else 1e-5)


def test_active_attention_equals_core_then_projection():
    N, nA, heads, dh = 1500, 600, 4, 128
    d = heads * dh
    g = torch.Generator(device=DEV).manual_seed(0)
    mk = lambda *s: torch.randn(*s, generator=g, device=DEV).to(torch.bfloat16)  # noqa: E731
    q, k, v, wo = mk(nA, d), mk(N, d), mk(N, d), mk(d, d) * 0.05
    idx = torch.sort(torch.randperm(N, device=DEV)[:nA])[0].to(torch.int32)
    out1, out2 = mk(N, d), None
    out2 = out1.clone()
    ws = torch.empty(H.hsa_attention_workspace_bytes(torch.bfloat16, nA, d) // 2, dtype=torch.bfloat16, device=DEV)
    H.hsa_active_attention(q, k, v, idx, nA, heads, dh, 1 / math.sqrt(dh), wo, out1, ws)
    o = torch.empty(nA, d, dtype=torch.bfloat16, device=DEV)
    H.hsa_attention_core(q, k, v, nA, heads, dh, 1 / math.sqrt(dh), o)
    H.hsa_out_scatter(o, idx, nA, wo, out2)
    torch.cuda.synchronize()
    assert torch.equal(out1, out2)
    assert torch.equal(ws.view(nA, d), o)


def _active_attention_with_parts(q_np, k_np, v_np, wo_np, out0, idx_np, heads, dh, scale, ws_bytes):
    """hsa_active_attention with a workspace of ws_bytes; returns (compact
    attention output, out)."""
    nA, d = q_np.shape
    ws = torch.zeros(ws_bytes, dtype=torch.uint8, device=DEV)
    out = to_dev(out0, "bf16")
    H.hsa_active_attention(to_dev(q_np, "bf16"), to_dev(k_np, "bf16"), to_dev(v_np, "bf16"), i32(idx_np), nA,
                           heads, dh, scale, to_dev(wo_np, "bf16"), out, ws)
    o = ws[: nA * d * 2].view(torch.bfloat16).view(nA, d)
    return host(o), out


@pytest.mark.parametrize("parts", [2, 3, 4])
@pytest.mark.parametrize("N,nA,heads,dh", [(1111, 777, 3, 128), (4100, 300, 2, 64), (130, 70, 2, 128),
                                           (65, 33, 1, 128), (2048, 256, 4, 128)])
def test_attention_key_parts(parts, N, nA, heads, dh, monkeypatch):
    """Cached rows split into key parts (forced count, clamped to the tiles)
    and merged: the attention output matches the oracle, the projection of
    it lands on the active rows only."""
    monkeypatch.setenv("HSA_ATTN_KV_PARTS", str(parts))
    d = heads * dh
    rng = np.random.default_rng(N * 10 + parts)
    q_np, k_np, v_np = (synth.to_bf16_values(rng.standard_normal((r, d)).astype(np.float32)) for r in (nA, N, N))
    wo_np = synth.to_bf16_values((rng.standard_normal((d, d)) / math.sqrt(d)).astype(np.float32))
    out0 = synth.to_bf16_values(rng.standard_normal((N, d)).astype(np.float32))
    idx_np = np.sort(rng.choice(N, nA, replace=False))
    scale = 1.0 / math.sqrt(dh)
    ws_bytes = H.hsa_attention_parts_workspace_bytes(torch.bfloat16, nA, heads, dh)
    o, out = _active_attention_with_parts(q_np, k_np, v_np, wo_np, out0, idx_np, heads, dh, scale, ws_bytes)
    ref = oracle.round_to(oracle.attention(q_np, k_np, v_np, heads, dh, scale), "bf16")
    assert rel_inf(o, ref) <= TOL["bf16"]
    skipped = np.setdiff1d(np.arange(N), idx_np)
    np.testing.assert_array_equal(host_bits(out)[skipped], host_bits(to_dev(out0, "bf16"))[skipped])
    assert rel_inf(host(out)[idx_np], oracle.project(o, wo_np, "bf16")) <= 1e-2


@pytest.mark.parametrize("parts", [None, "3"])
def test_attention_core_parts(parts, monkeypatch):
    """hsa_attention_core with a key-part scratch (the launcher's choice, or
    3 forced) matches the oracle."""
    if parts:
        monkeypatch.setenv("HSA_ATTN_KV_PARTS", parts)
    N, nA, heads, dh = 3000, 200, 2, 128
    d = heads * dh
    rng = np.random.default_rng(21)
    q_np, k_np, v_np = (synth.to_bf16_values(rng.standard_normal((r, d)).astype(np.float32)) for r in (nA, N, N))
    scale = 1.0 / math.sqrt(dh)
    nb = H.hsa_attention_parts_workspace_bytes(torch.bfloat16, nA, heads, dh) - \
        H.hsa_attention_workspace_bytes(torch.bfloat16, nA, d)
    scratch = torch.empty(nb, dtype=torch.uint8, device=DEV)
    o = torch.empty(nA, d, dtype=torch.bfloat16, device=DEV)
    H.hsa_attention_core(to_dev(q_np, "bf16"), to_dev(k_np, "bf16"), to_dev(v_np, "bf16"), nA, heads, dh, scale, o,
                         parts=scratch)
    ref = oracle.round_to(oracle.attention(q_np, k_np, v_np, heads, dh, scale), "bf16")
    assert rel_inf(host(o), ref) <= TOL["bf16"]


def test_attention_key_parts_shift_safe(monkeypatch):
    """Parts whose maxima differ by hundreds (log2 units) merge without
    overflow or underflow of the kept terms."""
    monkeypatch.setenv("HSA_ATTN_KV_PARTS", "4")
    N, nA, heads, dh = 2048, 130, 1, 128
    rng = np.random.default_rng(5)
    q_np = synth.to_bf16_values(rng.standard_normal((nA, dh)).astype(np.float32) * 8)
    k_np = rng.standard_normal((N, dh)).astype(np.float32) * 8
    k_np[: N // 2] *= 0.05  # the first parts see far smaller scores than the last
    k_np = synth.to_bf16_values(k_np)
    v_np = synth.to_bf16_values(rng.standard_normal((N, dh)).astype(np.float32))
    wo_np = synth.to_bf16_values(np.eye(dh, dtype=np.float32))
    idx_np = np.arange(nA)
    out0 = np.zeros((N, dh), np.float32)
    ws_bytes = H.hsa_attention_parts_workspace_bytes(torch.bfloat16, nA, heads, dh)
    o, _ = _active_attention_with_parts(q_np, k_np, v_np, wo_np, out0, idx_np, heads, dh, 1.0, ws_bytes)
    ref = oracle.round_to(oracle.attention(q_np, k_np, v_np, heads, dh, 1.0), "bf16")
    assert np.all(np.isfinite(o))
    assert rel_inf(o, ref) <= TOL["bf16"]


def test_attention_key_parts_auto_and_minimum_workspace():
    """A launch of few workgroups (one head, 256 queries, 4096 keys) splits
    on its own with the key-part workspace and matches the oracle; with the
    minimum workspace it does not split and equals hsa_attention_core bit for
    bit."""
    N, nA, heads, dh = 4096, 256, 1, 128
    rng = np.random.default_rng(11)
    q_np, k_np, v_np = (synth.to_bf16_values(rng.standard_normal((r, dh)).astype(np.float32)) for r in (nA, N, N))
    wo_np = synth.to_bf16_values((rng.standard_normal((dh, dh)) / math.sqrt(dh)).astype(np.float32))
    out0 = np.zeros((N, dh), np.float32)
    idx_np = np.arange(nA)
    scale = 1.0 / math.sqrt(dh)
    ref = oracle.round_to(oracle.attention(q_np, k_np, v_np, heads, dh, scale), "bf16")
    split = H.hsa_attention_parts_workspace_bytes(torch.bfloat16, nA, heads, dh)
    o_split, _ = _active_attention_with_parts(q_np, k_np, v_np, wo_np, out0, idx_np, heads, dh, scale, split)
    assert rel_inf(o_split, ref) <= TOL["bf16"]
    minimum = H.hsa_attention_workspace_bytes(torch.bfloat16, nA, heads * dh)
    o_min, _ = _active_attention_with_parts(q_np, k_np, v_np, wo_np, out0, idx_np, heads, dh, scale, minimum)
    o_core = torch.empty(nA, dh, dtype=torch.bfloat16, device=DEV)
    H.hsa_attention_core(to_dev(q_np, "bf16"), to_dev(k_np, "bf16"), to_dev(v_np, "bf16"), nA, heads, dh, scale,
                         o_core)
    np.testing.assert_array_equal(o_min, host(o_core))
    assert not np.array_equal(o_split, o_min)  # the split path ran (different rounding order)


@pytest.mark.parametrize("waves", [4, 8])
@pytest.mark.parametrize("dh", [64, 128])
def test_attention_every_tile_config(waves, dh, monkeypatch):
    """Each workgroup shape the launcher can pick (4 or 8 waves of 32 queries)
    on ragged sizes."""
    monkeypatch.setenv("HSA_ATTN_WAVES", str(waves))
    N, nA, heads = 1111, 777, 3
    d = heads * dh
    rng = np.random.default_rng(waves * 1000 + dh)
    q_np, k_np, v_np = (synth.to_bf16_values(rng.standard_normal((r, d)).astype(np.float32)) for r in (nA, N, N))
    scale = 1.0 / math.sqrt(dh)
    o = torch.empty(nA, d, dtype=torch.bfloat16, device=DEV)
    H.hsa_attention_core(to_dev(q_np, "bf16"), to_dev(k_np, "bf16"), to_dev(v_np, "bf16"), nA, heads, dh, scale, o)
    ref = oracle.round_to(oracle.attention(q_np, k_np, v_np, heads, dh, scale), "bf16")
    assert rel_inf(host(o), ref) <= TOL["bf16"]
