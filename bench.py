"""Benchmark of the HSA active-token layer step on one MI355X.

A step is one pass of the whole hot path over one batch of synthetic input:
  active set (with its one host read-back) -> Q/K/V + cache overwrite ->
  active-query attention -> output projection + scatter -> cached Euler update
of the N x 16 fp32 latents.

Default workload: a Wan-2.1-14B-shaped block, N = 21 x 30 x 52 = 32760 tokens,
d = 5120 (40 heads x 128), bf16, T = 40 with budgets {40, 20, 10, 5} on
quarters of the tokens ranked by a seeded velocity norm; timed at iteration 1
(25% of the tokens active) and, as a second line item, iteration 2 (50%).
The KV cache is filled by a dense iteration 0 first (every token is active at
i = 0). Inputs are synthetic (seeded normal latents and N(0, 1/d) weights);
everything is resident in HBM before the timed region.

Prints ONE JSON line. `value` is the layer-step time in ms (Q/K/V + cache
overwrite + attention + output projection and scatter, GPU event time) at
25% active; per-kernel times, the attention TFLOP/s at 25% and 50% active,
the roofline of the attention kernel and the CPU oracle baseline are extra
fields.

    python bench.py [--steps K] [--warmup W] [--workload wan14b] [--no-cpu-baseline]
    python bench.py --only attention --steps 3     # one kernel, for rocprofv3 counter passes
"""

from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

METRIC = "HSA layer-step ms + active-attention TFLOP/s at N=32760, 25%/50% active"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
EULER_CHANNELS = 16         # latent channels advanced by the cached Euler update
MI355X_SIMDS = 1024         # 256 CUs x 4 SIMDs
MI355X_XCDS = 8
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "attention_wan14b_traffic.txt")
ATTN_SRC = os.path.join(ROOT, "paper_2605_06892_amd", "csrc", "attention_bf16.hip")


def parse():
    p = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=50)
    p.add_argument("--warmup", type=int, default=5)
    p.add_argument("--workload", default="wan14b", choices=["wan14b", "wan1.3b", "wan14b_720p"])
    p.add_argument("--iteration", type=int, default=1, help="timed iteration (1: 25%% active)")
    p.add_argument("--second-iteration", type=int, default=2, help="also time this iteration (-1: skip)")
    p.add_argument("--layout", default="scattered", choices=["scattered", "contiguous"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--no-schedules", action="store_true", help="skip the preset-schedule trajectories")
    p.add_argument("--no-euler-stress", action="store_true",
                   help="skip the Euler and gather bandwidth-stress shapes")
    p.add_argument("--no-extra-timings", action="store_true",
                   help="skip the 100%%-active, cold-cache and other-layout timings of the step")
    p.add_argument("--no-other-workloads", action="store_true",
                   help="skip the 720p-shaped block (N = 75600) and the Wan-1.3B-shaped block at 50%%")
    p.add_argument("--no-end-to-end", action="store_true",
                   help="skip the 30-layer sampling loops (HSA vs dense, T = 40)")
    p.add_argument("--end-to-end-only", action="store_true", help="run only the 30-layer sampling loops")
    p.add_argument("--no-blocks", action="store_true",
                   help="skip the full-block (cross-attention + FFN) loops with the Appendix C presets")
    p.add_argument("--summarize", metavar="DIR", default=None,
                   help="print a text summary of the rocprofv3 csv output under DIR and exit")
    p.add_argument("--write-traffic", metavar="DIR", default=None,
                   help="from counter passes DIR/{attn,copy}_{fetch,write} write the attention HBM traffic file")
    p.add_argument("--only", default=None,
                   choices=["active_set", "qkv", "attention", "out", "euler", "copy", "stress", "stress_c64"],
                   help="launch only this kernel --steps times after setup (profiling passes); "
                        "stress / stress_c64: only the gather and Euler bandwidth-stress shapes at 16 / 64 channels")
    return p.parse_args()


def setup(wl, layout, dev):
    import torch

    import synth
    from paper_2605_06892_amd import layer as L

    blk = synth.draw_block(wl, 0)
    budget = synth.assign_budgets(blk["v_group"], wl.groups, layout)
    b = L.BlockBuffers.allocate(wl.N, wl.d, wl.heads, wl.dh, torch.bfloat16, device=dev)
    b.x.copy_(synth.bf16_tensor(blk["x"]))
    for k in ("wq", "wk", "wv", "wo"):
        getattr(b, k).copy_(synth.bf16_tensor(blk[k]))
    b.budget.copy_(torch.from_numpy(budget))
    b.out.zero_()
    st = synth.draw_euler_state(wl.N, EULER_CHANNELS, wl.N, seed=5)
    eul = {k: torch.from_numpy(v).to(dev) for k, v in st.items()}
    # iteration 0 activates every token: its Q/K/V pass fills the whole cache
    n0 = L.active_set(b, wl.T, 0)
    assert n0 == wl.N
    L.qkv(b, n0)
    torch.cuda.synchronize()
    return blk, budget, b, eul


def run_step(b, eul, T, it, sigmas, ev=None, margin=0, outside_period=1):
    """One full pass of the hot path; if ev is given, record events between calls."""
    from paper_2605_06892_amd import hsa_step as H
    from paper_2605_06892_amd import layer as L

    rec = (lambda k: ev[k].record()) if ev is not None else (lambda k: None)  # noqa: E731
    rec(0)
    n = L.active_set(b, T, it, margin, outside_period)
    rec(1)
    L.qkv(b, n)
    rec(2)
    L.attention(b, n)
    rec(3)
    L.out_projection(b, n)
    rec(4)
    H.hsa_cached_euler(eul["x"], eul["v_cache"], eul["v_fresh"], b.idx, n, float(sigmas[it]), float(sigmas[it + 1]))
    rec(5)
    return n


KERNEL_NAMES = ["active_set", "qkv_scatter", "attention", "out_scatter", "cached_euler"]


def time_iteration(b, eul, wl, it, sigmas, steps, warmup, flush=None):
    """Mean per-call event times over `steps` passes of iteration `it`, the
    host wall time per pass and the layer-step time (Q/K/V + attention +
    output) of every pass. With `flush` (a device buffer of at least the
    MALL's size) it is overwritten before every pass (cold caches)."""
    import torch

    for _ in range(warmup):
        run_step(b, eul, wl.T, it, sigmas)
    torch.cuda.synchronize()
    evs = [[torch.cuda.Event(enable_timing=True) for _ in range(6)] for _ in range(steps)]
    t0 = time.perf_counter()
    n = 0
    for s in range(steps):
        if flush is not None:
            flush.zero_()
        n = run_step(b, eul, wl.T, it, sigmas, evs[s])
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) / steps * 1e3
    per = {nm: float(np.mean([evs[s][k].elapsed_time(evs[s][k + 1]) for s in range(steps)]))
           for k, nm in enumerate(KERNEL_NAMES)}
    layer = [evs[s][1].elapsed_time(evs[s][4]) for s in range(steps)]
    return n, wall, per, layer


def workload_item(dev, name, it, steps, warmup=2):
    """One whole HSA iteration of another single-block workload (its own
    buffers, KV cache filled by a dense iteration 0): active set with its
    read-back, Q/K/V + cache overwrite, attention, output projection +
    scatter and the cached Euler update of N x 16 fp32 latents. Per-call event
    times, the layer step, the iteration and the attention rate."""
    import torch

    import synth

    wl = synth.WORKLOADS[name]
    sig = synth.linear_sigmas(wl.T)
    _, _, b, eul = setup(wl, "scattered", dev)
    n, wall, per, layer = time_iteration(b, eul, wl, it, sig, steps, warmup)
    layer_ms = per["qkv_scatter"] + per["attention"] + per["out_scatter"]
    res = {
        "workload": f"{wl.name} single block: N={wl.N} ({'x'.join(map(str, wl.grid))} latent tokens), d={wl.d} "
                    f"({wl.heads}x{wl.dh} heads), T={wl.T}, budgets {{{','.join(str(g[0]) for g in wl.groups)}}} "
                    f"by velocity-norm rank, iteration {it}",
        "n_active": n,
        "active_fraction": round(n / wl.N, 4),
        "layer_step_ms": round(layer_ms, 4),
        "layer_step_ms_dist": dist(layer),
        "iteration_ms": round(sum(per.values()), 4),
        "ms_per_step": round(wall, 4),
        "kernels_ms": {k: round(v, 4) for k, v in per.items()},
        "active_attention_tflops": round(attention_flops(n, wl.N, wl.d) / (per["attention"] * 1e-3) / 1e12, 2),
        "qkv_out_gemm_tflops": round(gemm_flops(n, wl.d) / ((per["qkv_scatter"] + per["out_scatter"]) * 1e-3) / 1e12, 2),
        "euler_state": f"{wl.N}x{EULER_CHANNELS} fp32",
        "euler_gbs": round(euler_bytes(wl.N, EULER_CHANNELS, n) / (per["cached_euler"] * 1e-3) / 1e9, 1),
    }
    del b, eul
    torch.cuda.empty_cache()
    return res


def dist(xs):
    """Median, 10th and 90th percentile (ms)."""
    return {"median": round(float(np.median(xs)), 4), "p10": round(float(np.percentile(xs, 10)), 4),
            "p90": round(float(np.percentile(xs, 90)), 4)}


def attention_flops(n_active, N, d):
    return 4.0 * n_active * N * d  # QK^T and PV, 2 FLOP per multiply-add


def gemm_flops(n_active, d):
    return 2.0 * n_active * d * (3 * d) + 2.0 * n_active * d * d


def traffic_from_profile(workload, layout, iteration):
    """HBM bytes per attention launch from the committed rocprofv3 counter
    summary, if it was taken on the current kernel source and this is the
    launch it measured (the Wan-14B block, scattered budgets, iteration 1);
    else None."""
    if (workload, layout, iteration) != ("wan14b", "scattered", 1) or not os.path.exists(TRAFFIC_FILE):
        return None
    src_sha = hashlib.sha256(open(ATTN_SRC, "rb").read()).hexdigest()
    vals = {}
    for line in open(TRAFFIC_FILE):
        if ":" in line and not line.startswith("#"):
            k, v = line.split(":", 1)
            vals[k.strip()] = v.strip()
    if vals.get("kernel_source_sha256") != src_sha:
        return None
    try:
        return float(vals["hbm_bytes_per_launch"])
    except (KeyError, ValueError):
        return None


def _csv_rows(path):
    import csv

    with open(path, newline="") as f:
        return list(csv.DictReader(f))


def _find(d, suffix):
    out = []
    for root, _, files in os.walk(d):
        out += [os.path.join(root, f) for f in files if f.endswith(suffix)]
    return sorted(out)


def _short(name, n=100):
    name = name.replace("hsa::(anonymous namespace)::", "").replace("void ", "", 1)
    return name if len(name) <= n else name[: n - 3] + "..."


def counter_values(d):
    """{(kernel, counter): [value per dispatch]} from rocprofv3 counter csv files."""
    acc = {}
    for f in _find(d, "counter_collection.csv"):
        for r in _csv_rows(f):
            key = (r["Kernel_Name"], r["Counter_Name"])
            acc.setdefault(key, []).append(float(r["Counter_Value"]))
    return acc


def counter_means(d):
    """{(kernel, counter): (mean value per dispatch, dispatches)}."""
    return {k: (float(np.mean(v)), len(v)) for k, v in counter_values(d).items()}


def summarize(d):
    lines = []
    for f in _find(d, "kernel_stats.csv"):
        lines.append(f"kernel statistics ({os.path.relpath(f, d)})")
        lines.append(f"{'calls':>6} {'avg_us':>10} {'min_us':>10} {'max_us':>10} {'pct':>6}  kernel")
        for r in _csv_rows(f):
            lines.append(f"{int(r['Calls']):>6} {float(r['AverageNs'])/1e3:>10.1f} {float(r['MinNs'])/1e3:>10.1f} "
                         f"{float(r['MaxNs'])/1e3:>10.1f} {float(r['Percentage']):>6.2f}  {_short(r['Name'])}")
    cm = counter_means(d)
    if cm:
        lines.append("counters (mean per dispatch)")
        for (k, c), (v, n) in sorted(cm.items()):
            lines.append(f"{c:>28} {v:>18.1f}  dispatches={n}  {_short(k)}")
        cv = counter_values(d)
        busy = {k: v for (k, c), v in cv.items() if c == "SQ_VALU_MFMA_BUSY_CYCLES"}
        gui = {k: v for (k, c), v in cv.items() if c == "GRBM_GUI_ACTIVE"}
        both = sorted(k for k in busy if k in gui and len(busy[k]) == len(gui[k]))
        if both:
            lines.append(f"MFMA busy per dispatch: SQ_VALU_MFMA_BUSY_CYCLES / ({MI355X_SIMDS} SIMDs x "
                         f"GRBM_GUI_ACTIVE / {MI355X_XCDS} XCDs)")
            for k in both:
                fr = [b / (MI355X_SIMDS * g / MI355X_XCDS) for b, g in zip(busy[k], gui[k]) if g > 0]
                if any(f > 0 for f in fr):
                    lines.append("  " + " ".join(f"{f:.3f}" for f in fr) + f"  {_short(k)}")
    return "\n".join(lines)


def write_traffic(d):
    """HBM bytes per attention launch: FETCH_SIZE and WRITE_SIZE (KiB per
    dispatch) of the attention kernel, each scaled by expected/measured bytes
    of a plain 1 GiB device copy profiled the same way."""
    def values(sub, counter, kernel_pred):
        vals = [v for (k, c), vs in counter_values(os.path.join(d, sub)).items()
                if c == counter and kernel_pred(k) for v in vs]
        if not vals:
            raise SystemExit(f"no {counter} data in {sub}")
        return vals
    is_attn = lambda k: "attention_bf16_kernel" in k  # noqa: E731
    is_copy = lambda k: "copyBuffer" in k  # noqa: E731
    copy_bytes = float(256 << 20) * 4
    f_att = float(np.mean(values("attn_fetch", "FETCH_SIZE", is_attn))) * 1024
    w_att = float(np.mean(values("attn_write", "WRITE_SIZE", is_attn))) * 1024
    # the 1 GiB copies are the largest copy dispatches of their runs
    f_cpy = max(values("copy_fetch", "FETCH_SIZE", is_copy)) * 1024
    w_cpy = max(values("copy_write", "WRITE_SIZE", is_copy)) * 1024
    fetch_scale, write_scale = copy_bytes / f_cpy, copy_bytes / w_cpy
    total = f_att * fetch_scale + w_att * write_scale
    sha = hashlib.sha256(open(ATTN_SRC, "rb").read()).hexdigest()
    text = (
        "# HBM traffic of one attention launch (Wan-14B-shaped block, N=32760, d=5120, 25% active)\n"
        "# from rocprofv3 counter passes, each command run from the repository root:\n"
        "#   rocprofv3 --pmc FETCH_SIZE --output-format csv -d <out>/attn_fetch -o run -- python3 bench.py --only attention --steps 3\n"
        "#   rocprofv3 --pmc WRITE_SIZE --output-format csv -d <out>/attn_write -o run -- python3 bench.py --only attention --steps 3\n"
        "#   rocprofv3 --pmc FETCH_SIZE --output-format csv -d <out>/copy_fetch -o run -- python3 bench.py --only copy --steps 3\n"
        "#   rocprofv3 --pmc WRITE_SIZE --output-format csv -d <out>/copy_write -o run -- python3 bench.py --only copy --steps 3\n"
        "#   python3 bench.py --write-traffic <out>\n"
        "# the copy passes move 1 GiB each way; their counters calibrate bytes per KiB unit\n"
        f"attention_fetch_kib_per_dispatch: {f_att / 1024:.1f}\n"
        f"attention_write_kib_per_dispatch: {w_att / 1024:.1f}\n"
        f"copy_fetch_kib_per_dispatch: {f_cpy / 1024:.1f}\n"
        f"copy_write_kib_per_dispatch: {w_cpy / 1024:.1f}\n"
        f"fetch_scale: {fetch_scale:.4f}\n"
        f"write_scale: {write_scale:.4f}\n"
        f"hbm_bytes_per_launch: {total:.0f}\n"
        f"kernel_source_sha256: {sha}\n"
    )
    with open(TRAFFIC_FILE, "w") as f:
        f.write(text)
    return text


def schedule_runtimes(dev, name="wan1.3b"):
    """Wall time of a whole T = 40 sampling trajectory of one layer (active set,
    layer step, cached Euler update at every iteration) for each budget preset
    of the paper's Appendix C, relative to the uniform schedule (every token at
    every iteration, FM with T = 40). Presets with strategy D use the
    velocity-norm ranking stand-in; HSA-25 uses random allocation (R)."""
    import torch

    import synth
    from paper_2605_06892_amd import hsa_step as H

    wl = synth.WORKLOADS[name]
    blk, _, b, eul = setup(wl, "scattered", dev)
    T = 40
    sig = synth.linear_sigmas(T)

    def trajectory(budget, margin, outside_period=1):
        b.budget.copy_(torch.from_numpy(budget))
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        steps = 0
        for i in range(T):
            steps += run_step(b, eul, T, i, sig, margin=margin, outside_period=outside_period)
        torch.cuda.synchronize()
        return (time.perf_counter() - t0) * 1e3, steps / (wl.N * T)

    full = np.full(wl.N, T, dtype=np.int32)
    trajectory(full, 0)  # warm-up
    fm_ms, _ = trajectory(full, 0)
    out = {"workload": f"{name} single layer, N={wl.N}, d={wl.d}, T={T}", "fm_T40_ms": round(fm_ms, 2)}
    for pname, pre in synth.PRESETS.items():
        layout = "random" if pre["strategy"] == "R" else "scattered"
        budget = synth.assign_budgets(blk["v_group"], pre["groups"], layout)
        m = H.hsa_window_margin(pre["window"], T)
        ms, frac = trajectory(budget, m)
        out[pname] = {"ms": round(ms, 2), "runtime_vs_fm": round(ms / fm_ms, 4),
                      "token_step_fraction": round(frac, 4), "paper_runtime": pre["printed_runtime"]}
        s_max = max(g[0] for g in pre["groups"])
        if s_max < T:  # the other reading of the window: the largest budget's schedule outside it
            ms, frac = trajectory(budget, m, T // s_max)
            out[pname]["outside_period_T_over_smax"] = {
                "ms": round(ms, 2), "runtime_vs_fm": round(ms / fm_ms, 4), "token_step_fraction": round(frac, 4)}
    return out


BURST = 10  # launches per event pair in the stress timings: per-launch time without the event overhead


def euler_bytes(n_tokens, channels, n_fresh):
    """Bytes the one-pass cached Euler update must move: x read and written and
    one velocity row read per token (cached or fresh), the fresh rows written
    to the velocity cache, and the index list."""
    return n_tokens * channels * 4 * 3 + n_fresh * (channels * 4 + 4)


def euler_stress(dev, n_tokens=1 << 24, channels=EULER_CHANNELS, reps=10):
    """The cached Euler update at a bandwidth-stress shape (16M tokens x 16 fp32
    channels, every 4th token fresh), far above the 256 MB last-level cache:
    algorithmic bytes per launch (euler_bytes) over its time (median over reps
    of BURST back-to-back launches between two events), against the HBM peak."""
    import torch

    from paper_2605_06892_amd import hsa_step as H

    x = torch.zeros(n_tokens, channels, device=dev)
    vc = torch.ones(n_tokens, channels, device=dev)
    idx = torch.arange(0, n_tokens, 4, dtype=torch.int32, device=dev)
    na = idx.numel()
    vf = torch.ones(na, channels, device=dev)
    ts = []
    for r in range(reps + 2):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(BURST):
            H.hsa_cached_euler(x, vc, vf, idx, na, 0.5, 0.25)
        b.record()
        torch.cuda.synchronize()
        if r >= 2:
            ts.append(a.elapsed_time(b) / BURST)
    ms = float(np.median(ts))
    nbytes = euler_bytes(n_tokens, channels, na)
    gbs = nbytes / (ms * 1e-3) / 1e9
    del x, vc, vf, idx
    return {"tokens": n_tokens, "channels": channels, "fresh_rows": na, "ms": round(ms, 4),
            "bytes": nbytes, "gbs": round(gbs, 1), "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)}


def gather_stress(dev, n_tokens=1 << 24, channels=EULER_CHANNELS, reps=10):
    """The index-driven row gather of the stack's latent (hsa_gather_rows) at the
    same bandwidth-stress shape: every 4th of 16M fp32 rows of 16 channels
    gathered into compact bf16 rows. HBM bytes per launch (the index, the rows
    read, the compact rows written) over its event time, against the HBM peak."""
    import torch

    from paper_2605_06892_amd import hsa_step as H

    x = torch.ones(n_tokens, channels, device=dev)
    idx = torch.arange(0, n_tokens, 4, dtype=torch.int32, device=dev)
    na = idx.numel()
    xa = torch.empty(na, channels, device=dev, dtype=torch.bfloat16)
    ts = []
    for r in range(reps + 2):
        a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        a.record()
        for _ in range(BURST):
            H.hsa_gather_rows(x, idx, na, xa)
        b.record()
        torch.cuda.synchronize()
        if r >= 2:
            ts.append(a.elapsed_time(b) / BURST)
    ms = float(np.median(ts))
    nbytes = na * (4 + channels * 4 + channels * 2)
    gbs = nbytes / (ms * 1e-3) / 1e9
    del x, idx, xa
    return {"tokens": n_tokens, "channels": channels, "rows": na, "ms": round(ms, 4), "bytes": nbytes,
            "gbs": round(gbs, 1), "hbm_frac": round(gbs / PEAK_HBM_GBS, 4)}


def stack_flops(n_active, N, d, C, layers, ffn=0, ctx=0):
    """Matrix-product FLOPs of one stack pass over n_active rows: embedding,
    per layer Q/K/V, attention against N cached rows and the output
    projection (plus, for full blocks, cross-attention to ctx rows and the
    FFN), velocity head."""
    per_layer = gemm_flops(n_active, d) + attention_flops(n_active, N, d)
    if ctx:
        per_layer += 4.0 * n_active * d * d + attention_flops(n_active, ctx, d)
    if ffn:
        per_layer += 4.0 * n_active * d * ffn
    return 2.0 * n_active * C * d * 2 + layers * per_layer


def end_to_end(dev, name="wan1.3b_stack", presets=False, rope=False):
    """Whole T = 40 sampling loops of a 30-layer Wan-1.3B-shaped stack on the
    same seed and weights: the dense loop (every token at every iteration:
    flow matching with T = 40) and the HSA loop with budgets {40, 20, 10, 5}
    on quarters of the tokens, groups refreshed from velocity norms where
    every schedule fires; with presets, also the Appendix C presets with
    their windows (strategy D from L1_rel for HSA-75A/75B/50, random
    allocation for HSA-25). Each loop is timed on the host clock between two
    device synchronizations, so it includes the per-iteration read-back of
    |A_i|."""
    import torch

    import synth
    from paper_2605_06892_amd import hsa_step as H
    from paper_2605_06892_amd import stack as S

    wl = synth.WORKLOADS[name]
    N, C, L, d, T = wl.N, wl.euler_channels, wl.layers, wl.d, wl.T
    t_draw = time.perf_counter()
    wts = synth.draw_stack(wl, seed=0)
    b = S.StackBuffers.allocate(N, C, L, wl.heads, wl.dh, torch.bfloat16, device=dev, ffn=wl.ffn, ctx=wl.ctx)
    bf = synth.bf16_tensor
    b.w_embed.copy_(bf(wts["w_embed"]))
    b.w_head.copy_(bf(wts["w_head"]))
    for dst, lw in zip(b.layers, wts["layers"]):
        for t, k in zip(dst, ("wq", "wk", "wv", "wo")):
            t.copy_(bf(lw[k]))
    if wl.ctx:
        for dst, lw in zip(b.cross, wts["layers"]):
            dst[0].copy_(bf(lw["wq_c"]))
            dst[1].copy_(bf(lw["wo_c"]))
        ctx = bf(wts["ctx"]).to(dev)
        b.set_context(ctx, [bf(lw["wk_c"]).to(dev) for lw in wts["layers"]],
                      [bf(lw["wv_c"]).to(dev) for lw in wts["layers"]])
    if wl.ffn:
        for dst, lw in zip(b.ffn, wts["layers"]):
            dst[0].copy_(bf(lw["w1"]))
            dst[1].copy_(bf(lw["w2"]))
    if rope:
        b.enable_rope(wl.grid)
    x0 = torch.from_numpy(wts["x0"]).to(dev)
    del wts
    t_draw = time.perf_counter() - t_draw
    sig = synth.linear_sigmas(T)

    def loop(groups, budget0=None, margin=0, outside_period=1, selection=H.SELECT_VELOCITY_NORM, iterations=T,
             bufs=None, reorder=False):
        bb = b if bufs is None else bufs
        bb.x.copy_(x0)
        bb.v_hat.zero_()
        if budget0 is None:
            bb.budget.fill_(T)
        else:
            bb.budget.copy_(torch.from_numpy(budget0))
        if reorder:
            if bb.pos is not None:
                bb.pos.copy_(torch.arange(N, dtype=torch.int32, device=dev))
            S.reorder(bb, T)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        res = S.run(bb, T, sig, groups, margin=margin, iterations=iterations, outside_period=outside_period,
                    selection=selection)
        torch.cuda.synchronize()
        ms = (time.perf_counter() - t0) * 1e3
        fl = sum(stack_flops(n, N, d, C, L, wl.ffn, wl.ctx) for n, _ in res)
        return ms, {"token_step_fraction": round(sum(n for n, _ in res) / (N * T), 4),
                    "refreshes": int(sum(r for _, r in res)), "tflops": round(fl / (ms * 1e-3) / 1e12, 1),
                    "final_latent_finite": bool(torch.isfinite(bb.x).all())}

    sizes = synth.group_sizes(N, wl.groups)
    loop(sizes, iterations=2)  # warm-up: a dense and a partial iteration
    dense_ms, dense = loop(None)
    hsa_ms, hsa = loop(sizes)
    out = {
        "workload": (f"{name}: {L} {'full blocks (FFN ' + str(wl.ffn) + ', context ' + str(wl.ctx) + ')' if wl.ffn else 'layers'}"
                     f"{', 3D RoPE by token position' if rope else ''}, "
                     f"N={N} ({'x'.join(map(str, wl.grid))}), d={d} ({wl.heads}x{wl.dh}), C={C} fp32 latent, bf16 model, "
                     f"T={T}, budgets {{40,20,10,5}} on quarters by velocity-norm rank, refreshed every "
                     f"{math.lcm(*[T // s for s, _ in sizes])} iterations"),
        "dense_T40_ms": round(dense_ms, 1),
        "hsa_ms": round(hsa_ms, 1),
        "runtime_vs_dense": round(hsa_ms / dense_ms, 4),
        "token_step_fraction": hsa["token_step_fraction"],
        "refreshes": hsa["refreshes"],
        "final_latents_finite": dense["final_latent_finite"] and hsa["final_latent_finite"],
        "dense_tflops": dense["tflops"],
        "hsa_tflops": hsa["tflops"],
        "setup_s": round(t_draw, 1),
    }
    if presets:
        for pname, pre in synth.PRESETS.items():
            psizes = synth.group_sizes(N, pre["groups"])
            m = H.hsa_window_margin(pre["window"], T)
            if pre["strategy"] == "D":
                ms, r = loop(psizes, margin=m, selection=H.SELECT_L1_REL)
                how = f"strategy D (L1_rel over iterations 0-{m - 1})"
            else:  # random allocation, fixed for the trajectory
                budget0 = synth.random_budgets(N, pre["groups"], seed=0)
                ms, r = loop(None, budget0=budget0, margin=m)
                how = "random allocation"
            r.update({"ms": round(ms, 1), "runtime_vs_dense": round(ms / dense_ms, 4), "selection": how,
                      "window_margin": m, "paper_runtime": pre["printed_runtime"]})
            out[pname] = r
            s_max = max(g[0] for g in pre["groups"])
            if s_max < T and pre["strategy"] != "D":  # the other window reading (strategy D needs period 1)
                ms, r2 = loop(None, budget0=budget0, margin=m, outside_period=T // s_max)
                r2.update({"ms": round(ms, 1), "runtime_vs_dense": round(ms / dense_ms, 4)})
                out[pname]["outside_period_T_over_smax"] = r2
        # token reordering + prefix-only cache (Section 2.5): HSA-75A groups with the first
        # frame reserved for the baseline group (strategy F), same loop with full and prefix caches
        pre = synth.PRESETS["HSA-75A"]
        budget0 = synth.assign_budgets(np.zeros((N, 1), np.float32), pre["groups"], "first_frame",
                                       frame_tokens=wl.grid[1] * wl.grid[2], seed=0)
        m = H.hsa_window_margin(pre["window"], T)
        n_cached = S.prefix_rows(int(np.sum(budget0 < T)), N)
        pb = S.StackBuffers.allocate(N, C, L, wl.heads, wl.dh, torch.bfloat16, device=dev, ffn=wl.ffn,
                                     ctx=wl.ctx, n_cached=n_cached)
        for f in ("w_embed", "w_head", "layers", "cross", "ffn", "rope_cs", "grid"):
            setattr(pb, f, getattr(b, f))  # the same weights and tables
        if pb.rope_cs is not None:
            pb.pos = torch.arange(N, dtype=torch.int32, device=dev)
        full_ms, rf = loop(None, budget0=budget0, margin=m, reorder=True)
        full_x = b.x.clone()
        pre_ms, rp = loop(None, budget0=budget0, margin=m, bufs=pb, reorder=True)
        es = 2
        out["reordered_prefix_cache"] = {
            "groups": "HSA-75A, first frame reserved (strategy F), reordered once before the loop",
            "cache_bytes_full": 2 * L * N * d * es, "cache_bytes_prefix": 2 * L * n_cached * d * es,
            "tail_bytes": 2 * (N - n_cached) * d * es,
            "full_cache_ms": round(full_ms, 1), "prefix_cache_ms": round(pre_ms, 1),
            "runtime_vs_dense": round(pre_ms / dense_ms, 4), "token_step_fraction": rp["token_step_fraction"],
            "latents_bit_identical": bool(torch.equal(full_x, pb.x)),
        }
        del pb
    return out


def cpu_baseline(wl, blk, budget, it):
    """The oracle's layer step timed on this host over every active row: the
    fresh Q/K/V rows and the cache overwrite, attention of all active queries
    against the whole N-row cache, the output projection and the scatter
    (oracle.layer_step, float64, queries in blocks of at most 512 rows)."""
    import oracle
    import synth

    try:
        from threadpoolctl import threadpool_info
        threads = max((i.get("num_threads", 1) for i in threadpool_info() if i.get("user_api") == "blas"), default=1)
    except Exception:  # pragma: no cover
        threads = 1
    idx = oracle.active_set(budget, wl.T, it)
    k0, v0 = synth.draw_cache(wl.N, wl.d, seed=1, dtype="bf16")
    out0 = np.zeros((wl.N, wl.d), np.float32)
    w = {k: blk[k] for k in ("wq", "wk", "wv", "wo")}
    t0 = time.perf_counter()
    oracle.layer_step(blk["x"], idx, w, k0, v0, out0, wl.heads, wl.dh, 1 / math.sqrt(wl.dh), "bf16")
    ms = (time.perf_counter() - t0) * 1e3
    return {"value": round(ms, 1), "unit": "ms", "cores": int(threads), "kind": "oracle",
            "host_cpus": os.cpu_count(),
            "sample": (f"full step, {idx.size} rows: one oracle.layer_step over all {idx.size} active rows "
                       f"(iteration {it}) against all {wl.N} cached rows, {wl.heads} heads, float64, timed once")}


def main():
    args = parse()
    if args.summarize:
        print(summarize(args.summarize))
        return
    if args.write_traffic:
        print(write_traffic(args.write_traffic))
        return
    if args.gpus != 1:
        print(f"bench.py runs on one GPU only (got --gpus {args.gpus}); the layer step has no "
              "multi-GPU path in this build", file=sys.stderr)
        sys.exit(2)
    import torch

    import synth
    from paper_2605_06892_amd import hsa_step as H
    from paper_2605_06892_amd import layer as L

    H.lib()  # fail loudly if the HIP library is missing
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(1)
    dev = "cuda:0"
    torch.cuda.set_device(0)
    if args.end_to_end_only:
        out = {"end_to_end": end_to_end(dev)}
        if not args.no_blocks:
            torch.cuda.empty_cache()
            out["end_to_end_blocks"] = end_to_end(dev, "wan1.3b_blocks", presets=True, rope=True)
        print(json.dumps(out))
        return
    if args.only == "stress":
        print(json.dumps({"gather_stress": gather_stress(dev), "euler_stress": euler_stress(dev)}))
        return
    if args.only == "stress_c64":
        print(json.dumps({"gather_stress_c64": gather_stress(dev, n_tokens=1 << 22, channels=64),
                          "euler_stress_c64": euler_stress(dev, n_tokens=1 << 22, channels=64)}))
        return
    wl = synth.WORKLOADS[args.workload]
    sigmas = synth.linear_sigmas(wl.T)
    blk, budget, b, eul = setup(wl, args.layout, dev)

    if args.only:
        n = L.active_set(b, wl.T, args.iteration)
        big = None
        if args.only == "copy":
            big = torch.empty(256 << 20, dtype=torch.float32, device=dev)  # 1 GiB
            dst = torch.empty_like(big)
        torch.cuda.synchronize()
        for _ in range(args.steps):
            if args.only == "active_set":
                L.active_set(b, wl.T, args.iteration)
            elif args.only == "qkv":
                L.qkv(b, n)
            elif args.only == "attention":
                L.attention(b, n)
            elif args.only == "out":
                L.out_projection(b, n)
            elif args.only == "euler":
                H.hsa_cached_euler(eul["x"], eul["v_cache"], eul["v_fresh"], b.idx, n, float(sigmas[1]), float(sigmas[2]))
            elif args.only == "copy":
                dst.copy_(big)
        torch.cuda.synchronize()
        print(json.dumps({"only": args.only, "steps": args.steps, "n_active": n,
                          "copy_bytes": None if big is None else big.numel() * 4}))
        return

    n, wall, per, layer = time_iteration(b, eul, wl, args.iteration, sigmas, args.steps, args.warmup)
    layer_ms = per["qkv_scatter"] + per["attention"] + per["out_scatter"]
    attn_fl = attention_flops(n, wl.N, wl.d)
    attn_tflops = attn_fl / (per["attention"] * 1e-3) / 1e12
    gemm_tf = gemm_flops(n, wl.d) / ((per["qkv_scatter"] + per["out_scatter"]) * 1e-3) / 1e12
    eb = euler_bytes(wl.N, EULER_CHANNELS, n)
    out = {
        "metric": METRIC,
        "value": round(layer_ms, 4),
        "unit": "ms",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(wall, 4),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {
            "workload": f"{wl.name} single block: N={wl.N} ({'x'.join(map(str, wl.grid))} latent tokens), "
                        f"d={wl.d} ({wl.heads}x{wl.dh} heads), T={wl.T}, budgets "
                        f"{{{','.join(str(g[0]) for g in wl.groups)}}} by velocity-norm rank ({args.layout}), "
                        f"iteration {args.iteration}",
            "n_active": n,
            "active_fraction": round(n / wl.N, 4),
            "euler_state": f"{wl.N}x{EULER_CHANNELS} fp32",
        },
        "kernels_ms": {k: round(v, 4) for k, v in per.items()},
        "layer_step_ms_dist": dist(layer),
        "active_attention_tflops": round(attn_tflops, 2),
        "qkv_out_gemm_tflops": round(gemm_tf, 2),
        "euler_gbs": round(eb / (per["cached_euler"] * 1e-3) / 1e9, 1),
    }
    out["roofline"] = {
        "kernel": "attention_bf16",
        "bound": "mfma",
        "achieved": round(attn_tflops, 2),
        "peak": PEAK_BF16_TFLOPS,
        "unit": "TFLOP/s",
        "frac": round(attn_tflops / PEAK_BF16_TFLOPS, 4),
        "traffic": traffic_from_profile(args.workload, args.layout, args.iteration),
        "flops_per_launch": attn_fl,
    }
    def item(it, steps, flush=None):
        n2, wall2, per2, layer2 = time_iteration(b, eul, wl, it, sigmas, steps, 1, flush)
        return {
            "iteration": it,
            "n_active": n2,
            "active_fraction": round(n2 / wl.N, 4),
            "layer_step_ms": round(per2["qkv_scatter"] + per2["attention"] + per2["out_scatter"], 4),
            "layer_step_ms_dist": dist(layer2),
            "ms_per_step": round(wall2, 4),
            "kernels_ms": {k: round(v, 4) for k, v in per2.items()},
            "active_attention_tflops": round(attention_flops(n2, wl.N, wl.d) / (per2["attention"] * 1e-3) / 1e12, 2),
        }

    if args.second_iteration >= 0:
        out["second"] = item(args.second_iteration, args.steps)
    if not args.no_extra_timings:
        # the same step with every token active (iteration T/s_min: the dense comparator, same kernels)
        full_it = wl.T // min(g[0] for g in wl.groups)
        out["full_active"] = item(full_it, max(3, args.steps // 4))
        out["full_active"]["hsa_step_over_full"] = round(layer_ms / out["full_active"]["layer_step_ms"], 4)
        # cold caches: a 1 GiB buffer (4x the 256 MB MALL) overwritten before every pass
        flush = torch.empty(256 << 20, dtype=torch.float32, device=dev)
        out["cold"] = item(args.iteration, max(5, args.steps // 2), flush)
        del flush
        # the other budget layout: groups as consecutive index ranges
        other = "contiguous" if args.layout == "scattered" else "scattered"
        b.budget.copy_(torch.from_numpy(synth.assign_budgets(blk["v_group"], wl.groups, other)))
        out["layout_" + other] = item(args.iteration, args.steps)
        b.budget.copy_(torch.from_numpy(budget))
    if not args.no_euler_stress:
        out["euler_stress"] = euler_stress(dev)
        # 64 fp32 channels: the stack's latent rows, 256 bytes, whole cache lines
        out["euler_stress_c64"] = euler_stress(dev, n_tokens=1 << 22, channels=64)
        out["gather_stress"] = gather_stress(dev)
        # the stack's real latent rows: 64 fp32 channels (256-byte rows, whole cache lines)
        out["gather_stress_c64"] = gather_stress(dev, n_tokens=1 << 22, channels=64)
    if not args.no_schedules or not args.no_end_to_end or not args.no_other_workloads:
        del b, eul
        torch.cuda.empty_cache()
    if not args.no_other_workloads:
        # the 720p-shaped block (N = 75600, 25% active) and the Wan-1.3B-shaped block at 50%
        out["wan14b_720p"] = workload_item(dev, "wan14b_720p", 1, max(5, args.steps // 4))
        out["wan13b_50"] = workload_item(dev, "wan1.3b", 2, args.steps)
    if not args.no_schedules:
        out["schedules"] = schedule_runtimes(dev)
        torch.cuda.empty_cache()
    if not args.no_end_to_end:
        out["end_to_end"] = end_to_end(dev)
        torch.cuda.empty_cache()
        if not args.no_blocks:
            out["end_to_end_blocks"] = end_to_end(dev, "wan1.3b_blocks", presets=True, rope=True)
            torch.cuda.empty_cache()
    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(wl, blk, budget, args.iteration)
    print(json.dumps(out))


if __name__ == "__main__":
    main()
