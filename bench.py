#!/usr/bin/env python3
"""Benchmark: seconds per ACID-gated denoise loop at the Wan-2.1-1.3B shape.

    python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME]
    python bench.py --workload small-dit-bf16 --sweep      (gate sweep: PSNR vs no-cache)

One bench "step" is one whole denoise loop (timestep-modulation table, per
step TEMNI + drift + gate, computed steps through all DiT blocks with the
residual stored, skipped steps through the residual cache, head + Euler on
every step) over one synthetic input.  W untimed loops, then K timed loops
bracketed by device synchronisation; rank 0 prints one JSON line.

Workload: 30 blocks, hidden 1536, 12 heads x 128, FFN 8960, 21 x 30 x 52 =
32760 video tokens, batch 1, 50 flow-matching steps, ACID gate
(tau_low 0.05, tau_high 0.2, delta 0.01), random-init weights N(0, 0.02^2)
and N(0, 1) latents (synthetic stand-ins for the trained model and prompts).

Other workloads (--workload): tiny-dit-f32, small-dit-bf16,
cogvideox-5b-shape, hunyuanvideo-slice (acid_inputs.CONFIGS).

Per-kernel durations come from the library's HIP-event timer on the stream
the kernels run on, over the timed loops.  The CPU baseline is the oracle
(fp64 NumPy) timed on this host: the whole loop for workloads of at most
2048 tokens, else a bounded sample (one block at full K/V for a few query
rows) extrapolated.
"""
from __future__ import annotations

import argparse
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "s per denoise loop; attention/GEMM TFLOP/s (% MFMA peak) at Wan-1.3B shape"
PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0       # MI355X HBM3E
PEAK_F32_TFLOPS = 157.3     # MI355X fp32 vector


def log(msg: str) -> None:
    print(f"[bench {time.strftime('%H:%M:%S')}] {msg}", file=sys.stderr, flush=True)


def work_per_class(cfg, n_computed: int, n_steps: int) -> dict:
    """Algorithmic flops / bytes per kernel class for one loop (skipped work
    not counted)."""
    L, Lv, H, F, nb = cfg.n_tokens, cfg.n_video, cfg.hidden, cfg.ffn, cfg.n_blocks
    es = 2 if cfg.dtype == "bf16" else 4
    kc = n_computed
    if getattr(cfg, "block", "sequential") == "parallel":
        # [W_qkv | W_1] in one GEMM (class gemm_qkv), [W_o ; W_2] in one
        # (class gemm_proj), one LN-modulate per block
        gemms = {"gemm_qkv": ("flop", kc * nb * 2.0 * L * H * (3 * H + F)),
                 "gemm_proj": ("flop", kc * nb * 2.0 * L * (H + F) * H)}
        ln_per_block = 1
    else:
        gemms = {"gemm_qkv": ("flop", kc * nb * 2.0 * L * H * 3 * H),
                 "gemm_proj": ("flop", kc * nb * 2.0 * L * H * H),
                 "gemm_ffn1": ("flop", kc * nb * 2.0 * L * H * F),
                 "gemm_ffn2": ("flop", kc * nb * 2.0 * L * F * H)}
        ln_per_block = 2
    return {
        "attention": ("flop", kc * nb * 4.0 * L * L * H),
        **gemms,
        "gemm_head": ("flop", n_steps * 2.0 * Lv * H * H),
        # TEMNI reads x, writes m; with a previous m also reads it (all fp32)
        "drift": ("byte", (8.0 + 12.0 * (n_steps - 1)) * Lv * H),
        # store: read x, h_out; write r.  apply: read x, r; write h_out.
        "cache": ("byte", n_steps * 12.0 * Lv * H),
        "ln_mod": ("byte", (kc * nb * ln_per_block * L + n_steps * Lv) * H * (4.0 + es)),
    }


def measured_traffic(kernel_source: str, record: str):
    """HBM bytes per launch of the dominant kernel from the committed counter
    record (rocprofv3 FETCH_SIZE / WRITE_SIZE passes scaled by the copy
    calibration), or None if the kernel source changed since it was taken."""
    import hashlib
    try:
        rec = json.load(open(os.path.join(ROOT, record)))
        sha = hashlib.sha256(open(os.path.join(ROOT, kernel_source), "rb").read()).hexdigest()
    except (OSError, ValueError):
        return None
    if rec.get("source_sha256") != sha:
        return None
    return rec["hbm_bytes_per_dispatch"]


def cpu_baseline_full(ai, cfg, schedule, gate: dict, threads: int, x_gpu,
                      mode: str = "acid", probe_blocks: int = 1) -> dict:
    """The oracle's whole denoise loop (small workloads), forced to the GPU
    run's schedule; also reports the relative error of the GPU's x_N."""
    import numpy as np

    import oracle as O

    om = O.DiTModel(cfg, ai.weights(cfg))
    x0 = ai.latents(cfg)
    text = ai.text_tokens(cfg)
    t0 = time.perf_counter()
    if mode == "dicache":
        xr, _ = O.dicache_loop(om, x0, ai.sigmas(cfg.n_steps), text,
                               gate=O.GateParams(gate["tau_low"], gate["tau_high"],
                                                 gate["delta"]),
                               n_probe=probe_blocks, forced_schedule=schedule)
    elif mode == "easycache":
        xr, _ = O.easycache_loop(lambda x, s: om.forward(x, s, text)[0], x0,
                                 ai.sigmas(cfg.n_steps),
                                 gate=O.GateParams(gate["tau_low"], gate["tau_high"],
                                                   gate["delta"], 2),
                                 forced_schedule=schedule)
    else:
        xr, _ = O.denoise_loop(om, x0, ai.sigmas(cfg.n_steps), text, mode="acid",
                               gate=O.GateParams(gate["tau_low"], gate["tau_high"],
                                                 gate["delta"]),
                               forced_schedule=schedule)
    t = time.perf_counter() - t0
    d = np.asarray(x_gpu, np.float64) - x0
    rel = float(np.linalg.norm(d - (xr - x0)) / np.linalg.norm(xr - x0))
    log(f"cpu baseline: full oracle loop {t:.2f} s, GPU x_N - x_0 rel err {rel:.2e}")
    return {"value": t, "unit": "s/loop", "cores": threads, "kind": "oracle",
            "sample": (f"fp64 NumPy oracle: the whole denoise loop ({cfg.n_steps} steps, "
                       f"{int(np.sum(schedule))} computed, schedule forced to the GPU run's)"),
            "gpu_rel_err_x": rel}


def cpu_baseline(ai, cfg, n_computed: int, n_steps: int, threads: int) -> dict:
    """The oracle on a bounded sample: one DiT block (full keys/values, R query
    rows at two values of R, extrapolated linearly to all rows), plus TEMNI,
    drift and head on all video rows; scaled to seconds per loop with the GPU
    run's computed-step count."""
    import numpy as np

    import oracle as O

    c1 = cfg.replace(n_blocks=1)
    params = ai.weights(c1)
    om = O.DiTModel(c1, params)
    x0 = ai.latents(cfg).astype(np.float64)
    text = ai.text_tokens(cfg)
    h = x0 if text is None else np.concatenate([text.astype(np.float64), x0])
    mod = om.modulation(0.5)
    L = h.shape[0]
    ts = {}
    for R in (64, 256):
        rows = np.arange(R)
        t0 = time.perf_counter()
        om.block(h, 0, mod["blocks"][0], rows=rows)
        ts[R] = time.perf_counter() - t0
        log(f"cpu baseline: block with {R} query rows {ts[R]:.2f} s")
    slope = (ts[256] - ts[64]) / (256 - 64)
    t_block = ts[64] + slope * (L - 64)
    t0 = time.perf_counter()
    m_prev = om.temni(x0, 0.5)
    m_cur = om.temni(x0 * 1.01, 0.48)
    O.relative_l1_drift(m_cur, m_prev)
    om.head(x0, 0.5)
    t_every = time.perf_counter() - t0
    log(f"cpu baseline: temni+drift+head {t_every:.2f} s")
    s_loop = n_computed * cfg.n_blocks * t_block + n_steps * t_every
    return {"value": s_loop, "unit": "s/loop", "cores": threads, "kind": "oracle",
            "sample": (f"fp64 NumPy oracle: one DiT block at full K/V for 64 and 256 query rows "
                       f"(extrapolated linearly to {L} rows = {t_block:.1f} s/block), plus TEMNI, "
                       f"drift and head on all {cfg.n_video} video rows ({t_every:.2f} s/step); "
                       f"loop = {n_computed} computed steps x {cfg.n_blocks} blocks + {n_steps} "
                       f"steps of per-step work (extrapolated)")}


def psnr(x, ref) -> float:
    """PSNR of x against ref with peak = max(ref) - min(ref), on final latents
    (device tensors; the quality measure of the gate sweep)."""
    x64, r64 = x.double(), ref.double()
    mse = float(((x64 - r64) ** 2).mean())
    rng = float(r64.max() - r64.min())
    return math.inf if mse == 0.0 else 10.0 * math.log10(rng * rng / mse)


def stream_ceilings(P, m, n: int, reps: int = 10) -> dict:
    """Attainable streaming rates on this part, measured with the library's
    own streaming kernels over three fp32 buffers of n elements: the cache
    STORE kernel (two streams in, one out: the drift's and the cache's
    mix) and the L1 sums (three streams in, nothing out)."""
    import torch

    bufs = [torch.randn(n, device="cuda") for _ in range(3)]

    def timed(fn):
        fn()
        torch.cuda.synchronize()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record()
        for _ in range(reps):
            fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps * 1e-3

    t21 = timed(lambda: P.cache_apply(P.ACID_CACHE_STORE, bufs[0], bufs[1], bufs[2]))
    # the L1 call reads its sums back to the host: time its kernels alone
    # with the library's event timer (the drift class)
    m.l1_norms(bufs[0], bufs[1], bufs[2])
    m.reset_timing()
    m.set_timing(True)
    for _ in range(reps):
        m.l1_norms(bufs[0], bufs[1], bufs[2])
    ms, launches = m.timing()["drift"]
    m.set_timing(False)
    m.reset_timing()
    t_ro = ms * 1e-3 / launches
    del bufs
    torch.cuda.empty_cache()
    return {"rw_2to1_gbs": 12.0 * n / t21 / 1e9, "read_only_gbs": 12.0 * n / t_ro / 1e9,
            "buffer_bytes": 4 * n,
            "kernels": "cache STORE (2 in, 1 out); L1 sums (3 in, two kernels: partial "
                       "sums and the one-block final reduction)"}


def parse_list(text: str):
    return [float(v) for v in text.split(",") if v]


def sweep_grid(taus: str, pairs: str, deltas: str, delta_fixed: float):
    """(kind, tau_low, tau_high, delta) points: fixed thresholds, then each
    ACID pair with each delta."""
    grid = [("fixed", t, t, delta_fixed) for t in parse_list(taus)]
    for pair in pairs.split(","):
        lo, hi = (float(v) for v in pair.split(":"))
        grid += [("acid", lo, hi, d) for d in parse_list(deltas)]
    return grid


def sweep(m, cfg, x0, text_d, sig, grid, mode: str = "acid", warmup: int = 0, steps: int = 1,
          outputs=None):
    """No-cache, then each grid point: computed steps, PSNR of x_N against the
    no-cache x_N, seconds per loop (median of `steps` timed loops after
    `warmup`).  Each run dict carries its trace; with `outputs` (a list) the
    x_N of every run (no-cache first) is appended to it."""
    import statistics

    import torch

    x = torch.empty_like(x0)

    def timed(mode, **gate):
        times, tr = [], None
        for k in range(warmup + steps):
            x.copy_(x0)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            tr = m.denoise_loop(x, sig, text_d, mode=mode, **gate)
            torch.cuda.synchronize()
            if k >= warmup:
                times.append(time.perf_counter() - t0)
        return statistics.median(times), tr

    t_ref, tr_ref = timed("nocache")
    ref = x.clone()
    if outputs is not None:
        outputs.append(ref)
    runs = [{"mode": "nocache", "computed_steps": cfg.n_steps, "s_per_loop": t_ref,
             "psnr_db": math.inf, "trace": tr_ref}]
    for kind, lo, hi, delta in grid:
        t, tr = timed(mode, tau_low=lo, tau_high=hi, delta=delta)
        if outputs is not None:
            outputs.append(x.clone())
        n_comp = int(tr["compute"].sum())
        sv = [float(v) for v in tr["s"] if math.isfinite(v)]
        ds = [abs(a - b) for a, b in zip(sv[1:], sv[:-1])]
        run = {"mode": kind, "tau_low": lo, "tau_high": hi, "delta": delta,
               "computed_steps": n_comp, "s_per_loop": t, "speedup_vs_nocache": t_ref / t,
               "psnr_db": psnr(x, ref),
               "steps_tau_high": int(sum(1 for v in tr["tau_used"][1:] if v == hi)),
               "steps_tau_low": int(sum(1 for v in tr["tau_used"][1:] if v == lo)),
               "drift_s_min_max": [min(sv), max(sv)] if sv else None,
               "drift_step_change_median_max": ([float(sorted(ds)[len(ds) // 2]), float(max(ds))]
                                                if ds else None),
               "schedule": "".join("C" if c else "S" for c in tr["compute"]),
               "trace": tr}
        runs.append(run)
        log(f"{kind} tau=({lo}, {hi}) delta={delta}: {n_comp}/{cfg.n_steps} computed, "
            f"{t * 1e3:.2f} ms/loop, PSNR {run['psnr_db']:.2f} dB")
    return runs


def run_sweep(args, m, cfg, x0, text_d, sig, mode: str = "acid") -> int:
    """The gate sweep of one workload as one JSON line (no traces)."""
    grid = sweep_grid(args.sweep_taus, args.sweep_pairs, args.sweep_deltas,
                      args.sweep_deltas_fixed)
    runs = sweep(m, cfg, x0, text_d, sig, grid, mode, args.warmup, args.steps)
    for r in runs:
        del r["trace"]
    print(json.dumps({"sweep": {"workload": cfg.name, "signal": args.signal,
                                "denoise_steps": cfg.n_steps,
                                "loops_timed": args.steps, "runs": runs}}), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5, help="timed denoise loops")
    ap.add_argument("--warmup", type=int, default=1, help="untimed denoise loops")
    ap.add_argument("--workload", default="wan2.1-1.3b-shape")
    ap.add_argument("--n-steps", type=int, default=None, help="denoising steps per loop")
    ap.add_argument("--signal", choices=["teacache", "easycache", "dicache"], default="teacache",
                    help="drift signal under the adaptive gate")
    ap.add_argument("--probe-blocks", type=int, default=1, help="DiCache probe depth")
    ap.add_argument("--tau-low", type=float, default=None,
                    help="default 0.05 (teacache) / 0.1 (easycache)")
    ap.add_argument("--tau-high", type=float, default=None,
                    help="default 0.2 (both signals)")
    ap.add_argument("--delta", type=float, default=0.01)
    ap.add_argument("--loop", choices=["host", "graph"], default="host",
                    help="host: gate on the host, one signal read-back per step; graph: gate "
                         "on the device, the loop captured once as a HIP graph and replayed")
    ap.add_argument("--graph-context", action="store_true",
                    help="also time the other loop variant (host gate / captured graph)")
    ap.add_argument("--attention-context", action="store_true",
                    help="also time PyTorch's scaled_dot_product_attention (flash backend only) "
                         "at the workload's attention shape, as context")
    ap.add_argument("--no-nocache", action="store_true", help="skip the uncached context loop")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-timing", action="store_true", help="disable the per-kernel event timer")
    ap.add_argument("--sweep", action="store_true",
                    help="gate sweep on --workload: no-cache, fixed tau, ACID tau pairs x delta "
                         "(computed steps, PSNR vs no-cache, s/loop)")
    ap.add_argument("--sweep-taus", default="0.05,0.1,0.2", help="fixed thresholds")
    ap.add_argument("--sweep-pairs", default="0.05:0.2", help="ACID tau_low:tau_high pairs")
    ap.add_argument("--sweep-deltas", default="0.0002,0.0005,0.001,0.002,0.005,0.01,0.02")
    ap.add_argument("--sweep-deltas-fixed", type=float, default=0.01,
                    help="delta for fixed-tau runs (unused when tau_low == tau_high)")
    ap.add_argument("--copy-calibration", action="store_true",
                    help="only run the residual-cache store over three 1 GiB fp32 arrays (reads "
                         "2 GiB, writes 1 GiB): the reference for scaling HBM byte counters")
    args = ap.parse_args()

    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py runs on exactly one GPU: the ACID-gated denoise loop here has no "
              "multi-GPU path (no sharding, no collectives); use --gpus 1.", file=sys.stderr)
        return 2

    import numpy as np
    import torch

    import acid_inputs as ai
    import paper_2607_12358_amd as P

    if args.copy_calibration:
        n = 1 << 28
        x = torch.randn(n, device="cuda")
        h = torch.randn(n, device="cuda")
        r = torch.empty(n, device="cuda")
        torch.cuda.synchronize()
        P.cache_apply(P.ACID_CACHE_STORE, x, h, r)
        torch.cuda.synchronize()
        print(json.dumps({"copy_calibration": {"elements": n, "read_bytes": 8 * n,
                                               "write_bytes": 4 * n}}), flush=True)
        return 0

    cfg = ai.CONFIGS[args.workload]
    if args.n_steps:
        cfg = cfg.replace(n_steps=args.n_steps)
    N = cfg.n_steps
    torch.cuda.set_device(0)
    log(f"libacid {P.version()} on {torch.cuda.get_device_name(0)}; workload {cfg.name}")

    t0 = time.perf_counter()
    m = P.Model(cfg, max_steps=N)

    def progress(it):
        last = time.perf_counter()
        for i, item in enumerate(it):
            if time.perf_counter() - last > 20:
                last = time.perf_counter()
                log(f"weights: tensor {i} of {m.tensor_count()}")
            yield item

    m.load_weights(progress(ai.iter_weights(cfg)))
    torch.cuda.synchronize()
    log(f"weights generated and loaded in {time.perf_counter() - t0:.1f} s "
        f"(arena {m.arena.numel() / 2**30:.2f} GiB, workspace {m.workspace.numel() / 2**30:.2f} GiB)")
    x0 = torch.from_numpy(ai.latents(cfg)).cuda()
    text = ai.text_tokens(cfg)
    text_d = torch.from_numpy(text).cuda() if text is not None else None
    sig = ai.sigmas(N)
    x = torch.empty_like(x0)
    if args.tau_low is None:
        # EasyCache's per-step signal on these random-weight stacks is about
        # 0.04 (k |dsigma| with k near 2), so the pair is set above it.
        args.tau_low = 0.05 if args.signal == "teacache" else 0.1
    if args.tau_high is None:
        args.tau_high = 0.2
    mode = {"teacache": "acid", "easycache": "easycache", "dicache": "dicache"}[args.signal]
    if mode == "dicache":
        m.set_probe_blocks(args.probe_blocks)
    gate = dict(tau_low=args.tau_low, tau_high=args.tau_high, delta=args.delta)

    if args.sweep:
        return run_sweep(args, m, cfg, x0, text_d, sig, mode)
    graph = args.loop == "graph"

    def loops(count, use_graph, timed_kernels, label):
        """count loops back to back; returns (seconds per loop, traces, timing)."""
        if timed_kernels:
            m.reset_timing()
            m.set_timing(True)
        torch.cuda.synchronize()
        t_start = time.perf_counter()
        trs = []
        for k in range(count):
            x.copy_(x0)
            if use_graph:
                # the captured loop returns without waiting; one trace suffices
                tr = m.denoise_loop(x, sig, text_d, mode=mode, **gate, graph=True,
                                    trace=(k == count - 1))
            else:
                tr = m.denoise_loop(x, sig, text_d, mode=mode, **gate)
            if tr is not None:
                trs.append(tr)
            log(f"{label} loop {k} issued")
        torch.cuda.synchronize()
        el = time.perf_counter() - t_start
        tim = m.timing() if timed_kernels else {}
        m.set_timing(False)
        return el / count, trs, tim

    for w in range(args.warmup):
        x.copy_(x0)
        tr = m.denoise_loop(x, sig, text_d, mode=mode, **gate, graph=graph)
        torch.cuda.synchronize()
        log(f"warmup loop {w} done: {int(tr['compute'].sum())}/{N} computed")

    s_per_loop, traces, timing = loops(args.steps, graph, not args.no_timing and not graph,
                                       "timed")
    if graph and not args.no_timing:
        # the event timer does not see kernels inside a graph: the per-kernel
        # table comes from one host-gated loop (same kernels, same schedule)
        _, host_tr, timing = loops(1, False, True, "kernel-table")
        assert np.array_equal(host_tr[0]["compute"], traces[-1]["compute"])
        kernel_loops = 1
    else:
        kernel_loops = args.steps
    n_comp = int(traces[-1]["compute"].sum())
    assert all(np.array_equal(t["compute"], traces[0]["compute"]) for t in traces)
    log(f"{args.steps} loops ({args.loop}) -> {s_per_loop:.4f} s/loop, {n_comp}/{N} computed")

    other = None
    if args.graph_context:
        x.copy_(x0)
        m.denoise_loop(x, sig, text_d, mode=mode, **gate, graph=not graph)  # warm / capture
        other, _, _ = loops(args.steps, not graph, False, "context")
        log(f"context: {'host' if graph else 'graph'} loop {other:.4f} s/loop")

    # per-kernel-class rates over the timed region
    work = work_per_class(cfg, n_comp, N)
    kernels = {}
    for name, (ms, launches) in timing.items():
        if launches == 0:
            continue
        ent = {"ms_per_loop": ms / kernel_loops, "launches_per_loop": launches / kernel_loops,
               "avg_us": 1e3 * ms / launches}
        if name in work:
            kind, amount = work[name]
            rate = amount * kernel_loops / (ms * 1e-3)
            if kind == "flop":
                ent["tflops"] = rate / 1e12
                if cfg.dtype == "bf16":
                    ent["frac_bf16_peak"] = rate / 1e12 / PEAK_BF16_TFLOPS
                else:
                    ent["frac_f32_peak"] = rate / 1e12 / PEAK_F32_TFLOPS
            else:
                ent["gbs"] = rate / 1e9
                ent["frac_hbm_peak"] = rate / 1e9 / PEAK_HBM_GBS
        kernels[name] = ent
    ceilings = None
    if cfg.dtype == "bf16":
        ceilings = stream_ceilings(P, m, cfg.n_video * cfg.hidden)
        for name in ("drift", "cache"):  # two streams in, one out
            if name in kernels and "gbs" in kernels[name]:
                kernels[name]["frac_measured_2to1"] = kernels[name]["gbs"] / ceilings["rw_2to1_gbs"]
        log(f"streaming ceilings: {ceilings['rw_2to1_gbs']:.0f} GB/s (2:1), "
            f"{ceilings['read_only_gbs']:.0f} GB/s (read-only)")
    gemm_ms = sum(timing[k][0] for k in timing if k.startswith("gemm_"))
    gemm_flop = sum(work[k][1] for k in work if k.startswith("gemm_"))
    gemm_tflops = gemm_flop * kernel_loops / (gemm_ms * 1e-3) / 1e12 if gemm_ms else None

    roofline = None
    if "attention" in kernels:
        L, H = cfg.n_tokens, cfg.hidden
        per_launch = 4.0 * L * L * H
        avg_s = kernels["attention"]["avg_us"] * 1e-6
        ach = per_launch / avg_s / 1e12
        traffic = None
        if cfg.head_dim == 128 and cfg.name == "wan2.1-1.3b-shape":
            traffic = measured_traffic("paper_2607_12358_amd/csrc/attention.hip",
                                       "profiles/attention_counters.json")
        if cfg.dtype == "bf16":
            bound, peak, kname = "mfma", PEAK_BF16_TFLOPS, f"attn_bf16_kernel<{cfg.head_dim}>"
        else:  # fp32 attention runs on the vector ALUs
            bound, peak, kname = "alu", PEAK_F32_TFLOPS, f"attn_f32_kernel<{cfg.head_dim}>"
        roofline = {"bound": bound, "achieved": ach, "peak": peak, "unit": "TFLOP/s",
                    "frac": ach / peak, "traffic": traffic, "kernel": kname,
                    "flop_per_launch": per_launch, "avg_launch_us": avg_s * 1e6}

    nocache = None
    if not args.no_nocache:
        if graph:  # capture first, time a replay
            x.copy_(x0)
            m.denoise_loop(x, sig, text_d, mode="nocache", graph=True, trace=False)
        x.copy_(x0)
        torch.cuda.synchronize()
        t1 = time.perf_counter()
        m.denoise_loop(x, sig, text_d, mode="nocache", graph=graph)
        torch.cuda.synchronize()
        nocache = time.perf_counter() - t1
        log(f"uncached loop: {nocache:.3f} s ({N} computed steps)")

    library_attention = None
    if args.attention_context and cfg.dtype == "bf16":
        from torch.nn.attention import SDPBackend, sdpa_kernel
        L, nh, d = cfg.n_tokens, cfg.n_heads, cfg.head_dim
        g = torch.Generator(device="cuda")
        g.manual_seed(7)
        q, k, v = (torch.randn((1, nh, L, d), generator=g, device="cuda").to(torch.bfloat16)
                   for _ in range(3))
        try:
            # flash backend only: no silent fallback to the batched-matmul path
            with sdpa_kernel([SDPBackend.FLASH_ATTENTION]):
                torch.nn.functional.scaled_dot_product_attention(q, k, v)
                torch.cuda.synchronize()
                t1 = time.perf_counter()
                for _ in range(3):
                    torch.nn.functional.scaled_dot_product_attention(q, k, v)
                torch.cuda.synchronize()
            ms = (time.perf_counter() - t1) / 3 * 1e3
            library_attention = {"backend": "torch sdpa (flash)", "ms": ms,
                                 "tflops": 4.0 * L * L * nh * d / (ms * 1e-3) / 1e12}
        except RuntimeError as e:
            library_attention = {"backend": "torch sdpa (flash)", "unavailable": str(e)[:200]}
        del q, k, v
        log(f"library attention: {library_attention}")

    cpu = None
    if not args.no_cpu_baseline:
        try:
            from threadpoolctl import threadpool_info
            threads = max((i.get("num_threads", 1) for i in threadpool_info()
                           if i.get("user_api") == "blas"), default=1)
        except Exception:
            threads = len(os.sched_getaffinity(0))
        if cfg.n_tokens <= 2048:
            x.copy_(x0)
            m.denoise_loop(x, sig, text_d, mode=mode, **gate)
            cpu = cpu_baseline_full(ai, cfg, traces[-1]["compute"], gate, threads,
                                    x.cpu().numpy(), mode, args.probe_blocks)
        else:
            cpu = cpu_baseline(ai, cfg, n_comp, N, threads)

    out = {
        "metric": METRIC,
        "value": s_per_loop,
        "unit": "s/loop",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": 1e3 * s_per_loop,
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": cfg.dtype,
        "data": "synthetic",
        "config": {"workload": cfg.name, "n_blocks": cfg.n_blocks, "hidden": cfg.hidden,
                   "heads": cfg.n_heads, "head_dim": cfg.head_dim, "ffn": cfg.ffn,
                   "video_tokens": cfg.n_video, "text_tokens": cfg.n_text, "batch": 1,
                   "block": cfg.block,
                   "denoise_steps": N,
                   "gate": {"mode": "acid", "signal": args.signal, **gate,
                            "n_warmup": 2 if mode == "easycache" else 1,
                            **({"probe_blocks": args.probe_blocks} if mode == "dicache"
                               else {})},
                   "parallelism": "single-gpu"},
        "loop": args.loop,
        "host_loop_s_per_loop": other if graph else s_per_loop,
        "graph_loop_s_per_loop": s_per_loop if graph else other,
        "computed_steps": n_comp,
        "schedule": "".join("C" if c else "S" for c in traces[-1]["compute"]),
        "gemm_tflops": gemm_tflops,
        "gemm_frac_peak": (gemm_tflops / (PEAK_BF16_TFLOPS if cfg.dtype == "bf16" else
                                          PEAK_F32_TFLOPS)) if gemm_tflops else None,
        "kernels": kernels,
        "stream_ceilings": ceilings,
        "nocache_s_per_loop": nocache,
        "speedup_vs_nocache": (nocache / s_per_loop) if nocache else None,
        "roofline": roofline,
        **({"library_attention": library_attention} if library_attention else {}),
        "cpu_baseline": cpu,
    }
    print(json.dumps(out), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
