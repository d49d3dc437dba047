#!/usr/bin/env python3
"""Benchmark: HeadCast routed attention on one MI355X.

One *step* is one autoregressive denoising step of the whole model on the hot
path: for each of the 30 layers, write the current block's K/V into the
layer's per-archetype buffers (hc_append_block) and run the head-specific
attention of all 12 heads (hc_attention).  The same step is timed on a second
context whose heads are all Global -- this library's own full-window attention
-- for the speedup.  The one-time classification (hc_classify_heads) is timed
separately on one layer.

Inputs are synthetic (N(0,1) rounded to bf16, drawn on the device from a seed)
with the shapes of a Wan-1.3B-class backbone at the chosen latent grid.  All
inputs are resident in HBM before the timed region starts.

Prints one JSON line: the metric, the roofline of the dominant kernel, the CPU
baseline, the variants and the per-path and per-layer figures.
"""
import argparse
import json
import math
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

from synth import inputs as S  # noqa: E402

METRIC = "routed attention ms/layer-step + TFLOP/s (% MFMA peak); speedup vs full-window"
PEAK_BF16_TFLOPS = 2500.0     # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0         # MI355X HBM3E
CALIB_BYTES = 512 * 2**20     # calibration copy for the profiler's byte counters
CSRC = os.path.join(ROOT, "paper_2607_20125_amd", "csrc")
# sources that determine each kernel's code: a counter profile is only
# reported while their hash matches the one it was taken with
KERNEL_SOURCES = {
    "dense": ("hc_device.h", "hc_internal.h", "hc_geometry.h", "hc_units.h", "hc_dense.hip"),
    "spatial": ("hc_device.h", "hc_internal.h", "hc_geometry.h", "hc_units.h", "hc_spatial.hip"),
}
TRAFFIC_FILES = {
    "dense": os.path.join(ROOT, "profiles", "attn_dense_routed_720p_traffic.txt"),
    "spatial": os.path.join(ROOT, "profiles", "attn_spatial_routed_720p_traffic.txt"),
}


def kernel_source_hash(kind: str = "dense") -> str:
    import hashlib
    h = hashlib.sha256()
    for name in KERNEL_SOURCES[kind]:
        h.update(open(os.path.join(CSRC, name), "rb").read())
    return h.hexdigest()[:16]


def counter_profile(workload: str, kind: str):
    """Key-value lines of the committed counter profile of a kernel of the
    routed 720P step, or None if the workload differs or the kernel's sources
    changed since the profile was taken."""
    path = TRAFFIC_FILES[kind]
    if workload != "720p" or not os.path.exists(path):
        return None
    kv = {}
    for ln in open(path):
        if "=" in ln and not ln.lstrip().startswith("#"):
            k, v = ln.split("=", 1)
            kv[k.strip()] = v.strip()
    if kv.get("kernel_source_sha256_16") != kernel_source_hash(kind):
        return None
    return kv


def measured_traffic(workload: str, kind: str = "dense"):
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, calibrated) of a routed
    720P kernel from its committed profile, or None (see counter_profile)."""
    kv = counter_profile(workload, kind)
    return None if kv is None else float(kv["hbm_bytes_per_launch"])


def parse():
    p = argparse.ArgumentParser(description=__doc__.split("\n")[0])
    p.add_argument("--gpus", type=int, default=1)
    p.add_argument("--steps", type=int, default=10)
    p.add_argument("--warmup", type=int, default=3)
    p.add_argument("--workload", default="720p", choices=["480p", "720p", "1080p"])
    p.add_argument("--no-cpu-baseline", action="store_true")
    p.add_argument("--cpu-rows", type=int, default=None,
                   help="query rows per head in the CPU oracle sample (default 1024; "
                        "2048 at 1080P)")
    p.add_argument("--spatial-cell", type=int, default=10,
                   help="cell size of the cell variant of the Spatial path, timed as an "
                        "extra routed step (0: skip)")
    p.add_argument("--no-sd2", action="store_true",
                   help="skip the extra routed step with two-block Sink / Dummy heads")
    p.add_argument("--no-paths", action="store_true",
                   help="skip the per-path isolation runs (every layer all Sink/Dummy, "
                        "then all Spatial; all Global is the full-window step)")
    p.add_argument("--no-workloads", action="store_true",
                   help="skip the routed and full-window steps of the other latent grids "
                        "(the `workloads` object of the JSON line)")
    p.add_argument("--prewarm-s", type=float, default=1.0,
                   help="seconds of untimed routed + full-window steps before the first measurement")
    p.add_argument("--no-fallback", action="store_true",
                   help="skip the routed step on queries scaled by 40, whose logits put every "
                        "work group on the running-max pass")
    p.add_argument("--ar-loop", type=int, default=0, metavar="BLOCKS",
                   help="also run the autoregressive schedule over BLOCKS blocks of 4 "
                        "denoising steps (full-window while the window fills, the "
                        "workload's head tables from then on) and report ms per block")
    return p.parse_args()


def seed_of(w, layer, tensor):
    return (w.seed * 1000 + layer) * 16 + tensor


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU only; --gpus {args.gpus} is not supported "
              "(the routed-attention path runs on a single MI355X).", file=sys.stderr)
        sys.exit(2)
    import torch
    assert torch.cuda.is_available(), "bench.py needs a GPU"
    out = measure(args.workload, args, primary=True)
    if not args.no_workloads:
        others = {}
        for wl in ("480p", "720p", "1080p"):
            if wl != args.workload:
                torch.cuda.empty_cache()
                others[wl] = measure(wl, args, primary=False)
        out["workloads"] = others
    print(json.dumps(out), flush=True)


def measure(workload, args, primary):
    """Routed and full-window steps of one workload.  The primary workload gives
    the whole JSON line (variants, per-path and per-layer figures, the
    classification and the CPU baseline); the others a compact entry."""
    import numpy as np
    import torch

    from paper_2607_20125_amd import costs as C
    from paper_2607_20125_amd import headcast as hcb

    dev = torch.device("cuda:0")
    w = S.WORKLOADS[workload]
    H, L, d, W = w.n_heads, w.block_tokens, w.head_dim, w.window_blocks
    NL = w.n_layers
    types = S.head_types(w)
    all_g = np.full(H, S.GLOBAL, np.uint8)
    cur = W - 1
    cfg = hcb.config_from_workload(w)
    routed = hcb.Context(cfg, 0)
    full = hcb.Context(cfg, 0)

    t_setup = time.time()
    q, kb, vb = [], [], []
    keep = None
    for layer in range(NL):
        kw = S.device_normal_bf16((H, W * L, d), seed_of(w, layer, 1), dev)
        vw = S.device_normal_bf16((H, W * L, d), seed_of(w, layer, 2), dev)
        routed.set_head_types(layer, types[layer], cur, kw, vw)
        full.set_head_types(layer, all_g, cur, kw, vw)
        q.append(S.device_normal_bf16((H, L, d), seed_of(w, layer, 3), dev))
        kb.append(S.device_normal_bf16((H, L, d), seed_of(w, layer, 4), dev))
        vb.append(S.device_normal_bf16((H, L, d), seed_of(w, layer, 5), dev))
        if layer == 0:
            keep = (kw, vw)
        else:
            del kw, vw
    # a device copy of known size, outside the timed region: profiler byte
    # counters of the kernels are scaled by what the same counters read for it
    calib = torch.empty(CALIB_BYTES // 4, dtype=torch.float32, device=dev)
    calib.copy_(torch.empty_like(calib))
    del calib
    torch.cuda.synchronize()
    print(f"# {workload} setup {time.time() - t_setup:.1f}s: {NL} layers, routed buffers "
          f"{routed.memory_bytes() / 2**30:.2f} GiB, full-window buffers "
          f"{full.memory_bytes() / 2**30:.2f} GiB", file=sys.stderr, flush=True)
    o = torch.empty((H, L, d), dtype=torch.float32, device=dev)

    def step(ctx, tables, qs=None):
        qs = q if qs is None else qs
        for layer in range(NL):
            ctx.append_block(layer, cur, kb[layer], vb[layer])
            ctx.attention(layer, qs[layer], tables[layer], o)

    def timed(ctx, tables, qs=None):
        """ms per step over `steps` steps with the library's per-launch events off
        (their host cost would show at small workloads), then the same number of
        steps with them on for the per-kernel launch averages."""
        for _ in range(args.warmup):
            step(ctx, tables, qs)
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(args.steps):
            step(ctx, tables, qs)
        e1.record()
        torch.cuda.synchronize()
        ms = e0.elapsed_time(e1) / args.steps
        for k in range(hcb.K_COMBINE + 1):
            ctx.profile_read(k)              # reset
        ctx.profile_enable(True)
        for _ in range(args.steps):
            step(ctx, tables, qs)
        torch.cuda.synchronize()
        ctx.profile_enable(False)
        prof = {k: ctx.profile_read(k)
                for k in (hcb.K_DENSE, hcb.K_SPATIAL, hcb.K_SCATTER, hcb.K_COMBINE)}
        return ms, prof

    # A fresh GPU takes a while to reach its steady clock under this load: about
    # a second of untimed routed and full-window steps first, so that neither
    # measurement below (each with its own warm-up) carries the ramp.
    if primary and args.prewarm_s > 0:
        t_end = time.perf_counter() + args.prewarm_s
        while time.perf_counter() < t_end:
            step(routed, types)
            step(full, [all_g] * NL)
            torch.cuda.synchronize()
    ms_routed, prof_r = timed(routed, types)
    print(f"# {workload} routed: {ms_routed:.3f} ms/step", file=sys.stderr, flush=True)
    ms_full, prof_f = timed(full, [all_g] * NL)
    print(f"# {workload} full-window: {ms_full:.3f} ms/step", file=sys.stderr, flush=True)

    geo = (w.grid_h, w.grid_w, w.frames_per_block, W)
    r = w.spatial_radius
    fl_routed = sum(C.layer_flops(types[l], *geo, r, d) for l in range(NL))
    fl_dense = sum(C.layer_flops(types[l], *geo, r, d, kinds=(S.SINK, S.DUMMY, S.GLOBAL))
                   for l in range(NL))
    by_sp = sum(C.layer_bytes(types[l], *geo, d, kinds=(S.SPATIAL,)) for l in range(NL))
    fl_sp = sum(C.layer_flops(types[l], *geo, r, d, kinds=(S.SPATIAL,)) for l in range(NL))
    fl_full = NL * C.layer_flops(all_g, *geo, r, d)
    by_app = C.append_bytes(H, w.grid_h, w.grid_w, w.frames_per_block, d)

    def per_launch(prof, kind, work_per_step):
        ms, n = prof[kind]
        if n == 0:
            return None, None
        avg_ms = ms / n
        work = work_per_step * args.steps / n
        return avg_ms, work

    dense_ms, dense_fl = per_launch(prof_r, hcb.K_DENSE, fl_dense)
    sp_ms, sp_by = per_launch(prof_r, hcb.K_SPATIAL, by_sp)
    _, sp_fl = per_launch(prof_r, hcb.K_SPATIAL, fl_sp)
    full_ms, full_fl = per_launch(prof_f, hcb.K_DENSE, fl_full)
    dense_tf = dense_fl / (dense_ms * 1e-3) / 1e12
    full_tf = full_fl / (full_ms * 1e-3) / 1e12
    sp_gbs = sp_by / (sp_ms * 1e-3) / 1e9 if sp_ms else None

    if not primary:
        routed.close()
        full.close()
        del q, kb, vb, keep
        entry = {
            "config": {"grid": [w.grid_h, w.grid_w], "block_tokens": L, "window_blocks": W,
                       "window_tokens": W * L, "head_mix_sink_dummy_spatial_global": list(w.mix)},
            "routed_ms_per_layer_step": round(ms_routed / NL, 4),
            "full_window_ms_per_layer_step": round(ms_full / NL, 4),
            "speedup_vs_full": round(ms_full / ms_routed, 3),
            "ideal_speedup_flops": round(fl_full / fl_routed, 3),
            "tflops": round(fl_routed / (ms_routed * 1e-3) / 1e12, 2),
            "dense_roofline_frac": round(dense_tf / PEAK_BF16_TFLOPS, 4),
            "dense_tflops": round(dense_tf, 2), "dense_avg_launch_ms": round(dense_ms, 4),
            "full_window_dense_frac": round(full_tf / PEAK_BF16_TFLOPS, 4),
            "spatial_roofline_frac": sp_gbs and round(sp_gbs / PEAK_HBM_GBS, 4),
            "spatial_GB/s": sp_gbs and round(sp_gbs, 1),
            "spatial_avg_launch_ms": sp_ms and round(sp_ms, 4),
        }
        if not args.no_cpu_baseline:
            rows = args.cpu_rows or (2048 if workload == "1080p" else 1024)
            q0 = S.device_normal_bf16((H, L, d), seed_of(w, 0, 3), dev)
            kw = S.device_normal_bf16((H, W * L, d), seed_of(w, 0, 1), dev)
            vw = S.device_normal_bf16((H, W * L, d), seed_of(w, 0, 2), dev)
            entry["cpu_baseline"] = cpu_baseline(w, types[0], q0, kw, vw, rows)
            del q0, kw, vw
        print(f"# {workload}: {json.dumps(entry)}", file=sys.stderr, flush=True)
        return entry

    # the same routed step on queries scaled by 40: logits of ~60 log2 units
    # spread overflow the fixed-offset pass in every work group, so every
    # group runs its keys a second time with the running max (not part of `value`)
    fallback = None
    if not args.no_fallback:
        q40 = [(t.float() * 40.0).to(torch.bfloat16) for t in q]
        ms_fb, prof_fb = timed(routed, types, q40)
        del q40
        fb_dense, _ = per_launch(prof_fb, hcb.K_DENSE, 0.0)
        fb_sp, _ = per_launch(prof_fb, hcb.K_SPATIAL, 0.0)
        fallback = {"ms_per_layer_step": round(ms_fb / NL, 4),
                    "slowdown_vs_value": round(ms_fb / ms_routed, 3),
                    "dense_avg_launch_ms": fb_dense and round(fb_dense, 4),
                    "spatial_avg_launch_ms": fb_sp and round(fb_sp, 4),
                    "note": "routed step on queries scaled by 40 (logits ~60 log2 units "
                            "spread): every work group fails the fixed-offset check and "
                            "reruns its keys with the running max"}
        print(f"# routed, fall-back pass: {ms_fb:.3f} ms/step", file=sys.stderr, flush=True)

    # the same routed step captured once into a HIP graph and replayed: the
    # library only enqueues kernels at a fixed window fill (not part of `value`)
    def graph_timed(ctx, tables):
        g = torch.cuda.CUDAGraph()
        torch.cuda.synchronize()
        with torch.cuda.graph(g):
            step(ctx, tables)
        for _ in range(args.warmup):
            g.replay()
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(args.steps):
            g.replay()
        e1.record()
        torch.cuda.synchronize()
        del g
        return e0.elapsed_time(e1) / args.steps

    ms_graph = graph_timed(routed, types)
    print(f"# routed, graph replay: {ms_graph:.3f} ms/step", file=sys.stderr, flush=True)

    # per-layer distribution of the routed step: events around every layer's
    # append + attention, over a few extra steps (not part of `value`)
    def per_layer(ctx, tables, reps=3):
        evs = [[(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
                for _ in range(NL)] for _ in range(reps)]
        for rep in range(reps):
            for layer in range(NL):
                e0, e1 = evs[rep][layer]
                e0.record()
                ctx.append_block(layer, cur, kb[layer], vb[layer])
                ctx.attention(layer, q[layer], tables[layer], o)
                e1.record()
        torch.cuda.synchronize()
        per = [statistics.median(evs[rep][l][0].elapsed_time(evs[rep][l][1]) for rep in range(reps))
               for l in range(NL)]
        qs = np.percentile(per, [10, 50, 90])
        return {"median": round(float(qs[1]), 4), "p10": round(float(qs[0]), 4),
                "p90": round(float(qs[2]), 4), "mean": round(sum(per) / NL, 4)}

    layer_stats = {"routed": per_layer(routed, types), "full_window": per_layer(full, [all_g] * NL)}

    # the same routed step with a variant of the paths (same inputs)
    full.close()

    def variant(label, **cfg_kw):
        ctx = hcb.Context(hcb.config_from_workload(w, **cfg_kw), 0)
        for layer in range(NL):
            kw = S.device_normal_bf16((H, W * L, d), seed_of(w, layer, 1), dev)
            vw = S.device_normal_bf16((H, W * L, d), seed_of(w, layer, 2), dev)
            ctx.set_head_types(layer, types[layer], cur, kw, vw)
            del kw, vw
        torch.cuda.synchronize()
        ms, prof = timed(ctx, types)
        print(f"# routed, {label}: {ms:.3f} ms/step", file=sys.stderr, flush=True)
        ctx.close()
        return ms, prof

    ar = None
    if args.ar_loop > 0:
        from paper_2607_20125_amd import ar_loop
        pool = [(S.device_normal_bf16((H, L, d), seed_of(w, l, 6), dev),
                 S.device_normal_bf16((H, L, d), seed_of(w, l, 7), dev),
                 S.device_normal_bf16((H, L, d), seed_of(w, l, 8), dev)) for l in range(NL)]
        data = lambda layer, b, si: pool[layer]
        runs = {}
        for label, tables in (("routed", types), ("full_window", [all_g] * NL)):
            ctx = hcb.Context(cfg, 0)
            res = ar_loop.run(ctx, args.ar_loop, data, o, classify=False, tables_at_fill=tables)
            ctx.close()
            runs[label] = [round(x, 3) for x in res.ms_per_block]
            print(f"# AR loop {label}: ms per block {runs[label]}", file=sys.stderr, flush=True)
        steady = lambda xs: sum(xs[W:]) / max(len(xs[W:]), 1)
        ar = {"blocks": args.ar_loop, "steps_per_block": len(ar_loop.TIMESTEPS),
              "ms_per_block_routed": runs["routed"], "ms_per_block_full_window": runs["full_window"],
              "steady_speedup": round(steady(runs["full_window"]) / steady(runs["routed"]), 3)
              if args.ar_loop > W else None,
              "note": "attention + appends only (no model); head tables installed when the "
                      "window first fills; classification timed separately"}
        del pool

    ms_cell = prof_c = ms_sd2 = prof_s2 = None
    if args.spatial_cell > 0:
        ms_cell, prof_c = variant(f"{args.spatial_cell}x{args.spatial_cell} Spatial cells",
                                  spatial_cell=args.spatial_cell)
    if not args.no_sd2:
        ms_sd2, prof_s2 = variant("two-block Sink/Dummy", sd_blocks=2)

    # per-path isolation: every layer's table homogeneous, so one path runs
    paths = None
    if not args.no_paths:
        sd_tab = np.array([S.SINK, S.DUMMY] * (H // 2) + [S.SINK] * (H % 2), np.uint8)
        sp_tab = np.full(H, S.SPATIAL, np.uint8)
        paths = {}
        for label, tab in (("sink_dummy", sd_tab), ("spatial", sp_tab)):
            ctx = hcb.Context(cfg, 0)
            for layer in range(NL):
                kw = S.device_normal_bf16((H, W * L, d), seed_of(w, layer, 1), dev)
                vw = S.device_normal_bf16((H, W * L, d), seed_of(w, layer, 2), dev)
                ctx.set_head_types(layer, tab, cur, kw, vw)
                del kw, vw
            torch.cuda.synchronize()
            ms_p, prof_p = timed(ctx, [tab] * NL)
            ctx.close()
            paths[label] = (ms_p, prof_p, tab)
            print(f"# all layers {label}: {ms_p:.3f} ms/step", file=sys.stderr, flush=True)

    app_ms, app_by = per_launch(prof_r, hcb.K_SCATTER, NL * by_app)

    roofline = {"kernel": "attn_dense (Global + Sink/Dummy work items of the routed step)",
                "bound": "mfma", "achieved": round(dense_tf, 2), "peak": PEAK_BF16_TFLOPS,
                "unit": "TFLOP/s", "frac": round(dense_tf / PEAK_BF16_TFLOPS, 4),
                "traffic": measured_traffic(workload), "avg_launch_ms": round(dense_ms, 4),
                "flop_per_launch": dense_fl}
    extra = {}
    if sp_ms:
        gbs = sp_gbs
        extra["roofline_spatial"] = {
            "kernel": "attn_spatial", "bound": "hbm", "achieved": round(gbs, 1),
            "peak": PEAK_HBM_GBS, "unit": "GB/s", "frac": round(gbs / PEAK_HBM_GBS, 4),
            "traffic": measured_traffic(workload, "spatial"),
            "avg_launch_ms": round(sp_ms, 4), "compulsory_bytes_per_launch": sp_by,
            "tflops_algorithmic": round(sp_fl / (sp_ms * 1e-3) / 1e12, 2)}
        kv = counter_profile(workload, "spatial")
        if kv is not None:
            # matrix work the kernel issues (SQ_INSTS_MFMA x 32768 flops) over the
            # in-window pairs' 4 d flops: masked scores of the rectangular tiles
            extra["roofline_spatial"]["mfma_executed_over_algorithmic"] = float(
                kv["mfma_executed_over_algorithmic"])
    extra["graph_replay"] = {
        "ms_per_layer_step": round(ms_graph / NL, 4),
        "note": "the routed step captured once into a HIP graph and replayed (no host launch cost)"}
    extra["full_window_dense"] = {
        "kernel": "attn_dense (all heads Global)", "bound": "mfma",
        "achieved": round(full_tf, 2), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
        "frac": round(full_tf / PEAK_BF16_TFLOPS, 4), "avg_launch_ms": round(full_ms, 4)}
    if app_ms:
        extra["append"] = {"avg_launch_ms": round(app_ms, 4),
                           "GB/s": round(app_by / (app_ms * 1e-3) / 1e9, 1)}
    if ms_cell:
        fl_cell = sum(C.layer_flops(types[l], *geo, r, d, cell=args.spatial_cell)
                      for l in range(NL))
        cd_ms, _ = per_launch(prof_c, hcb.K_DENSE, 0.0)
        extra["cell_variant"] = {
            "spatial_cell": args.spatial_cell,
            "ms_per_layer_step": round(ms_cell / NL, 4),
            "speedup_vs_full": round(ms_full / ms_cell, 3),
            "ideal_speedup_flops": round(fl_full / fl_cell, 3),
            "tflops": round(fl_cell / (ms_cell * 1e-3) / 1e12, 2),
            "dense_avg_launch_ms": cd_ms and round(cd_ms, 4),
            "note": "Spatial heads attend to their own cell in every window frame "
                    "(Sec. 4.4 deployed form); cells run as dense units of attn_dense"}
    if ms_sd2:
        fl_sd2 = sum(C.layer_flops(types[l], *geo, r, d, sd_blocks=2) for l in range(NL))
        extra["sd2_variant"] = {
            "ms_per_layer_step": round(ms_sd2 / NL, 4),
            "speedup_vs_full": round(ms_full / ms_sd2, 3),
            "ideal_speedup_flops": round(fl_full / fl_sd2, 3),
            "tflops": round(fl_sd2 / (ms_sd2 * 1e-3) / 1e12, 2),
            "note": "Sink = block 0 + current, Dummy = previous + current (App. B / C)"}
    if fallback:
        extra["fallback"] = fallback
    if ar:
        extra["ar_loop"] = ar
    extra["per_layer_ms"] = {**layer_stats, "note": "routed / full-window append + attention "
                             "per layer, median of 3 steps per layer, then p10/p50/p90 over "
                             "the layers"}
    if paths:
        iso = {"global": {"ms_per_layer_step": round(ms_full / NL, 4),
                          "dense_tflops": round(full_tf, 2), "note": "the full-window step"}}
        for label, (ms_p, prof_p, tab) in paths.items():
            fl_p = NL * C.layer_flops(tab, *geo, r, d)
            entry = {"ms_per_layer_step": round(ms_p / NL, 4),
                     "tflops_algorithmic": round(fl_p / (ms_p * 1e-3) / 1e12, 2)}
            if label == "spatial":
                s_ms, s_by = per_launch(prof_p, hcb.K_SPATIAL, NL * C.layer_bytes(tab, *geo, d))
                entry["spatial_avg_launch_ms"] = round(s_ms, 4)
                entry["spatial_compulsory_GB/s"] = round(s_by / (s_ms * 1e-3) / 1e9, 1)
            else:
                p_ms, p_fl = per_launch(prof_p, hcb.K_DENSE, fl_p)
                entry["dense_avg_launch_ms"] = round(p_ms, 4)
                entry["dense_tflops"] = round(p_fl / (p_ms * 1e-3) / 1e12, 2)
            iso[label] = entry
        extra["paths"] = iso
    comb_r, _ = per_launch(prof_r, hcb.K_COMBINE, 0.0)
    comb_f, _ = per_launch(prof_f, hcb.K_COMBINE, 0.0)
    extra["combine"] = {"routed_avg_launch_ms": comb_r and round(comb_r, 4),
                        "full_window_avg_launch_ms": comb_f and round(comb_f, 4)}

    # one-time classification of one layer (synchronising call), second call timed
    cls = hcb.Context(hcb.config_from_workload(w, n_layers=1), 0)
    kw, vw = keep
    t_cls = []
    for _ in range(2):
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        cls.classify_heads(0, cur, q[0], kw, vw)
        t_cls.append((time.perf_counter() - t0) * 1e3)
    cls.close()

    cpu = None
    if not args.no_cpu_baseline:
        rows = args.cpu_rows or (2048 if workload == "1080p" else 1024)
        cpu = cpu_baseline(w, types[0], q[0], kw, vw, rows)
    del keep, kw, vw
    routed.close()

    tflops = fl_routed / (ms_routed * 1e-3) / 1e12
    out = {
        "metric": METRIC,
        "value": round(ms_routed / NL, 4),
        "unit": "ms/layer-step",
        "n_gpus": 1, "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(ms_routed, 3),
        "higher_is_better": False,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic (N(0,1) bf16 drawn on device; random-init, no model weights)",
        "config": {"workload": f"{workload} Wan-1.3B-shaped routed attention",
                   "layers": NL, "heads": H, "head_dim": d,
                   "grid": [w.grid_h, w.grid_w], "frames_per_block": w.frames_per_block,
                   "block_tokens": L, "window_blocks": W, "window_tokens": W * L,
                   "spatial_radius": r, "head_mix_sink_dummy_spatial_global": list(w.mix),
                   "parallelism": "single-gpu"},
        "tflops": round(tflops, 2),
        "mfma_frac_of_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
        "full_window_ms_per_layer_step": round(ms_full / NL, 4),
        "speedup_vs_full": round(ms_full / ms_routed, 3),
        "ideal_speedup_flops": round(fl_full / fl_routed, 3),
        "classify_ms_per_layer": round(t_cls[-1], 2),
        "roofline": roofline,
        **extra,
        "cpu_baseline": cpu,
        "device": torch.cuda.get_device_name(0),
    }
    return out


def cpu_baseline(w, types, q_dev, kw_dev, vw_dev, rows_per_head):
    """The oracle on a bounded sample of layer 0: `rows_per_head` query rows of
    every head, scaled to all L rows (oracle cost is linear in the rows)."""
    import numpy as np
    import torch

    from oracle import headcast_oracle as O

    bits = lambda t: t.view(torch.int16).cpu().numpy().view(np.uint16)
    q, k, v = bits(q_dev), bits(kw_dev), bits(vw_dev)
    L = w.block_tokens
    rows = np.sort(np.random.default_rng(0).choice(L, size=min(rows_per_head, L), replace=False))
    # every CPU this process may run on (the CPU affinity set; os.cpu_count()
    # counts the whole host, which a container's share can be far below)
    host_cpus = os.cpu_count() or 1
    usable = len(os.sched_getaffinity(0)) if hasattr(os, "sched_getaffinity") else host_cpus
    prev = torch.get_num_threads()
    torch.set_num_threads(usable)
    per_rep = []
    try:
        for _ in range(3):
            t0 = time.perf_counter()
            O.routed_attention(types, q, k, v, w.grid_h, w.grid_w, w.frames_per_block,
                               w.spatial_radius, rows=rows)
            per_rep.append(time.perf_counter() - t0)
        used = torch.get_num_threads()
    finally:
        torch.set_num_threads(prev)
    med = statistics.median(per_rep)
    ms_layer = med * 1e3 * L / rows.size
    return {"value": round(ms_layer, 1), "unit": "ms/layer-step", "cores": used,
            "host_cpus": host_cpus, "affinity_cpus": usable, "kind": "oracle",
            "sample": f"layer 0 of the same workload: {rows.size} of {L} query rows per head "
                      f"x {w.n_heads} heads (fp64), median of 3 runs of {med:.2f}s, "
                      f"scaled linearly to {L} rows (extrapolated)"}


if __name__ == "__main__":
    main()
