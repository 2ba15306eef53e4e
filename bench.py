"""Benchmark of the region-reuse DiT denoising step on one MI355X.

Workload: the 28-block PixArt-alpha-shaped model at 1024 px (latent
4x128x128 -> 64x64 = 4096 tokens), bf16, a 20-step sampler schedule with
timesteps linearly spaced 999 -> 0, and an edit mask of seeded elliptical
blobs covering 10-20 % of the tokens.  Turn 0 fills the cache pool with 20
dense steps; turn 1 (new prompt with edited tokens) runs 4 dense steps and 16
region-reuse steps.  Everything is synthetic and seeded (random-init weights,
N(0,1) text features and latents).

One timed "step" is one region-reuse denoising step of turn 1 (gather + patch
embedding, 28 blocks with the fused K/V scatter and the merge into the cached
hidden state, final layer, DDIM update of the active patches).  The line also
reports the dense step, the speedup of reuse over dense, and the whole 20-step
editing turn (text preparation, 4 dense steps with map emission, edit-region
localisation, 16 reuse steps) against an all-dense turn; without --quick also
the 1024 px localisation read-out from raw logits, a batch-4 active-fraction
sweep and a 512/1024/2048 px resolution sweep.

Prints ONE JSON line.  `--gpus` above 1 is not supported (single-GPU build).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "DiT denoising steps/sec at 1024px, 10-20% active tokens; speedup vs dense"
PEAK_BF16_TFLOPS = 2500.0
PEAK_HBM_GBS = 8000.0


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=32)
    ap.add_argument("--warmup", type=int, default=4)
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--frac", type=float, default=None, help="active fraction (default: seeded in [0.10, 0.20])")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-layers", type=int, default=28, help="blocks in the oracle timing sample (28: the whole step)")
    ap.add_argument("--quick", action="store_true", help="skip the schedule legs (profiling runs)")
    ap.add_argument("--graph", action="store_true",
                    help="replay one captured HIP graph per reuse step instead of host launches")
    ap.add_argument("--copy-calibrate", type=int, default=0, metavar="MIB",
                    help="only run one plain device-to-device copy of MIB MiB (HBM counter calibration)")
    return ap.parse_args()


def log(*a):
    print(*a, file=sys.stderr, flush=True)


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: only --gpus 1 is supported; the library runs one process on one GPU (asked for {args.gpus})",
              file=sys.stderr)
        sys.exit(2)
    import torch
    if args.copy_calibrate:
        n = args.copy_calibrate * (1 << 20) // 4
        x = torch.ones(n, dtype=torch.float32, device="cuda")
        y = torch.empty_like(x)
        torch.cuda.synchronize()
        y.copy_(x)
        torch.cuda.synchronize()
        print(json.dumps({"copy_bytes_read": n * 4, "copy_bytes_written": n * 4}))
        return
    import synth
    from paper_2608_29809_amd import abi
    from paper_2608_29809_amd.runtime import ActiveSet, RegionCacheModel

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    dev = "cuda"
    shape = synth.shape_c3()
    T = 20
    n_dense = 4                        # floor(0.2 * 20) dense steps, the rest reuse
    tgrid = synth.timestep_grid(T)
    mask, frac, n_blobs = synth.c3_edit_region(args.seed, args.frac)
    idx = np.flatnonzero(mask)
    R = int(idx.size)
    log(f"workload: 1024px, {shape.layers} blocks, N={shape.tokens}, R={R} ({R / shape.tokens:.1%}), blobs={n_blobs}")

    t0 = time.time()
    W = synth.make_weights(shape, seed=args.seed)
    model = RegionCacheModel(shape, W)
    cache = model.alloc_cache(1, T)
    txt0 = synth.make_text(shape, 1, args.seed)
    txt1, delta = synth.edit_text(shape, txt0, 5, args.seed)
    noise = torch.from_numpy(synth.make_latent(shape, 1, args.seed)).to(dev)
    tkv0 = model.prepare_text(model.to_storage(txt0))
    lat = [torch.empty_like(noise) for _ in range(T + 1)]
    lat[0].copy_(noise)
    for s in range(T):  # turn 0: dense trajectory fills the cache pool
        tn = int(tgrid[s + 1]) if s + 1 < T else -1
        model.build_cache(cache, s, lat[s], int(tgrid[s]), tn, tkv0, latent_out=lat[s + 1])
    torch.cuda.synchronize()
    log(f"setup + turn 0 in {time.time() - t0:.1f}s")

    act = ActiveSet.from_lists([idx])
    tkv1 = model.prepare_text(model.to_storage(txt1))
    maps = torch.zeros((1, shape.tokens, len(delta)), device=dev)
    lat1 = [torch.empty_like(noise) for _ in range(T + 1)]
    lat1[0].copy_(noise)
    for s in range(n_dense):
        model.build_cache(cache, s, lat1[s], int(tgrid[s]), int(tgrid[s + 1]), tkv1, delta,
                          maps if s == n_dense - 1 else None, lat1[s + 1])
    torch.cuda.synchronize()

    reuse_steps = list(range(n_dense, T))

    def reuse(k):
        s = reuse_steps[k % len(reuse_steps)]
        tn = int(tgrid[s + 1]) if s + 1 < T else -1
        model.reuse_step(cache, s, act, lat1[s], int(tgrid[s]), tn, tkv1, latent_out=lat1[s + 1])

    def dense(k):
        s = reuse_steps[k % len(reuse_steps)]
        tn = int(tgrid[s + 1]) if s + 1 < T else -1
        model.build_cache(cache, s, lat1[s], int(tgrid[s]), tn, tkv1, latent_out=lat1[s + 1])

    def time_loop(fn, steps, warmup):
        for k in range(warmup):
            fn(k)
        torch.cuda.synchronize()
        ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        w0 = time.perf_counter()
        ev0.record()
        for k in range(steps):
            fn(k)
        ev1.record()
        torch.cuda.synchronize()
        wall = time.perf_counter() - w0
        return ev0.elapsed_time(ev1) / 1000.0, wall

    # ---------------------------------------------------------------- headline: reuse steps
    # The active set is fixed for the 16 reuse steps of a turn, so every
    # launch of a reuse step is known after localisation: each step is
    # captured once into a HIP graph (kernel nodes only) and replayed.
    t_eager, _ = time_loop(reuse, args.steps, args.warmup)
    ms_eager = 1000.0 * t_eager / args.steps
    log(f"reuse step (host launches): {ms_eager:.3f} ms ({args.steps / t_eager:.1f} steps/s)")
    graphs = None
    if args.graph:
        graphs = []
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for k in range(len(reuse_steps)):
                gr = torch.cuda.CUDAGraph()
                with torch.cuda.graph(gr, stream=side):
                    reuse(k)
                graphs.append(gr)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()

        def reuse_graph(k):
            graphs[k % len(graphs)].replay()

        t_reuse, wall_reuse = time_loop(reuse_graph, args.steps, args.warmup)
    else:
        t_reuse, wall_reuse = t_eager, 0.0
    ms_reuse = 1000.0 * t_reuse / args.steps
    log(f"reuse step: {ms_reuse:.3f} ms ({args.steps / t_reuse:.1f} steps/s; wall {wall_reuse:.3f}s)")

    # ---------------------------------------------------------------- dense steps
    n_d = max(4, args.steps // 4)
    t_dense, _ = time_loop(dense, n_d, 2)
    ms_dense = 1000.0 * t_dense / n_d
    log(f"dense step: {ms_dense:.3f} ms")

    # ---------------------------------------------------------------- per-kernel timing (HIP events)
    model.set_kernel_timing(True)
    n_prof = max(4, min(args.steps, 16))
    for k in range(n_prof):
        reuse(k)
    torch.cuda.synchronize()
    per = {}
    for c, name in enumerate(abi.KERNEL_CLASSES):
        ms, n = model.kernel_timing(c)
        if n:
            per[name] = dict(total_ms=ms / n_prof, launches=n // n_prof, avg_us=1000.0 * ms / n)
    model.set_kernel_timing(False)
    log("per-step kernel time by class: " + ", ".join(f"{k} {v['total_ms']:.3f}ms/{v['launches']}"
                                                      for k, v in sorted(per.items(), key=lambda kv: -kv[1]['total_ms'])))

    # the dense step's kernel classes, for the vendor comparison below
    model.set_kernel_timing(True)
    for k in range(4):
        dense(k)
    torch.cuda.synchronize()
    per_dense = {}
    for c, name in enumerate(abi.KERNEL_CLASSES):
        ms, n = model.kernel_timing(c)
        if n:
            per_dense[name] = dict(total_ms=ms / 4, launches=n // 4, avg_us=1000.0 * ms / n)
    model.set_kernel_timing(False)
    vendor = None if args.quick else vendor_leg(shape, R, per, per_dense, ms_reuse, ms_dense)

    C, N, F, M = shape.hidden, shape.tokens, shape.mlp, shape.text_len
    work = class_work(shape, R, 1)
    by_class = {}
    for k, w in work.items():
        if k not in per:
            continue
        sec = per[k]["avg_us"] * 1e-6
        e = dict(bound=w["bound"], avg_launch_us=round(per[k]["avg_us"], 3), launches_per_step=per[k]["launches"],
                 flops_per_launch=w["flops"], bytes_per_launch=w["bytes"],
                 tflops=round(w["flops"] / sec / 1e12, 2), gbs=round(w["bytes"] / sec / 1e9, 1))
        e["frac"] = round(e["tflops"] / PEAK_BF16_TFLOPS if w["bound"] == "mfma" else e["gbs"] / PEAK_HBM_GBS, 4)
        by_class[k] = e
    mfma_classes = [k for k in by_class if by_class[k]["bound"] == "mfma"]
    dom = max(mfma_classes, key=lambda k: per[k]["total_ms"])
    achieved = by_class[dom]["tflops"]
    traffic = _committed_traffic(dom, R)
    roofline = dict(bound="mfma", kernel=dom, achieved=achieved, peak=PEAK_BF16_TFLOPS,
                    unit="TFLOP/s", frac=round(achieved / PEAK_BF16_TFLOPS, 4), traffic=traffic,
                    flops_per_launch=work[dom]["flops"], avg_launch_us=by_class[dom]["avg_launch_us"])
    log("roofline by class: " + ", ".join(f"{k} {v['frac']:.3f}" for k, v in sorted(by_class.items(), key=lambda kv: -per[kv[0]]["total_ms"])))

    # ---------------------------------------------------------------- whole editing turn
    schedule = None
    if not args.quick:
        def turn(all_dense: bool):
            tk = model.prepare_text(model.to_storage(txt1))
            mp = torch.zeros((1, shape.tokens, len(delta)), device=dev)
            for s in range(T):
                tn = int(tgrid[s + 1]) if s + 1 < T else -1
                if all_dense or s < n_dense:
                    model.build_cache(cache, s, lat1[s], int(tgrid[s]), tn, tk, delta,
                                      mp if s == n_dense - 1 else None, lat1[s + 1])
                    if s == n_dense - 1 and not all_dense:
                        model.localize(mp, len(delta), 0.3, 1)  # the region read-out of Sec. 3.2
                else:
                    model.reuse_step(cache, s, act, lat1[s], int(tgrid[s]), tn, tk, latent_out=lat1[s + 1])

        turn(False)
        torch.cuda.synchronize()
        w0 = time.perf_counter()
        turn(False)
        torch.cuda.synchronize()
        t_turn = time.perf_counter() - w0
        w0 = time.perf_counter()
        turn(True)
        torch.cuda.synchronize()
        t_turn_dense = time.perf_counter() - w0
        schedule = dict(turn_s=round(t_turn, 5), all_dense_turn_s=round(t_turn_dense, 5),
                        steps_per_s=round(T / t_turn, 2), speedup_vs_all_dense=round(t_turn_dense / t_turn, 3),
                        plan="4 dense (maps at step 3) + localisation + 16 reuse")
        log(f"turn: {t_turn * 1000:.1f} ms vs all-dense {t_turn_dense * 1000:.1f} ms")

    # ---------------------------------------------------------------- host-resident pool
    hosted = None
    if not args.quick:
        hosted = hosted_leg(model, shape, cache, act, lat1, tgrid, tkv1, n_dense, ms_reuse, R)

    # ---------------------------------------------------------------- localisation workload
    loc = None
    sweep = None
    res = None
    if not args.quick:
        loc = localize_leg(args)
        del cache
        torch.cuda.empty_cache()
        sweep = sweep_leg(model, args)
        res = resolution_leg(W, args)

    # ---------------------------------------------------------------- oracle on the host cores
    cpu = None
    if not args.no_cpu_baseline:
        cpu = cpu_baseline(shape, W, idx, args)
        if not args.quick:
            cpu["by_config"] = cpu_baseline_configs(shape, W, args)

    value = args.steps / t_reuse
    out = {
        "metric": METRIC,
        "value": round(value, 3),
        "unit": "steps/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_reuse, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "bf16",
        "data": "synthetic",
        "config": {"workload": "1024px 28-block PixArt-alpha-shaped DiT, region-reuse denoising step",
                   "tokens": N, "active_tokens": R, "active_frac": round(R / N, 4), "blobs": n_blobs,
                   "batch": 1, "layers": shape.layers, "sampler_steps": T, "dense_steps": n_dense,
                   "parallelism": "single GPU"},
        "launch": "hip_graph_per_step" if graphs else "host",
        "host_launch_ms_per_step": round(ms_eager, 4),
        "dense_step_ms": round(ms_dense, 4),
        "dense_steps_per_s": round(1000.0 / ms_dense, 3),
        "speedup_vs_dense": round(ms_dense / ms_reuse, 3),
        "vendor_gemm_reference": vendor,
        "schedule": schedule,
        "kernels_ms_per_step": {k: round(v["total_ms"], 4) for k, v in per.items()},
        "roofline": roofline,
        "roofline_by_class": by_class,
        "localize": loc,
        "fraction_sweep": sweep,
        "resolution_sweep": res,
        "hosted_pool": hosted,
        "cpu_baseline": cpu,
        # the paper's own figures (one RTX L20, trained PixArt-alpha on editing
        # datasets, precision unstated): context for the speedups above, not a target
        "paper_context": {"hardware": "one NVIDIA RTX L20 (Sec. 4.1), precision not stated",
                          "end_to_end_speedup_range": [1.43, 2.55],
                          "table2_speedup": {"total": 1.57, "self_attention": 2.89},
                          "fig9_self_attention_speedup": {"512px": 2.7, "1024px": 4.7, "2048px": ">6"},
                          "comparable_here": ["schedule.speedup_vs_all_dense", "speedup_vs_dense",
                                              "resolution_sweep.*.speedup"]},
    }
    print(json.dumps(out), flush=True)


def vendor_leg(shape, R, per, per_dense, ms_reuse, ms_dense):
    """Each GEMM class of the step timed beside the vendor's bf16 GEMM
    (torch.mm, served by hipBLASLt) on the same shape, at the region step's R
    rows and the dense step's N rows.  The dense step is then also stated as
    if every one of its GEMMs ran at the faster of the two, and the reuse
    step's speedup against that step: a check on the dense denominator, not
    part of the path (the library runs its own kernels only)."""
    import torch
    C, N, F = shape.hidden, shape.tokens, shape.mlp
    shapes = {"gemm_qkv": (3 * C, C), "gemm_proj": (C, C), "gemm_xproj": (C, C), "gemm_fc1": (F, C),
              "gemm_fc2": (C, F)}
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def mm_us(m, n, k):
        a = torch.randn(m, k, device="cuda", dtype=torch.bfloat16)
        b = torch.randn(k, n, device="cuda", dtype=torch.bfloat16).contiguous()
        for _ in range(3):
            torch.mm(a, b)
        torch.cuda.synchronize()
        e0.record()
        for _ in range(20):
            torch.mm(a, b)
        e1.record()
        torch.cuda.synchronize()
        return 1000.0 * e0.elapsed_time(e1) / 20

    out = {"rows": {"region": R, "dense": N}, "classes": {}}
    saved_us = 0.0
    for cls, (n, k) in shapes.items():
        row = {}
        for tag, m, table in (("region", R, per), ("dense", N, per_dense)):
            v = mm_us(m, n, k)
            ours = table.get(cls, {}).get("avg_us")
            row[tag] = dict(ours_us=round(ours, 2) if ours else None, vendor_us=round(v, 2))
            if tag == "dense" and ours:
                saved_us += max(0.0, ours - v) * table[cls]["launches"]
        out["classes"][cls] = row
    dense_best = ms_dense - saved_us / 1000.0
    out["dense_step_ms_at_faster_gemms"] = round(dense_best, 4)
    out["speedup_vs_that_dense_step"] = round(dense_best / ms_reuse, 3)
    log(f"vendor GEMM check: dense step at the faster GEMM of each class {dense_best:.3f} ms "
        f"(ours {ms_dense:.3f}); reuse speedup against it {dense_best / ms_reuse:.2f}x")
    return out


def hosted_leg(model, shape, cache, act, lat1, tgrid, tkv1, s_from, ms_device, R):
    """The same 1024 px reuse step with the cache pool in pinned host memory
    (pipelined execution: per block, keys/values uploaded by the copy engine
    ahead of the compute, computed rows written back behind it).  A two-step
    pool holds the device pool's slot of step `s_from` and its trajectory
    entries; the step is timed against the device-pool step, beside a
    transfer-only pass (the 28 blocks' key/value uploads alone), which bounds
    it from below."""
    import torch
    from paper_2608_29809_amd import abi as _abi  # noqa: F401  (library loaded)

    L, H, N, C = shape.layers, shape.heads, shape.tokens, shape.hidden
    host = model.alloc_cache(1, 2, host=True)
    for l in range(L):
        host.K(0, 1, l).copy_(cache.K(0, s_from, l))
        host.V(0, 1, l).copy_(cache.V(0, s_from, l))
        host.H(0, 1, l).copy_(cache.H(0, s_from, l))
    host.latent(0, 2).copy_(cache.latent(0, s_from + 1))
    torch.cuda.synchronize()
    t, tn = int(tgrid[s_from]), int(tgrid[s_from + 1])
    out = torch.empty_like(lat1[s_from])

    def step():
        model.reuse_step(host, 1, act, lat1[s_from], t, tn, tkv1, latent_out=out)

    for _ in range(2):
        step()
    torch.cuda.synchronize()
    n = 8
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for _ in range(n):
        step()
    e1.record()
    torch.cuda.synchronize()
    ms_hosted = e0.elapsed_time(e1) / n
    kv_bytes = 2 * H * N * 72 * 2
    dst = torch.empty(kv_bytes, dtype=torch.uint8, device="cuda")
    src = [host.buf[host.offsets(0, 1, l)[0]:host.offsets(0, 1, l)[0] + kv_bytes] for l in range(L)]
    for x in src[:2]:
        dst.copy_(x, non_blocking=True)
    torch.cuda.synchronize()
    e0.record()
    for x in src:
        dst.copy_(x, non_blocking=True)
    e1.record()
    torch.cuda.synchronize()
    ms_h2d = e0.elapsed_time(e1)
    up = L * kv_bytes
    wb = L * 3 * R * C * 2
    log(f"host-resident pool: reuse step {ms_hosted:.3f} ms (device pool {ms_device:.3f} ms); "
        f"uploads alone {ms_h2d:.3f} ms ({up / ms_h2d / 1e6:.1f} GB/s)")
    return dict(pool="pinned host memory, 3-entry device staging ring",
                reuse_step_ms=round(ms_hosted, 3), device_pool_reuse_step_ms=round(ms_device, 3),
                slowdown_vs_device_pool=round(ms_hosted / ms_device, 3),
                upload_bytes_per_step=up, writeback_bytes_per_step=wb,
                uploads_alone_ms=round(ms_h2d, 3), upload_gbs=round(up / ms_h2d / 1e6, 1),
                overlap=round(ms_h2d / ms_hosted, 3))


def localize_leg(args):
    """Edit-region localisation at 1024 px: bf16 logits [28, 16, 4096, 120]
    (N(0,1), +3 on 6 delta columns over a seeded blob) -> per-token maps ->
    range-normalised threshold 0.3, union, 3x3 dilation -> mask + indices.
    The logits pass is HBM-bound; its rate is reported against 8 TB/s."""
    import torch
    import synth
    from paper_2608_29809_amd.runtime import RegionCacheModel, maps_from_logits
    gh = gw = 64
    Z, delta, blob = synth.make_logits(28, 16, gh * gw, 120, gh, gw, n_delta=6, seed=args.seed, frac=0.12)
    Zt = torch.from_numpy(Z).to(torch.bfloat16).cuda()
    del Z
    shp = synth.ModelShape(layers=1, grid_h=gh, grid_w=gw, dtype="bf16")
    m = RegionCacheModel(shp, synth.make_weights(shp, seed=0))
    for _ in range(2):
        maps = maps_from_logits(Zt, delta)
        mask, act = m.localize(maps[None].contiguous(), len(delta), 0.3, 1)
    torch.cuda.synchronize()
    e0, e1, e2 = (torch.cuda.Event(enable_timing=True) for _ in range(3))
    reps = 10
    e0.record()
    for _ in range(reps):
        maps = maps_from_logits(Zt, delta)
    e1.record()
    for _ in range(reps):
        mask, act = m.localize(maps[None].contiguous(), len(delta), 0.3, 1)  # includes one host sync
    e2.record()
    torch.cuda.synchronize()
    t_maps = e0.elapsed_time(e1) / reps
    t_loc = e1.elapsed_time(e2) / reps
    nbytes = Zt.numel() * 2
    gbs = nbytes / (t_maps * 1e-3) / 1e9
    log(f"localisation: maps {t_maps * 1000:.1f} us ({gbs:.0f} GB/s), mask+compaction {t_loc * 1000:.1f} us, "
        f"{act.total} active tokens")
    return dict(workload="logits bf16 [28,16,4096,120], 6 delta columns", maps_us=round(t_maps * 1000, 2),
                logits_gbs=round(gbs, 1), hbm_frac=round(gbs / PEAK_HBM_GBS, 4),
                mask_and_compaction_us=round(t_loc * 1000, 2), active_tokens=int(act.total))


def resolution_leg(W, args):
    """One chain at 512, 1024 and 2048 px (32x32, 64x64, 128x128 tokens), the
    28-block model (same weights, position table of the grid), a seeded
    15 % blob region: reuse-step and dense-step times."""
    import dataclasses
    import torch
    import synth
    from paper_2608_29809_amd.runtime import ActiveSet, RegionCacheModel
    out = {}
    for px, g in ((512, 32), (1024, 64), (2048, 128)):
        shape = dataclasses.replace(synth.shape_c3(), grid_h=g, grid_w=g)
        model = RegionCacheModel(shape, W)
        cache = model.alloc_cache(1, 2)
        txt = synth.make_text(shape, 1, args.seed + 2)
        tkv = model.prepare_text(model.to_storage(txt))
        lat = torch.from_numpy(synth.make_latent(shape, 1, args.seed + 2)).cuda()
        nxt = torch.empty_like(lat)
        act = ActiveSet.from_lists([synth.resolution_region(args.seed, g)])
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

        def timed(fn, n=6):
            fn()
            torch.cuda.synchronize()
            ev[0].record()
            for _ in range(n):
                fn()
            ev[1].record()
            torch.cuda.synchronize()
            return ev[0].elapsed_time(ev[1]) / n

        dense_ms = timed(lambda: model.build_cache(cache, 0, lat, 842, 789, tkv, latent_out=nxt))
        reuse_ms = timed(lambda: model.reuse_step(cache, 0, act, lat, 842, 789, tkv, latent_out=nxt))
        # bytes a reuse step must move: every block's weights once, the slot's
        # keys and values, the fresh keys, values and hidden rows written back
        C_, L_, R_ = shape.hidden, shape.layers, int(act.total)
        nbytes = L_ * 14 * C_ * C_ * 2 + 2 * L_ * g * g * C_ * 2 + 3 * L_ * R_ * C_ * 2
        gbs = nbytes / (reuse_ms * 1e-3) / 1e9
        out[f"{px}px"] = dict(tokens=g * g, active=int(act.total), reuse_step_ms=round(reuse_ms, 3),
                              dense_step_ms=round(dense_ms, 3), speedup=round(dense_ms / reuse_ms, 3),
                              reuse_bytes=nbytes, reuse_gbs=round(gbs, 1), hbm_frac=round(gbs / PEAK_HBM_GBS, 4))
        log(f"{px} px: {g * g} tokens, {act.total} active: reuse {reuse_ms:.3f} ms, dense {dense_ms:.3f} ms")
        del cache, model
        torch.cuda.empty_cache()
    return out


def sweep_leg(model1, args):
    """Batch-4 active-fraction sweep at 1024 px: four chains, fresh blob masks
    at 5/10/25/50/100 % of 4096 tokens; reuse-step and dense-step times."""
    import torch
    import synth
    from paper_2608_29809_amd.runtime import ActiveSet
    shape = synth.shape_c3()
    B, T = 4, 20
    tgrid = synth.timestep_grid(T)
    model = model1
    cache = model.alloc_cache(B, T)
    txt = synth.make_text(shape, B, args.seed + 1)
    tkv = model.prepare_text(model.to_storage(txt))
    lat = [torch.from_numpy(synth.make_latent(shape, B, args.seed + 1)).cuda()]
    for s in range(T):
        lat.append(torch.empty_like(lat[0]))
        model.build_cache(cache, s, lat[s], int(tgrid[s]), int(tgrid[s + 1]) if s + 1 < T else -1, tkv,
                          latent_out=lat[s + 1])
    torch.cuda.synchronize()
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(2)]

    def timed(fn, n):
        fn(0)
        torch.cuda.synchronize()
        ev[0].record()
        for k in range(n):
            fn(k)
        ev[1].record()
        torch.cuda.synchronize()
        return ev[0].elapsed_time(ev[1]) / n

    out, rows = {}, {}
    steps = list(range(4, T))
    for f in (0.05, 0.10, 0.25, 0.50, 1.00):
        act = ActiveSet.from_lists(synth.sweep_regions(args.seed, f, B))

        def rs(k, act=act):
            s = steps[k % len(steps)]
            model.reuse_step(cache, s, act, lat[s], int(tgrid[s]), int(tgrid[s + 1]) if s + 1 < T else -1, tkv,
                             latent_out=lat[s + 1])

        out[f"{int(f * 100)}%"] = round(timed(rs, 8), 3)
        rows[f"{int(f * 100)}%"] = act.total
    def ds(k):
        s = steps[k % len(steps)]
        model.build_cache(cache, s, lat[s], int(tgrid[s]), int(tgrid[s + 1]) if s + 1 < T else -1, tkv,
                          latent_out=lat[s + 1])
    dense_ms = round(timed(ds, 4), 3)
    log("fraction sweep (batch 4, ms per step): " + ", ".join(f"{k} {v}" for k, v in out.items()) +
        f"; dense {dense_ms}")
    # fixed per-step cost: least-squares line t = a + b * rows over the
    # partial fractions (5-50 %); a is the step time at zero active rows
    keys = [k for k in out if k != "100%"]
    xs = np.array([rows[k] for k in keys], float)
    ys = np.array([out[k] for k in keys], float)
    b_ms, a_ms = np.polyfit(xs, ys, 1)
    log(f"fraction sweep intercept: {a_ms:.3f} ms + {b_ms * 1000:.3f} us per active row")

    # the configured workload: per fraction, four edit turns (turn 0 is the
    # dense trajectory above), each with fresh blob masks and fresh delta
    # tokens, a 20-step schedule of 4 dense steps then 16 region-reuse steps;
    # against all-dense turns
    sched = {}
    n_dense = 4
    txt_prev = txt

    def one_turn(txt_t, act_t, all_dense):
        tk = model.prepare_text(model.to_storage(txt_t))
        for s in range(T):
            tn = int(tgrid[s + 1]) if s + 1 < T else -1
            if all_dense or s < n_dense:
                model.build_cache(cache, s, lat[s], int(tgrid[s]), tn, tk, latent_out=lat[s + 1])
            else:
                model.reuse_step(cache, s, act_t, lat[s], int(tgrid[s]), tn, tk, latent_out=lat[s + 1])

    for f in (0.05, 0.10, 0.25, 0.50, 1.00):
        per_turn = []
        for turn in range(1, 5):
            txt_t, _ = synth.edit_text(shape, txt_prev, 5, args.seed + 100 * turn + int(f * 100))
            act_t = ActiveSet.from_lists(synth.sweep_regions(args.seed + turn, f, B))
            torch.cuda.synchronize()
            ev[0].record()
            one_turn(txt_t, act_t, False)
            ev[1].record()
            torch.cuda.synchronize()
            per_turn.append(ev[0].elapsed_time(ev[1]))
            txt_prev = txt_t
        sched[f"{int(f * 100)}%"] = round(float(np.mean(per_turn)), 2)
    ev[0].record()
    one_turn(txt_prev, None, True)
    ev[1].record()
    torch.cuda.synchronize()
    dense_turn_ms = ev[0].elapsed_time(ev[1])
    log("edit turns (batch 4, 4 dense + 16 reuse, ms per turn): " + ", ".join(f"{k} {v}" for k, v in sched.items()) +
        f"; all-dense turn {dense_turn_ms:.1f}")
    del cache
    torch.cuda.empty_cache()
    return dict(batch=B, active_rows=rows, reuse_step_ms=out, dense_step_ms=dense_ms,
                speedup_vs_dense={k: round(dense_ms / v, 3) for k, v in out.items()},
                fixed_ms=round(float(a_ms), 3), per_active_row_us=round(float(b_ms) * 1000, 4),
                edit_turns=dict(turns_per_fraction=4, steps=T, dense_steps=n_dense, masks="fresh blob masks per turn",
                                turn_ms=sched, all_dense_turn_ms=round(dense_turn_ms, 2),
                                speedup_vs_all_dense={k: round(dense_turn_ms / v, 3) for k, v in sched.items()}))


def class_work(shape, R, B):
    """Algorithmic work of one launch of each kernel class of a region step
    over R active rows in B chains (one chain's worth of keys per chain):
    flops for the matrix-core classes, bytes every launch must move at least
    once for the memory-bound ones (and for the GEMMs, whose weights are
    streamed from HBM once per launch).  bf16 operands, fp32 residual stream."""
    C, N, F, M, H = shape.hidden, shape.tokens, shape.mlp, shape.text_len, shape.heads
    e = 2  # bf16

    def g(m, n, k, out_bytes, extra_in=0):
        return dict(bound="mfma", flops=2.0 * m * n * k, bytes=n * k * e + m * k * e + out_bytes + extra_in)
    w = {
        "gemm_qkv": g(R, 3 * C, C, R * 3 * C * e),                      # q compact, k/v scattered into the slot
        "gemm_proj": g(R, C, C, R * C * (4 + e), R * C * 4),            # X read + written, bf16 copy
        "gemm_xq": g(R, C, C, R * C * e),
        "gemm_xproj": g(R, C, C, R * C * 4, R * C * 4),                 # X read + written
        "gemm_fc1": g(R, F, C, R * F * e),
        "gemm_fc2": g(R, C, F, 2 * R * C * 4),                          # two fp32 split partials
        "attn_self": dict(bound="mfma", flops=4.0 * R * N * C,
                          bytes=B * 2 * H * N * 72 * e + R * C * e + 5 * R * C * e),  # K,V of the slot, Q, split outputs
        # the cross query projection runs inside the bf16 cross-attention kernel
        "attn_cross": dict(bound="mfma", flops=4.0 * R * M * C + 2.0 * R * C * C,
                           bytes=B * 2 * C * 128 * e + C * C * e + 2 * R * C * e),  # text K/V, Wq, rows in, out
        "attn_combine": dict(bound="hbm", flops=0.0, bytes=5 * R * C * e + R * C * e),
        "split_finish": dict(bound="hbm", flops=0.0, bytes=2 * R * C * 4 + 2 * R * C * 4 + 2 * R * C * e),
        "norm": dict(bound="hbm", flops=0.0, bytes=R * C * (4 + e)),
        "embed": dict(bound="hbm", flops=0.0, bytes=R * C * 4 + R * 16 * 4),
    }
    return w


KERNEL_SOURCES = {  # sources whose text fixes a kernel class's code
    "attn_self": ["rc_attn3.hip", "rc_common.h", "rc_internal.h", "rc_launch.h"],
    "attn_cross": ["rc_attn2.hip", "rc_common.h", "rc_internal.h", "rc_launch.h"],
    "gemm": ["rc_gemm2.hip", "rc_common.h", "rc_internal.h", "rc_launch.h"],
}
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "hbm_traffic_reuse_step_1024px.md")


def kernel_source_hash(cls):
    import hashlib
    h = hashlib.sha256()
    for f in KERNEL_SOURCES.get(cls, KERNEL_SOURCES["gemm"]):
        h.update(open(os.path.join(ROOT, "paper_2608_29809_amd", "csrc", f), "rb").read())
    return h.hexdigest()[:16]


def _committed_traffic(cls, R):
    """HBM bytes per launch of a kernel class from the committed counter
    summary (FETCH_SIZE and WRITE_SIZE runs, scaled by a plain copy's
    counts), or None when there is none for this class and active-row count
    or the kernel's sources have changed since the counters were taken."""
    if not os.path.exists(TRAFFIC_SUMMARY):
        return None
    for line in open(TRAFFIC_SUMMARY):
        if not line.startswith("traffic-record: "):
            continue
        try:
            rec = json.loads(line[len("traffic-record: "):])
        except ValueError:
            continue
        if rec.get("kernel") == cls and rec.get("R") == R and rec.get("source_hash") == kernel_source_hash(cls):
            return rec.get("bytes_per_launch")
    return None


def _cpu_model():
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def cpu_baseline(shape, W, idx, args):
    """The oracle, in its float32 mode, timed on this machine's host cores on
    a bounded sample of the same reuse step: the first `--cpu-layers` blocks
    of the step for one chain; the per-step time is scaled by
    layers/sampled-layers."""
    import dataclasses
    import oracle as O
    import synth
    try:
        from threadpoolctl import threadpool_info
        threads = max([i.get("num_threads", 1) for i in threadpool_info()] + [1])
        blas = sorted({i.get("internal_api", "?") for i in threadpool_info()})
    except Exception:
        threads, blas = os.cpu_count(), []
    Ls = max(1, min(args.cpu_layers, shape.layers))
    sub = dataclasses.replace(shape, layers=Ls)
    Wsub = dict(W)
    Wsub["layers"] = W["layers"][:Ls]
    txt = synth.make_text(shape, 1, args.seed)
    lat = synth.make_latent(shape, 1, args.seed)
    slot = synth.make_cache_slot(sub, 1, args.seed)
    cache = dict(K=slot["K"][:, 0], V=slot["V"][:, 0], H=slot["H"][:, 0])
    f32 = np.float32
    y = O.caption_projection(Wsub, txt[0], dt=f32)
    tkv = [O.text_kv(lw, y, shape.heads, dt=f32) for lw in Wsub["layers"]]
    w0 = time.perf_counter()
    O.reuse_step(sub, Wsub, lat[0], 842, 789, tkv, idx, cache, lat[0], dt=f32)
    dt = time.perf_counter() - w0
    per_step = dt * shape.layers / Ls
    log(f"oracle (float32): {Ls} blocks in {dt:.2f}s -> {per_step:.2f}s per {shape.layers}-block reuse step")
    blocks = (f"all {Ls} blocks" if Ls == shape.layers
              else f"first {Ls} of {shape.layers} blocks, time x {shape.layers}/{Ls}")
    return dict(value=round(1.0 / per_step, 5), unit="steps/s", cores=int(threads), kind="oracle",
                sample=f"one region-reuse step of one chain, {blocks} (R={len(idx)} of {shape.tokens} tokens), "
                       f"float32 NumPy",
                sample_seconds=round(dt, 3), nproc=len(os.sched_getaffinity(0)), cpu_model=_cpu_model(),
                blas=blas)


def cpu_baseline_configs(shape, W, args):
    """The oracle (float32, host cores) on the other workloads the GPU legs
    time, each on a bounded sample scaled to the whole: the 512 px region
    step of the resolution sweep (all blocks) and its dense step (first 4
    blocks), the 1024 px dense step (first block) and the 1024 px
    localisation read-out (4 of the 28 layers of logits, same per-layer shape
    and distribution as the GPU leg's)."""
    import dataclasses
    import oracle as O
    import synth
    f32 = np.float32
    L = shape.layers

    def first_blocks(sh, n):
        n = max(1, min(n, sh.layers))
        Wn = dict(W)
        Wn["layers"] = W["layers"][:n]
        return dataclasses.replace(sh, layers=n), Wn, n

    def text_kv(sh, Wn, seed):
        y = O.caption_projection(Wn, synth.make_text(sh, 1, seed)[0], dt=f32)
        return [O.text_kv(lw, y, sh.heads, dt=f32) for lw in Wn["layers"]]

    out = {}
    # 512 px: the resolution sweep's 15 % blob region
    s2 = dataclasses.replace(shape, grid_h=32, grid_w=32)
    idx2 = synth.resolution_region(args.seed, 32)
    lat = synth.make_latent(s2, 1, args.seed + 2)
    slot = synth.make_cache_slot(s2, 1, args.seed)
    cache = dict(K=slot["K"][:, 0], V=slot["V"][:, 0], H=slot["H"][:, 0])
    w0 = time.perf_counter()
    O.reuse_step(s2, W, lat[0], 842, 789, text_kv(s2, W, args.seed + 2), idx2, cache, lat[0], dt=f32)
    t_r = time.perf_counter() - w0
    del slot, cache
    sd, Wd, nd = first_blocks(s2, 4)
    tkv = text_kv(sd, Wd, args.seed + 2)
    w0 = time.perf_counter()
    O.dense_step(sd, Wd, lat[0], 842, 789, tkv, dt=f32)
    t_d = (time.perf_counter() - w0) * L / nd
    out["512px"] = dict(tokens=s2.tokens, active=int(len(idx2)), reuse_step_s=round(t_r, 3), dense_step_s=round(t_d, 3),
                        sample=f"region step: all {L} blocks; dense step: first {nd} blocks, time x {L}/{nd}")
    # 1024 px dense step
    s3, W3, n3 = first_blocks(shape, 1)
    lat = synth.make_latent(shape, 1, args.seed)
    tkv = text_kv(s3, W3, args.seed)
    w0 = time.perf_counter()
    O.dense_step(s3, W3, lat[0], 842, 789, tkv, dt=f32)
    t_d3 = (time.perf_counter() - w0) * L / n3
    out["1024px_dense"] = dict(tokens=shape.tokens, dense_step_s=round(t_d3, 3),
                               sample=f"first {n3} of {L} blocks, time x {L}/{n3}")
    # localisation read-out at 1024 px
    nl = 4
    Z, delta, blob = synth.make_logits(nl, 16, 4096, 120, 64, 64, n_delta=6, seed=args.seed, frac=0.12)
    w0 = time.perf_counter()
    maps = O.maps_from_logits(Z, delta, dt=f32)
    t_m = (time.perf_counter() - w0) * 28 / nl
    w0 = time.perf_counter()
    O.localize(maps, 64, 64, theta=0.3, radius=1)
    t_l = time.perf_counter() - w0
    out["localize_1024px"] = dict(maps_s=round(t_m, 3), mask_and_compaction_s=round(t_l, 3),
                                  sample=f"logits [{nl},16,4096,120] as float32, maps time x 28/{nl}; 6 delta columns")
    log("oracle (float32) on the other workloads: " + json.dumps(out))
    return out


if __name__ == "__main__":
    main()
