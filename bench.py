#!/usr/bin/env python3
"""Benchmark of the 3DGART hot path on one MI355X.

A step is one pass of the whole path over the 1M-Gaussian synthetic scene
(1,000,000 Gaussians, SH degree 3, 1237x822, 8x8 tiles): gart_bounds ->
gart_build_tile_map -> gart_forward -> gart_backward, inputs resident in
HBM.  The headline value is backward Gaussian-pixel gradients per second
(composited hits / backward time); ms_per_step is the whole fwd+bwd
iteration.  Kernel times come from HIP events that the library records on
its own stream around each kernel.

Prints one JSON line.  ``--gpus N`` with N > 1 exits: this path runs on one
GPU.
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

HBM_PEAK_GBS = 8000.0          # MI355X HBM3E, published
FP32_PEAK_TFLOPS = 157.3       # MI355X vector fp32, published
FP64_PEAK_TFLOPS = 78.6        # MI355X vector fp64, published

# Algorithmic cost per unit of work: what the method must move or compute,
# independent of how the kernels do it.
#   composited hit, backward: 16 B (L,T) read; 12K + 90 fp32 flops
#   composited hit, forward: 16 B (L,T) write; 6K fp32 flops (colour)
#   (pixel, Gaussian) ray test (fwd and bwd): 45 fp64 flops
#   pixel: 40 B read by the backward (dL/dC 12, C 12, end marker 16); 12 B image written by the forward
#   Gaussian: 4P B of parameters read by the backward, 4P B of gradients written by the reduction
#             (P = 11 + 3K values), ~200 fp64 flops of chain rule
LT_BYTES_PER_HIT = 16
PIXEL_BYTES_BWD = 40
PIXEL_BYTES_FWD = 12
F64_PER_TEST = 45
F64_PER_CHAIN = 200


def f32_per_hit_bwd(K):
    return 12 * K + 90


def f32_per_hit_fwd(K):
    return 6 * K


def param_bytes(K):
    return 4 * (11 + 3 * K)


# Implementation cost model (the bytes these kernels' designs must move, as
# opposed to the algorithmic figures above), reported beside them.
IMPL_GEOM_BYTES = 128 + 16 + 8 + 4  # per staged pair in the forward: fp64 geometry row, rect, O_prim, pair index
IMPL_UNIT_BYTES = 104 + 8 + 16 + 8 + 8  # per gather unit: W and o_g, sigma, rect, O_prim, pair offset


ALL_MODES = ("gather", "gather_wave", "gather_atomic", "scatter", "hybrid")
# backward mode + intermediate-buffer precision pairs timed beside the default
STORAGE_VARIANTS = (("gather", "fixed16"), ("gather", "half"), ("hybrid", "fixed16"))


def parse():
    ap = argparse.ArgumentParser(description=__doc__)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", default="1m", choices=["tiny", "small", "1m", "4m", "stress"])
    ap.add_argument("--mode", default="gather", choices=["gather", "gather_atomic", "scatter", "hybrid"])
    ap.add_argument("--compare-modes", type=int, default=1, help="also time the other backward modes")
    ap.add_argument("--cpu-baseline", type=int, default=1)
    ap.add_argument("--cpu-pixels", type=int, default=0, help="oracle sample size in pixels (0 = whole frame)")
    ap.add_argument("--train-steps", type=int, default=12,
                    help="also time this many multi-view training iterations (0 = skip)")
    ap.add_argument("--train-views", type=int, default=4, help="orbit views of the training loop")
    ap.add_argument("--copy-probe-mib", type=int, default=0,
                    help="only run a device copy of this size (HBM counter calibration) and exit")
    ap.add_argument("--out", default=None, help="also write the JSON line to this file")
    return ap.parse_args()


def copy_probe(mib):
    import torch
    n = mib * (1 << 20) // 4
    a = torch.ones(n, device="cuda", dtype=torch.float32)
    b = torch.empty_like(a)
    for _ in range(5):
        b.copy_(a)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_per_dispatch": n * 4}))


def source_hash(files):
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(ROOT, f), "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()[:16]


KERNEL_SOURCES = {
    "gather": ["paper_2608_17298_amd/csrc/backward.hip", "paper_2608_17298_amd/csrc/common.h"],
    "forward": ["paper_2608_17298_amd/csrc/forward.hip", "paper_2608_17298_amd/csrc/common.h"],
}


def recorded_profile(kernel, workload):
    """The committed rocprofv3 counter record of a kernel (HBM bytes per launch,
    VALU busy / utilisation), or {} if absent or if the kernel source changed
    since the counters were taken."""
    path = os.path.join(ROOT, "profiles", "traffic.json")
    try:
        with open(path) as f:
            rec = json.load(f).get(f"{kernel}/{workload}")
    except (OSError, ValueError):
        return {}
    if not rec or rec.get("source_sha256") != source_hash(KERNEL_SOURCES[kernel]):
        return {}
    return rec


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py: this build runs on one GPU; --gpus {args.gpus} is not supported "
              "(the multi-GPU sharding is a design only).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2608_17298_amd import gart
    from paper_2608_17298_amd.scenes import make_scene

    if not torch.cuda.is_available():
        print("bench.py: no GPU visible", file=sys.stderr)
        sys.exit(1)
    if args.copy_probe_mib:
        copy_probe(args.copy_probe_mib)
        return

    t0 = time.time()
    sc = make_scene(args.workload)
    K = sc.sh_k
    cam = gart.make_camera(sc.camera)
    st = gart.make_settings(sc.tile, args.mode)
    g = gart.Gaussians.from_scene(sc)
    stream = torch.cuda.current_stream()
    H, W = sc.camera.height, sc.camera.width
    print(f"[bench] scene {args.workload}: N={sc.n} K={K} {W}x{H} tile {sc.tile}, generated in "
          f"{time.time() - t0:.1f}s", file=sys.stderr, flush=True)

    # Upstream gradient: L1 loss against a render of the perturbed-means copy
    # (rendered once with the same pipeline, outside the timed region); the
    # tiny workload draws it instead (N(0,1)).
    target = None
    if sc.means_perturbed is not None:
        gp = gart.Gaussians.from_scene(sc)
        gp.means = torch.from_numpy(sc.means_perturbed).cuda()
        fp = gart.prepare(gp, cam, st)
        target = torch.empty((H, W, 3), dtype=torch.float32, device="cuda")
        gart.gart_forward(gp, cam, st, fp, target)
        del fp

    # 16-byte intermediate entries, so that every backward mode can render
    # into this frame (the hybrid forward uses the first 4 bytes of each)
    frame = gart.prepare(g, cam, gart.make_settings(sc.tile, "gather"), slack=1.05)
    image = torch.empty((H, W, 3), dtype=torch.float32, device="cuda")
    gart.gart_forward(g, cam, st, frame, image)
    if target is not None:
        dl = torch.sign(image - target).contiguous()
    else:
        dl = torch.from_numpy(sc.dl_dimage).cuda().contiguous()
    grads = gart.empty_grads(g)

    # Counting run (device counters; not timed).
    frame.counters = torch.zeros(gart.NUM_COUNTERS, dtype=torch.int64, device="cuda")
    counts = {}
    for mode in (ALL_MODES if args.compare_modes else [args.mode]):
        frame.counters.zero_()
        stm = gart.make_settings(sc.tile, mode)
        gart.gart_bounds(g, cam, stm, frame)
        gart.gart_build_tile_map(cam, stm, frame)
        gart.gart_forward(g, cam, stm, frame, image)
        gart.gart_backward(g, cam, stm, frame, dl, grads)
        torch.cuda.synchronize()
        counts[mode] = frame.counters.cpu().numpy().astype(np.int64)
    frame.counters = None
    c = counts[args.mode]
    vram = frame_vram(frame, sc)
    hits = int(c[gart.CNT_FWD_HITS])

    def make_events(n):
        evs = [torch.cuda.Event(enable_timing=True) for _ in range(n)]
        for e in evs:
            e.record(stream)  # materialise the underlying hipEvent_t
        return evs

    def run_steps(settings, n_steps, n_warm, backward_only=False):
        per = []
        for s in range(n_warm + n_steps):
            timed = s >= n_warm
            if timed:
                call = make_events(5)
                kern = make_events(gart.NUM_EVENTS)
                frame.set_events([e.cuda_event for e in kern])
            else:
                frame.set_events([])
            if not backward_only:
                if timed:
                    call[0].record(stream)
                gart.gart_bounds(g, cam, settings, frame)
                if timed:
                    call[1].record(stream)
                gart.gart_build_tile_map(cam, settings, frame)
                if timed:
                    call[2].record(stream)
                gart.gart_forward(g, cam, settings, frame, image)
            if timed:
                call[3].record(stream)
            gart.gart_backward(g, cam, settings, frame, dl, grads)
            if timed:
                call[4].record(stream)
                per.append((call, kern))
        frame.set_events([])
        torch.cuda.synchronize()
        return per

    def ms(a, b):
        return a.elapsed_time(b)

    # Warm-up, then exactly K timed steps bracketed by synchronisation.
    run_steps(st, 0, args.warmup)
    torch.cuda.synchronize()
    t_start = time.perf_counter()
    per = run_steps(st, args.steps, 0)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t_start
    ms_per_step = 1e3 * wall / args.steps
    fwd_status = gart.gart_frame_status(frame)
    if fwd_status != 0:
        print(f"bench.py: forward status {fwd_status:#x} (incomplete trace)", file=sys.stderr)
        sys.exit(3)

    def avg(fn):
        return float(np.mean([fn(cl, kr) for cl, kr in per]))

    call_ms = dict(
        bounds=avg(lambda cl, kr: ms(cl[0], cl[1])), tile_map=avg(lambda cl, kr: ms(cl[1], cl[2])),
        forward=avg(lambda cl, kr: ms(cl[2], cl[3])), backward=avg(lambda cl, kr: ms(cl[3], cl[4])))
    kern_ms = dict(
        pair_sort=avg(lambda cl, kr: ms(kr[0], kr[1])), forward_trace=avg(lambda cl, kr: ms(kr[2], kr[3])),
        backward_main=avg(lambda cl, kr: ms(kr[4], kr[5])), reduce_chain=avg(lambda cl, kr: ms(kr[6], kr[7])))

    # Work of the dominant kernels per launch, from the counting run's unit
    # counts and the algorithmic costs per unit.
    npix = W * H
    AW = 10 + 3 * K
    AS = 16 if AW <= 16 else (AW + 31) // 32 * 32  # partial-row stride in floats (whole 128-byte lines)
    bwd_tests, bwd_hits = int(c[gart.CNT_BWD_TESTS]), int(c[gart.CNT_BWD_HITS])
    bwd_pairs, bwd_active = int(c[gart.CNT_BWD_PAIRS]), int(c[gart.CNT_BWD_ACTIVE])
    fwd_tests = int(c[gart.CNT_FWD_TESTS])
    N = sc.n
    work = {
        "backward_main": dict(
            bytes=LT_BYTES_PER_HIT * bwd_hits + PIXEL_BYTES_BWD * npix + param_bytes(K) * N,
            f64=F64_PER_TEST * bwd_tests, f32=f32_per_hit_bwd(K) * bwd_hits),
        "backward": dict(
            bytes=LT_BYTES_PER_HIT * bwd_hits + PIXEL_BYTES_BWD * npix + 2 * param_bytes(K) * N,
            f64=F64_PER_TEST * bwd_tests + F64_PER_CHAIN * N, f32=f32_per_hit_bwd(K) * bwd_hits),
        "forward_trace": dict(
            bytes=LT_BYTES_PER_HIT * hits + PIXEL_BYTES_FWD * npix,
            f64=F64_PER_TEST * fwd_tests, f32=f32_per_hit_fwd(K) * hits),
    }
    # bytes the kernels' own designs move (staged geometry, SH, partial rows,
    # hit lists), for comparison with the algorithmic figures
    impl_bytes = {
        "backward_main": 20 * bwd_hits + 12 * bwd_pairs + bwd_active * (IMPL_UNIT_BYTES + 12 * K + 4 * AS + 1)
        + npix * (12 + 32),
        "forward_trace": 20 * hits + bwd_pairs * IMPL_GEOM_BYTES + bwd_active * 12 * K + npix * (12 + 32),
    }
    times_ms = {"backward_main": kern_ms["backward_main"], "backward": call_ms["backward"],
                "forward_trace": kern_ms["forward_trace"]}

    def roofline(name):
        w = work[name]
        t = times_ms[name] * 1e-3
        t_hbm = w["bytes"] / (HBM_PEAK_GBS * 1e9)
        t_alu = w["f32"] / (FP32_PEAK_TFLOPS * 1e12) + w["f64"] / (FP64_PEAK_TFLOPS * 1e12)
        common = dict(algorithmic_bytes=w["bytes"], f32_flops=w["f32"], f64_flops=w["f64"],
                      time_ms=round(times_ms[name], 4), roofline_ms=round(1e3 * max(t_hbm, t_alu), 4))
        if t_hbm >= t_alu:
            achieved = w["bytes"] / t / 1e9
            return dict(bound="hbm", achieved=round(achieved, 1), peak=HBM_PEAK_GBS, unit="GB/s",
                        frac=round(achieved / HBM_PEAK_GBS, 4), **common)
        flops = w["f32"] + w["f64"]
        peak = flops / t_alu / 1e12  # the published fp32 / fp64 peaks weighted by this kernel's mix
        achieved = flops / t / 1e12
        return dict(bound="alu", achieved=round(achieved, 3), peak=round(peak, 1), unit="TFLOP/s",
                    frac=round(achieved / peak, 4), **common)

    def with_counters(name):
        r = roofline(name)
        prof = {"backward_main": "gather", "forward_trace": "forward"}.get(name)
        rec = recorded_profile(prof, args.workload) if prof else {}
        r["traffic"] = rec.get("hbm_bytes_per_launch")
        vb = rec.get("valu_busy_pct")
        r["valu_busy"] = None if vb is None else round(vb / 100.0, 4)
        vu = rec.get("valu_utilization_pct")
        r["valu_utilization"] = None if vu is None else round(vu / 100.0, 4)
        if name in impl_bytes:
            r["implementation_bytes"] = impl_bytes[name]
        return r

    # Headline: the gather backward's main kernel, whose throughput `value`
    # measures and whose roofline fraction the target is set on; the whole
    # backward (with the reduction) and the forward are reported beside it.
    roof = with_counters("backward_main")
    roof["kernel"] = "gather_kernel"

    value = bwd_hits / (call_ms["backward"] * 1e-3)

    modes = {}
    if args.compare_modes:
        for mode in ALL_MODES:
            stm = gart.make_settings(sc.tile, mode)
            # render once with this mode's intermediate-buffer format (the
            # hybrid forward writes T only), then time the backward alone
            gart.gart_forward(g, cam, stm, frame, image)
            per_m = run_steps(stm, max(5, args.steps // 2), 2, backward_only=True)
            bms = float(np.mean([ms(cl[3], cl[4]) for cl, kr in per_m]))
            kms = float(np.mean([ms(kr[4], kr[5]) for cl, kr in per_m]))
            cm = counts[mode]
            modes[mode] = dict(backward_ms=round(bms, 4), main_kernel_ms=round(kms, 4),
                               grads_per_s=round(int(cm[gart.CNT_BWD_HITS]) / (bms * 1e-3), 1),
                               float_atomics=int(cm[gart.CNT_BWD_ATOMICS]),
                               wave_units=int(cm[gart.CNT_BWD_WAVE_UNITS]),
                               lt_bytes=int(frame.lt_entries) * gart.gart_lt_entry_bytes(stm))
        for mode, prec in STORAGE_VARIANTS:
            stm = gart.make_settings(sc.tile, mode, lt_precision=prec)
            per_m = run_steps(stm, max(5, args.steps // 2), 2)
            fms = float(np.mean([ms(cl[2], cl[3]) for cl, kr in per_m]))
            bms = float(np.mean([ms(cl[3], cl[4]) for cl, kr in per_m]))
            modes[f"{mode}+{prec}"] = dict(forward_ms=round(fms, 4), backward_ms=round(bms, 4),
                                           lt_bytes=int(frame.lt_entries) * gart.gart_lt_entry_bytes(stm))
        gart.gart_forward(g, cam, st, frame, image)

    train = None
    if args.train_steps > 0 and sc.means_perturbed is not None:
        train = train_timing(sc, args.train_steps, args.train_views)

    cpu = None
    if args.cpu_baseline:
        cpu = cpu_baseline(sc, dl.cpu().numpy(), args.cpu_pixels)

    line = {
        "metric": "backward Gaussian-pixel grads/sec; ms per fwd+bwd iter @1M Gaussians",
        "value": round(value, 1),
        "unit": "grads/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": "f32+f64",
        "data": "synthetic (seeded generator; stands in for Mip-NeRF 360)",
        "config": {"workload": f"{args.workload}: {sc.n} Gaussians, SH{sc.sh_degree}, {W}x{H}, "
                               f"{sc.tile}x{sc.tile} tiles", "backward_mode": args.mode,
                   "composited_hits": hits, "pairs": int(frame.pair_count), "lt_entries": int(frame.lt_entries)},
        "roofline": roof,
        "roofline_backward_with_reduction": with_counters("backward"),
        "roofline_forward": dict(with_counters("forward_trace"), kernel="forward_kernel"),
        "cpu_baseline": cpu,
        "call_ms": {k: round(v, 4) for k, v in call_ms.items()},
        "kernel_ms": {k: round(v, 4) for k, v in kern_ms.items()},
        "grads_per_s_full_step": round(hits / (ms_per_step * 1e-3), 1),
        "backward_modes": modes,
        "forward_rescans": int(c[gart.CNT_FWD_RESCANS]),
        "counters": {name: int(c[i]) for i, name in enumerate(
            ["fwd_hits", "fwd_tests", "fwd_rescans", "bwd_hits", "bwd_tests", "bwd_atomics", "bwd_pairs",
             "bwd_active_units", "fwd_drops", "bwd_hybrid_steps", "bwd_wave_units"])},
        "vram_bytes": vram,
        "train_step": train,
    }
    s = json.dumps(line)
    print(s, flush=True)
    if args.out:
        with open(args.out, "w") as f:
            f.write(s + "\n")


def frame_vram(frame, sc):
    """Device bytes of the frame's buffers as allocated (capacities with the
    bench's slack, scratch sized for every backward mode) and as used by this
    workload (counts from gart_bounds)."""
    nb = lambda t: int(t.numel() * t.element_size())
    alloc = dict(lt=nb(frame.lt), hit_list=nb(frame.hit_list),
                 pairs=nb(frame.pair_tile) + nb(frame.pair_prim) + nb(frame.pair_key),
                 scratch=nb(frame.scratch),
                 per_gaussian=nb(frame.rect) + nb(frame.lt_offset) + nb(frame.prim_geom) + nb(frame.tile_count)
                 + nb(frame.pair_offset),
                 pixel_state=nb(frame.pixel_state), tile_range=nb(frame.tile_range))
    alloc["total"] = sum(alloc.values())
    P, E = frame.pair_count, frame.lt_entries
    from paper_2608_17298_amd import gart
    used = dict(lt=16 * E, hit_list=4 * gart.gart_hit_list_slots(P, frame.camera, frame.settings), pairs=12 * P)
    return {"allocated": alloc, "used_by_workload": used,
            "torch_max_allocated": int(__import__("torch").cuda.max_memory_allocated())}


def train_timing(sc, steps, n_views):
    """Synthetic multi-view training on the same scene: `n_views` orbit
    cameras, targets rendered (untimed) from the perturbed-means copy, Adam
    over L1; per-stage HIP-event times over `steps` iterations after two
    warm-up iterations."""
    import dataclasses
    import torch
    from paper_2608_17298_amd import gart
    from paper_2608_17298_amd.scenes import orbit_camera
    from paper_2608_17298_amd.train import Trainer
    W, H = sc.camera.width, sc.camera.height
    cams = [orbit_camera(W, H, 360.0 * k / n_views) for k in range(n_views)]
    pert = dataclasses.replace(sc, means=sc.means_perturbed)
    gp = gart.Gaussians.from_scene(pert)
    st = gart.make_settings(sc.tile, "gather")
    targets, fr = [], None
    for c in cams:
        gc = gart.make_camera(c)
        fr = gart.prepare(gp, gc, st, fr)
        t = torch.empty((H, W, 3), dtype=torch.float32, device="cuda")
        gart.gart_forward(gp, gc, st, fr, t)
        targets.append(t)
    del fr, gp
    tr = Trainer(sc, cams, targets)
    for it in range(2):
        tr.step(it % n_views)
    torch.cuda.synchronize()
    per, losses = [], []
    for it in range(steps):
        ev = [torch.cuda.Event(enable_timing=True) for _ in range(6)]
        tr.step(it % n_views, events=ev)
        per.append(ev)
        losses.append(tr.loss.clone())
    torch.cuda.synchronize()
    names = ["bounds_tile_map", "forward", "l1", "backward", "adam"]
    stage = {nm: float(np.mean([e[k].elapsed_time(e[k + 1]) for e in per])) for k, nm in enumerate(names)}
    total = float(np.mean([e[0].elapsed_time(e[5]) for e in per]))
    return {"views": n_views, "iterations": steps, "ms_per_iteration": round(total, 4),
            "stage_ms": {k: round(v, 4) for k, v in stage.items()},
            "l1_loss_first": round(losses[0].item(), 3), "l1_loss_last": round(losses[-1].item(), 3),
            "adam": "3DGS-style per-group learning rates (paper_2608_17298_amd/train.py)"}


def cpu_baseline(sc, dl, npix):
    """The fp64 oracle (untuned) on a bounded pixel sample of the same workload:
    its per-pixel forward + analytic backward over every candidate."""
    import oracle
    rng = np.random.default_rng(7)
    W, H = sc.camera.width, sc.camera.height
    if npix <= 0 or npix >= W * H:
        pix = np.arange(W * H)
    else:
        pix = np.sort(rng.choice(W * H, size=npix, replace=False))
    o = oracle.OracleScene(sc)
    hits = int(o.render(pix)["n_included"].sum())
    t = time.perf_counter()
    o.backward(dl, pixels=pix)
    dt = time.perf_counter() - t
    return {"value": round(hits / dt, 1), "unit": "grads/s", "cores": oracle.num_threads(), "kind": "oracle",
            "sample": f"{len(pix)} pixels of the same frame ({hits} composited hits), "
                      f"fp64 forward+backward per pixel, {dt:.1f}s"}


if __name__ == "__main__":
    main()
