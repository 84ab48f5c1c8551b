"""Benchmark of the TemporalGS hot path on one MI355X.

One step = one pass of the whole hot path over the 120-frame camera path of
the room workload (1.5M Gaussians, SH degree 3, 1920x1080): the frame
schedule renders true references, pseudo references and TemporalGS frames
(adaptive frustum + occlusion culling, selective rendering, stitching), every
one through the HIP kernels of libtgs.  The scene is resident in HBM before
the timed region starts.

Printed (one JSON line): temporal-mode FPS (value), full-render FPS over the
same path (both with the 3DGS 3-sigma tile rule and the paper-literal empty
pixels; the same timings with the alpha-footprint tile rule and with empty
pixels on the far plane alongside), PSNR of temporal vs full, the roofline of the dominant kernel (its
launch durations from HIP events attached to its dispatches inside the timed
region), a per-stage breakdown from an untimed pass, and the CPU oracle timed
on a bounded sample of the same workload.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import math
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "ms/frame & FPS (full vs temporal) at 1080p, 1.5M Gaussians; PSNR temporal-vs-full"
# Algorithmic VALU lane-operations per blended (pixel, Gaussian) pair, i.e. a
# pair whose alpha reaches 1/255 (it is composited or stops the pixel):
# offset 2, quadratic form 5, exp 1, alpha and its cap 2, threshold 1,
# T(1 - alpha) 2, stop test 1, weight 1, colour 3 FMAs, T update 1 = 19;
# reference frames add the Eq. 1/2 moments around the pivot (weight sum,
# depth offset, two moment updates: 5) = 24.  Pairs below the threshold cost
# nothing algorithmically (a blender may reject them by footprint bounds).
BLEND_OPS_PER_HIT = {"blend_ref": 24, "blend_tgs": 19, "blend_full": 19}
# non-packed fp32 VALU issue rate: 256 CUs x 64 lanes x 2.4 GHz
VALU_PEAK_TOPS = 256 * 64 * 2.4e9 / 1e12
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "blend_traffic_room.json")
# sources the blend kernel is compiled from (its traffic counters are valid
# for these exact files)
BLEND_SRCS = [os.path.join(ROOT, "paper_2607_03390_amd", "csrc", f)
              for f in ("k_blend.hip", "stitch.h", "tgs_internal.h")]


def log(msg):
    print(msg, file=sys.stderr, flush=True)


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=5)
    ap.add_argument("--warmup", type=int, default=1)
    ap.add_argument("--workload", default="room")
    ap.add_argument("--frames", type=int, default=None, help="truncate the camera path")
    ap.add_argument("--cpu-frames", type=int, default=3,
                    help="frames of the path the CPU oracle renders for its baseline")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-psnr", action="store_true")
    ap.add_argument("--no-footprint", action="store_true",
                    help="skip the variant timings (footprint tile rule, empty pixels at z_far)")
    ap.add_argument("--ablation", action="store_true",
                    help="also run the ablation and sensitivity study (culling and selective "
                         "rendering toggles, lambda / eta sweeps, camera speed)")
    ap.add_argument("--tgb-downscale", type=int, default=None,
                    help="geometry-buffer downscale (1 or 2); default: 2 for the large-scale "
                         "city workload (the paper's large-scene setting), 1 otherwise")
    ap.add_argument("--sort-path", default="auto", choices=["auto", "depth_first", "per_tile"],
                    help="how per-tile depth order is produced (tgs_set_sort_path)")
    ap.add_argument("--blend-split", type=int, default=12,
                    help="tiles with at least 2**N list entries are blended as four quadrant "
                         "blocks (tgs_set_blend_split; -1: never)")
    ap.add_argument("--copy-calibration-mb", type=int, default=0,
                    help="run one device copy of this size (for HBM counter calibration)")
    return ap.parse_args()


def kernel_source_hash():
    h = hashlib.sha256()
    for f in BLEND_SRCS:
        h.update(open(f, "rb").read())
    return h.hexdigest()[:16]


def main():
    args = parse()
    if args.tgb_downscale is None:
        args.tgb_downscale = 2 if args.workload == "city" else 1
    if args.gpus != 1:
        print(json.dumps({"error": "this build targets one GPU: the TemporalGS hot path runs "
                                   "on a single MI355X; run with --gpus 1"}))
        sys.exit(2)
    import numpy as np
    import torch

    from paper_2607_03390_amd import metrics, synth, tgs

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    torch.cuda.set_device(0)
    SORT_MODES = {"auto": tgs.SORT_AUTO, "depth_first": tgs.SORT_DEPTH_FIRST,
                  "per_tile": tgs.SORT_PER_TILE}
    tgs.tgs_set_sort_path(SORT_MODES[args.sort_path])
    tgs.tgs_set_blend_split(args.blend_split)
    log(f"[bench] generating workload {args.workload}")
    wl = synth.workload(args.workload, n_frames=args.frames)
    cams = wl.cameras
    W, H = cams[0].width, cams[0].height
    TX, TY = cams[0].tiles
    n = wl.scene.n
    out_t = tgs.alloc_frame(W, H)
    out_f = tgs.alloc_frame(W, H)
    torch.cuda.synchronize()

    def used():
        free, total = torch.cuda.mem_get_info()
        return total - free

    # device memory of each path (the library allocates with hipMalloc, so
    # the device-wide figure is read): scene, then the full render's own
    # buffers, then the temporal state's (priors and its frame buffers)
    mem0 = used()
    scene_h = tgs.tgs_scene_upload(wl.scene)
    torch.cuda.synchronize()
    mem_scene = used() - mem0
    tgs.tgs_render_full(scene_h, cams[0], **out_f)
    torch.cuda.synchronize()
    mem_full_ws = used() - mem0 - mem_scene
    state_h = tgs.tgs_state_create(scene_h, W, H, tgs.params(tgb_downscale=args.tgb_downscale))
    for cam in cams:
        tgs.tgs_render_temporal(state_h, cam, **out_t)
    torch.cuda.synchronize()
    mem_state = used() - mem0 - mem_scene - mem_full_ws
    memory = {"scene_bytes": mem_scene, "full_render_bytes": mem_scene + mem_full_ws,
              "temporal_bytes": mem_scene + mem_state,
              "temporal_over_full": round((mem_scene + mem_state) / max(1, mem_scene + mem_full_ws), 4),
              "note": "device memory held by the library (scene + its render buffers; scene + "
                      "temporal state with priors and render buffers), from hipMemGetInfo; "
                      "output images excluded"}
    log(f"[bench] {n} Gaussians, {W}x{H}, {len(cams)} frames uploaded; memory {memory}")

    def temporal_step(record=None):
        tgs.tgs_state_reset(state_h)
        for cam in cams:
            info = tgs.tgs_render_temporal(state_h, cam, **out_t)
            if record is not None:
                record.append(info)

    def full_step():
        for cam in cams:
            tgs.tgs_render_full(scene_h, cam, **out_f)

    if args.copy_calibration_mb:
        nb = args.copy_calibration_mb << 20
        src = torch.empty(nb // 4, dtype=torch.float32, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        log(f"[bench] calibration copy of {nb} bytes done")
        del src, dst

    for w in range(args.warmup):
        temporal_step()
        full_step()
        torch.cuda.synchronize()
        log(f"[bench] warmup {w + 1}/{args.warmup} done")

    # untimed: evaluated pixel-Gaussian pairs per blend stage (deterministic)
    tgs.tgs_profile_start(count_pairs=True)
    kinds = []
    temporal_step(kinds)
    full_step()
    counted = tgs.tgs_profile_stop()
    log("[bench] pair counts done")

    # untimed: per-stage breakdown (stage events add queue barriers)
    tgs.tgs_profile_start(stages=True)
    temporal_step()
    detail = tgs.tgs_profile_stop()
    tgs.tgs_profile_start(stages=True)
    full_step()
    detail_full = tgs.tgs_profile_stop()
    log("[bench] stage breakdown done")

    # timed: temporal mode; the blend dispatches carry their own timing events
    torch.cuda.synchronize()
    tgs.tgs_profile_start(count_pairs=False)
    t0 = time.perf_counter()
    for k in range(args.steps):
        temporal_step()
    torch.cuda.synchronize()
    t_temporal = time.perf_counter() - t0
    prof = tgs.tgs_profile_stop()
    log(f"[bench] temporal timed: {t_temporal:.3f}s for {args.steps} steps")

    # timed: full render of the same path
    torch.cuda.synchronize()
    tgs.tgs_profile_start(count_pairs=False)
    t0 = time.perf_counter()
    for k in range(args.steps):
        full_step()
    torch.cuda.synchronize()
    t_full = time.perf_counter() - t0
    prof_full = tgs.tgs_profile_stop()
    log(f"[bench] full timed: {t_full:.3f}s for {args.steps} steps")

    n_frames = len(cams)
    fps_t = n_frames * args.steps / t_temporal
    fps_f = n_frames * args.steps / t_full

    # per-kind frame times (untimed pass, events around each frame)
    per_kind = {0: [], 1: [], 2: []}
    tgs.tgs_state_reset(state_h)
    for cam in cams:
        e0 = torch.cuda.Event(enable_timing=True)
        e1 = torch.cuda.Event(enable_timing=True)
        e0.record()
        info = tgs.tgs_render_temporal(state_h, cam, **out_t)
        e1.record()
        torch.cuda.synchronize()
        per_kind[info["frame_kind"]].append(e0.elapsed_time(e1))

    # PSNR and SSIM temporal vs full (images clamped to [0,1]); identical
    # frames are excluded from the PSNR mean (infinite)
    psnr = ssim = None
    if not args.no_psnr:
        vals, svals = [], []
        tgs.tgs_state_reset(state_h)
        for cam in cams:
            tgs.tgs_render_temporal(state_h, cam, **out_t)
            tgs.tgs_render_full(scene_h, cam, **out_f)
            p = metrics.psnr(out_t["rgb"], out_f["rgb"])
            if math.isfinite(p):
                vals.append(p)
            svals.append(metrics.ssim(out_t["rgb"], out_f["rgb"]))
        psnr = dict(mean_db=float(np.mean(vals)) if vals else None,
                    min_db=float(np.min(vals)) if vals else None,
                    frames_compared=len(vals), identical_frames=n_frames - len(vals))
        ssim = dict(mean=round(float(np.mean(svals)), 6), min=round(float(np.min(svals)), 6),
                    frames=len(svals))

    def variant(label, cams_v, tile_bound=tgs.TGS_TILES_3SIGMA, steps=None, full=False,
                sort_path=None, **pkw):
        """Temporal FPS, frame mix and PSNR vs the full render of one setting."""
        steps = steps or args.steps
        tgs.tgs_scene_set_tile_bound(scene_h, tile_bound)
        if sort_path is not None:
            tgs.tgs_set_sort_path(SORT_MODES[sort_path])
        pkw = {"tgb_downscale": args.tgb_downscale, **pkw}
        sv = tgs.tgs_state_create(scene_h, W, H, tgs.params(**pkw))

        def run(rec=None):
            tgs.tgs_state_reset(sv)
            for cam in cams_v:
                info = tgs.tgs_render_temporal(sv, cam, **out_t)
                if rec is not None:
                    rec.append(info)

        run()
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        for _ in range(steps):
            run()
        torch.cuda.synchronize()
        dt = time.perf_counter() - t0
        rec = []
        run(rec)
        nv = len(cams_v)
        sel = [100.0 * i["n_selected"] / (TX * TY) for i in rec if i["frame_kind"] == tgs.TGS_FRAME_TGS]
        r = {"label": label, "params": pkw, "tile_rule": "footprint" if tile_bound else "3sigma",
             "frames": nv, "temporal_fps": round(nv * steps / dt, 2),
             "temporal_ms_per_frame": round(1e3 * dt / (steps * nv), 4),
             "tgsf_pct": round(100.0 * sum(i["frame_kind"] == tgs.TGS_FRAME_TGS for i in rec) / nv, 2),
             "sr_tile_pct": round(float(np.mean(sel)), 2) if sel else None}
        if full:
            for cam in cams_v:
                tgs.tgs_render_full(scene_h, cam, **out_f)
            torch.cuda.synchronize()
            t0 = time.perf_counter()
            for _ in range(steps):
                for cam in cams_v:
                    tgs.tgs_render_full(scene_h, cam, **out_f)
            torch.cuda.synchronize()
            dtf = time.perf_counter() - t0
            r["full_fps"] = round(nv * steps / dtf, 2)
            r["full_ms_per_frame"] = round(1e3 * dtf / (steps * nv), 4)
            r["speedup_temporal_vs_full"] = round(dtf / dt, 3)
        if not args.no_psnr:
            vals, svals = [], []
            tgs.tgs_state_reset(sv)
            for cam in cams_v:
                tgs.tgs_render_temporal(sv, cam, **out_t)
                tgs.tgs_render_full(scene_h, cam, **out_f)
                p = metrics.psnr(out_t["rgb"], out_f["rgb"])
                if math.isfinite(p):
                    vals.append(p)
                svals.append(metrics.ssim(out_t["rgb"], out_f["rgb"]))
            r["psnr_mean_db"] = round(float(np.mean(vals)), 2) if vals else None
            r["psnr_min_db"] = round(float(np.min(vals)), 2) if vals else None
            r["ssim_mean"] = round(float(np.mean(svals)), 5)
        tgs.tgs_state_free(sv)
        tgs.tgs_scene_set_tile_bound(scene_h, tgs.TGS_TILES_3SIGMA)
        tgs.tgs_set_sort_path(SORT_MODES[args.sort_path])
        if sort_path is not None:
            r["sort_path"] = sort_path
        log(f"[bench] variant {label}: {r}")
        return r

    variants = {}
    if not args.no_footprint:
        # the alpha-footprint tile rule (same contributions up to the 3-sigma
        # clipping, fewer Gaussian-tile keys) and empty pixels on the far plane
        variants["footprint_tile_rule"] = variant("footprint tile rule", cams,
                                                  tile_bound=tgs.TGS_TILES_FOOTPRINT, full=True)
        variants["empty_far"] = variant("empty pixels at z_far", cams, empty_far=1)
        for sp in ("depth_first", "per_tile"):
            if sp != args.sort_path:
                variants[f"sort_{sp}"] = variant(f"{sp} sort", cams, full=True, sort_path=sp)
        other = 2 if args.tgb_downscale == 1 else 1
        variants[f"tgb_downscale_{other}"] = variant(f"geometry buffer downscale x{other}", cams,
                                                     tgb_downscale=other)
    ablation = None
    if args.ablation:
        ablation = []
        for label, kw in (("all on", {}), ("no AFC", dict(enable_afc=0)),
                          ("no TOC", dict(enable_toc=0)), ("no SR", dict(enable_sr=0)),
                          ("lambda_SR 2", dict(lambda_sr=2)), ("lambda_SR 10", dict(lambda_sr=10)),
                          ("lambda_TDC 25", dict(lambda_tdc=25)), ("lambda_TDC 100", dict(lambda_tdc=100)),
                          ("eta 0.2", dict(eta=0.2)), ("eta 0.6", dict(eta=0.6)),
                          ("empty_far, footprint", dict(empty_far=1))):
            tb = tgs.TGS_TILES_FOOTPRINT if "footprint" in label else tgs.TGS_TILES_3SIGMA
            ablation.append(variant(label, cams, tile_bound=tb, steps=2, **kw))
        for v in (2.0, 4.0):
            cv = synth.workload(args.workload, n_frames=args.frames, speed=v).cameras
            ablation.append(variant(f"camera speed x{v:g}", cv, steps=2))
        if args.workload == "room":
            # the paper's interval study: one curve through key poses, sampled
            # at growing intervals of eye travel (faster camera)
            for iv in (0.01, 0.02, 0.04):
                cv = synth.keyframe_path(synth.ROOM_KEY_EYES, synth.ROOM_KEY_TARGETS, iv, W, H,
                                         n_frames=len(cams))
                ablation.append(variant(f"key-pose curve, interval {iv:g}", cv, steps=2,
                                        full=True))
        log("[bench] ablation done")

    n_tgs = sum(1 for i in kinds if i["frame_kind"] == tgs.TGS_FRAME_TGS)
    sr_pct = [100.0 * i["n_selected"] / (TX * TY) for i in kinds if i["frame_kind"] == tgs.TGS_FRAME_TGS]

    # roofline of the dominant kernel (largest summed time in the timed region)
    stage_ms = {k: v["ms"] for k, v in prof.items()}
    dom = max(("blend_ref", "blend_tgs"), key=lambda s: stage_ms[s])
    launches = prof[dom]["launches"]
    avg_s = stage_ms[dom] / launches * 1e-3
    pairs_per_launch = counted[dom]["pairs"] / max(1, counted[dom]["launches"])
    hits_per_launch = counted[dom]["hits"] / max(1, counted[dom]["launches"])
    achieved = BLEND_OPS_PER_HIT[dom] * hits_per_launch / avg_s / 1e12
    traffic = None
    if os.path.exists(TRAFFIC_FILE):
        tr = json.load(open(TRAFFIC_FILE))
        if tr.get("kernel_source_sha") == kernel_source_hash() and dom in tr.get("bytes_per_launch", {}):
            traffic = tr["bytes_per_launch"][dom]
    roofline = {"bound": "alu", "kernel": f"blend ({dom})", "achieved": round(achieved, 3),
                "peak": round(VALU_PEAK_TOPS, 2), "unit": "Tlane-op/s",
                "frac": round(achieved / VALU_PEAK_TOPS, 4), "traffic": traffic,
                "avg_launch_ms": round(avg_s * 1e3, 4), "hits_per_launch": int(hits_per_launch),
                "ops_per_hit": BLEND_OPS_PER_HIT[dom], "list_pairs_per_launch": int(pairs_per_launch)}

    # CPU oracle on a bounded sample of the same workload
    cpu = None
    if not args.no_cpu_baseline:
        from oracle import oracle as O
        nf = min(args.cpu_frames, n_frames)
        ora = O.TemporalOracle(wl.scene, W, H)
        t0 = time.perf_counter()
        for cam in cams[:nf]:
            ora.render(cam)
        dt = time.perf_counter() - t0
        cpu = {"value": round(nf / dt, 5), "unit": "frames/s", "cores": 1, "kind": "oracle",
               "sample": f"frames 0-{nf - 1} of the {n_frames}-frame temporal sequence "
                         f"(1 true reference + {nf - 1} TemporalGS frames), single-threaded C "
                         f"oracle, {dt:.1f} s on {os.cpu_count()} host cores"}
        log(f"[bench] cpu oracle: {nf} frames in {dt:.1f}s")

    per_frame = lambda s: round(detail[s]["ms"] / n_frames, 4)
    res = {
        "metric": METRIC, "value": round(fps_t, 2), "unit": "frames/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup,
        "ms_per_step": round(1e3 * t_temporal / args.steps, 3),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": synth.WORKLOADS.get(args.workload, args.workload),
                   "frames_per_step": n_frames, "gaussians": n, "width": W, "height": H,
                   "lambda_tdc": 50, "lambda_sr": 5, "eta": 0.4,
                   "tgb_downscale": args.tgb_downscale},
        "temporal": {"fps": round(fps_t, 2), "ms_per_frame": round(1e3 * t_temporal / (args.steps * n_frames), 4),
                     "ms_per_kind": {name: round(float(np.mean(v)), 4) if v else None
                                     for name, v in zip(("true_ref", "pseudo_ref", "tgs"),
                                                        (per_kind[0], per_kind[1], per_kind[2]))},
                     "tgsf_pct": round(100.0 * n_tgs / n_frames, 2),
                     "sr_tile_pct": round(float(np.mean(sr_pct)), 2) if sr_pct else None},
        "full": {"fps": round(fps_f, 2), "ms_per_frame": round(1e3 * t_full / (args.steps * n_frames), 4)},
        "speedup_temporal_vs_full": round(fps_t / fps_f, 3),
        "tile_rule": "3DGS 3-sigma square",
        "sort_path": args.sort_path,
        "blend_split_log2": args.blend_split,
        **variants,
        "psnr_temporal_vs_full": psnr,
        "ssim_temporal_vs_full": ssim,
        "memory": memory,
        "stage_ms_per_frame": {s: per_frame(s) for s in tgs.PROF_STAGES if detail[s]["ms"] > 0},
        "stage_full_ms_per_frame": {s: round(v["ms"] / n_frames, 4)
                                    for s, v in detail_full.items() if v["ms"] > 0},
        "stage_breakdown_note": "untimed pass with every stage bracketed by separately "
                                "recorded HIP events (each adds a queue barrier)",
        "roofline": roofline,
        "cpu_baseline": cpu,
    }
    if ablation is not None:
        res["ablation"] = ablation
    tgs.tgs_state_free(state_h)
    tgs.tgs_scene_free(scene_h)
    print(json.dumps(res), flush=True)


if __name__ == "__main__":
    main()
