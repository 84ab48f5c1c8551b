"""Helpers shared by the GPU parity tests: run the HIP path through the
C-ABI, run the oracle on the same inputs, compare element by element."""
from __future__ import annotations

import numpy as np

from oracle import oracle as O
from paper_2607_03390_amd import tgs

# Per-channel colour tolerance (absolute, on [0,1] colours).
RGB_TOL = 2e-4
# Eq. 1/2 tolerances: fp32 one-pass moments on the GPU vs two-pass fp64.
DEPTH_RTOL = 1e-5
SIGMA_TOL = 1e-4
ALPHA_TOL = 2e-4
# fp32 SH colour of the preprocess vs fp64.
COLOUR_TOL = 1e-5
# stitched pixels: fp32 bilinear vs fp64 of the same fp32 samples
STITCH_TOL = 1e-5


def log(msg):
    print(msg, flush=True)


def gpu_full(scene_h, cam, n, depth=True, contrib=True):
    import torch
    out = tgs.alloc_frame(cam.width, cam.height, n, depth=depth, contrib=contrib, tile_mask=True)
    info = tgs.tgs_render_full(scene_h, cam, **out)
    torch.cuda.synchronize()
    res = {k: v.cpu().numpy() for k, v in out.items()}
    res.update(info)
    return res


def dumps(scene_h, state_h, n):
    d = {}
    d["vals"] = tgs.tgs_debug_dump(scene_h, state_h, tgs.TGS_DUMP_SORTED_VALUES)
    d["keys"] = tgs.tgs_debug_dump(scene_h, state_h, tgs.TGS_DUMP_SORTED_KEYS)
    d["ranges"] = tgs.tgs_debug_dump(scene_h, state_h, tgs.TGS_DUMP_TILE_RANGES).reshape(-1, 2)
    d["records"] = tgs.tgs_debug_dump(scene_h, state_h, tgs.TGS_DUMP_RECORDS).reshape(n, 12)
    d["rects"] = tgs.tgs_debug_dump(scene_h, state_h, tgs.TGS_DUMP_RECTS).reshape(n, 4)
    d["status"] = tgs.tgs_debug_dump(scene_h, state_h, tgs.TGS_DUMP_STATUS)
    return d


def check_records(d, g):
    """Projection, conic, depth and rectangle bit-exact; colour within tol."""
    vis = g["status"] == O.VISIBLE
    gpu_vis = d["rects"][:, 0] <= d["rects"][:, 2]
    assert np.array_equal(vis, gpu_vis), f"visible sets differ: {np.flatnonzero(vis != gpu_vis)[:10]}"
    surv = g["status"] >= O.DEGENERATE
    assert np.array_equal(surv, (d["status"] & 1) > 0), "survivor flags differ"
    assert np.array_equal(g["newly_visible"] > 0, (d["status"] & 2) > 0), "newly-visible flags differ"
    r = d["records"][vis]
    assert np.array_equal(d["rects"][vis].astype(np.int32), g["rect"][vis]), "tile rectangles differ"
    assert np.array_equal(r[:, 0:2].view(np.uint32), g["mean2d"][vis].view(np.uint32)), "means differ"
    conic = np.stack([r[:, 2], r[:, 3], r[:, 4]], 1)
    assert np.array_equal(conic.view(np.uint32), g["conic"][vis].view(np.uint32)), "conics differ"
    assert np.array_equal(r[:, 6].view(np.uint32), g["depth"][vis].view(np.uint32)), "depths differ"
    if vis.any():
        err = np.abs(r[:, 8:11].astype(np.float64) - g["rgb"][vis]).max()
        assert err <= COLOUR_TOL, f"SH colour error {err}"


def check_lists(d, ts, items, tiles=None):
    """Per-tile front-to-back lists bit-exact (all tiles, or `tiles`)."""
    nt = ts.size - 1
    K = int(ts[-1])
    assert d["vals"].size == K, f"key count {d['vals'].size} vs {K}"
    keys = d["keys"]
    assert np.all(keys[1:] >= keys[:-1]), "keys not sorted"
    for t in (range(nt) if tiles is None else tiles):
        a, b = d["ranges"][t]
        want = items[ts[t]:ts[t + 1]]
        if b - a != want.size or not np.array_equal(d["vals"][a:b].astype(np.int64), want):
            raise AssertionError(f"tile {t}: list differs (gpu {b - a}, oracle {want.size})")


def check_image(rgb, ref_rgb, ok_mask, tol=RGB_TOL, where=""):
    err = np.abs(rgb.astype(np.float64) - ref_rgb)
    worst = err[:, ok_mask].max() if ok_mask.any() else 0.0
    assert worst <= tol, f"{where} max |drgb| {worst:.3e} > {tol}"
    return worst


def check_moments(res, b, ok):
    hit = ok & (b["D"] != float(O.NOHIT))
    gD = res["depth"].astype(np.float64)
    assert np.array_equal(res["depth"][ok & ~hit], np.full((ok & ~hit).sum(), O.NOHIT, np.float32))
    if hit.any():
        rel = (np.abs(gD[hit] - b["D"][hit]) / b["D"][hit]).max()
        assert rel <= DEPTH_RTOL, f"depth rel err {rel}"
        serr = (np.abs(res["sigma"].astype(np.float64)[hit] - b["sigma"][hit]) / np.maximum(1.0, b["D"][hit])).max()
        assert serr <= SIGMA_TOL, f"sigma err {serr}"
    aerr = np.abs(res["alpha"].astype(np.float64)[ok] - b["alpha"][ok]).max()
    assert aerr <= ALPHA_TOL, f"alpha err {aerr}"


def check_gaussian_buffer(gpu_flag, b):
    """Temporal Gaussian buffer: certain members and certain non-members."""
    certain = b["g_certain"] > 0
    never = (b["maxw"] == 0) & (b["g_uncertain"] == 0)
    assert np.all(gpu_flag[certain]), f"{(~gpu_flag[certain]).sum()} certain members missing"
    assert not np.any(gpu_flag[never]), f"{gpu_flag[never].sum()} spurious members"


def import_into_oracle(ora, blob):
    st = tgs.parse_state(blob)
    ora.import_state(st["D"], st["S"], st["tab"], st["g_rendered"], st["fbox"], st["ref_w2c"],
                     st["ref_intr"], st["frame_index"], st["since_true"], st["since_ref"],
                     st["force_pseudo"])
    return st


def tile_pixels(mask_tiles, W, H):
    m = np.repeat(np.repeat(mask_tiles.astype(bool), 16, 0), 16, 1)
    return m[:H, :W]


def check_pooled_tgb(st, ora, margin_px):
    """Geometry buffer downscaled by 2: the GPU's Eq. 1/2 pooled over each
    2x2 block (exported state) against the oracle's, blocks that hold a
    margin pixel excluded; empty blocks carry the same empty depth."""
    Dg, Sg = st["D"].astype(np.float64), st["S"].astype(np.float64)
    Do, So = ora.D.astype(np.float64), ora.S.astype(np.float64)
    assert Dg.shape == Do.shape, (Dg.shape, Do.shape)
    H, W = margin_px.shape
    m = np.zeros((2 * Do.shape[0], 2 * Do.shape[1]), bool)
    m[:H, :W] = margin_px
    ok = ~m.reshape(Do.shape[0], 2, Do.shape[1], 2).any(axis=(1, 3))
    empty = ok & ((Do == float(O.NOHIT)) | (Do == float(O.Z_FAR)))
    assert np.array_equal(Dg[empty], Do[empty]) and np.all(Sg[empty] == 0.0), "empty blocks differ"
    hit = ok & ~empty
    if hit.any():
        rel = (np.abs(Dg[hit] - Do[hit]) / Do[hit]).max()
        assert rel <= DEPTH_RTOL, f"pooled depth rel err {rel}"
        serr = (np.abs(Sg[hit] - So[hit]) / np.maximum(1.0, Do[hit])).max()
        assert serr <= SIGMA_TOL, f"pooled sigma err {serr}"
