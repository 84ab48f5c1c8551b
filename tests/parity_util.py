"""Helpers shared by the GPU parity tests: run the HIP path through the
C-ABI, run the oracle on the same inputs, compare element by element."""
from __future__ import annotations

import numpy as np

from oracle import oracle as O
from paper_2607_03390_amd import tgs

# Per-channel colour tolerance (absolute, on [0,1] colours).
RGB_TOL = 2e-4
# Eq. 1/2 tolerances: fp32 one-pass moments on the GPU vs two-pass fp64.
# Depth: 1e-5 D, or, where larger, the first-order bound of the fp32
# pivot form D = d0 + S1 / sum(w) over k composited Gaussians with depth
# spread s = max |d - d0| (depth_tol).
DEPTH_RTOL = 1e-5
U32 = 2.0 ** -24
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


def dumps(scene_h, state_h, n, lists=True):
    """Per-Gaussian records and flags of the last frame, and (``lists``) its
    sorted keys, values and tile ranges."""
    d = {}
    if lists:
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


def check_lists(d, ts, items, tiles=None, K=None):
    """Per-tile front-to-back lists bit-exact (all tiles, or `tiles`); K: the
    frame's key count when ts / items cover only `tiles`."""
    nt = ts.size - 1
    K = int(ts[-1]) if K is None else int(K)
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


def depth_tol(b):
    """Per-pixel tolerance of Eq. 1 depth: 1e-5 D, or the first-order bound
    of the fp32 arithmetic where that is larger.  The weights themselves
    differ by relative errors up to w_rel (the oracle's per-pixel bound: each
    alpha's exp2 on the two sides, carried through the transmittance chain
    before it), which move the weighted mean by at most 2 w_rel s,
    s = max |d - d0|.  Then the GPU's one-pass pivot form: S1 = sum w (d - d0)
    and sum(w) are sequential fp32 sums of k non-negative terms (lists are
    depth-ordered, so d >= d0), so m = S1 / sum(w) <= s carries about
    (2k + 16) u of relative error, and D = d0 + m one more rounding
    (u = 2^-24)."""
    D = b["D"]
    s = b["spread"].astype(np.float64)
    derived = U32 * (D + (2.0 * b["ninc"] + 16.0) * s) + 2.0 * b["wrel"].astype(np.float64) * s
    return np.maximum(DEPTH_RTOL * D, derived)


def check_moments(res, b, ok):
    hit = ok & (b["D"] != float(O.NOHIT))
    gD = res["depth"].astype(np.float64)
    assert np.array_equal(res["depth"][ok & ~hit], np.full((ok & ~hit).sum(), O.NOHIT, np.float32))
    if hit.any():
        r = np.where(hit, np.abs(gD - b["D"]) / depth_tol(b), 0.0)
        rel = np.where(hit, np.abs(gD - b["D"]) / b["D"], 0.0)
        log(f"    depth: worst error {r.max():.3f} of its tolerance, worst relative error {rel.max():.2e}")
        if r.max() > 1.0:
            y, x = np.unravel_index(np.argmax(r), r.shape)
            raise AssertionError(
                f"depth at pixel ({x}, {y}): gpu {gD[y, x]!r} oracle {b['D'][y, x]!r}, "
                f"{r[y, x]:.3f} of its tolerance; composited {b['ninc'][y, x]}, spread "
                f"{b['spread'][y, x]}, alpha gpu {res['alpha'][y, x]!r} oracle {b['alpha'][y, x]!r}, "
                f"rgb gpu {res['rgb'][:, y, x]} oracle {b['rgb'][:, y, x]}")
        serr = (np.abs(res["sigma"].astype(np.float64)[hit] - b["sigma"][hit]) / np.maximum(1.0, b["D"][hit])).max()
        assert serr <= SIGMA_TOL, f"sigma err {serr}"
    if ok.any():
        aerr = np.abs(res["alpha"].astype(np.float64)[ok] - b["alpha"][ok]).max()
        assert aerr <= ALPHA_TOL, f"alpha err {aerr}"


def check_gaussian_buffer(gpu_flag, b):
    """Temporal Gaussian buffer: certain members and certain non-members."""
    certain = b["g_certain"] > 0
    never = (b["maxw"] == 0) & (b["g_uncertain"] == 0)
    assert np.all(gpu_flag[certain]), f"{(~gpu_flag[certain]).sum()} certain members missing"
    assert not np.any(gpu_flag[never]), f"{gpu_flag[never].sum()} spurious members"


def import_into_oracle(ora, blob):
    """State injection: the GPU's priors after frame t replace the oracle's
    (its fp32 Eq. 1/2 and exp-driven blend would otherwise cascade ULP
    differences into the warp).  The schedule counters are not injected:
    the oracle's own drive its frame kinds, and compare_state has checked
    that the GPU's equal them."""
    st = tgs.parse_state(blob)
    ora.import_priors(st["D"], st["S"], st["tab"], st["g_rendered"], st["fbox"], st["ref_w2c"],
                      st["ref_intr"])
    return st


def compare_state(st, ora, prev, prev_kind, tgb_downscale=1, sample_px=None):
    """The GPU's exported state after frame t against the oracle's own state
    after the same frame, before any import for frame t+1.

    * counters and the reference pose: exact;
    * after a TemporalGS frame the priors are carried unchanged: exactly the
      ones imported before it;
    * after a reference frame: the temporal Gaussian buffer holds every
      Gaussian the oracle composites before a margin event and none it never
      composites; the adaptive frustum of a true reference is bit-equal to
      the oracle's (to the oracle's reduction over the GPU's buffer where the
      buffers differ at margin Gaussians); TGB depth / sigma at the Eq. 1/2
      tolerances and the TAB within the colour tolerance, margin pixels
      excluded.
    ``sample_px``: the pixels the oracle rendered (all if None); the buffer's
    non-members and the adaptive frustum are then checked through the
    reduction only.  Returns the margin pixels excluded."""
    counters = (st["frame_index"], st["since_true"], st["since_ref"], bool(st["force_pseudo"]))
    want = (ora.frame_index, ora.since_true, ora.since_ref, bool(ora.force_pseudo))
    assert counters == want, f"schedule counters: gpu {counters}, oracle {want}"
    assert st["has_reference"] == 1
    assert np.array_equal(st["ref_w2c"], ora.ref_w2c), "reference pose"
    assert np.array_equal(st["ref_intr"], ora.ref_intr), "reference intrinsics"
    if prev_kind == O.TGS_FRAME:
        assert np.array_equal(st["D"].view(np.uint32), ora.D.view(np.uint32)), "TGB depth changed"
        assert np.array_equal(st["S"].view(np.uint32), ora.S.view(np.uint32)), "TGB sigma changed"
        assert np.array_equal(st["tab"].view(np.uint32), ora.tab.view(np.uint32)), "TAB changed"
        assert np.array_equal(st["g_rendered"], ora.g_rendered), "Gaussian buffer changed"
        assert np.array_equal(st["fbox"].view(np.uint32), ora.fbox.view(np.uint32)), "frustum changed"
        return 0
    H, W = prev["margin_pos"].shape
    rendered = np.ones((H, W), bool) if sample_px is None else sample_px
    margin = rendered & (prev["margin_pos"] >= 0)
    ok = rendered & ~margin
    gpu_flag = st["g_rendered"] > 0
    certain = prev["g_certain"] > 0
    assert np.all(gpu_flag[certain]), f"{(~gpu_flag[certain]).sum()} certain members missing from the state"
    if sample_px is None:
        never = (prev["maxw"] == 0) & (prev["g_uncertain"] == 0)
        assert not np.any(gpu_flag[never]), f"{gpu_flag[never].sum()} spurious members in the state"
    # members are Gaussians with a tile rectangle this frame
    assert np.all(prev["g"]["status"][gpu_flag] == O.VISIBLE), "member without tiles"
    if prev_kind == O.TRUE_REF:
        if sample_px is None and np.array_equal(gpu_flag, ora.g_rendered > 0):
            want_box = ora.fbox
        else:
            want_box, _ = O.afc_bounds(st["g_rendered"], prev["g"]["ndc"])
        assert np.array_equal(st["fbox"].view(np.uint32), want_box.view(np.uint32)), \
            f"adaptive frustum {st['fbox']} vs {want_box}"
    else:
        assert np.array_equal(st["fbox"].view(np.uint32), ora.fbox.view(np.uint32)), \
            "frustum of a pseudo reference must be the imported one"
    if tgb_downscale == 2:
        check_pooled_tgb(st, ora, ~ok, prev)
    else:
        Dg, Sg = st["D"].astype(np.float64), st["S"].astype(np.float64)
        Do, So = ora.D.astype(np.float64), ora.S.astype(np.float64)
        empty = ok & ((Do == float(O.NOHIT)) | (Do == float(O.Z_FAR)))
        assert np.array_equal(Dg[empty], Do[empty]) and np.all(Sg[empty] == 0.0), "empty TGB pixels"
        hit = ok & ~empty
        if hit.any():
            tol = depth_tol(prev)
            ratio = (np.abs(Dg[hit] - Do[hit]) / tol[hit]).max()
            assert ratio <= 1.0, f"TGB depth err {ratio:.3f} of its tolerance"
            serr = (np.abs(Sg[hit] - So[hit]) / np.maximum(1.0, Do[hit])).max()
            assert serr <= SIGMA_TOL, f"TGB sigma err {serr}"
    check_image(st["tab"], ora.tab.astype(np.float64), ok, RGB_TOL, "TAB")
    return int(margin.sum())


# Bounds on what the margin rules may exclude (pixels whose blend takes a
# decision within the oracle's margin of a threshold; occluded-tile flags
# decided within it): a tolerance or margin bug that flagged many would
# otherwise weaken every check silently.
MARGIN_PX_FRAC = 1e-3
MARGIN_TILE_FRAC = 1e-3


def check_margin_bounds(stats, label="", px_frac=MARGIN_PX_FRAC):
    px, mpx = stats.get("px_checked", 0), stats.get("margin_px", 0)
    tl, mtl = stats.get("tiles_checked", 0), stats.get("margin_tiles", 0)
    log(f"    margins {label}: {mpx} of {px} pixels, {mtl} of {tl} tiles")
    assert mpx <= px_frac * max(px, 1), f"margin pixels {mpx} of {px}"
    assert mtl <= MARGIN_TILE_FRAC * max(tl, 1), f"margin tiles {mtl} of {tl}"


def tile_pixels(mask_tiles, W, H):
    m = np.repeat(np.repeat(mask_tiles.astype(bool), 16, 0), 16, 1)
    return m[:H, :W]


def check_pooled_tgb(st, ora, margin_px, prev=None):
    """Geometry buffer downscaled by 2: the GPU's Eq. 1/2 pooled over each
    2x2 block (exported state) against the oracle's, blocks that hold a
    margin pixel excluded; empty blocks carry the same empty depth.  Depth
    tolerance: the largest depth_tol of the block's pixels (the pooled
    depth is a weighted mean of theirs) plus the pooling's own roundings
    (8 u D), given the reference frame's oracle output ``prev``; else
    1e-5 D."""
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
        tol = DEPTH_RTOL * Do
        if prev is not None:
            pt = np.zeros((2 * Do.shape[0], 2 * Do.shape[1]))
            pt[:H, :W] = np.where(prev["ninc"] == 0, 0.0, depth_tol(prev))
            blk = pt.reshape(Do.shape[0], 2, Do.shape[1], 2).max(axis=(1, 3))
            tol = np.maximum(tol, blk + 8 * U32 * Do)
        ratio = (np.abs(Dg[hit] - Do[hit]) / tol[hit]).max()
        assert ratio <= 1.0, f"pooled depth err {ratio:.3f} of its tolerance"
        serr = (np.abs(Sg[hit] - So[hit]) / np.maximum(1.0, Do[hit])).max()
        assert serr <= SIGMA_TOL, f"pooled sigma err {serr}"


def check_lists_by_range(scene_h, state_h, counts, ts, items, tiles):
    """Lists of a frame with too many keys to copy whole: every tile's range
    length against the oracle's per-tile counts (``counts``: tile_start of
    all tiles), the ranges tiling [0, K) in tile order, and the lists of
    ``tiles`` (oracle lists ``ts``/``items``) copied range by range."""
    rng = tgs.tgs_debug_dump(scene_h, state_h, tgs.TGS_DUMP_TILE_RANGES).reshape(-1, 2).astype(np.int64)
    ln = rng[:, 1] - rng[:, 0]
    want = np.diff(counts)
    assert np.array_equal(ln, want), f"range lengths differ at {np.flatnonzero(ln != want)[:10]}"
    nz = ln > 0
    starts, ends = rng[nz, 0], rng[nz, 1]
    assert starts.size == 0 or (starts[0] == 0 and ends[-1] == counts[-1] and
                                np.array_equal(starts[1:], ends[:-1])), "ranges do not tile the keys"
    for t in tiles:
        a, b = int(rng[t, 0]), int(rng[t, 1])
        want_t = items[ts[t]:ts[t + 1]]
        assert b - a == want_t.size, f"tile {t}: {b - a} entries vs {want_t.size}"
        if b > a:
            v = tgs.tgs_debug_dump_range(scene_h, state_h, tgs.TGS_DUMP_SORTED_VALUES, a, b - a)
            k = tgs.tgs_debug_dump_range(scene_h, state_h, tgs.TGS_DUMP_SORTED_KEYS, a, b - a)
            assert np.all(k == t), f"tile {t}: foreign keys in its range"
            assert np.array_equal(v.astype(np.int64), want_t), f"tile {t}: list differs"


def sample_tiles_for(counts, TX, TY, seed=0, heavy=12, rand=40):
    """Tiles to check at sizes the oracle cannot blend whole: the longest
    lists, a random set and every 13th tile of the last (ragged) row."""
    rng = np.random.default_rng(seed)
    lens = np.diff(counts)
    top = np.argsort(lens, kind="stable")[-heavy:]
    return np.unique(np.concatenate([top, rng.choice(TX * TY, rand, replace=False),
                                     np.arange((TY - 1) * TX, TY * TX, 13)])).astype(np.int64)


# Per-scene settings of the library under test.
DEFAULT_SPLIT = (tgs.BLEND_SPLIT_DEFAULT, tgs.BLEND_SPLIT_MAX)


class Uploaded:
    """A scene on the device with its tile rule, sort path and blend split."""

    def __init__(self, scene, bound=tgs.TGS_TILES_3SIGMA, sort=tgs.SORT_AUTO, split=DEFAULT_SPLIT):
        self.scene, self.bound, self.sort, self.split = scene, bound, sort, split

    def __enter__(self):
        self.h = tgs.tgs_scene_upload(self.scene)
        tgs.tgs_scene_set_tile_bound(self.h, self.bound)
        tgs.tgs_scene_set_sort_path(self.h, self.sort)
        tgs.tgs_scene_set_blend_split(self.h, *self.split)
        return self.h

    def __exit__(self, *a):
        tgs.tgs_scene_free(self.h)


def full_parity(scene, cams, sample_tiles=None, label="", bound=tgs.TGS_TILES_3SIGMA,
                sort=tgs.SORT_AUTO, split=DEFAULT_SPLIT, by_range=False,
                margin_px_frac=MARGIN_PX_FRAC):
    """tgs_render_full against the oracle: records, lists (every tile; or, with
    ``by_range``, range lengths of every tile and the lists of the sampled
    ones), colour and moments (all tiles or ``sample_tiles``), the Gaussian
    buffer; margin exclusions bounded."""
    n = scene.n
    stats = dict(px_checked=0, margin_px=0)
    with Uploaded(scene, bound, sort, split) as h:
        for k, cam in enumerate(cams):
            W, H = cam.width, cam.height
            TX, TY = cam.tiles
            log(f"[full parity {label}] cam {k} {W}x{H} n={n} tile bound {bound}")
            res = gpu_full(h, cam, n)
            g = O.gaussians(scene, cam, tile_bound=bound)
            d = dumps(h, None, n, lists=not by_range)
            check_records(d, g)
            counts = O.tile_counts(g, TX, TY)
            assert res["n_keys"] == counts[-1] and res["n_survivors"] == g["n_survivors"]
            assert res["frame_kind"] == tgs.TGS_FRAME_FULL and np.all(res["tile_mask"] == 1)
            sample = None if sample_tiles is None else np.asarray(sample_tiles, np.int64)
            if by_range:
                ts, items = O.tile_lists(g, TX, TY, O.sample_mask(sample, TX, TY))
                check_lists_by_range(h, None, counts, ts, items, sample)
            else:
                ts, items = O.tile_lists(g, TX, TY)
                check_lists(d, ts, items)
            b = O.blend(W, H, ts, items, g, None if sample is None else sample.astype(np.int32),
                        bg=O.camera_bg(cam))
            rendered = O.sample_mask(sample, TX, TY).astype(bool)
            ok = tile_pixels(rendered, W, H) & (b["margin_pos"] < 0)
            worst = check_image(res["rgb"], b["rgb"], ok, where=f"cam {k}")
            check_moments(res, b, ok)
            if sample is None:
                check_gaussian_buffer(res["contrib"][:n] > 0, b)
            stats["px_checked"] += int(tile_pixels(rendered, W, H).sum())
            stats["margin_px"] += int((b["margin_pos"] >= 0).sum())
            log(f"    keys {int(counts[-1])} pairs {b['pairs']} max|drgb| {worst:.2e} "
                f"margin px {(b['margin_pos'] >= 0).sum()}")
    check_margin_bounds(stats, label, margin_px_frac)
    return stats


def temporal_parity(scene, cams, W, H, label, bound=tgs.TGS_TILES_3SIGMA, sort=tgs.SORT_AUTO,
                    split=DEFAULT_SPLIT, sample_tiles=None, by_range=False,
                    margin_px_frac=MARGIN_PX_FRAC, **pkw):
    """tgs_render_temporal over a camera stream against the oracle's own
    schedule.  Before every frame after the first, the GPU's exported state
    is compared with the oracle's (compare_state) and its priors, never its
    counters, are imported.  Per frame: frame kind, records, lists, warp /
    fill / correspondence buffers, unmatched / occluded / selected tiles,
    counts, colour of the rendered tiles and of the stitched ones.  With
    ``sample_tiles`` the oracle lists and blends only those tiles (the
    selected ones among them); ``by_range`` checks lists as in
    full_parity."""
    import torch
    n = scene.n
    tgb = pkw.get("tgb_downscale", 1)
    stats = dict(frames=0, tgs=0, kinds=[], margin_tiles=0, margin_px=0, px_checked=0,
                 tiles_checked=0)
    TX, TY = (W + 15) // 16, (H + 15) // 16
    sample = None if sample_tiles is None else np.asarray(sample_tiles, np.int64)
    smask = O.sample_mask(sample, TX, TY).astype(bool)
    spx = None if sample is None else tile_pixels(smask, W, H)
    with Uploaded(scene, bound, sort, split) as h:
        s = tgs.tgs_state_create(h, W, H, tgs.params(**pkw))
        ora = O.TemporalOracle(scene, W, H, O.Params(tile_bound=bound, **pkw))
        prev = prev_kind = None
        try:
            for k, cam in enumerate(cams):
                if k > 0:
                    # the GPU's state after frame k-1 against the oracle's
                    # own, then its priors (never the counters) injected
                    blob = tgs.tgs_state_export(s)
                    stats["margin_px_state"] = stats.get("margin_px_state", 0) + compare_state(
                        tgs.parse_state(blob), ora, prev, prev_kind, tgb, spx)
                    import_into_oracle(ora, blob)
                out = tgs.alloc_frame(W, H, n, depth=True, contrib=True, tile_mask=True)
                log(f"[temporal parity {label}] frame {k}")
                info = tgs.tgs_render_temporal(s, cam, **out)
                torch.cuda.synchronize()
                res = {kk: v.cpu().numpy() for kk, v in out.items()}
                ref = ora.render(cam, sample_tiles=sample)
                assert info["frame_kind"] == ref["kind"], (k, info["frame_kind"], ref["kind"])
                prev, prev_kind = ref, ref["kind"]
                stats["kinds"].append(ref["kind"])
                d = dumps(None, s, n, lists=not by_range)
                check_records(d, ref["g"])
                stats["frames"] += 1
                sel_tiles = res["tile_mask"].astype(bool)
                sel_ref = ref["tile_sel"].astype(bool)
                counts = O.tile_counts(ref["g"], TX, TY, ref["tile_sel"])
                listed = np.flatnonzero((sel_ref & smask).ravel())

                def lists_equal():
                    if by_range:
                        check_lists_by_range(None, s, counts, ref["tile_start"], ref["items"], listed)
                    else:
                        check_lists(d, ref["tile_start"], ref["items"], tiles=listed, K=counts[-1])
                    assert info["n_keys"] == counts[-1]

                if ref["kind"] == O.TGS_FRAME:
                    stats["tgs"] += 1
                    Hg, Wg = ref["dmin"].shape   # the geometry buffer's grid
                    dm = tgs.tgs_debug_dump(None, s, tgs.TGS_DUMP_WARP_DEPTH).reshape(Hg, Wg)
                    sm = tgs.tgs_debug_dump(None, s, tgs.TGS_DUMP_WARP_SIGMA).reshape(Hg, Wg)
                    df = tgs.tgs_debug_dump(None, s, tgs.TGS_DUMP_FILLED_DEPTH).reshape(Hg, Wg)
                    uv = tgs.tgs_debug_dump(None, s, tgs.TGS_DUMP_CORRESPONDENCE).reshape(Hg, Wg, 2)
                    um = tgs.tgs_debug_dump(None, s, tgs.TGS_DUMP_UNMATCHED).reshape(TY, TX)
                    oc = tgs.tgs_debug_dump(None, s, tgs.TGS_DUMP_OCCLUDED).reshape(TY, TX)
                    assert np.array_equal(dm.view(np.uint32), ref["dmin"].view(np.uint32)), "warped depth"
                    assert np.array_equal(sm, ref["smax"]), "warped sigma"
                    assert np.array_equal(df.view(np.uint32), ref["dfill"].view(np.uint32)), "filled depth"
                    assert np.array_equal(uv.view(np.uint32), ref["uv"].view(np.uint32)), "correspondences"
                    assert np.array_equal(um, ref["um"]), "unmatched tiles"
                    differ = oc != ref["oc"]
                    assert not np.any(differ & (ref["oc_margin"] == 0)), "occluded tiles"
                    stats["margin_tiles"] += int(differ.sum())
                    stats["tiles_checked"] += TX * TY
                    if np.array_equal(sel_tiles, sel_ref):
                        lists_equal()
                    else:
                        log(f"    selection differs only at margin tiles {np.flatnonzero(differ.ravel())}")
                    assert info["n_selected"] == int(sel_tiles.sum())
                    assert info["n_survivors"] == ref["n_survivors"]
                    assert info["n_newly_visible"] == int(ref["g"]["newly_visible"].sum())
                    rend = tile_pixels(sel_tiles & sel_ref & smask, W, H)
                    stitched = tile_pixels(~sel_tiles & ~sel_ref, W, H)
                    ok = rend & (ref["margin_pos"] < 0)
                    check_image(res["rgb"], ref["rgb"], ok, RGB_TOL, f"frame {k} rendered tiles")
                    check_image(res["rgb"], ref["rgb"], stitched, STITCH_TOL, f"frame {k} stitched tiles")
                    stats["margin_px"] += int((rend & (ref["margin_pos"] >= 0)).sum())
                    stats["px_checked"] += int(rend.sum())
                else:
                    assert np.all(sel_tiles)
                    lists_equal()
                    assert info["n_survivors"] == ref["n_survivors"]
                    rend = tile_pixels(smask, W, H)
                    ok = rend & (ref["margin_pos"] < 0)
                    check_image(res["rgb"], ref["rgb"], ok, RGB_TOL, f"frame {k} reference")
                    check_moments(res, ref, ok)
                    if sample is None:
                        check_gaussian_buffer(res["contrib"][:n] > 0, ref)
                    else:
                        assert np.all(res["contrib"][:n][ref["g_certain"] > 0] > 0)
                    stats["margin_px"] += int((rend & ~ok).sum())
                    stats["px_checked"] += int(rend.sum())
                log(f"    kind {info['frame_kind']} sel {info['n_selected']} keys {info['n_keys']} "
                    f"surv {info['n_survivors']} newly {info['n_newly_visible']}")
            # the state after the last frame as well
            compare_state(tgs.parse_state(tgs.tgs_state_export(s)), ora, prev, prev_kind, tgb, spx)
        finally:
            tgs.tgs_state_free(s)
    log(f"[temporal parity {label}] {stats}")
    check_margin_bounds(stats, label, margin_px_frac)
    return stats
