"""GPU parity: the HIP path through the C-ABI against the CPU oracle on the
same seeded inputs.

Bit-exact: survivors, newly-visible flags, projected means, conics, depths,
tile rectangles, key counts, every per-tile sorted list, the warped depth and
sigma buffers, the repaired depth, correspondences, unmatched / occluded /
selected tile masks.  Within tolerance: colour (2e-4), Eq. 1/2 moments,
alpha, stitched pixels.  Pixels (and occluded tiles) whose blending takes a
decision within the oracle's margin of a threshold are excluded and counted.
Temporal frames use state injection: the GPU's priors after frame t are
imported into the oracle before both render frame t+1, after the GPU's
exported state has been compared with the oracle's own (schedule counters,
adaptive frustum, temporal Gaussian buffer, TGB, TAB); the schedule counters
are never injected, so the oracle's own decide every frame kind.  Margin
exclusions are bounded per test.
"""
import numpy as np
import pytest

from oracle import oracle as O
from paper_2607_03390_amd import synth, tgs
from tests.parity_util import Uploaded as Up
from tests.parity_util import full_parity, gpu_full, log, temporal_parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    torch.cuda.set_device(0)
    tgs.lib()


# Per-scene settings applied by Uploaded: the sort path and the blend split.
SETTINGS = dict(sort=tgs.SORT_AUTO, split=(tgs.BLEND_SPLIT_DEFAULT, tgs.BLEND_SPLIT_MAX))


# Every parity case runs with both ways of producing per-tile depth order
# (global depth sort first; per-tile sort after the tile sort): the lists
# must be the oracle's either way.
@pytest.fixture(autouse=True, params=[tgs.SORT_DEPTH_FIRST, tgs.SORT_PER_TILE],
                ids=["depth_first", "per_tile"])
def sort_path(request):
    SETTINGS["sort"] = request.param
    yield request.param
    SETTINGS["sort"] = tgs.SORT_AUTO


class Uploaded(Up):
    def __init__(self, scene, bound=tgs.TGS_TILES_3SIGMA):
        super().__init__(scene, bound, SETTINGS["sort"], SETTINGS["split"])


def _full_parity(scene, cams, sample_tiles=None, label="", bound=tgs.TGS_TILES_3SIGMA, **kw):
    return full_parity(scene, cams, sample_tiles, label, bound, SETTINGS["sort"], SETTINGS["split"],
                       **kw)


def _temporal_parity(scene, cams, W, H, label, bound=tgs.TGS_TILES_3SIGMA, **pkw):
    return temporal_parity(scene, cams, W, H, label, bound, SETTINGS["sort"], SETTINGS["split"],
                           **pkw)


def test_full_parity_tiny_orbit():
    w = synth.workload("tiny")
    _full_parity(w.scene, w.cameras, label="tiny")


@pytest.mark.parametrize("n,seed,deg,W,H", [(3000, 1, 3, 200, 136), (500, 2, 2, 37, 53),
                                            (50, 3, 1, 1, 1), (2000, 4, 0, 300, 17),
                                            (4000, 5, 3, 64, 64)])
def test_full_parity_ragged(n, seed, deg, W, H):
    sc = synth.small_scene(n, seed, degree=deg)
    cams = [synth.make_camera(synth.look_at(e, (0, 0, 0)), W, H)
            for e in ((0.2, -3.0, 0.7), (2.5, 1.0, -0.4), (0.0, -1.2, 0.1))]
    _full_parity(sc, cams, label=f"ragged {W}x{H}")


def test_full_render_independent_of_earlier_sizes():
    """A render depends on its inputs only, not on the frames before it (the
    scene's workspace, blend order and split set are the frame's own):
    renders at changing sizes on one scene equal, bit for bit, the renders
    of a scene that sees each camera once."""
    sc = synth.small_scene(3000, 1, degree=3)
    eyes = ((0.2, -3.0, 0.7), (2.5, 1.0, -0.4), (0.0, -1.2, 0.1), (1.0, 2.0, 0.3), (-2.0, 0.5, 0.2))
    sizes = ((200, 136), (64, 64), (200, 136), (200, 136), (37, 53))
    cams = [synth.make_camera(synth.look_at(e, (0, 0, 0)), W, H) for e, (W, H) in zip(eyes, sizes)]
    with Uploaded(sc) as h:
        seq = [gpu_full(h, c, sc.n) for c in cams]
    for c, got in zip(cams, seq):
        with Uploaded(sc) as h:
            ref = gpu_full(h, c, sc.n)
        for k in ("rgb", "depth", "sigma", "alpha", "contrib", "tile_mask"):
            assert np.array_equal(got[k], ref[k]), (k, c.width, c.height)


def test_full_render_after_split_change():
    """The quadrant split follows the scene's current setting: alternating
    split caps on one scene of long lists give the renders of fresh scenes
    with each cap."""
    sc = synth.scene_uniform_cube(24_000, 11, degree=0, log_scale_mean=-2.6)
    cam = synth.make_camera(synth.look_at((0.0, -7.0, 0.5), (0, 0, 0)), 48, 40)
    caps = ((0, 40), (0, 8), (0, 40), (0, 8))
    with Uploaded(sc) as h:
        seq = []
        for split in caps:
            tgs.tgs_scene_set_blend_split(h, *split)
            seq.append(gpu_full(h, cam, sc.n))
    for split, got in zip(caps, seq):
        with Uploaded(sc) as h:
            tgs.tgs_scene_set_blend_split(h, *split)
            ref = gpu_full(h, cam, sc.n)
        for k in ("rgb", "depth", "sigma", "alpha", "contrib", "tile_mask"):
            assert np.array_equal(got[k], ref[k]), (k, split)


@pytest.mark.parametrize("n,seed,deg,W,H", [(3000, 1, 3, 200, 136), (2000, 4, 0, 300, 17)])
def test_full_parity_footprint_tiles(n, seed, deg, W, H):
    sc = synth.small_scene(n, seed, degree=deg)
    rng = np.random.default_rng(seed)
    low = rng.random(n) < 0.2          # opacities around the 1/255 cut
    sc.opacities[low] = rng.uniform(0.002, 0.01, low.sum()).astype(np.float32)
    cams = [synth.make_camera(synth.look_at(e, (0, 0, 0)), W, H)
            for e in ((0.2, -3.0, 0.7), (2.5, 1.0, -0.4))]
    _full_parity(sc, cams, label=f"footprint {W}x{H}", bound=tgs.TGS_TILES_FOOTPRINT)


def test_long_tile_lists(sort_path):
    """Tile lists above the per-tile sort's LDS bound (4096 entries): its
    in-block radix path, against the oracle's lists."""
    sc = synth.scene_uniform_cube(24_000, 11, degree=0, log_scale_mean=-2.6)
    cam = synth.make_camera(synth.look_at((0.0, -7.0, 0.5), (0, 0, 0)), 48, 40)
    g = O.gaussians(sc, cam)
    ts, _ = O.tile_lists(g, *cam.tiles)
    longest = int(np.diff(ts).max())
    log(f"    longest tile list {longest}")
    assert longest > 4096
    _full_parity(sc, [cam], label="long lists")


def test_long_lists_after_short_ones(sort_path):
    """Long lists in a frame after one whose lists were all short: the
    per-tile sort then has no launch for long lists and sorts them in its
    short-list kernel over global memory."""
    sc = synth.scene_uniform_cube(24_000, 11, degree=0, log_scale_mean=-2.6)
    # the first camera looks away from the cube at a corner of it
    away = synth.make_camera(synth.look_at((0.0, -7.0, 0.5), (6.0, -14.0, 0.5)), 48, 40)
    near = synth.make_camera(synth.look_at((0.0, -7.0, 0.5), (0, 0, 0)), 48, 40)
    lengths = []
    for cam in (away, near):
        ts, _ = O.tile_lists(O.gaussians(sc, cam), *cam.tiles)
        lengths.append(int(np.diff(ts).max()))
    log(f"    longest tile lists {lengths}")
    assert lengths[0] < 1024 and lengths[1] > 4096
    _full_parity(sc, [away, near], label="long after short")


@pytest.fixture(params=[(0, tgs.BLEND_SPLIT_MAX), (0, 40)], ids=["split_all", "split_capped"])
def split_all(request):
    """Quadrant blocks for every tile with a non-empty list, or (capped) for
    the tiles of the longest length classes that hold at most 40 tiles, the
    other tiles whole."""
    SETTINGS["split"] = request.param
    yield request.param
    SETTINGS["split"] = (tgs.BLEND_SPLIT_DEFAULT, tgs.BLEND_SPLIT_MAX)


@pytest.mark.parametrize("n,seed,deg,W,H", [(3000, 1, 3, 200, 136), (500, 2, 2, 37, 53),
                                            (4000, 5, 3, 64, 64)])
def test_split_blend_full_parity(split_all, n, seed, deg, W, H):
    """Quadrant blocks (the first 64 tiles of the blend order) next to whole
    tiles, ragged images: colour, moments and the Gaussian buffer against the
    oracle."""
    sc = synth.small_scene(n, seed, degree=deg)
    cams = [synth.make_camera(synth.look_at(e, (0, 0, 0)), W, H)
            for e in ((0.2, -3.0, 0.7), (2.5, 1.0, -0.4))]
    _full_parity(sc, cams, label=f"split {W}x{H}")


def test_split_blend_long_lists(split_all):
    """Quadrant blocks on lists of several thousand entries (many batches,
    pixels stopping inside a group of four entries)."""
    sc = synth.scene_uniform_cube(24_000, 11, degree=0, log_scale_mean=-2.6)
    cam = synth.make_camera(synth.look_at((0.0, -7.0, 0.5), (0, 0, 0)), 48, 40)
    _full_parity(sc, [cam], label="split long lists")


@pytest.mark.parametrize("pkw", [dict(), dict(tgb_downscale=2)])
def test_split_blend_temporal_parity(split_all, pkw):
    """Reference frames (capture of Eq. 1/2, pooled 2x2 geometry buffer on a
    ragged grid) and TemporalGS frames (split selected tiles, stitched tiles
    shifted past the quadrant blocks) with quadrant blocks."""
    sc = synth.scene_room(60_000, 2)
    cams = synth.handheld_path(10, (0.0, -5.0, 0.3), (0.0, 0.0, 0.0), 0.3, 0.01, 401, 233)
    st = _temporal_parity(sc, cams, 401, 233, f"split room60k {pkw}", **pkw)
    assert st["tgs"] >= 3


def test_split_blend_determinism(split_all):
    """Which tiles are split depends on whole length classes, never on the
    order of tiles within one: a replay gives the same bits."""
    import torch
    w = synth.workload("tiny", n_frames=4)
    with Uploaded(w.scene) as h:
        runs = []
        for rep in range(2):
            frames = []
            for cam in w.cameras:
                o = tgs.alloc_frame(256, 256, w.scene.n, depth=True)
                tgs.tgs_render_full(h, cam, **o)
                torch.cuda.synchronize()
                frames.append(torch.cat([o["rgb"].flatten(), o["depth"].flatten(),
                                         o["sigma"].flatten()]).cpu().numpy())
            runs.append(frames)
        for a, b in zip(*runs):
            assert np.array_equal(a.view(np.uint32), b.view(np.uint32))


def test_split_blend_pair_count(split_all):
    """Evaluated pairs and hits of quadrant blocks: one count per pixel for
    the entries up to its stopping one, one per entry for the hits."""
    w = synth.workload("tiny", n_frames=2)
    with Uploaded(w.scene) as h:
        for cam in w.cameras:
            tgs.tgs_profile_start(count_pairs=True)
            gpu_full(h, cam, w.scene.n, depth=False, contrib=False)
            prof = tgs.tgs_profile_stop()
            r = O.render_full(w.scene, cam)
            got, hits = prof["blend_full"]["pairs"], prof["blend_full"]["hits"]
            log(f"    split: pairs gpu {got} oracle {r['pairs']}; hits gpu {hits} oracle {r['hits']}")
            assert abs(got - r["pairs"]) <= 1e-3 * r["pairs"]
            assert abs(hits - r["hits"]) <= 1e-3 * r["hits"]


@pytest.mark.parametrize("W,H,log_scale", [(3840, 2160, -3.6), (7680, 4320, -3.6),
                                           (3840, 2160, -2.2)])
def test_full_parity_large_grids(W, H, log_scale):
    """Tile grids of 240 x 135 and 480 x 270 (tile-sort passes of 8 + 7 and
    6 + 6 + 5 bits over 15- and 17-bit tile ids; the tile order in several
    rounds), and 35M keys on the first (the radix column scan's long-table
    path, key buffers grown after an overflow): lists bit-exact, colour on
    sampled tiles."""
    sc = synth.small_scene(20_000, 13, degree=1, log_scale_mean=log_scale)
    cam = synth.make_camera(synth.look_at((0.0, -3.0, 1.0), (0, 0, 0)), W, H)
    TX, TY = cam.tiles
    sample = np.random.default_rng(1).choice(TX * TY, 60, replace=False)
    _full_parity(sc, [cam], sample_tiles=sample, label=f"grid {TX}x{TY}")


def test_full_parity_object_subset():
    w = synth.workload("object", n_gaussians=40_000)
    _full_parity(w.scene, [w.cameras[0], w.cameras[37]], label="object 40k")


def test_key_capacity_growth():
    """Frames whose Gaussian-tile keys exceed the key buffers (first sized
    4N + 65536) render again after the buffers grow: a few thousand large
    Gaussians seen from ever closer, so the capacity grows more than once."""
    sc = synth.small_scene(3000, 11, degree=1, log_scale_mean=-1.6)
    cams = [synth.make_camera(synth.look_at((0.0, -d, 0.4 * d), (0, 0, 0)), 512, 384)
            for d in (3.2, 2.2, 1.5)]
    g = O.gaussians(sc, cams[-1])
    vis = g["status"] == O.VISIBLE
    r = g["rect"][vis]
    K = int(((r[:, 2] - r[:, 0] + 1) * (r[:, 3] - r[:, 1] + 1)).sum())
    assert K > 2 * (4 * sc.n + 65536), K
    # pixels here evaluate hundreds of large Gaussians each, so more of them
    # take a decision within the oracle's margin (1.2e-3 measured)
    _full_parity(sc, cams, label="capacity growth", margin_px_frac=2e-3)
    st = _temporal_parity(sc, cams, 512, 384, "capacity growth", margin_px_frac=2e-3)
    assert st["frames"] == 3


def test_empty_and_invisible_scenes():
    import torch
    sc = synth.small_scene(0, 0, degree=0)
    cam = synth.make_camera(synth.look_at((0, -3, 0), (0, 0, 0)), 48, 40)
    with Uploaded(sc) as h:
        res = gpu_full(h, cam, 0)
        assert res["n_keys"] == 0 and np.all(res["rgb"] == 0) and np.all(res["depth"] == O.NOHIT)
        assert np.all(res["alpha"] == 0) and np.all(res["sigma"] == 0)
    sc = synth.small_scene(300, 1, degree=1)
    back = synth.make_camera(synth.look_at((0, -3, 0), (0, -6, 0)), 48, 40)   # looks away
    with Uploaded(sc) as h:
        res = gpu_full(h, back, sc.n)
        assert res["n_keys"] == 0 and res["n_survivors"] == 0 and np.all(res["rgb"] == 0)
        s = tgs.tgs_state_create(h, 48, 40, tgs.params())
        out = tgs.alloc_frame(48, 40, sc.n)
        for _ in range(3):
            info = tgs.tgs_render_temporal(s, back, **out)
            torch.cuda.synchronize()
            assert info["n_keys"] == 0 and torch.all(out["rgb"] == 0)
        tgs.tgs_state_free(s)


def test_temporal_parity_tiny():
    w = synth.workload("tiny")
    st = _temporal_parity(w.scene, w.cameras, 256, 256, "tiny")
    assert st["tgs"] >= 1


def test_parity_background_colour():
    """A camera background (rgb = sum of w c + T bg): full renders and a
    temporal sequence, whose stitched pixels carry the reference's
    background."""
    w = synth.workload("tiny", n_frames=6)
    for c in w.cameras:
        c.bg = (0.25, 0.5, 0.125)
    _full_parity(w.scene, w.cameras[:2], label="tiny background")
    st = _temporal_parity(w.scene, w.cameras, 256, 256, "tiny background")
    assert st["tgs"] >= 1


def test_temporal_parity_tiny_empty_far():
    w = synth.workload("tiny")
    st = _temporal_parity(w.scene, w.cameras, 256, 256, "tiny empty_far", empty_far=1)
    assert st["tgs"] >= 4


@pytest.mark.parametrize("pkw", [dict(), dict(lambda_sr=2), dict(enable_toc=0),
                                 dict(enable_afc=0, eta=1.0), dict(enable_sr=0),
                                 dict(empty_far=1), dict(tgb_downscale=2),
                                 dict(tgb_downscale=2, empty_far=1)])
def test_temporal_parity_room_subset(pkw):
    sc = synth.scene_room(60_000, 2)
    cams = synth.handheld_path(12, (0.0, -5.0, 0.3), (0.0, 0.0, 0.0), 0.3, 0.01, 400, 232)
    st = _temporal_parity(sc, cams, 400, 232, f"room60k {pkw}", **pkw)
    assert st["tgs"] >= 3


def test_temporal_parity_tgb_half_ragged():
    # odd width and height: partial 2x2 blocks on the last column and row
    sc = synth.scene_room(60_000, 2)
    cams = synth.handheld_path(10, (0.0, -5.0, 0.3), (0.0, 0.0, 0.0), 0.3, 0.01, 401, 233)
    st = _temporal_parity(sc, cams, 401, 233, "room60k ragged tgb/2", tgb_downscale=2)
    assert st["tgs"] >= 3


def test_temporal_parity_tiny_tgb_half():
    w = synth.workload("tiny")
    st = _temporal_parity(w.scene, w.cameras, 256, 256, "tiny tgb/2", tgb_downscale=2, empty_far=1)
    assert st["tgs"] >= 4


def test_temporal_parity_room_subset_footprint_tiles():
    sc = synth.scene_room(60_000, 2)
    cams = synth.handheld_path(12, (0.0, -5.0, 0.3), (0.0, 0.0, 0.0), 0.3, 0.01, 400, 232)
    st = _temporal_parity(sc, cams, 400, 232, "room60k footprint", bound=tgs.TGS_TILES_FOOTPRINT)
    assert st["tgs"] >= 3


def test_temporal_parity_cube_occlusion():
    sc = synth.scene_uniform_cube(20_000, 7, degree=1, log_scale_mean=-3.3)
    cams = synth.orbit_path(10, 3.0, 15.0, 1.0, 144, 120)
    st = _temporal_parity(sc, cams, 144, 120, "cube20k", eta=1.0)
    assert st["tgs"] >= 5


def test_temporal_parity_eta_insertion():
    """A sequence whose pseudo references all come from the eta rule
    (Sec. III-E adaptive reference insertion): slow orbit steps select
    under 80 % of the tiles, every fourth step jumps 6 degrees and selects
    more, and lambda_SR = 10 is never reached.  Frame kinds come from the
    oracle's own counters."""
    sc = synth.scene_room(60_000, 2)
    cams = synth.orbit_path(16, 5.0, 10.0, 0.0, 400, 232, steps=(0.3, 0.3, 0.3, 6.0))
    st = _temporal_parity(sc, cams, 400, 232, "room60k eta", empty_far=1, lambda_sr=10, eta=0.8)
    kinds = st["kinds"]
    assert kinds.count(O.PSEUDO_REF) >= 3 and kinds.count(O.TGS_FRAME) >= 6
    # a pseudo reference follows a TemporalGS frame before lambda_SR frames
    # have passed: only the eta rule inserts it
    assert all(kinds[i - 1] == O.TGS_FRAME for i, kd in enumerate(kinds) if kd == O.PSEUDO_REF)
    # and the rule does not fire on every TemporalGS frame
    assert any(kinds[i] == O.TGS_FRAME and kinds[i + 1] == O.TGS_FRAME for i in range(len(kinds) - 1))


def test_force_all_dirty_no_cull_equals_full():
    import torch
    w = synth.workload("tiny", n_frames=5)
    with Uploaded(w.scene) as h:
        s = tgs.tgs_state_create(h, 256, 256, tgs.params(enable_afc=0, enable_toc=0, force_all_dirty=1))
        for cam in w.cameras:
            a = tgs.alloc_frame(256, 256)
            tgs.tgs_render_temporal(s, cam, **a)
            b = gpu_full(h, cam, w.scene.n, depth=False, contrib=False)
            torch.cuda.synchronize()
            assert np.array_equal(a["rgb"].cpu().numpy(), b["rgb"])
        tgs.tgs_state_free(s)


def test_determinism():
    import torch
    w = synth.workload("tiny", n_frames=6)
    with Uploaded(w.scene) as h:
        s = tgs.tgs_state_create(h, 256, 256, tgs.params())
        runs = []
        for rep in range(2):
            tgs.tgs_state_reset(s)
            frames = []
            for cam in w.cameras:
                o = tgs.alloc_frame(256, 256)
                tgs.tgs_render_temporal(s, cam, **o)
                torch.cuda.synchronize()
                frames.append((o["rgb"].cpu().numpy(), tgs.tgs_debug_dump(None, s, tgs.TGS_DUMP_SORTED_KEYS).copy()))
            runs.append(frames)
        for (a, ka), (b, kb) in zip(*runs):
            assert np.array_equal(a, b) and np.array_equal(ka, kb)
        tgs.tgs_state_free(s)


def test_state_errors_on_device():
    w = synth.workload("tiny", n_frames=1)
    with Uploaded(w.scene) as h:
        s = tgs.tgs_state_create(h, 256, 256)
        other = synth.make_camera(w.cameras[0].w2c, 128, 256)
        with pytest.raises(tgs.TgsError) as e:
            tgs.tgs_render_temporal(s, other, **tgs.alloc_frame(128, 256))
        assert e.value.status == tgs.TGS_ERR_STATE_MISMATCH
        blob = tgs.tgs_state_export(s)
        with pytest.raises(tgs.TgsError):
            tgs.tgs_state_import(s, blob[:-1])
        tgs.tgs_state_import(s, blob)
        tgs.tgs_state_free(s)


def test_full_size_room_frame():
    """The 1.5M-Gaussian 1920x1080 workload in the benchmark's launch
    configuration: every list bit-exact, colour and moments on sampled tiles,
    then one TemporalGS frame by state injection."""
    import torch
    w = synth.workload("room", n_frames=2)
    sc, cams = w.scene, w.cameras
    TX, TY = cams[0].tiles
    rng = np.random.default_rng(0)
    g = O.gaussians(sc, cams[0])
    ts, _ = O.tile_lists(g, TX, TY)
    heavy = np.argsort(np.diff(ts))[-12:]
    sample = np.unique(np.concatenate([heavy, rng.choice(TX * TY, 40, replace=False),
                                       np.arange((TY - 1) * TX, TY * TX, 13)]))
    _full_parity(sc, cams[:1], sample_tiles=sample, label="room 1.5M")
    _full_parity(sc, cams[1:2], sample_tiles=sample, label="room 1.5M footprint",
                 bound=tgs.TGS_TILES_FOOTPRINT)
    _temporal_parity(sc, cams[:2], 1920, 1080, "room 1.5M")
    torch.cuda.synchronize()


def test_pair_count_matches_oracle():
    """The blend's evaluated (pixel, Gaussian) pairs and its hits (pairs with
    alpha >= 1/255, the unit of the blend roofline) equal the oracle's counts
    up to margin pixels."""
    w = synth.workload("tiny", n_frames=2)
    with Uploaded(w.scene) as h:
        for cam in w.cameras:
            tgs.tgs_profile_start(count_pairs=True)
            gpu_full(h, cam, w.scene.n, depth=False, contrib=False)
            prof = tgs.tgs_profile_stop()
            r = O.render_full(w.scene, cam)
            got = prof["blend_full"]["pairs"]
            hits = prof["blend_full"]["hits"]
            log(f"    pairs gpu {got} oracle {r['pairs']}; hits gpu {hits} oracle {r['hits']}")
            assert prof["blend_full"]["launches"] == 1
            assert abs(got - r["pairs"]) <= 1e-3 * r["pairs"]
            assert abs(hits - r["hits"]) <= 1e-3 * r["hits"]
