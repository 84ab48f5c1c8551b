"""The allocation-free full render (tgs_render_full_noalloc, workspace in the
library's fixed device array) against tgs_render_full through the C-ABI:
the same kernels on the same inputs, so every output is bit-identical.
Two calls in a row, the second with a smaller input; a frame whose keys do
not fit the array is refused with TGS_ERR_CAPACITY, and the call after it
is exact again (the array keeps the last call's contents)."""
import numpy as np
import pytest

from paper_2607_03390_amd import synth, tgs

pytestmark = pytest.mark.gpu


def _render(fn, h, cam, n):
    import torch
    out = tgs.alloc_frame(cam.width, cam.height, n, depth=True, contrib=True, tile_mask=True)
    info = fn(h, cam, **out)
    torch.cuda.synchronize()
    return info, {k: v.cpu().numpy() for k, v in out.items()}


def _same(h, cam, n, label):
    a_info, a = _render(tgs.tgs_render_full, h, cam, n)
    b_info, b = _render(tgs.tgs_render_full_noalloc, h, cam, n)
    print(f"[no-alloc {label}] keys {b_info['n_keys']} survivors {b_info['n_survivors']}", flush=True)
    assert a_info == b_info, (a_info, b_info)
    for k in ("rgb", "depth", "sigma", "alpha", "tile_mask"):
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k
    assert np.array_equal(a["contrib"][:n].view(np.uint32), b["contrib"][:n].view(np.uint32))


def test_noalloc_matches_render_full():
    import torch
    assert torch.cuda.is_available()
    torch.cuda.set_device(0)
    tiny = synth.workload("tiny", n_frames=2)
    small = synth.small_scene(3000, 1, degree=3)
    small_cam = synth.make_camera(synth.look_at((0.2, -3.0, 0.7), (0, 0, 0)), 200, 136)
    small_cam.bg = (0.1, 0.2, 0.3)
    big = synth.small_scene(20_000, 13, degree=1, log_scale_mean=-2.2)
    big_cam = synth.make_camera(synth.look_at((0.0, -3.0, 1.0), (0, 0, 0)), 3840, 2160)
    hs = [tgs.tgs_scene_upload(sc) for sc in (tiny.scene, small, big)]
    try:
        # the larger input, then a smaller one
        _same(hs[0], tiny.cameras[0], tiny.scene.n, "tiny 256x256")
        _same(hs[1], small_cam, small.n, "3000 at 200x136")
        # a frame of 35M keys does not fit: refused, and the next call is exact
        out = tgs.alloc_frame(big_cam.width, big_cam.height, big.n)
        with pytest.raises(tgs.TgsError) as e:
            tgs.tgs_render_full_noalloc(hs[2], big_cam, **out)
        torch.cuda.synchronize()
        assert e.value.status == tgs.TGS_ERR_CAPACITY
        _same(hs[0], tiny.cameras[1], tiny.scene.n, "tiny after the refused frame")
        # too many Gaussians for the array: refused before any launch
        huge = synth.small_scene(1_000_000, 2, degree=0)
        hh = tgs.tgs_scene_upload(huge)
        try:
            with pytest.raises(tgs.TgsError) as e:
                tgs.tgs_render_full_noalloc(hh, tiny.cameras[0], **tgs.alloc_frame(256, 256))
            assert e.value.status == tgs.TGS_ERR_CAPACITY
        finally:
            tgs.tgs_scene_free(hh)
    finally:
        for h in hs:
            tgs.tgs_scene_free(h)
