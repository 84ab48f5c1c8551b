"""CPU checks of the C-ABI library: it loads, exports every function that
include/tgs.h declares, and rejects bad arguments before touching a GPU."""
import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2607_03390_amd import synth, tgs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tgs.h")


def _declared():
    src = open(HEADER).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    names = set(re.findall(r"\b(tgs_[a-z_]+)\s*\(", src))
    return sorted(names)


def test_header_declares_the_boundary():
    names = _declared()
    for must in ("tgs_scene_upload", "tgs_render_full", "tgs_state_create", "tgs_render_temporal"):
        assert must in names
    assert sorted(tgs.EXPORTED) == names


def test_library_exports_every_declared_symbol():
    out = subprocess.run(["nm", "-D", "--defined-only", tgs.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r" T (tgs_[a-z_]+)$", out, flags=re.M))
    missing = [n for n in _declared() if n not in exported]
    assert not missing, missing
    L = tgs.lib()
    for n in _declared():
        assert hasattr(L, n)


_STRUCTS = ("tgs_camera", "tgs_params", "tgs_frame_out", "tgs_scene_desc", "tgs_state_header",
            "tgs_profile")


def test_struct_layouts_match_header(tmp_path):
    # the binding's ctypes structs against the C compiler's layout of the header
    src = tmp_path / "sizes.c"
    src.write_text('#include <stdio.h>\n#include "tgs.h"\nint main(void) {\n' +
                   "".join(f'    printf("%zu\\n", sizeof({n}));\n' for n in _STRUCTS) +
                   "    return 0;\n}\n")
    exe = tmp_path / "sizes"
    subprocess.run(["gcc", "-std=c99", "-I", os.path.join(ROOT, "include"), "-o", str(exe), str(src)],
                   check=True)
    sizes = [int(v) for v in subprocess.run([str(exe)], capture_output=True, text=True,
                                            check=True).stdout.split()]
    for name, size in zip(_STRUCTS, sizes):
        assert C.sizeof(getattr(tgs, name)) == size, name


def test_params_default_are_the_papers():
    p = tgs.params()
    assert (p.lambda_tdc, p.lambda_sr) == (50, 5)
    assert abs(p.eta - 0.40) < 1e-7 and p.lambda1 == 3.0 and p.lambda2 == 0.0
    assert abs(p.z_near - 0.2) < 1e-7
    assert p.enable_afc == p.enable_toc == p.enable_sr == 1 and p.force_all_dirty == 0
    assert p.empty_far == 0


def _bad_upload(**kw):
    sc = synth.small_scene(4, 0, degree=1)
    d = tgs.tgs_scene_desc()
    arrs = [np.ascontiguousarray(a, np.float32) for a in
            (sc.means, sc.scales, sc.rotations, sc.opacities, sc.sh)]
    d.n, d.sh_degree = 4, 1
    d.means, d.scales, d.rotations, d.opacities, d.sh = [a.ctypes.data for a in arrs]
    for k, v in kw.items():
        if k in ("nan_mean", "zero_quat"):
            if k == "nan_mean":
                arrs[0][1, 2] = np.nan
            else:
                arrs[2][3] = 0.0
        else:
            setattr(d, k, v)
    h = C.c_void_p()
    st = tgs.lib().tgs_scene_upload(C.byref(d), None, C.byref(h))
    return st, tgs.lib().tgs_last_error().decode()


@pytest.mark.parametrize("kw", [dict(n=-1), dict(sh_degree=4), dict(sh_degree=-1),
                                dict(means=None), dict(nan_mean=True), dict(zero_quat=True)])
def test_scene_upload_rejects_bad_input_on_host(kw):
    st, msg = _bad_upload(**kw)
    assert st == tgs.TGS_ERR_INVALID_ARG and msg


def test_render_rejects_bad_camera_on_host():
    L = tgs.lib()
    o = tgs.tgs_frame_out()
    o.rgb = 1  # never dereferenced: validation fails first
    cam = tgs.camera(synth.make_camera(np.eye(4), 32, 32))
    cam.world_to_cam[0] = 2.0                  # not a rotation
    dummy = C.c_void_p(1)
    assert L.tgs_render_full(dummy, C.byref(cam), C.byref(o), None) == tgs.TGS_ERR_INVALID_ARG
    assert "orthonormal" in L.tgs_last_error().decode()
    cam = tgs.camera(synth.make_camera(np.eye(4), 32, 32))
    cam.fx = 0.0
    assert L.tgs_render_full(dummy, C.byref(cam), C.byref(o), None) == tgs.TGS_ERR_INVALID_ARG
    cam = tgs.camera(synth.make_camera(np.eye(4), 0, 32))
    assert L.tgs_render_full(dummy, C.byref(cam), C.byref(o), None) == tgs.TGS_ERR_INVALID_ARG
    o.rgb = None
    cam = tgs.camera(synth.make_camera(np.eye(4), 32, 32))
    assert L.tgs_render_full(dummy, C.byref(cam), C.byref(o), None) == tgs.TGS_ERR_INVALID_ARG


def test_tile_bound_rejects_bad_input_on_host():
    L = tgs.lib()
    assert L.tgs_scene_set_tile_bound(None, tgs.TGS_TILES_FOOTPRINT) == tgs.TGS_ERR_INVALID_ARG
    dummy = C.c_void_p(1)      # never dereferenced: the rule is checked first
    for bad in (-1, 2):
        assert L.tgs_scene_set_tile_bound(dummy, bad) == tgs.TGS_ERR_INVALID_ARG
        assert "tile bound" in L.tgs_last_error().decode()


def test_scene_settings_reject_bad_values():
    """The sort path and blend split are per-scene settings: a NULL scene
    and out-of-range values are rejected before the scene is touched."""
    L = tgs.lib()
    dummy = C.c_void_p(1)      # never dereferenced: the values are checked first
    assert L.tgs_scene_set_sort_path(None, tgs.SORT_AUTO) == tgs.TGS_ERR_INVALID_ARG
    assert L.tgs_scene_set_blend_split(None, 12, 16) == tgs.TGS_ERR_INVALID_ARG
    for bad in (-1, 3):
        assert L.tgs_scene_set_sort_path(dummy, bad) == tgs.TGS_ERR_INVALID_ARG
    for bad in (-2, 32):
        assert L.tgs_scene_set_blend_split(dummy, bad, 16) == tgs.TGS_ERR_INVALID_ARG
        assert "log2_min" in L.tgs_last_error().decode()
    for bad in (-1, tgs.BLEND_SPLIT_MAX + 1):
        assert L.tgs_scene_set_blend_split(dummy, 0, bad) == tgs.TGS_ERR_INVALID_ARG
        assert "max_tiles" in L.tgs_last_error().decode()


def test_dump_range_rejects_bad_input_on_host():
    L = tgs.lib()
    dummy = C.c_void_p(1)      # never dereferenced: the arguments are checked first
    assert L.tgs_debug_dump_range(None, None, tgs.TGS_DUMP_SORTED_VALUES, 0, 1, dummy) == \
        tgs.TGS_ERR_INVALID_ARG
    for bad in (tgs.TGS_DUMP_TILE_RANGES, tgs.TGS_DUMP_RECORDS, 99):
        assert L.tgs_debug_dump_range(dummy, None, bad, 0, 1, dummy) == tgs.TGS_ERR_INVALID_ARG
    assert L.tgs_debug_dump_range(dummy, None, tgs.TGS_DUMP_SORTED_KEYS, 0, 4, None) == \
        tgs.TGS_ERR_INVALID_ARG


def test_noalloc_render_rejects_bad_input_on_host():
    L = tgs.lib()
    dummy = C.c_void_p(1)      # rejected before the scene is touched
    o = tgs.tgs_frame_out()
    cam = tgs.camera(synth.make_camera(np.eye(4), 32, 32))
    assert L.tgs_render_full_noalloc(None, C.byref(cam), C.byref(o), None) == tgs.TGS_ERR_INVALID_ARG
    assert L.tgs_render_full_noalloc(dummy, C.byref(cam), C.byref(o), None) == tgs.TGS_ERR_INVALID_ARG
    o.rgb = C.c_void_p(1)
    cam.width = 0
    assert L.tgs_render_full_noalloc(dummy, C.byref(cam), C.byref(o), None) == tgs.TGS_ERR_INVALID_ARG


def test_camera_background_must_be_finite():
    L = tgs.lib()
    dummy = C.c_void_p(1)      # rejected before the scene is touched
    o = tgs.tgs_frame_out()
    o.rgb = C.c_void_p(1)
    cam = tgs.camera(synth.make_camera(np.eye(4), 32, 32))
    cam.bg[1] = float("nan")
    assert L.tgs_render_full(dummy, C.byref(cam), C.byref(o), None) == tgs.TGS_ERR_INVALID_ARG
    assert "background" in L.tgs_last_error().decode()


def test_state_create_rejects_bad_params_on_host():
    L = tgs.lib()
    h = C.c_void_p()
    dummy = C.c_void_p(1)
    for kw in (dict(lambda_sr=0), dict(lambda_tdc=0), dict(eta=float("nan")), dict(z_near=0.0)):
        p = tgs.params(**kw)
        assert L.tgs_state_create(dummy, 64, 64, C.byref(p), C.byref(h)) == tgs.TGS_ERR_INVALID_ARG
    assert L.tgs_state_create(dummy, 0, 64, None, C.byref(h)) == tgs.TGS_ERR_INVALID_ARG


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(tgs, "_LIB", None)
    monkeypatch.setattr(tgs, "LIB_PATH", str(tmp_path / "missing.so"))
    with pytest.raises(ImportError):
        tgs.lib()
