"""ctypes binding of libtgs (include/tgs.h), same names as the C-ABI.

Argument marshalling only: every step of a frame runs in the HIP kernels of
``libtgs.so``.  Device buffers are torch tensors (PyTorch supplies device
memory and the current HIP stream); scenes are host arrays copied once by
``tgs_scene_upload``.  There is no CPU fallback: a missing library raises.
"""
from __future__ import annotations

import ctypes as C
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libtgs.so")

TGS_OK, TGS_ERR_INVALID_ARG, TGS_ERR_OUT_OF_MEMORY, TGS_ERR_DEVICE, TGS_ERR_STATE_MISMATCH, \
    TGS_ERR_CAPACITY = range(6)
TGS_FRAME_TRUE_REF, TGS_FRAME_PSEUDO_REF, TGS_FRAME_TGS, TGS_FRAME_FULL = range(4)
TGS_TILES_3SIGMA, TGS_TILES_FOOTPRINT = 0, 1
(TGS_DUMP_SORTED_VALUES, TGS_DUMP_SORTED_KEYS, TGS_DUMP_TILE_RANGES, TGS_DUMP_RECORDS,
 TGS_DUMP_RECTS, TGS_DUMP_STATUS, TGS_DUMP_WARP_DEPTH, TGS_DUMP_WARP_SIGMA,
 TGS_DUMP_FILLED_DEPTH, TGS_DUMP_CORRESPONDENCE, TGS_DUMP_UNMATCHED, TGS_DUMP_OCCLUDED,
 TGS_DUMP_SELECTED) = range(13)

EXPORTED = ["tgs_params_default", "tgs_scene_upload", "tgs_scene_free", "tgs_scene_count",
            "tgs_scene_set_tile_bound",
            "tgs_render_full", "tgs_state_create", "tgs_state_reset", "tgs_state_free",
            "tgs_render_temporal", "tgs_state_export", "tgs_state_import", "tgs_debug_dump",
            "tgs_debug_dump_range", "tgs_render_full_noalloc",
            "tgs_profile_start", "tgs_profile_stop", "tgs_scene_set_sort_path",
            "tgs_scene_set_blend_split",
            "tgs_last_error"]

# tgs_scene_set_sort_path modes
SORT_AUTO, SORT_DEPTH_FIRST, SORT_PER_TILE = 0, 1, 2
# tgs_scene_set_blend_split: default log2 of the list length from which tiles are
# split into quadrant blocks, and the most tiles split per frame
BLEND_SPLIT_DEFAULT, BLEND_SPLIT_MAX = 12, 1024

PROF_STAGES = ["preprocess", "scan", "readback", "duplicate", "sort", "ranges", "blend_full",
               "blend_ref", "blend_tgs", "warp", "fill_query", "occluded", "select", "stitch",
               "capture"]


class TgsError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__(f"tgs status {status}: {msg}")
        self.status = status


class tgs_scene_desc(C.Structure):
    _fields_ = [("n", C.c_int32), ("sh_degree", C.c_int32), ("means", C.c_void_p),
                ("scales", C.c_void_p), ("rotations", C.c_void_p), ("opacities", C.c_void_p),
                ("sh", C.c_void_p)]


class tgs_camera(C.Structure):
    _fields_ = [("world_to_cam", C.c_float * 16), ("fx", C.c_float), ("fy", C.c_float),
                ("cx", C.c_float), ("cy", C.c_float), ("width", C.c_int32), ("height", C.c_int32),
                ("bg", C.c_float * 3)]


class tgs_params(C.Structure):
    _fields_ = [("lambda_tdc", C.c_int32), ("lambda_sr", C.c_int32), ("eta", C.c_float),
                ("lambda1", C.c_float), ("lambda2", C.c_float), ("z_near", C.c_float),
                ("enable_afc", C.c_int32), ("enable_toc", C.c_int32), ("enable_sr", C.c_int32),
                ("force_all_dirty", C.c_int32), ("empty_far", C.c_int32),
                ("tgb_downscale", C.c_int32)]


class tgs_frame_out(C.Structure):
    _fields_ = [("rgb", C.c_void_p), ("depth", C.c_void_p), ("sigma", C.c_void_p),
                ("alpha", C.c_void_p), ("contrib", C.c_void_p), ("tile_mask", C.c_void_p),
                ("frame_kind", C.c_int32), ("n_selected", C.c_int32), ("n_survivors", C.c_int32),
                ("n_newly_visible", C.c_int32), ("n_keys", C.c_int64)]


class tgs_profile(C.Structure):
    _fields_ = [("ms", C.c_double * 16), ("launches", C.c_int64 * 16), ("pairs", C.c_int64 * 16),
                ("hits", C.c_int64 * 16)]


class tgs_state_header(C.Structure):
    _fields_ = [("magic", C.c_uint32), ("width", C.c_int32), ("height", C.c_int32),
                ("n", C.c_int32), ("frame_index", C.c_int32), ("since_true_ref", C.c_int32),
                ("since_ref", C.c_int32), ("force_pseudo", C.c_int32),
                ("has_reference", C.c_int32), ("fbox", C.c_float * 4),
                ("ref_world_to_cam", C.c_float * 16), ("ref_intrinsics", C.c_float * 4),
                ("tgb_width", C.c_int32), ("tgb_height", C.c_int32)]


_LIB = None


def lib():
    global _LIB
    if _LIB is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                              "(the HIP library is required, there is no CPU fallback)")
        L = C.CDLL(LIB_PATH)
        vp, i32, sz = C.c_void_p, C.c_int32, C.c_size_t
        L.tgs_last_error.restype = C.c_char_p
        L.tgs_params_default.argtypes = [C.POINTER(tgs_params)]
        L.tgs_scene_upload.argtypes = [C.POINTER(tgs_scene_desc), vp, C.POINTER(vp)]
        L.tgs_scene_free.argtypes = [vp]
        L.tgs_scene_count.argtypes = [vp]
        L.tgs_scene_set_tile_bound.argtypes = [vp, C.c_int32]
        L.tgs_render_full.argtypes = [vp, C.POINTER(tgs_camera), C.POINTER(tgs_frame_out), vp]
        L.tgs_render_full_noalloc.argtypes = [vp, C.POINTER(tgs_camera), C.POINTER(tgs_frame_out), vp]
        L.tgs_state_create.argtypes = [vp, i32, i32, C.POINTER(tgs_params), C.POINTER(vp)]
        L.tgs_state_reset.argtypes = [vp]
        L.tgs_state_free.argtypes = [vp]
        L.tgs_render_temporal.argtypes = [vp, C.POINTER(tgs_camera), C.POINTER(tgs_frame_out), vp]
        L.tgs_state_export.argtypes = [vp, vp, C.POINTER(sz)]
        L.tgs_state_import.argtypes = [vp, vp, sz]
        L.tgs_debug_dump.argtypes = [vp, vp, i32, vp, C.POINTER(sz)]
        L.tgs_debug_dump_range.argtypes = [vp, vp, i32, sz, sz, vp]
        L.tgs_profile_start.argtypes = [i32]
        L.tgs_profile_stop.argtypes = [C.POINTER(tgs_profile)]
        L.tgs_scene_set_sort_path.argtypes = [vp, i32]
        L.tgs_scene_set_blend_split.argtypes = [vp, i32, i32]
        for name in EXPORTED:
            if name not in ("tgs_last_error", "tgs_params_default", "tgs_scene_free",
                            "tgs_state_free", "tgs_scene_count"):
                getattr(L, name).restype = C.c_int
        L.tgs_scene_count.restype = C.c_int32
        _LIB = L
    return _LIB


def _check(status):
    if status != TGS_OK:
        raise TgsError(status, lib().tgs_last_error().decode())


def _stream(stream):
    if stream is None:
        import torch
        return C.c_void_p(torch.cuda.current_stream().cuda_stream)
    return C.c_void_p(stream)


def _ptr(t):
    return None if t is None else C.c_void_p(t.data_ptr())


def camera(cam) -> tgs_camera:
    """tgs_camera from any object with w2c, fx, fy, cx, cy, width, height
    (and optionally bg, the background colour; black otherwise)."""
    c = tgs_camera()
    w = np.ascontiguousarray(cam.w2c, np.float32).ravel()
    for k in range(16):
        c.world_to_cam[k] = float(w[k])
    c.fx, c.fy, c.cx, c.cy = float(cam.fx), float(cam.fy), float(cam.cx), float(cam.cy)
    c.width, c.height = int(cam.width), int(cam.height)
    bg = getattr(cam, "bg", (0.0, 0.0, 0.0))
    for k in range(3):
        c.bg[k] = float(bg[k])
    return c


def params(**kw) -> tgs_params:
    p = tgs_params()
    lib().tgs_params_default(C.byref(p))
    for k, v in kw.items():
        setattr(p, k, v)
    return p


def _frame_out(rgb, depth, sigma, alpha, contrib, tile_mask):
    o = tgs_frame_out()
    o.rgb, o.depth, o.sigma, o.alpha = _ptr(rgb), _ptr(depth), _ptr(sigma), _ptr(alpha)
    o.contrib, o.tile_mask = _ptr(contrib), _ptr(tile_mask)
    return o


def _scalars(o):
    return dict(frame_kind=o.frame_kind, n_selected=o.n_selected, n_survivors=o.n_survivors,
                n_newly_visible=o.n_newly_visible, n_keys=o.n_keys)


def tgs_scene_upload(scene, stream=None):
    """Upload a host scene (synth.Scene-like arrays); returns the handle."""
    arrs = [np.ascontiguousarray(a, np.float32) for a in
            (scene.means, scene.scales, scene.rotations, scene.opacities, scene.sh)]
    d = tgs_scene_desc()
    d.n, d.sh_degree = int(arrs[0].shape[0]), int(scene.sh_degree)
    d.means, d.scales, d.rotations, d.opacities, d.sh = [a.ctypes.data for a in arrs]
    h = C.c_void_p()
    _check(lib().tgs_scene_upload(C.byref(d), _stream(stream), C.byref(h)))
    return h


def tgs_scene_free(h):
    lib().tgs_scene_free(h)


def tgs_scene_count(h):
    return int(lib().tgs_scene_count(h))


def tgs_scene_set_tile_bound(h, bound):
    """TGS_TILES_3SIGMA (default) or TGS_TILES_FOOTPRINT for later renders."""
    _check(lib().tgs_scene_set_tile_bound(h, int(bound)))


def tgs_render_full(scene_h, cam, rgb, depth=None, sigma=None, alpha=None, contrib=None,
                    tile_mask=None, stream=None):
    o = _frame_out(rgb, depth, sigma, alpha, contrib, tile_mask)
    c = camera(cam)
    _check(lib().tgs_render_full(scene_h, C.byref(c), C.byref(o), _stream(stream)))
    return _scalars(o)


# bytes of the device array that holds the workspace of tgs_render_full_noalloc
NOALLOC_SCRATCH_BYTES = 64 << 20


def tgs_render_full_noalloc(scene_h, cam, rgb, depth=None, sigma=None, alpha=None, contrib=None,
                            tile_mask=None, stream=None):
    """tgs_render_full with the workspace in the library's fixed device array
    (no allocation; raises TgsError with TGS_ERR_CAPACITY beyond it)."""
    o = _frame_out(rgb, depth, sigma, alpha, contrib, tile_mask)
    c = camera(cam)
    _check(lib().tgs_render_full_noalloc(scene_h, C.byref(c), C.byref(o), _stream(stream)))
    return _scalars(o)


def tgs_state_create(scene_h, width, height, p: tgs_params | None = None):
    h = C.c_void_p()
    _check(lib().tgs_state_create(scene_h, int(width), int(height),
                                  None if p is None else C.byref(p), C.byref(h)))
    return h


def tgs_state_reset(h):
    _check(lib().tgs_state_reset(h))


def tgs_state_free(h):
    lib().tgs_state_free(h)


def tgs_render_temporal(state_h, cam, rgb, depth=None, sigma=None, alpha=None, contrib=None,
                        tile_mask=None, stream=None):
    o = _frame_out(rgb, depth, sigma, alpha, contrib, tile_mask)
    c = camera(cam)
    _check(lib().tgs_render_temporal(state_h, C.byref(c), C.byref(o), _stream(stream)))
    return _scalars(o)


def tgs_state_export(h) -> bytes:
    n = C.c_size_t(0)
    _check(lib().tgs_state_export(h, None, C.byref(n)))
    buf = C.create_string_buffer(n.value)
    _check(lib().tgs_state_export(h, buf, C.byref(n)))
    return buf.raw[:n.value]


def tgs_state_import(h, blob: bytes):
    buf = C.create_string_buffer(blob, len(blob))
    _check(lib().tgs_state_import(h, buf, len(blob)))


def parse_state(blob: bytes):
    """Split an exported state into its header fields and arrays."""
    hdr = tgs_state_header.from_buffer_copy(blob[:C.sizeof(tgs_state_header)])
    W, H, n = hdr.width, hdr.height, hdr.n
    off = C.sizeof(tgs_state_header)
    px = W * H
    Wg, Hg = hdr.tgb_width, hdr.tgb_height
    D = np.frombuffer(blob, np.float32, Wg * Hg, off).reshape(Hg, Wg); off += 4 * Wg * Hg
    S = np.frombuffer(blob, np.float32, Wg * Hg, off).reshape(Hg, Wg); off += 4 * Wg * Hg
    tab = np.frombuffer(blob, np.float32, 3 * px, off).reshape(3, H, W); off += 12 * px
    g = np.frombuffer(blob, np.uint8, n, off)
    return dict(width=W, height=H, n=n, frame_index=hdr.frame_index,
                since_true=hdr.since_true_ref, since_ref=hdr.since_ref,
                force_pseudo=hdr.force_pseudo, has_reference=hdr.has_reference,
                fbox=np.array(hdr.fbox, np.float32),
                ref_w2c=np.array(hdr.ref_world_to_cam, np.float32).reshape(4, 4),
                ref_intr=np.array(hdr.ref_intrinsics, np.float32), D=D, S=S, tab=tab,
                g_rendered=g)


_DUMP_DTYPE = {TGS_DUMP_SORTED_VALUES: np.uint32, TGS_DUMP_SORTED_KEYS: np.uint32,
               TGS_DUMP_TILE_RANGES: np.uint32, TGS_DUMP_RECORDS: np.float32,
               TGS_DUMP_RECTS: np.uint16, TGS_DUMP_STATUS: np.uint8,
               TGS_DUMP_WARP_DEPTH: np.float32, TGS_DUMP_WARP_SIGMA: np.float32,
               TGS_DUMP_FILLED_DEPTH: np.float32, TGS_DUMP_CORRESPONDENCE: np.float32,
               TGS_DUMP_UNMATCHED: np.uint8, TGS_DUMP_OCCLUDED: np.uint8,
               TGS_DUMP_SELECTED: np.uint8}


def tgs_debug_dump(scene_h, state_h, what) -> np.ndarray:
    n = C.c_size_t(0)
    _check(lib().tgs_debug_dump(scene_h, state_h, int(what), None, C.byref(n)))
    out = np.zeros(n.value, np.uint8)
    _check(lib().tgs_debug_dump(scene_h, state_h, int(what), out.ctypes.data, C.byref(n)))
    return out.view(_DUMP_DTYPE[what])


def tgs_debug_dump_range(scene_h, state_h, what, first, count) -> np.ndarray:
    """Sorted values or keys [first, first + count) of the last frame."""
    out = np.zeros(max(int(count), 0), np.uint32)
    _check(lib().tgs_debug_dump_range(scene_h, state_h, int(what), int(first), int(count),
                                      out.ctypes.data if count else None))
    return out


TGS_PROFILE_COUNT_PAIRS, TGS_PROFILE_STAGES = 1, 2


def tgs_scene_set_sort_path(h, mode):
    """How per-tile depth order is produced for later renders through the
    scene: SORT_AUTO, SORT_DEPTH_FIRST (global depth sort, keys emitted in
    depth order) or SORT_PER_TILE (keys in index order, each tile's list
    sorted)."""
    _check(lib().tgs_scene_set_sort_path(h, int(mode)))


def tgs_scene_set_blend_split(h, log2_min=BLEND_SPLIT_DEFAULT, max_tiles=BLEND_SPLIT_MAX):
    """For later renders through the scene, tiles with at least 2**log2_min
    list entries are blended as four quadrant blocks (-1: never); if more
    than max_tiles tiles qualify, the threshold doubles until at most
    max_tiles do."""
    _check(lib().tgs_scene_set_blend_split(h, int(log2_min), int(max_tiles)))


def tgs_profile_start(count_pairs=False, stages=False):
    """Blend dispatches are always timed; ``stages`` also brackets every other
    stage with separately recorded events (adds queue barriers)."""
    flags = (TGS_PROFILE_COUNT_PAIRS if count_pairs else 0) | (TGS_PROFILE_STAGES if stages else 0)
    _check(lib().tgs_profile_start(flags))


def tgs_profile_stop():
    """Per stage: summed event ms, launches, counted pairs and hits."""
    p = tgs_profile()
    _check(lib().tgs_profile_stop(C.byref(p)))
    return {name: dict(ms=p.ms[k], launches=p.launches[k], pairs=p.pairs[k], hits=p.hits[k])
            for k, name in enumerate(PROF_STAGES)}


def alloc_frame(width, height, n=0, depth=False, contrib=False, tile_mask=False, device="cuda"):
    """Device output buffers for one frame (torch tensors)."""
    import torch
    t = dict(rgb=torch.empty((3, height, width), dtype=torch.float32, device=device))
    if depth:
        for k in ("depth", "sigma", "alpha"):
            t[k] = torch.empty((height, width), dtype=torch.float32, device=device)
    if contrib:
        t["contrib"] = torch.empty((max(n, 1),), dtype=torch.float32, device=device)
    if tile_mask:
        t["tile_mask"] = torch.empty(((height + 15) // 16, (width + 15) // 16), dtype=torch.uint8,
                                     device=device)
    return t
