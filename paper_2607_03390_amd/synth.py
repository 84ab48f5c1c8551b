"""Seeded synthetic scenes and camera paths (inputs only).

This module draws the inputs that both the HIP path and the CPU oracle consume:
3D Gaussian scenes (means, linear scales, unit quaternions in w,x,y,z order,
activated opacities, SH coefficients) and rigid world-to-camera matrices along
a camera path.  It holds none of the rendering arithmetic: no projection, no
covariance, no blending.  Every array is produced by numpy's PCG64 generator
from a fixed seed, so the same call always returns the same bytes.

Camera convention: camera x points right, y down, z forward; world up is +z.
Pixel centres sit at integer coordinates, so the principal point of a W x H
image is ((W-1)/2, (H-1)/2); the vertical field of view is 60 degrees and
pixels are square (fx = fy = H / (2 tan 30deg)).

The five workloads follow the scene and path descriptions of the paper's
evaluation setting (Sec. IV-A: small object-centred scenes, unbounded rooms,
large city-like scenes, fast camera motion), scaled to seeded synthetic
stand-ins because the paper's datasets and trained checkpoints are not used.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

FOVY_DEG = 60.0


@dataclass
class Scene:
    means: np.ndarray       # [N,3] float32, world space
    scales: np.ndarray      # [N,3] float32, linear (post-exp) axis scales
    rotations: np.ndarray   # [N,4] float32, unit quaternions (w,x,y,z)
    opacities: np.ndarray   # [N]   float32, activated (post-sigmoid)
    sh: np.ndarray          # [N,(deg+1)^2,3] float32, coefficient-major
    sh_degree: int

    @property
    def n(self) -> int:
        return int(self.means.shape[0])

    def subset(self, idx) -> "Scene":
        return Scene(self.means[idx].copy(), self.scales[idx].copy(),
                     self.rotations[idx].copy(), self.opacities[idx].copy(),
                     self.sh[idx].copy(), self.sh_degree)


@dataclass
class Camera:
    w2c: np.ndarray          # [4,4] float32 row-major rigid world->camera
    fx: float
    fy: float
    cx: float
    cy: float
    width: int
    height: int
    bg: tuple = (0.0, 0.0, 0.0)   # background colour

    @property
    def tiles(self) -> tuple[int, int]:
        return (self.width + 15) // 16, (self.height + 15) // 16


@dataclass
class Workload:
    name: str
    scene: Scene
    cameras: list = field(default_factory=list)


# --------------------------------------------------------------------------
# elementary draws
# --------------------------------------------------------------------------

def _rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def _unit_quaternions(rng, n):
    q = rng.standard_normal((n, 4))
    q /= np.linalg.norm(q, axis=1, keepdims=True)
    return q.astype(np.float32)


def _sigmoid(x):
    return 1.0 / (1.0 + np.exp(-x))


def _sh(rng, n, degree, dc_std=0.5, rest_std=0.05):
    k = (degree + 1) ** 2
    sh = np.empty((n, k, 3), np.float32)
    sh[:, 0, :] = rng.normal(0.0, dc_std, (n, 3))
    if k > 1:
        sh[:, 1:, :] = rng.normal(0.0, rest_std, (n, k - 1, 3))
    return sh


def _unit_vectors(rng, n):
    v = rng.standard_normal((n, 3))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    return v


# --------------------------------------------------------------------------
# cameras
# --------------------------------------------------------------------------

def focal_for_height(height: int) -> float:
    return height / (2.0 * math.tan(math.radians(FOVY_DEG) / 2.0))


def look_at(eye, target, up=(0.0, 0.0, 1.0)) -> np.ndarray:
    """Rigid world->camera matrix (x right, y down, z forward)."""
    eye = np.asarray(eye, np.float64)
    f = np.asarray(target, np.float64) - eye
    f /= np.linalg.norm(f)
    r = np.cross(f, np.asarray(up, np.float64))
    r /= np.linalg.norm(r)
    d = np.cross(f, r)
    R = np.stack([r, d, f])
    m = np.eye(4)
    m[:3, :3] = R
    m[:3, 3] = -R @ eye
    return m


def make_camera(w2c, width, height) -> Camera:
    f = focal_for_height(height)
    return Camera(np.asarray(w2c, np.float64).astype(np.float32), float(np.float32(f)),
                  float(np.float32(f)), (width - 1) / 2.0, (height - 1) / 2.0, width, height)


def orbit_path(n_frames, radius, elevation_deg, step_deg, width, height,
               start_deg=-90.0, target=(0.0, 0.0, 0.0), steps=None):
    cams = []
    ang = start_deg
    el = math.radians(elevation_deg)
    for k in range(n_frames):
        if k > 0:
            ang += steps[(k - 1) % len(steps)] if steps is not None else step_deg
        a = math.radians(ang)
        eye = (target[0] + radius * math.cos(el) * math.cos(a),
               target[1] + radius * math.cos(el) * math.sin(a),
               target[2] + radius * math.sin(el))
        cams.append(make_camera(look_at(eye, target), width, height))
    return cams


def handheld_path(n_frames, eye0, target, yaw_deg_per_frame, slide_per_frame,
                  width, height):
    """Yaw about world z plus a slide along the initial right vector."""
    eye0 = np.asarray(eye0, np.float64)
    f0 = np.asarray(target, np.float64) - eye0
    f0 /= np.linalg.norm(f0)
    right0 = np.cross(f0, [0.0, 0.0, 1.0])
    right0 /= np.linalg.norm(right0)
    cams = []
    for k in range(n_frames):
        a = math.radians(yaw_deg_per_frame * k)
        c, s = math.cos(a), math.sin(a)
        fk = np.array([c * f0[0] - s * f0[1], s * f0[0] + c * f0[1], f0[2]])
        eye = eye0 + slide_per_frame * k * right0
        cams.append(make_camera(look_at(eye, eye + fk), width, height))
    return cams


def walk_path(n_frames, eye0, heading_deg, step, yaw_deg_per_frame, width, height):
    cams = []
    eye = np.asarray(eye0, np.float64).copy()
    h = heading_deg
    for k in range(n_frames):
        if k > 0:
            a = math.radians(h)
            eye = eye + step * np.array([math.cos(a), math.sin(a), 0.0])
            h += yaw_deg_per_frame
        a = math.radians(h)
        fwd = np.array([math.cos(a), math.sin(a), -0.02])
        cams.append(make_camera(look_at(eye, eye + fwd), width, height))
    return cams


def catmull_rom(keys, u):
    """Uniform Catmull-Rom curve through keys[0..M-1] (M >= 2) at parameters
    u in [0, M-1]: cubic Hermite segments between consecutive keys with
    central-difference tangents (one-sided at the two ends), so the curve
    passes through every key with a continuous first derivative."""
    keys = np.asarray(keys, np.float64)
    m = len(keys)
    tan = np.empty_like(keys)
    tan[1:-1] = 0.5 * (keys[2:] - keys[:-2])
    tan[0] = keys[1] - keys[0]
    tan[-1] = keys[-1] - keys[-2]
    u = np.asarray(u, np.float64)
    seg = np.clip(np.floor(u).astype(np.int64), 0, m - 2)
    t = (u - seg)[:, None]
    t2, t3 = t * t, t * t * t
    return ((2 * t3 - 3 * t2 + 1) * keys[seg] + (t3 - 2 * t2 + t) * tan[seg] +
            (-2 * t3 + 3 * t2) * keys[seg + 1] + (t3 - t2) * tan[seg + 1])


def keyframe_path(key_eyes, key_targets, interval, width, height, n_frames=None,
                  samples_per_segment=512):
    """Cameras on curves fitted through consecutive key poses, sampled at a
    fixed interval of eye travel (the paper's synthetic test trajectories,
    Sec. IV-A; a larger interval is a faster camera, Table V).

    Eye positions and look-at targets each follow a Catmull-Rom curve over the
    key index; frame k sits where the eye curve's arc length (dense chord sum)
    reaches k * interval.  n_frames truncates the path."""
    m = len(key_eyes)
    u_dense = np.linspace(0.0, m - 1.0, (m - 1) * samples_per_segment + 1)
    p = catmull_rom(key_eyes, u_dense)
    arc = np.concatenate([[0.0], np.cumsum(np.linalg.norm(np.diff(p, axis=0), axis=1))])
    n = int(math.floor(arc[-1] / interval + 1e-9)) + 1
    if n_frames is not None:
        n = min(n, n_frames)
    u = np.interp(interval * np.arange(n), arc, u_dense)
    eyes = catmull_rom(key_eyes, u)
    targets = catmull_rom(key_targets, u)
    return [make_camera(look_at(e, t), width, height) for e, t in zip(eyes, targets)]


# key poses of the room walk-through: the eye circles the central cluster at
# about 5 units while the gaze drifts across it
ROOM_KEY_EYES = ((-1.5, -5.0, 0.3), (-0.5, -5.2, 0.4), (0.5, -5.1, 0.35),
                 (1.5, -4.8, 0.3), (2.4, -4.3, 0.45), (3.2, -3.6, 0.4))
ROOM_KEY_TARGETS = ((0.0, 0.0, 0.0), (0.1, 0.0, 0.05), (0.2, 0.1, 0.0),
                    (0.3, 0.1, 0.0), (0.3, 0.2, 0.05), (0.2, 0.3, 0.0))


# --------------------------------------------------------------------------
# scenes
# --------------------------------------------------------------------------

def scene_uniform_cube(n, seed, degree=0, log_scale_mean=-4.0, log_scale_std=0.5,
                       opacity_std=1.5, extent=1.0) -> Scene:
    rng = _rng(seed)
    means = rng.uniform(-extent, extent, (n, 3)).astype(np.float32)
    scales = np.exp(rng.normal(log_scale_mean, log_scale_std, (n, 3))).astype(np.float32)
    rots = _unit_quaternions(rng, n)
    opac = _sigmoid(rng.normal(0.0, opacity_std, n)).astype(np.float32)
    sh = _sh(rng, n, degree)
    return Scene(means, scales, rots, opac, sh, degree)


def scene_clusters(n, seed, n_clusters=32) -> Scene:
    rng = _rng(seed)
    centres = rng.uniform(-1.5, 1.5, (n_clusters, 3))
    axes = rng.uniform(0.1, 0.5, (n_clusters, 3))
    # random cluster orientations from the QR factorisation of Gaussian matrices
    Rc = np.empty((n_clusters, 3, 3))
    for c in range(n_clusters):
        q, r = np.linalg.qr(rng.standard_normal((3, 3)))
        Rc[c] = q * np.sign(np.diag(r))
    lab = rng.integers(0, n_clusters, n)
    local = rng.standard_normal((n, 3)) * axes[lab]
    means = centres[lab] + np.einsum("nij,nj->ni", Rc[lab], local)
    means = np.clip(means, -2.0, 2.0).astype(np.float32)
    scales = np.exp(rng.normal(-5.0, 0.7, (n, 3))).astype(np.float32)
    rots = _unit_quaternions(rng, n)
    opac = _sigmoid(rng.normal(0.0, 1.5, n)).astype(np.float32)
    sh = _sh(rng, n, 3)
    return Scene(means, scales, rots, opac, sh, 3)


def scene_room(n, seed, needle_fraction=0.0) -> Scene:
    rng = _rng(seed)
    n_core = int(round(0.7 * n))
    n_shell = n - n_core
    d = _unit_vectors(rng, n_core)
    rad = 2.0 * rng.uniform(0.0, 1.0, n_core) ** (1.0 / 3.0)
    core = d * rad[:, None]
    ds = _unit_vectors(rng, n_shell)
    shell = ds * rng.uniform(10.0, 50.0, n_shell)[:, None]
    means = np.concatenate([core, shell]).astype(np.float32)
    scales = np.exp(rng.normal(-5.0, 0.7, (n, 3)))
    scales[n_core:] *= 10.0
    if needle_fraction > 0.0:
        m = rng.uniform(0.0, 1.0, n) < needle_fraction
        ax = rng.integers(0, 3, n)
        scales[m, ax[m]] *= 50.0
    rots = _unit_quaternions(rng, n)
    opac = _sigmoid(rng.normal(0.0, 2.0, n)).astype(np.float32)
    sh = _sh(rng, n, 3)
    return Scene(means, scales.astype(np.float32), rots, opac, sh, 3)


def scene_city(n, seed, n_buildings=400, extent=100.0, street_half_width=6.0) -> Scene:
    """Ground plane of flat Gaussians plus Gaussians on the faces of boxes."""
    rng = _rng(seed)
    n_ground = int(round(0.4 * n))
    n_faces = n - n_ground
    # buildings: footprints placed uniformly, rejecting overlaps and the street
    placed = np.zeros((n_buildings, 5))
    m = 0
    tries = 0
    while m < n_buildings and tries < 200000:
        tries += 1
        w, dpt = rng.uniform(4.0, 12.0, 2)
        h = rng.uniform(5.0, 40.0)
        cx, cy = rng.uniform(-extent + 6.0, extent - 6.0, 2)
        x0, x1, y0, y1 = cx - w / 2, cx + w / 2, cy - dpt / 2, cy + dpt / 2
        if y0 < street_half_width and y1 > -street_half_width:
            continue
        pb = placed[:m]
        if np.any((x0 < pb[:, 1] + 1.0) & (x1 > pb[:, 0] - 1.0) & (y0 < pb[:, 3] + 1.0) &
                  (y1 > pb[:, 2] - 1.0)):
            continue
        placed[m] = (x0, x1, y0, y1, h)
        m += 1
    boxes = placed[:m]
    # ground
    g_means = np.stack([rng.uniform(-extent, extent, n_ground),
                        rng.uniform(-extent, extent, n_ground),
                        np.zeros(n_ground)], 1)
    g_in = np.exp(rng.normal(-2.5, 0.3, (n_ground, 2)))
    g_scales = np.concatenate([g_in, 0.01 * g_in.mean(1, keepdims=True)], 1)
    yaw = rng.uniform(0.0, math.pi, n_ground)
    g_rot = np.stack([np.cos(yaw / 2), np.zeros(n_ground), np.zeros(n_ground), np.sin(yaw / 2)], 1)
    # faces: 4 walls + roof per box, chosen proportionally to area
    x0, x1, y0, y1, h = boxes.T
    wx, wy = x1 - x0, y1 - y0
    areas = np.stack([wx * h, wx * h, wy * h, wy * h, wx * wy], 1).ravel()
    face = rng.choice(areas.size, n_faces, p=areas / areas.sum())
    b, f = face // 5, face % 5
    u, v = rng.uniform(0.0, 1.0, (2, n_faces))
    fm = np.empty((n_faces, 3))
    fm[:, 0] = np.where(f == 2, x0[b], np.where(f == 3, x1[b], x0[b] + u * wx[b]))
    fm[:, 1] = np.where(f == 0, y0[b], np.where(f == 1, y1[b], y0[b] + np.where(f >= 2, u, v) * wy[b]))
    fm[:, 2] = np.where(f == 4, h[b], v * h[b])
    fm[f == 4, 0] = x0[b[f == 4]] + u[f == 4] * wx[b[f == 4]]
    f_in = np.exp(rng.normal(-1.8, 0.3, (n_faces, 2)))
    f_scales = np.empty((n_faces, 3))
    normal_axis = np.where(f <= 1, 1, np.where(f <= 3, 0, 2))
    for a in range(3):
        sel = normal_axis == a
        others = [k for k in range(3) if k != a]
        f_scales[sel, others[0]] = f_in[sel, 0]
        f_scales[sel, others[1]] = f_in[sel, 1]
        f_scales[sel, a] = 0.01 * f_in[sel].mean(1)
    f_rot = np.tile(np.array([1.0, 0.0, 0.0, 0.0]), (n_faces, 1))
    means = np.concatenate([g_means, fm]).astype(np.float32)
    scales = np.concatenate([g_scales, f_scales]).astype(np.float32)
    rots = np.concatenate([g_rot, f_rot]).astype(np.float32)
    opac = _sigmoid(rng.normal(1.0, 1.5, n)).astype(np.float32)
    sh = _sh(rng, n, 3)
    return Scene(means, scales, rots, opac, sh, 3)


# --------------------------------------------------------------------------
# the five workloads
# --------------------------------------------------------------------------

WORKLOADS = {
    "tiny": "10k Gaussians, SH0, 256x256, 8-frame orbit (seed 0)",
    "object": "300k Gaussians, SH3, 1280x720, 60-frame orbit (seed 1)",
    "room": "1.5M Gaussians, SH3, 1920x1080, 120-frame handheld path (seed 2)",
    "city": "6M Gaussians, SH3, 1920x1080, 240-frame street walk (seed 3)",
    "stress": "3M Gaussians with 20% needles, SH3, 3840x2160, 60-frame jumpy orbit (seed 4)",
}


def workload(name: str, n_frames: int | None = None, n_gaussians: int | None = None,
             speed: float = 1.0, interval: float | None = None) -> Workload:
    """Build one of the five seeded workloads.

    ``n_frames`` truncates the camera path; ``n_gaussians`` overrides the scene
    size (used only by tests that want a smaller scene of the same structure);
    ``speed`` scales the per-frame camera motion (the motion-speed study);
    ``interval`` (room only) replaces the path by the curve fitted through the
    room's key poses, sampled every ``interval`` units of eye travel (120
    frames unless ``n_frames`` says otherwise).
    """
    if interval is not None:
        if name != "room":
            raise KeyError("key-pose paths are defined for the room workload only")
        scene = scene_room(n_gaussians or 1_500_000, 2)
        cams = keyframe_path(ROOM_KEY_EYES, ROOM_KEY_TARGETS, interval, 1920, 1080,
                             n_frames=n_frames or 120)
        return Workload(name, scene, cams)
    v = float(speed)
    if name == "tiny":
        n = n_gaussians or 10_000
        scene = scene_uniform_cube(n, 0, degree=0)
        cams = orbit_path(8, 3.0, 15.0, 1.0 * v, 256, 256)
    elif name == "object":
        n = n_gaussians or 300_000
        scene = scene_clusters(n, 1)
        cams = orbit_path(60, 6.0, 15.0, 0.5 * v, 1280, 720)
    elif name == "room":
        n = n_gaussians or 1_500_000
        scene = scene_room(n, 2)
        cams = handheld_path(120, (0.0, -5.0, 0.3), (0.0, 0.0, 0.0), 0.3 * v, 0.01 * v, 1920, 1080)
    elif name == "city":
        n = n_gaussians or 6_000_000
        scene = scene_city(n, 3)
        cams = walk_path(240, (-60.0, 0.0, 1.7), 0.0, 0.2 * v, 0.05 * v, 1920, 1080)
    elif name == "stress":
        n = n_gaussians or 3_000_000
        scene = scene_room(n, 4, needle_fraction=0.2)
        cams = orbit_path(60, 5.0, 10.0, 0.0, 3840, 2160, steps=(0.2 * v, 8.0 * v))
    else:
        raise KeyError(f"unknown workload {name!r}; choose from {sorted(WORKLOADS)}")
    if n_frames is not None:
        cams = cams[:n_frames]
    return Workload(name, scene, cams)


def small_scene(n, seed, degree=3, extent=1.0, log_scale_mean=-3.0):
    """Small random scene for unit-level parity cases."""
    return scene_uniform_cube(n, seed, degree=degree, log_scale_mean=log_scale_mean,
                              extent=extent)
