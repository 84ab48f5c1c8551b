"""CPU pins of the camera-path synthesis (inputs only): the key-pose curve
and its fixed-interval sampling (Sec. IV-A trajectory synthesis)."""
import numpy as np

from paper_2607_03390_amd import synth


def test_catmull_rom_passes_through_keys():
    rng = np.random.default_rng(0)
    keys = rng.standard_normal((7, 3))
    got = synth.catmull_rom(keys, np.arange(7.0))
    np.testing.assert_allclose(got, keys, atol=1e-12)


def test_catmull_rom_reproduces_lines():
    # equally spaced collinear keys: the curve is the line, uniformly parameterised
    a, d = np.array([1.0, -2.0, 0.5]), np.array([0.3, 0.1, -0.2])
    keys = a + np.arange(5.0)[:, None] * d
    u = np.linspace(0.0, 4.0, 37)
    np.testing.assert_allclose(synth.catmull_rom(keys, u), a + u[:, None] * d, atol=1e-12)


def test_catmull_rom_c1_at_keys():
    rng = np.random.default_rng(1)
    keys = rng.standard_normal((5, 3))
    h = 1e-6
    for k in (1, 2, 3):
        left = (synth.catmull_rom(keys, [k]) - synth.catmull_rom(keys, [k - h])) / h
        right = (synth.catmull_rom(keys, [k + h]) - synth.catmull_rom(keys, [k])) / h
        np.testing.assert_allclose(left, right, atol=1e-4)


def test_keyframe_path_fixed_interval():
    for interval in (0.01, 0.04):
        cams = synth.keyframe_path(synth.ROOM_KEY_EYES, synth.ROOM_KEY_TARGETS, interval, 64, 48)
        eyes = np.array([-c.w2c[:3, :3].astype(np.float64).T @ c.w2c[:3, 3] for c in cams])
        step = np.linalg.norm(np.diff(eyes, axis=0), axis=1)
        # chord of an arc step: within 1e-3 of the interval on this gentle curve
        assert np.all(np.abs(step - interval) < 1e-3 * interval + 2e-6)
        np.testing.assert_allclose(eyes[0], synth.ROOM_KEY_EYES[0], atol=1e-5)
        for c in cams:
            R = c.w2c[:3, :3].astype(np.float64)
            np.testing.assert_allclose(R @ R.T, np.eye(3), atol=1e-5)
    # twice the interval covers the same curve in half the frames
    a = synth.keyframe_path(synth.ROOM_KEY_EYES, synth.ROOM_KEY_TARGETS, 0.02, 64, 48)
    b = synth.keyframe_path(synth.ROOM_KEY_EYES, synth.ROOM_KEY_TARGETS, 0.04, 64, 48)
    assert abs(len(a) - 2 * len(b)) <= 2
    np.testing.assert_allclose(a[2].w2c, b[1].w2c, atol=2e-5)


def test_room_keyframe_workload():
    w = synth.workload("room", n_frames=5, n_gaussians=1000, interval=0.02)
    assert len(w.cameras) == 5 and w.scene.n == 1000
