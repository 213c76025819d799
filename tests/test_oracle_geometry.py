"""Pins for the oracle's per-Gaussian geometry and its screen-space bounds.

Sec. 3.1 (rotation, scale), Sec. 3.4 (clamped ellipsoid, Eq. 9-10) and
Sec. 4.2 (conservative perspective-correct bounds, Eq. 11-14).

Pinned against: scipy's quaternion->matrix routine; the closed-form
projected extent of a sphere (on and off the optical axis); a dense sampling
of an anisotropic ellipsoid's silhouette; and brute-force coverage, i.e.
every ray/Gaussian hit found WITHOUT rectangles lies inside the rectangle.
"""
import math

import numpy as np
import pytest
from scipy.spatial.transform import Rotation

import oracle
from helpers import dc_for_colour, random_tiny_scene, small_camera
from paper_2608_17298_amd.scenes import ALPHA_MIN, custom_scene, make_scene


def _one(means, ls, q, logit, cam, deg=0):
    n = len(means)
    K = (deg + 1) ** 2
    sh = np.zeros((n, K, 3))
    sh[:, 0, :] = dc_for_colour(0.5)
    return custom_scene(means, ls, q, logit, sh, cam)


def test_rotation_matches_scipy():
    rng = np.random.default_rng(3)
    n = 64
    q = rng.standard_normal((n, 4)) * rng.uniform(0.3, 3.0, (n, 1))  # unnormalised on purpose
    ls = rng.normal(-2, 0.5, (n, 3))
    cam = small_camera()
    sc = _one(rng.uniform(-1, 1, (n, 3)), ls, q, np.zeros(n), cam)
    o = oracle.OracleScene(sc, params=dict(quats=q, log_scales=ls))
    W = o.prim_info().W
    R_ref = Rotation.from_quat(q[:, [1, 2, 3, 0]]).as_matrix()  # scipy: scalar last
    S = np.exp(ls)
    R_or = np.transpose(S[:, :, None] * W, (0, 2, 1))  # W = S^-1 R^T
    assert np.abs(R_or - R_ref).max() < 1e-12


def _p_h(raw, axis):
    Qaa, Qa4, Q44 = raw[:, 2 * axis], raw[:, 2 * axis + 1], raw[:, 4]
    p = Qa4 / Q44
    return p, np.sqrt(p * p - Qaa / Q44)


def _skewed_camera(w=64, h=48):
    """Non-square pixels and an off-centre principal point."""
    cam = small_camera(w, h)
    cam.fx, cam.fy = float(np.float32(cam.fx * 1.3)), float(np.float32(cam.fy * 0.85))
    cam.cx, cam.cy = float(np.float32(cam.cx + 3.25)), float(np.float32(cam.cy - 2.5))
    return cam


@pytest.mark.parametrize("z0,ls,logit,skew", [(0.0, -2.0, 0.0, False), (1.5, -1.2, 2.0, True),
                                              (-2.5, -3.0, -1.0, True)])
def test_sphere_on_axis_closed_form(z0, ls, logit, skew):
    cam = _skewed_camera() if skew else small_camera(64, 48)
    # on the optical axis of the camera: pixel coordinate (cx, cy)
    m = np.array([[0.0, 0.0, z0]])
    sc = _one(m, np.full((1, 3), ls), [[1, 0, 0, 0]], [logit], cam)
    o = oracle.OracleScene(sc, params=dict(means=m, log_scales=np.full((1, 3), ls), opacity_logits=np.array([logit])))
    raw = o.bounds_raw()
    sigma = 1 / (1 + math.exp(-logit))
    r = math.sqrt(2 * math.log(sigma / ALPHA_MIN)) * math.exp(ls)
    z = z0 + 4.0
    for axis, (f, c) in enumerate(((cam.fx, cam.cx), (cam.fy, cam.cy))):
        p, h = _p_h(raw, axis)
        assert abs(p[0] - c) < 1e-9
        assert abs(h[0] - f * r / math.sqrt(z * z - r * r)) < 1e-9 * f


def test_sphere_off_axis_tangent_angles():
    cam = _skewed_camera()
    rng = np.random.default_rng(5)
    n = 20
    X = rng.uniform(-1.5, 1.5, n)
    Z = rng.uniform(-1.0, 2.0, n)
    m = np.stack([X, np.zeros(n), Z], 1)
    ls = np.repeat(rng.uniform(-2.5, -1.5, (n, 1)), 3, axis=1)
    logit = rng.normal(0, 1, n)
    sc = _one(m, ls, np.tile([1.0, 0, 0, 0], (n, 1)), logit, cam)
    o = oracle.OracleScene(sc, params=dict(means=m, log_scales=ls, opacity_logits=logit))
    p, h = _p_h(o.bounds_raw(), 0)
    sigma = 1 / (1 + np.exp(-logit))
    r = np.sqrt(2 * np.log(sigma / ALPHA_MIN)) * np.exp(ls[:, 0])
    Zc = Z + 4.0
    D = np.hypot(X, Zc)
    thc = np.arctan2(X, Zc)
    beta = np.arcsin(r / D)
    lo = cam.cx + cam.fx * np.tan(thc - beta)
    hi = cam.cx + cam.fx * np.tan(thc + beta)
    assert np.abs((p - h) - lo).max() < 1e-8
    assert np.abs((p + h) - hi).max() < 1e-8


def test_ellipsoid_silhouette_sampling():
    """x/y screen extent of an anisotropic clamped ellipsoid vs a dense sampling of its surface."""
    cam = _skewed_camera()
    rng = np.random.default_rng(11)
    n = 6
    m = rng.uniform(-0.8, 0.8, (n, 3))
    ls = rng.normal(-1.8, 0.5, (n, 3))
    q = rng.standard_normal((n, 4))
    logit = rng.normal(0, 1, n)
    sc = _one(m, ls, q, logit, cam)
    o = oracle.OracleScene(sc, params=dict(means=m, log_scales=ls, quats=q, opacity_logits=logit))
    raw = o.bounds_raw()
    th, ph = np.meshgrid(np.linspace(0, math.pi, 700), np.linspace(0, 2 * math.pi, 1400), indexing="ij")
    y = np.stack([np.sin(th) * np.cos(ph), np.sin(th) * np.sin(ph), np.cos(th)], -1).reshape(-1, 3)
    R = Rotation.from_quat(q[:, [1, 2, 3, 0]]).as_matrix()
    sigma = 1 / (1 + np.exp(-logit))
    ac = np.sqrt(2 * np.log(sigma / ALPHA_MIN))
    for i in range(n):
        pts = m[i] + (y * (np.exp(ls[i]) * ac[i])) @ R[i].T
        pc = pts + np.array([0, 0, 4.0])  # camera frame (R = I, t = (0,0,4))
        u = cam.fx * pc[:, 0] / pc[:, 2] + cam.cx
        v = cam.fy * pc[:, 1] / pc[:, 2] + cam.cy
        for axis, coord in ((0, u), (1, v)):
            p, h = _p_h(raw[i:i + 1], axis)
            assert coord.max() <= p[0] + h[0] + 1e-9
            assert coord.min() >= p[0] - h[0] - 1e-9
            tol = 1e-4 * max(h[0], 1.0)
            assert coord.max() >= p[0] + h[0] - tol
            assert coord.min() <= p[0] - h[0] + tol


def _assert_coverage(sc, params=None, pixels=None):
    o = oracle.OracleScene(sc, params=params)
    info = o.prim_info()
    if pixels is None:
        pixels = np.arange(o.W * o.H)
    off, prims = o.all_hits(pixels, brute=True)
    owner = np.repeat(pixels, np.diff(off))
    px, py = owner % o.W, owner // o.W
    r = info.rect[prims]
    inside = (px >= r[:, 0]) & (px <= r[:, 2]) & (py >= r[:, 1]) & (py <= r[:, 3])
    assert (info.state[prims] == oracle.STATE_ACTIVE).all(), "a culled Gaussian was hit"
    assert inside.all(), f"{(~inside).sum()} hits outside their rectangle"
    a = o.render(pixels, brute=False)
    b = o.render(pixels, brute=True)
    assert np.array_equal(a["color"], b["color"])
    assert np.array_equal(a["n_included"], b["n_included"])
    return len(prims)


def test_coverage_tiny_workload():
    nhits = _assert_coverage(make_scene("tiny"))
    assert nhits > 50_000


def test_coverage_small_workload_subset():
    sc = make_scene("small", n=3000, width=96, height=72)
    nhits = _assert_coverage(sc)
    assert nhits > 1000


def test_coverage_random_anisotropic():
    rng = np.random.default_rng(21)
    sc, params, _ = random_tiny_scene(rng, 40, 40, 30, 3, ls_sd=0.8)
    _assert_coverage(sc, params)


def test_eye_plane_crossing_behind_and_offscreen():
    """Ellipsoids that cross the eye plane (z = -4 here), contain the camera,
    lie behind it, or sit beside the frustum: rectangles stay conservative and
    the culled ones produce no hit anywhere."""
    cam = small_camera(48, 40)
    means = np.array([
        [0.0, 0.0, -4.0],   # contains the camera centre
        [0.6, 0.2, -3.9],   # straddles the eye plane inside the view cone
        [-0.5, -0.4, -4.2],
        [12.0, 0.0, -4.0],  # straddles the eye plane far to the side
        [0.0, -9.0, -3.8],
        [0.1, 0.1, -7.0],   # wholly behind the camera
        [0.3, -0.2, 1.0],   # ordinary, in front
        [5.0, 0.0, 0.0],    # in front but outside the view cone
    ])
    ls = np.log(np.array([[0.5, 0.4, 0.6], [0.3, 0.3, 0.3], [0.4, 0.2, 0.3], [0.5, 0.5, 0.5],
                          [0.4, 0.4, 0.4], [0.5, 0.5, 0.5], [0.2, 0.3, 0.25], [0.2, 0.2, 0.2]]))
    q = np.random.default_rng(2).standard_normal((len(means), 4))
    logit = np.array([1.0, 0.5, 2.0, 1.0, 1.0, 1.0, 0.5, 1.0])
    sh = np.zeros((len(means), 1, 3))
    sh[:, 0, :] = dc_for_colour(0.7)
    sc = custom_scene(means, ls, q, logit, sh, cam)
    params = dict(means=means, log_scales=ls, quats=q, opacity_logits=logit)
    o = oracle.OracleScene(sc, params=params)
    st = o.prim_info().state
    assert st[5] == oracle.STATE_CULLED_BEHIND
    assert st[3] == oracle.STATE_CULLED_OFFSCREEN and st[4] == oracle.STATE_CULLED_OFFSCREEN
    assert st[7] == oracle.STATE_CULLED_OFFSCREEN
    assert (st[[0, 1, 2, 6]] == oracle.STATE_ACTIVE).all()
    _assert_coverage(sc, params)


def test_random_eye_plane_crossings():
    """Many ellipsoids straddling the eye plane at random lateral offsets, so
    that the covered columns/rows are one-sided, two-sided or everything."""
    cam = _skewed_camera(40, 32)
    rng = np.random.default_rng(31)
    n = 300
    means = np.stack([rng.uniform(-3, 3, n), rng.uniform(-3, 3, n), -4.0 + rng.uniform(-0.6, 0.6, n)], 1)
    ls = np.log(rng.uniform(0.08, 0.5, (n, 3)))
    q = rng.standard_normal((n, 4))
    logit = rng.normal(0, 1.5, n)
    sh = np.zeros((n, 1, 3))
    sh[:, 0, :] = dc_for_colour(rng.uniform(0.2, 0.8, (n, 3)))
    sc = custom_scene(means, ls, q, logit, sh, cam)
    params = dict(means=means, log_scales=ls, quats=q, opacity_logits=logit)
    o = oracle.OracleScene(sc, params=params)
    raw = o.bounds_raw()
    st = o.prim_info().state
    crossing = (raw[:, 4] >= 0) & (st == oracle.STATE_ACTIVE)
    assert crossing.sum() > 20
    area = o.prim_info().area
    assert (area[crossing] < o.W * o.H).sum() > 5, "expected some partial rectangles"
    assert _assert_coverage(sc, params) > 100


def test_opacity_cull_and_nonfinite():
    cam = small_camera()
    means = np.array([[0, 0, 0], [0.1, 0, 0], [0.2, 0, 0.0]])
    ls = np.full((3, 3), -2.0)
    logit = np.array([math.log(ALPHA_MIN / (1 - ALPHA_MIN)) - 1e-6, 0.0, 0.0])
    means_nf = means.copy()
    means_nf[2, 0] = np.nan
    sh = np.zeros((3, 1, 3))
    sc = custom_scene(means, ls, np.tile([1.0, 0, 0, 0], (3, 1)), logit, sh, cam)
    o = oracle.OracleScene(sc, params=dict(means=means_nf, opacity_logits=logit))
    st = o.prim_info().state
    assert st[0] == oracle.STATE_CULLED_OPACITY
    assert st[1] == oracle.STATE_ACTIVE
    assert st[2] == oracle.STATE_CULLED_NONFINITE
