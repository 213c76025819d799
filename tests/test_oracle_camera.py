"""Pins for the oracle's camera and for the rounding of its pixel
rectangles, with general (non-identity) camera rotations.

Sec. 3.2 Eq. 3 (the camera ray r(tau) = o + tau d) and Sec. 4.2 Eq. 11-14
(projected bounds and the pixel rectangle they give).  Everything expected
here is derived independently of the oracle: rotations come from scipy,
camera centres and ray directions from numpy, the continuous screen extent
of a clamped ellipsoid from the support function of the ellipsoid in camera
coordinates (checked against dense sampling of its surface), and the pixel
rectangle from that extent by the rule "first / last pixel column whose
centre lies within 1e-4 px of the extent".  A transposed camera rotation in
the ray, in the camera centre or in the view matrix, or a floor / ceil / +-0.5
slip in the rectangle rounding, fails one of these tests.
"""
import math

import numpy as np
import pytest
from scipy.spatial.transform import Rotation

import oracle
from helpers import dc_for_colour, random_tiny_scene, rotated_camera
from paper_2608_17298_amd.scenes import ALPHA_MIN, custom_scene

EPS_PX = 1e-4  # rectangle padding in pixels (reading R11)


def _scene(means, ls, q, logit, cam, colour=0.6):
    n = len(means)
    sh = np.zeros((n, 1, 3))
    sh[:, 0, :] = dc_for_colour(colour)
    params = dict(means=np.asarray(means, np.float64), log_scales=np.asarray(ls, np.float64),
                  quats=np.asarray(q, np.float64), opacity_logits=np.asarray(logit, np.float64),
                  sh=sh)
    return custom_scene(means, ls, q, logit, sh, cam), params


def _random_camera(rng, w=57, h=43):
    cam = rotated_camera(w, h)
    cam.R = Rotation.random(random_state=int(rng.integers(1 << 30))).as_matrix().astype(np.float32)
    cam.t = rng.uniform(-1.0, 1.0, 3).astype(np.float32)
    cam.fx, cam.fy = float(np.float32(cam.fx * 1.2)), float(np.float32(cam.fy * 0.9))
    cam.cx, cam.cy = float(np.float32(cam.cx + 2.75)), float(np.float32(cam.cy - 1.5))
    return cam


def test_camera_centre_and_rays_general_rotation():
    """o = -R^T t and d = R^T (a, b, 1) / |.| with a = (x + .5 - cx) / fx,
    b = (y + .5 - cy) / fy, for random rotations and translations."""
    rng = np.random.default_rng(101)
    for _ in range(6):
        cam = _random_camera(rng)
        sc, params = _scene(np.zeros((1, 3)), np.full((1, 3), -2.0), [[1, 0, 0, 0]], [0.0], cam)
        o = oracle.OracleScene(sc, params=params)
        R = np.asarray(cam.R, np.float64)
        t = np.asarray(cam.t, np.float64)
        assert np.abs(o.camera_origin() - (-R.T @ t)).max() < 1e-14
        pix = rng.integers(0, cam.width * cam.height, 40)
        px, py = pix % cam.width, pix // cam.width
        dc = np.stack([(px + 0.5 - cam.cx) / cam.fx, (py + 0.5 - cam.cy) / cam.fy, np.ones(len(pix))], 1)
        d = dc @ R  # rows: R^T dc
        d /= np.linalg.norm(d, axis=1, keepdims=True)
        got = o.ray_prim(pix, np.zeros(len(pix), np.int64))["dir"]
        assert np.abs(got - d).max() < 1e-14


def test_gaussian_on_a_pixel_ray_rotated_camera():
    """A small isotropic Gaussian centred on the ray of pixel p (a point
    placed with numpy at depth s along o + s d) is hit at p with
    tau = s, D^2 = 0 and alpha = sigma, and renders C = sigma c there
    (Eq. 3-8); a pixel three columns away does not see its mean."""
    cam = rotated_camera(61, 47)
    R = np.asarray(cam.R, np.float64)
    o_ref = -R.T @ np.asarray(cam.t, np.float64)
    rng = np.random.default_rng(7)
    for k in range(10):
        x, y = int(rng.integers(3, cam.width - 4)), int(rng.integers(3, cam.height - 4))
        dc = np.array([(x + 0.5 - cam.cx) / cam.fx, (y + 0.5 - cam.cy) / cam.fy, 1.0])
        d = R.T @ dc
        d /= np.linalg.norm(d)
        s = rng.uniform(3.0, 5.0)
        mu = o_ref + s * d
        logit = rng.normal(0.5, 0.5)
        sc, params = _scene(mu[None], np.full((1, 3), math.log(0.02)), [[1, 0, 0, 0]], [logit], cam, 0.7)
        o = oracle.OracleScene(sc, params=params)
        p = y * cam.width + x
        r = o.ray_prim([p, p + 3], [0, 0])
        sigma = 1.0 / (1.0 + math.exp(-logit))
        assert r["hit"][0]
        assert abs(r["tau"][0] - s) < 1e-9 * s
        assert r["D2"][0] < 1e-16
        assert abs(r["alpha"][0] - sigma) < 1e-12
        assert r["D2"][1] > 1.0  # three pixels off: far from the mean in Gaussian units
        c = o.render([p])["color"][0]
        assert np.abs(c - sigma * 0.7).max() < 1e-12, k


def _support_extent(mu, ls, q, logit, cam):
    """Continuous pixel extent (u_lo, u_hi, v_lo, v_hi) of the clamped
    ellipsoid (radius alpha_c in Gaussian units, Eq. 9-10) seen by the
    pinhole camera.  In camera coordinates the ellipsoid is
    {x : (x - m)^T A (x - m) <= 1} with A^-1 = Sigma_c = (R Rq S ac)(R Rq S ac)^T;
    the plane n.x = 0 through the camera centre touches it where
    (n.m)^2 = n^T Sigma_c n (support function).  For the column planes
    n = (1, 0, -u) (pixel column fx u + cx) this is a quadratic in u."""
    R = np.asarray(cam.R, np.float64)
    t = np.asarray(cam.t, np.float64)
    Rq = Rotation.from_quat(np.asarray(q, np.float64)[[1, 2, 3, 0]]).as_matrix()
    sigma = 1.0 / (1.0 + math.exp(-logit))
    ac = math.sqrt(2.0 * math.log(sigma / ALPHA_MIN))
    M = R @ Rq @ np.diag(np.exp(ls) * ac)
    Sc = M @ M.T
    m = R @ mu + t
    out = []
    for a, f, c in ((0, cam.fx, cam.cx), (1, cam.fy, cam.cy)):
        # (m_a - u m_z)^2 = Saa - 2 u Saz + u^2 Szz
        A2 = m[2] ** 2 - Sc[2, 2]
        B1 = -2.0 * (m[a] * m[2] - Sc[a, 2])
        C0 = m[a] ** 2 - Sc[a, a]
        disc = B1 * B1 - 4.0 * A2 * C0
        r1 = (-B1 - math.sqrt(disc)) / (2.0 * A2)
        r2 = (-B1 + math.sqrt(disc)) / (2.0 * A2)
        out += [f * min(r1, r2) + c, f * max(r1, r2) + c]
    return out


def _sampled_extent(mu, ls, q, logit, cam, n=300):
    R = np.asarray(cam.R, np.float64)
    t = np.asarray(cam.t, np.float64)
    Rq = Rotation.from_quat(np.asarray(q, np.float64)[[1, 2, 3, 0]]).as_matrix()
    sigma = 1.0 / (1.0 + math.exp(-logit))
    ac = math.sqrt(2.0 * math.log(sigma / ALPHA_MIN))
    th, ph = np.meshgrid(np.linspace(0, math.pi, n), np.linspace(0, 2 * math.pi, 2 * n), indexing="ij")
    y = np.stack([np.sin(th) * np.cos(ph), np.sin(th) * np.sin(ph), np.cos(th)], -1).reshape(-1, 3)
    pts = mu + (y * (np.exp(ls) * ac)) @ Rq.T
    pc = pts @ R.T + t
    u = cam.fx * pc[:, 0] / pc[:, 2] + cam.cx
    v = cam.fy * pc[:, 1] / pc[:, 2] + cam.cy
    return u.min(), u.max(), v.min(), v.max()


def _ellipsoids(rng, n, cam, spread=1.2):
    means = rng.uniform(-spread, spread, (n, 3))
    ls = rng.normal(-2.0, 0.5, (n, 3))
    q = rng.standard_normal((n, 4))
    logit = rng.normal(0.5, 1.0, n)
    return means, ls, q, logit


@pytest.mark.parametrize("cam_kind", ["rotated", "random"])
def test_projected_extent_general_rotation(cam_kind):
    """p -+ h of Eq. 12-14 equals the support-function extent of each clamped
    ellipsoid in a rotated camera, which also bounds a dense sampling of
    its surface."""
    rng = np.random.default_rng(211)
    cam = rotated_camera(64, 48) if cam_kind == "rotated" else _random_camera(rng, 64, 48)
    if cam_kind == "random":  # keep the ellipsoids in front of this camera
        R = np.asarray(cam.R, np.float64)
        centre = -R.T @ np.asarray(cam.t, np.float64) + 4.0 * R.T @ np.array([0, 0, 1.0])
    else:
        centre = np.zeros(3)
    means, ls, q, logit = _ellipsoids(rng, 24, cam)
    means = means + centre
    sc, params = _scene(means, ls, q, logit, cam)
    o = oracle.OracleScene(sc, params=params)
    raw = o.bounds_raw()
    assert (raw[:, 4] < 0).all()  # every ellipsoid in front of the eye plane
    for i in range(len(means)):
        ulo, uhi, vlo, vhi = _support_extent(means[i], ls[i], q[i], logit[i], cam)
        for axis, (lo, hi) in enumerate(((ulo, uhi), (vlo, vhi))):
            Qaa, Qa4, Q44 = raw[i, 2 * axis], raw[i, 2 * axis + 1], raw[i, 4]
            p = Qa4 / Q44
            h = math.sqrt(p * p - Qaa / Q44)
            assert abs((p - h) - lo) < 1e-9 * max(1.0, abs(lo)), (i, axis)
            assert abs((p + h) - hi) < 1e-9 * max(1.0, abs(hi)), (i, axis)
        if i < 6:
            su = _sampled_extent(means[i], ls[i], q[i], logit[i], cam)
            ext = (ulo, uhi, vlo, vhi)
            tol = [1e-3 * max(1.0, uhi - ulo)] * 2 + [1e-3 * max(1.0, vhi - vlo)] * 2
            assert su[0] >= ext[0] - 1e-9 and su[1] <= ext[1] + 1e-9
            assert su[2] >= ext[2] - 1e-9 and su[3] <= ext[3] + 1e-9
            assert all(abs(a - b) < t for a, b, t in zip(su, ext, tol))


def test_rectangle_rounding_is_tight():
    """The pixel rectangle is exactly the columns / rows whose centre lies
    within EPS_PX of the continuous extent, clamped to the image:
    x0 = max(0, ceil(u_lo - 1/2 - eps)), x1 = min(W - 1, floor(u_hi - 1/2 + eps)),
    same for y (R11).  Ellipsoids partly outside the image are included, so
    the clamping is exercised; values within 1e-7 of a rounding boundary are
    skipped (none in practice)."""
    rng = np.random.default_rng(307)
    cam = rotated_camera(53, 41)
    means, ls, q, logit = _ellipsoids(rng, 400, cam, spread=2.2)
    sc, params = _scene(means, ls, q, logit, cam)
    o = oracle.OracleScene(sc, params=params)
    info = o.prim_info()
    W, H = cam.width, cam.height
    checked = clamped = 0
    for i in range(len(means)):
        ulo, uhi, vlo, vhi = _support_extent(means[i], ls[i], q[i], logit[i], cam)
        want = []
        for lo, hi, npix in ((ulo, uhi, W), (vlo, vhi, H)):
            a, b = lo - 0.5 - EPS_PX, hi - 0.5 + EPS_PX
            if min(abs(a - round(a)), abs(b - round(b))) < 1e-7:
                want = None
                break
            want.append((max(0, math.ceil(a)), min(npix - 1, math.floor(b))))
        if want is None:
            continue
        (x0, x1), (y0, y1) = want
        if x0 > x1 or y0 > y1:  # no pixel centre covered: culled
            assert info.state[i] == oracle.STATE_CULLED_OFFSCREEN, i
            assert info.area[i] == 0
            continue
        assert info.state[i] == oracle.STATE_ACTIVE, i
        assert tuple(info.rect[i]) == (x0, y0, x1, y1), (i, tuple(info.rect[i]), (x0, y0, x1, y1))
        assert info.area[i] == (x1 - x0 + 1) * (y1 - y0 + 1)
        checked += 1
        clamped += int(x0 == 0 or y0 == 0 or x1 == W - 1 or y1 == H - 1)
    assert checked > 250 and clamped > 20, (checked, clamped)


def test_coverage_rotated_cameras():
    """Brute force with rotated cameras: every hit found without rectangles
    lies inside its rectangle, and the bucketed render equals the brute one."""
    rng = np.random.default_rng(401)
    for cam in (rotated_camera(44, 34), rotated_camera(40, 36, axis=(-0.3, 0.2, 1.0), angle_deg=-70.0),
                _random_camera(rng, 38, 30)):
        R = np.asarray(cam.R, np.float64)
        centre = -R.T @ np.asarray(cam.t, np.float64) + 4.0 * R.T @ np.array([0, 0, 1.0])
        sc, params, _ = random_tiny_scene(rng, 60, cam.width, cam.height, 3, ls_sd=0.7, cam=cam)
        params["means"] = params["means"] + centre
        sc.means = params["means"].astype(np.float32)
        o = oracle.OracleScene(sc, params=params)
        info = o.prim_info()
        pixels = np.arange(cam.width * cam.height)
        off, prims = o.all_hits(pixels, brute=True)
        owner = np.repeat(pixels, np.diff(off))
        px, py = owner % o.W, owner // o.W
        r = info.rect[prims]
        assert len(prims) > 500
        assert ((px >= r[:, 0]) & (px <= r[:, 2]) & (py >= r[:, 1]) & (py <= r[:, 3])).all()
        a = o.render(pixels, brute=False)
        b = o.render(pixels, brute=True)
        assert np.array_equal(a["color"], b["color"])
