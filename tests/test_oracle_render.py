"""Pins for the oracle's forward trace (Sec. 3.2-3.3, Eq. 3-8).

Pinned against closed forms (a Gaussian hit through its mean has alpha equal
to its opacity; two stacked Gaussians composite by the hand formula), the
transmittance invariant (with unit colours C = 1 - T_final, and T_final is the
product of (1 - alpha)), an independent world-space Mahalanobis minimisation
along the ray (covariance from scipy's rotation and numpy's inverse), and the
compositing order / termination rule read from the recorded hits.
"""
import math

import numpy as np
import pytest
from scipy.spatial.transform import Rotation

import oracle
from helpers import Y00, dc_for_colour, pixel_ray_point, random_tiny_scene, small_camera
from paper_2608_17298_amd.scenes import ALPHA_MIN, T_MIN, custom_scene, make_scene


def _through_mean_scene(depths, logits, colours, px=13, py=17, ls=-2.0, w=32, h=32):
    cam = small_camera(w, h)
    means = np.stack([pixel_ray_point(cam, px, py, d) for d in depths])
    n = len(depths)
    q = np.random.default_rng(0).standard_normal((n, 4))
    lsa = np.full((n, 3), ls)
    sh = np.zeros((n, 1, 3))
    sh[:, 0, :] = dc_for_colour(np.asarray(colours))
    lg = np.asarray(logits, np.float64)
    sc = custom_scene(means, lsa, q, lg, sh, cam)
    params = dict(means=means, log_scales=lsa, quats=q, opacity_logits=lg, sh=sh)
    return sc, params, cam, py * w + px


def test_single_gaussian_through_mean():
    sc, params, cam, p = _through_mean_scene([4.0], [0.7], [[0.2, 0.5, 0.9]])
    o = oracle.OracleScene(sc, params=params)
    r = o.render([p])
    sigma = 1 / (1 + math.exp(-0.7))
    assert r["n_included"][0] == 1
    assert np.abs(r["color"][0] - sigma * np.array([0.2, 0.5, 0.9])).max() < 1e-12
    assert abs(r["T_final"][0] - (1 - sigma)) < 1e-12


def test_two_gaussians_hand_formula():
    c1, c2 = np.array([0.9, 0.1, 0.3]), np.array([0.2, 0.8, 0.6])
    # Listed back-to-front so that the depth sort, not the index, decides.
    sc, params, cam, p = _through_mean_scene([5.5, 3.5], [0.3, -0.4], [c2, c1])
    o = oracle.OracleScene(sc, params=params)
    r = o.render([p])
    a1 = 1 / (1 + math.exp(0.4))
    a2 = 1 / (1 + math.exp(-0.3))
    assert np.abs(r["color"][0] - (a1 * c1 + (1 - a1) * a2 * c2)).max() < 1e-12
    off, prim, LT, tau = o.records([p], r["n_included"])
    assert list(prim) == [1, 0]
    assert np.abs(LT[1, :3] - a1 * c1).max() < 1e-12 and abs(LT[1, 3] - (1 - a1)) < 1e-12


def test_termination_includes_crossing_hit():
    # Three nearly opaque Gaussians on one ray: T drops below T_MIN at the 2nd.
    lg = [8.0, 8.0, 8.0]
    sc, params, cam, p = _through_mean_scene([3.0, 4.0, 5.0], lg, [[0.5] * 3] * 3)
    o = oracle.OracleScene(sc, params=params)
    r = o.render([p])
    s = 1 / (1 + math.exp(-8.0))
    assert (1 - s) ** 2 < T_MIN <= (1 - s)
    assert r["n_included"][0] == 2 and r["id_end"][0] == 1
    assert abs(r["T_final"][0] - (1 - s) ** 2) < 1e-15


@pytest.mark.parametrize("which", ["tiny", "random"])
def test_transmittance_invariant_unit_colour(which):
    if which == "tiny":
        sc = make_scene("tiny")
        sh = np.zeros_like(sc.sh, dtype=np.float64)
        sh[:, 0, :] = dc_for_colour(1.0)
        params = dict(sh=sh)
    else:
        rng = np.random.default_rng(8)
        sc, params, _ = random_tiny_scene(rng, 60, 40, 36, 3, logit_mu=1.5)
        sh = np.zeros((60, 16, 3))
        sh[:, 0, :] = dc_for_colour(1.0)
        params = dict(params, sh=sh)
    o = oracle.OracleScene(sc, params=params)
    r = o.render()
    err = np.abs(r["color"] - (1.0 - r["T_final"])[:, None]).max()
    assert err < 1e-12
    # T_final = prod (1 - alpha_i) over the composited hits, alphas queried per hit.
    pix = np.nonzero(r["n_included"] > 0)[0][:500]
    off, prim, LT, tau = o.records(pix, r["n_included"][pix])
    q = o.ray_prim(np.repeat(pix, np.diff(off)), prim)
    logT = np.add.reduceat(np.log1p(-q["alpha"]), off[:-1])
    assert np.abs(np.exp(logT) - r["T_final"][pix]).max() < 1e-12


def test_records_order_and_termination_rule():
    sc = make_scene("small", n=60000, width=80, height=64)
    o = oracle.OracleScene(sc)
    r = o.render()
    pix = np.arange(o.W * o.H)
    off, prim, LT, tau = o.records(pix, r["n_included"])
    for j in np.nonzero(r["n_included"] > 1)[0][:2000]:
        t = tau[off[j]:off[j + 1]]
        assert (np.diff(t) >= 0).all()
        T = LT[off[j]:off[j + 1], 3]
        assert (np.diff(T) <= 0).all() and (T[:-1] >= T_MIN).all() and T[0] == 1.0
    term = np.isfinite(r["tau_end"])
    assert term.any() and (~term).any()
    assert (r["T_final"][term] < T_MIN).all()
    assert (r["T_final"][~term] >= T_MIN).all()
    last = off[1:][term] - 1
    assert np.array_equal(prim[last], r["id_end"][term])


def _mahalanobis_along(o_w, d, mu, ls, q, taus):
    R = Rotation.from_quat(q[[1, 2, 3, 0]]).as_matrix()
    Sigma = R @ np.diag(np.exp(2 * ls)) @ R.T
    Si = np.linalg.inv(Sigma)
    x = o_w[None, :] + taus[:, None] * d[None, :] - mu[None, :]
    return np.einsum("ni,ij,nj->n", x, Si, x), Si


def test_max_response_point_independent_route():
    rng = np.random.default_rng(4)
    sc, params, _ = random_tiny_scene(rng, 25, 30, 26, 1, ls_sd=0.6)
    o = oracle.OracleScene(sc, params=params)
    o_w = o.camera_origin()
    m = 3000
    pix = rng.integers(0, o.W * o.H, m)
    prim = rng.integers(0, 25, m)
    q = o.ray_prim(pix, prim)
    sigma = 1 / (1 + np.exp(-params["opacity_logits"]))
    for j in range(0, m, 7):
        i = prim[j]
        d = q["dir"][j]
        mu, ls, qq = params["means"][i], params["log_scales"][i], params["quats"][i] / np.linalg.norm(params["quats"][i])
        # 1-D quadratic in tau: minimum at -b/(2a) of (o + tau d - mu)^T Si (...)
        _, Si = _mahalanobis_along(o_w, d, mu, ls, qq, np.zeros(1))
        e = o_w - mu
        tau_star = -(d @ Si @ e) / (d @ Si @ d)
        scale = np.linalg.norm(mu - o_w)
        assert abs(q["tau"][j] - tau_star) < 1e-9 * scale
        D2s, _ = _mahalanobis_along(o_w, d, mu, ls, qq, np.array([tau_star]))
        assert abs(q["D2"][j] - D2s[0]) < 1e-9 * (1 + D2s[0])
        grid = tau_star + np.linspace(-0.5, 0.5, 2001)
        Dg, _ = _mahalanobis_along(o_w, d, mu, ls, qq, grid)
        assert Dg.min() >= D2s[0] - 1e-9 * (1 + D2s[0])
        D2c = 2 * math.log(sigma[i] / ALPHA_MIN) if sigma[i] > ALPHA_MIN else -1.0
        assert q["hit"][j] == bool(tau_star > 0 and D2s[0] <= D2c)
        assert abs(q["alpha"][j] - sigma[i] * math.exp(-0.5 * D2s[0])) < 1e-12


def test_colour_uses_ray_direction_sh():
    """SH colour is evaluated at the per-ray direction (degree-1 term sign flips across the image)."""
    cam = small_camera(32, 32)
    means = np.array([[0.0, 0.0, 0.0]])
    ls = np.log(np.full((1, 3), 0.35))
    sh = np.zeros((1, 4, 3))
    sh[0, 0, :] = dc_for_colour(0.5)
    sh[0, 3, :] = 0.3  # Y_1^1 ~ x component of the direction
    sc = custom_scene(means, ls, [[1, 0, 0, 0]], [3.0], sh, cam)
    o = oracle.OracleScene(sc, params=dict(means=means, log_scales=ls, sh=sh, opacity_logits=np.array([3.0])))
    left, right = 16 * 32 + 10, 16 * 32 + 21
    r = o.render([left, right])
    q = o.ray_prim([left, right], [0, 0])
    Y1 = math.sqrt(3 / (4 * math.pi))
    for j in range(2):
        c = 0.5 + 0.3 * Y1 * q["dir"][j][0]
        assert np.abs(r["color"][j] - q["alpha"][j] * c).max() < 1e-12


def test_clamped_colour_channel_and_barely_visible():
    """A negative raw colour clamps to zero (and carries no SH gradient); a
    Gaussian with opacity just above alpha_min is still hit through its mean."""
    cam = small_camera(32, 32)
    px, py = 13, 17
    means = np.stack([pixel_ray_point(cam, px, py, 4.0), pixel_ray_point(cam, px + 6, py, 4.0)])
    ls = np.full((2, 3), -2.0)
    sh = np.zeros((2, 1, 3))
    sh[0, 0, :] = dc_for_colour([-0.3, 0.4, 0.7])
    sh[1, 0, :] = dc_for_colour([0.6, 0.6, 0.6])
    s1 = 1.5 * ALPHA_MIN
    lg = np.array([0.5, math.log(s1 / (1 - s1))])
    q = np.tile([1.0, 0, 0, 0], (2, 1))
    dl = np.zeros((32, 32, 3))
    dl[py, px] = [1.0, 1.0, 1.0]
    sc = custom_scene(means, ls, q, lg, sh, cam, dl_dimage=dl)
    params = dict(means=means, log_scales=ls, quats=q, opacity_logits=lg, sh=sh)
    o = oracle.OracleScene(sc, params=params)
    assert o.prim_info().state[1] == oracle.STATE_ACTIVE
    r = o.render([py * 32 + px, py * 32 + px + 6])
    s0 = 1 / (1 + math.exp(-0.5))
    assert np.abs(r["color"][0] - s0 * np.array([0.0, 0.4, 0.7])).max() < 1e-12
    assert np.abs(r["color"][1] - s1 * 0.6).max() < 1e-14
    g = o.backward(dl)
    assert g["sh"][0, 0, 0] == 0.0 and abs(g["sh"][0, 0, 1] - s0 * Y00) < 1e-12
