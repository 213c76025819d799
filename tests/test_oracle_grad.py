"""Pins for the oracle's analytic gradient (pixel-centric backward, Sec. 3.5).

Central finite differences of the oracle's own fp64 forward on tiny scenes
(every parameter group, SH degree 0 and 3), closed forms for a Gaussian hit
through its mean and for two stacked Gaussians, and the gradient arity the
paper states (59 values per Gaussian at SH degree 3, 48 of them SH).
"""
import math
import os

import numpy as np
import pytest

import oracle
from helpers import Y00, dc_for_colour, pixel_ray_point, random_tiny_scene, small_camera
from paper_2608_17298_amd.scenes import custom_scene

GROUPS = [("means", "means"), ("log_scales", "log_scales"), ("quats", "quats"),
          ("opacity_logits", "logits"), ("sh", "sh")]


def _golden():
    out = {}
    with open(os.path.join(os.path.dirname(__file__), "golden", "paper_constants.txt")) as f:
        for line in f:
            line = line.split("#")[0].strip()
            if line:
                k, v = line.split()
                out[k] = float(v)
    return out


def _loss_and_decisions(sc, params, dl):
    o = oracle.OracleScene(sc, params=params)
    r = o.render()
    pix = np.arange(o.W * o.H)
    off, prim, _, _ = o.records(pix, r["n_included"])
    return float((r["color"] * dl.reshape(-1, 3)).sum()), (r["n_included"].copy(), prim.copy())


def _fd_check(sc, params, dl, groups_checked=None, rtol=1e-6):
    o = oracle.OracleScene(sc, params=params)
    an = o.backward(dl)
    _, base_dec = _loss_and_decisions(sc, params, dl)
    checked = skipped = 0
    for pkey, gkey in GROUPS:
        if groups_checked and gkey not in groups_checked:
            continue
        theta = params[pkey]
        a = an[gkey].reshape(-1)
        scale = max(np.abs(a).max(), 1e-12)
        for j in range(theta.size):
            t0 = theta.reshape(-1)[j]
            h = 1e-6 * max(1.0, abs(t0))
            vals = []
            same = True
            for sgn in (1, -1):
                th = theta.copy().reshape(-1)
                th[j] = t0 + sgn * h
                p2 = dict(params)
                p2[pkey] = th.reshape(theta.shape)
                L, dec = _loss_and_decisions(sc, p2, dl)
                same = same and np.array_equal(dec[0], base_dec[0]) and np.array_equal(dec[1], base_dec[1])
                vals.append(L)
            if not same:
                skipped += 1
                continue
            fd = (vals[0] - vals[1]) / (2 * h)
            assert abs(fd - a[j]) <= rtol * max(abs(a[j]), 1e-3 * scale), (gkey, j, fd, a[j])
            checked += 1
    return checked, skipped


@pytest.mark.parametrize("deg,n,seed", [(0, 12, 1), (3, 8, 2), (1, 16, 3)])
def test_finite_differences(deg, n, seed):
    rng = np.random.default_rng(seed)
    sc, params, dl = random_tiny_scene(rng, n, 24, 20, deg, logit_mu=0.5, ls_sd=0.4)
    checked, skipped = _fd_check(sc, params, dl)
    assert checked > 0.9 * (checked + skipped)


def test_finite_differences_dense_overlap():
    """Many overlapping, fairly opaque Gaussians so that termination is reached."""
    rng = np.random.default_rng(7)
    sc, params, dl = random_tiny_scene(rng, 24, 16, 16, 1, spread=0.25, ls_mu=-1.7, logit_mu=3.0,
                                       logit_sd=1.0)
    o = oracle.OracleScene(sc, params=params)
    assert np.isfinite(o.render()["tau_end"]).any(), "scene should terminate some rays"
    checked, skipped = _fd_check(sc, params, dl, groups_checked={"means", "logits", "log_scales"})
    assert checked > 0.8 * (checked + skipped)


def _through_mean(depths, logits, colours, px=9, py=7):
    cam = small_camera(20, 16)
    means = np.stack([pixel_ray_point(cam, px, py, d) for d in depths])
    n = len(depths)
    q = np.random.default_rng(1).standard_normal((n, 4))
    ls = np.full((n, 3), -2.2)
    sh = np.zeros((n, 1, 3))
    sh[:, 0, :] = dc_for_colour(np.asarray(colours))
    lg = np.asarray(logits, np.float64)
    dl = np.zeros((16, 20, 3))
    dl[py, px] = [1.0, -2.0, 0.5]
    sc = custom_scene(means, ls, q, lg, sh, cam, dl_dimage=dl)
    return sc, dict(means=means, log_scales=ls, quats=q, opacity_logits=lg, sh=sh), dl


def test_closed_form_single_gaussian_at_mean():
    c = np.array([0.3, 0.6, 0.45])
    sc, params, dl = _through_mean([4.0], [0.4], [c])
    g = oracle.OracleScene(sc, params=params).backward(dl)
    gp = np.array([1.0, -2.0, 0.5])
    s = 1 / (1 + math.exp(-0.4))
    assert abs(g["logits"][0] - s * (1 - s) * (c @ gp)) < 1e-12
    assert np.abs(g["sh"][0, 0] - s * Y00 * gp).max() < 1e-12
    # rho = 1 is stationary at the mean: no first-order change in shape or position.
    for k in ("means", "log_scales", "quats"):
        assert np.abs(g[k]).max() < 1e-9, k


def test_closed_form_two_gaussians():
    c1, c2 = np.array([0.8, 0.2, 0.4]), np.array([0.1, 0.7, 0.5])
    sc, params, dl = _through_mean([3.0, 5.0], [0.2, 1.1], [c1, c2])
    g = oracle.OracleScene(sc, params=params).backward(dl)
    gp = np.array([1.0, -2.0, 0.5])
    s1, s2 = 1 / (1 + math.exp(-0.2)), 1 / (1 + math.exp(-1.1))
    assert abs(g["logits"][0] - s1 * (1 - s1) * ((c1 - s2 * c2) @ gp)) < 1e-12
    assert abs(g["logits"][1] - s2 * (1 - s2) * (1 - s1) * (c2 @ gp)) < 1e-12


def test_arity_matches_paper():
    gold = _golden()
    rng = np.random.default_rng(0)
    sc, params, dl = random_tiny_scene(rng, 3, 8, 8, 3)
    g = oracle.OracleScene(sc, params=params).backward(dl)
    per = sum(int(np.prod(v.shape[1:])) if v.ndim > 1 else 1 for v in g.values())
    assert per == gold["params_per_gaussian_sh3"]
    assert int(np.prod(g["sh"].shape[1:])) == gold["sh_params_per_gaussian_sh3"]
    assert abs(gold["alpha_min"] - 1 / 255) < 1e-15
