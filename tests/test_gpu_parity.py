"""GPU parity: the HIP path (through the C ABI) against the fp64 oracle.

Bars: rectangles, areas, offsets and per-tile Gaussian sets bit-exact;
pixels within 1e-5 max-abs outside ambiguous pixels (decision margin below
1e-9, counted); each gradient group within 1e-4 relative L2.
Sizes span several tiles with a ragged edge; the oracle finishes in seconds.
"""
import numpy as np
import pytest

import oracle
from helpers import (dc_for_colour, l1_upstream, max_abs_over_rms, per_gaussian_err, random_tiny_scene, rel_l2,
                     rotated_camera, run_gpu, small_camera)
from paper_2608_17298_amd.scenes import custom_scene, make_scene

pytestmark = pytest.mark.gpu

PIX_TOL = 1e-5
GRAD_TOL = 1e-4
# Per-Gaussian bar: each hit's terms carry about 1e-6 relative error (fp32
# colour, SH and accumulation; fp64 geometry), so a Gaussian's gradient errs
# by about 1e-6 times the cancellation factor sum|terms| / |sum|; 1e-3
# allows a factor of 1000 against max(|g_i|, 1e-3 x the group's RMS).
ELEM_TOL = 1e-3
AMBIG = 1e-9
GROUPS = ["means", "log_scales", "quats", "logits", "sh"]


def _scene(name):
    if name == "tiny":
        return make_scene("tiny")
    if name == "small":  # the small workload at its full size, with its L1 upstream gradient
        sc = make_scene("small")
        sc.dl_dimage = l1_upstream(sc, oracle)
        return sc
    if name == "small_reduced":
        sc = make_scene("small", n=30000, width=203, height=157)
        sc.dl_dimage = l1_upstream(sc, oracle)
        return sc
    if name == "1m_reduced":
        sc = make_scene("1m", n=120000, width=171, height=115)
        sc.dl_dimage = l1_upstream(sc, oracle)
        return sc
    if name == "stress_reduced":
        sc = make_scene("stress", n=6000, width=97, height=75)
        sc.dl_dimage = l1_upstream(sc, oracle)
        return sc
    if name == "random_sh3":
        sc, _, _ = random_tiny_scene(np.random.default_rng(5), 300, 83, 61, 3, spread=1.0, ls_mu=-2.6,
                                     ls_sd=0.5, logit_mu=1.0)
        return sc
    if name in ("random_sh1", "random_sh2"):  # the K = 4 and K = 9 kernel instantiations
        deg = int(name[-1])
        sc, _, _ = random_tiny_scene(np.random.default_rng(40 + deg), 400, 75, 58, deg, spread=1.0, ls_mu=-2.5,
                                     ls_sd=0.5, logit_mu=0.5, high_sd=0.15)
        return sc
    if name == "random_sh3_tile16":  # 16x16 tiles (four pixel groups per tile) at SH degree 3
        sc, _, _ = random_tiny_scene(np.random.default_rng(7), 500, 97, 70, 3, tile=16, spread=1.0, ls_mu=-2.4,
                                     ls_sd=0.5, logit_mu=0.5)
        return sc
    if name == "rotated_sh3":  # camera turned about a non-axis-aligned axis (with roll), SH3, 8x8 tiles
        sc, _, _ = random_tiny_scene(np.random.default_rng(9), 600, 91, 67, 3, spread=1.0, ls_mu=-2.5, ls_sd=0.5,
                                     logit_mu=0.5, high_sd=0.15, cam=rotated_camera(91, 67))
        return sc
    if name == "opaque_sh3":  # nearly opaque Gaussians: logits ~ N(10, 2), 1 - alpha down to ~1e-8
        sc, _, _ = random_tiny_scene(np.random.default_rng(13), 400, 79, 61, 3, spread=1.0, ls_mu=-2.4,
                                     ls_sd=0.5, logit_mu=10.0, logit_sd=2.0, cam=rotated_camera(79, 61))
        return sc
    if name in ("large_sh3", "large_sh3_tile16"):  # large low-opacity footprints: a reduction block's
        # rows span several flag chunks (up to 6.3k rows at 8x8 tiles; four rows per pair at 16x16)
        # and Gaussians straddle chunk and share boundaries
        sc, _, _ = random_tiny_scene(np.random.default_rng(23), 160, 160, 120, 3, spread=0.6, ls_mu=-0.7,
                                     ls_sd=0.3, logit_mu=-2.5, high_sd=0.1, tile=16 if name.endswith("16") else 8)
        return sc
    if name == "nonfinite_sh3":  # NaN / inf parameters and zero-norm quaternions among ordinary Gaussians
        rng = np.random.default_rng(17)
        sc, _, _ = random_tiny_scene(rng, 400, 73, 59, 3, spread=1.0, ls_mu=-2.5, ls_sd=0.5, logit_mu=0.5)
        bad = rng.choice(sc.n, 48, replace=False)
        kinds = np.arange(len(bad)) % 8
        nan, inf = np.float32(np.nan), np.float32(np.inf)
        for i, k in zip(bad, kinds):
            if k == 0:
                sc.means[i, 0] = nan
            elif k == 1:
                sc.means[i, 2] = -inf
            elif k == 2:
                sc.log_scales[i, 1] = inf
            elif k == 3:
                sc.log_scales[i, 0] = -inf
            elif k == 4:
                sc.opacity_logits[i] = nan
            elif k == 5:
                sc.opacity_logits[i] = inf
            elif k == 6:
                sc.quats[i] = 0.0
            else:
                sc.quats[i, 3] = nan
        sc.bad = np.sort(bad)
        return sc
    raise KeyError(name)


_cache = {}


def _case(name, mode="gather", tile=None):
    key = (name, mode, tile)
    if key not in _cache:
        sc = _cache.get(("scene", name)) or _scene(name)
        _cache[("scene", name)] = sc
        if ("oracle", name) not in _cache:
            o = oracle.OracleScene(sc)
            _cache[("oracle", name)] = (o, o.prim_info(), o.render(), o.backward(sc.dl_dimage))
        _cache[key] = run_gpu(sc, mode=mode, tile=tile)
    o, info, ren, grads = _cache[("oracle", name)]
    return _cache[("scene", name)], o, info, ren, grads, _cache[key]


SCENES = ["tiny", "small", "small_reduced", "1m_reduced", "stress_reduced", "random_sh3", "random_sh1", "random_sh2",
          "random_sh3_tile16", "rotated_sh3", "opaque_sh3", "large_sh3", "large_sh3_tile16",
          "nonfinite_sh3"]


@pytest.mark.parametrize("name", SCENES)
def test_bounds_bit_exact(name):
    sc, o, info, ren, grads, gpu = _case(name)
    assert np.array_equal(gpu["rect"], info.rect)
    area = np.diff(gpu["lt_offset"])
    assert np.array_equal(area, info.area)
    assert gpu["lt_offset"][0] == 0 and gpu["lt_entries"] == info.area.sum()


@pytest.mark.parametrize("name", SCENES)
def test_tile_lists_bit_exact(name):
    sc, o, info, ren, grads, gpu = _case(name)
    ts = sc.tile
    off, prim = oracle.tile_lists(info.rect, info.state, o.W, o.H, ts)
    assert np.array_equal(gpu["tile_range"], off)
    assert gpu["pair_count"] == len(prim)
    key = gpu["pair_key"]
    gp = gpu["pair_prim"].astype(np.int64)
    for t in range(len(off) - 1):
        seg = gp[off[t]:off[t + 1]]
        assert np.array_equal(np.sort(seg), prim[off[t]:off[t + 1]]), t
        k = key[off[t]:off[t + 1]]
        # front-to-back order inside a tile: depth lower bound, then index
        assert np.all((np.diff(k) > 0) | ((np.diff(k) == 0) & (np.diff(seg) > 0))), t
    assert np.all(gpu["pair_tile"][:-1] <= gpu["pair_tile"][1:])
    # pair_offset: each Gaussian owns tile_count consecutive emission slots
    act = np.nonzero(info.area > 0)[0]
    po = gpu["pair_offset"]
    order = act[np.argsort(po[act], kind="stable")]
    assert np.array_equal(np.diff(np.append(po[order], po[-1])), gpu["tile_count"][order].astype(np.int64))


@pytest.mark.parametrize("name", ["small_reduced", "1m_reduced", "stress_reduced", "random_sh3_tile16",
                                  "rotated_sh3"])
def test_pair_keys_bound_every_hit(name):
    """Each pair's key is at most tau_q / s_q at every pixel q of its tile
    where the ray hits the Gaussian (gart_frame.pair_key): tau_q from the
    oracle's max-response point (Eq. 3-5), s_q = |R^T u_q| / (c . u_q) for
    the pixel's camera ray u_q = (a, b, 1) and c the unit camera-space
    direction through the tile centre.  The forward's early compositing and
    the backward's list cut-off rely on it."""
    sc, o, info, ren, grads, gpu = _case(name)
    ts, W = sc.tile, o.W
    cam = sc.camera
    tx_n = (W + ts - 1) // ts
    rng = np.random.default_rng(7)
    P = gpu["pair_count"]
    sel = rng.choice(P, min(P, 4000), replace=False)
    pix, prims, keys, axes = [], [], [], []
    for j in sel:
        t, i = int(gpu["pair_tile"][j]), int(gpu["pair_prim"][j])
        x0, y0, x1, y1 = info.rect[i]
        tx, ty = t % tx_n, t // tx_n
        xs = np.arange(max(x0, tx * ts), min(x1, tx * ts + ts - 1) + 1)
        ys = np.arange(max(y0, ty * ts), min(y1, ty * ts + ts - 1) + 1)
        assert len(xs) > 0 and len(ys) > 0, (j, t, i)
        p = (ys[:, None] * W + xs[None, :]).ravel()
        pix.append(p)
        prims.append(np.full(p.size, i))
        keys.append(np.full(p.size, gpu["pair_key"][j], np.float64))
        c = np.array([((tx + 0.5) * ts - cam.cx) / cam.fx, ((ty + 0.5) * ts - cam.cy) / cam.fy, 1.0])
        axes.append(np.tile(c / np.linalg.norm(c), (p.size, 1)))
    pix, prims, keys, axes = np.concatenate(pix), np.concatenate(prims), np.concatenate(keys), np.concatenate(axes)
    r = o.ray_prim(pix, prims)
    hit = r["hit"]
    assert hit.any()
    u = np.stack([(pix % W + 0.5 - cam.cx) / cam.fx, (pix // W + 0.5 - cam.cy) / cam.fy, np.ones(pix.size)], 1)
    s_q = np.linalg.norm(u @ np.asarray(cam.R, np.float64), axis=1) / np.einsum("ij,ij->i", u, axes)
    depth = r["tau"] / s_q
    assert np.all(keys[hit] <= depth[hit]), np.max(keys[hit] - depth[hit])
    # the per-tile bound is not vacuous: most hit pairs get a positive key
    assert np.mean(keys[hit] > 0) > 0.5


@pytest.mark.parametrize("name", SCENES)
def test_forward_pixels_and_markers(name):
    sc, o, info, ren, grads, gpu = _case(name)
    img = gpu["image"].reshape(-1, 3)
    ok = ren["margin"] >= AMBIG
    err = np.abs(img - ren["color"]).max(axis=1)
    assert err[ok].max() <= PIX_TOL, (err[ok].max(), np.argmax(np.where(ok, err, 0)))
    assert (~ok).sum() <= max(2, 1e-3 * ok.size)
    assert np.array_equal(gpu["n_hits"][ok], ren["n_included"][ok])
    term = np.isfinite(ren["tau_end"]) & ok
    assert np.array_equal(gpu["id_end"][term], ren["id_end"][term])
    assert np.all(~np.isfinite(gpu["tau_end"][~np.isfinite(ren["tau_end"]) & ok]))
    # final colour in the frame's fixed point (half a step of rounding) and
    # final transmittance, as the backward reads them
    assert np.abs(gpu["state_color"] - ren["color"])[ok].max() <= PIX_TOL
    slack = 0.5 * gpu["color_step"] + 1.2e-7 * np.maximum(1.0, np.abs(img))
    assert np.all(np.abs(gpu["state_color"] - img.astype(np.float64)) <= slack)
    assert np.abs(gpu["t_final"].astype(np.float64) - ren["T_final"])[ok].max() <= 1e-6


@pytest.mark.parametrize("name", ["tiny", "small_reduced", "random_sh3"])
def test_forward_lt_entries(name):
    """(L, T) written at idx(i,t,p) for every composited hit (Eq. 16)."""
    import torch
    sc, o, info, ren, grads, _ = _case(name)
    gpu = run_gpu(sc, keep_frame=True)
    ok = np.nonzero(ren["margin"] >= AMBIG)[0]
    pix = ok[ren["n_included"][ok] > 0][:20000]
    off, prim, LT, tau = o.records(pix, ren["n_included"][pix])
    owner = np.repeat(pix, np.diff(off))
    idx = o.lt_index(sc.tile, prim, owner)
    assert (idx >= 0).all()
    L, T = gpu["frame"].lt_entries_host(torch.from_numpy(idx).cuda())
    assert np.abs(L - LT[:, :3]).max() <= PIX_TOL
    assert np.abs(T.astype(np.float64) - LT[:, 3]).max() <= 1e-6


@pytest.mark.parametrize("mode", ["gather", "gather_wave", "gather_atomic", "scatter", "hybrid"])
@pytest.mark.parametrize("name", SCENES)
def test_backward_parity(name, mode):
    sc, o, info, ren, grads, gpu = _case(name, mode)
    for k in GROUPS:
        e = rel_l2(gpu["grads"][k], grads[k])
        assert e <= GRAD_TOL, (k, e)
        assert np.isfinite(gpu["grads"][k]).all(), k
        pe = per_gaussian_err(gpu["grads"][k], grads[k])
        assert pe <= ELEM_TOL, (k, pe)


def test_nonfinite_parameters_culled():
    """Gaussians with NaN or infinite means, log-scales or logits, or a
    zero-norm or NaN quaternion, are culled on both sides: empty rectangle,
    no pairs, zero gradients, and no NaN anywhere in the outputs."""
    sc, o, info, ren, grads, gpu = _case("nonfinite_sh3")
    bad = sc.bad
    assert (info.state[bad] == oracle.STATE_CULLED_NONFINITE).all()
    assert (gpu["rect"][bad, 0] > gpu["rect"][bad, 2]).all()
    assert (np.diff(gpu["lt_offset"])[bad] == 0).all() and (gpu["tile_count"][bad] == 0).all()
    assert not np.isin(gpu["pair_prim"], bad).any()
    assert np.isfinite(gpu["image"]).all()
    for k in GROUPS:
        assert np.isfinite(gpu["grads"][k]).all(), k
        assert (gpu["grads"][k][bad] == 0).all(), k
    assert (info.state != oracle.STATE_ACTIVE).sum() >= len(bad)
    assert (info.state == oracle.STATE_ACTIVE).sum() > 200


@pytest.mark.parametrize("name", ["tiny", "1m_reduced", "random_sh3"])
def test_hybrid_t_only_buffer(name):
    """Hybrid mode: the forward writes only T per entry (4 bytes, Sec. 4.4
    hybrid approach) at the same idx(i,t,p), the image is the gather mode's
    bit for bit, the pixel pass walks every composited hit (once per window
    of list positions), no global atomics are issued, and repeated runs
    agree to float rounding (LDS atomics vary the summation order)."""
    import torch
    from paper_2608_17298_amd import gart
    sc, o, info, ren, grads, gpu = _case(name, "hybrid")
    ref = _case(name, "gather")[5]
    assert np.array_equal(gpu["image"], ref["image"])
    assert np.array_equal(gpu["n_hits"], ref["n_hits"])
    c = gpu["counters"]
    assert c[gart.CNT_BWD_ATOMICS] == 0
    assert c[gart.CNT_BWD_HITS] == c[gart.CNT_FWD_HITS]
    assert c[gart.CNT_BWD_ACTIVE] == ref["counters"][gart.CNT_BWD_ACTIVE]
    assert c[gart.CNT_BWD_STEPS] >= c[gart.CNT_BWD_HITS]
    if np.diff(gpu["tile_range"]).max() <= (384 if sc.tile == 8 else 128):  # one window per tile
        assert c[gart.CNT_BWD_STEPS] == c[gart.CNT_BWD_HITS]
    h = run_gpu(sc, mode="hybrid", keep_frame=True)
    for k in GROUPS:
        assert rel_l2(h["grads"][k], gpu["grads"][k]) <= 1e-6, k
    fr = h["frame"]
    assert fr.lt.shape[1] * 2 == 4 and int(fr.c.lt_format) == gart.LT_T_ONLY
    ok = np.nonzero(ren["margin"] >= AMBIG)[0]
    pix = ok[ren["n_included"][ok] > 0][:20000]
    off, prim, LT, tau = o.records(pix, ren["n_included"][pix])
    idx = o.lt_index(sc.tile, prim, np.repeat(pix, np.diff(off)))
    L, T = fr.lt_entries_host(torch.from_numpy(idx).cuda())
    assert L is None
    assert np.abs(T.astype(np.float64) - LT[:, 3]).max() <= 1e-6


@pytest.mark.parametrize("name", ["tiny", "stress_reduced", "1m_reduced"])
def test_gather_wave_units(name):
    """GATHER_WAVE evaluates the units with at least 48 hits by a whole wave
    (Sec. 4.4, a warp per primitive) and the rest per lane: the dense path
    is taken where such units exist, every unit is still visited once, and
    the gradients match the per-lane gather to float rounding."""
    from paper_2608_17298_amd import gart
    sc, o, info, ren, grads, gpu = _case(name, "gather_wave")
    ref = _case(name, "gather")[5]
    c, cr = gpu["counters"], ref["counters"]
    assert c[gart.CNT_BWD_ACTIVE] == cr[gart.CNT_BWD_ACTIVE]
    assert c[gart.CNT_BWD_HITS] == cr[gart.CNT_BWD_HITS]
    if name == "stress_reduced":  # large footprints: many units cover most of their pixels
        assert c[gart.CNT_BWD_WAVE_UNITS] > 0
    assert c[gart.CNT_BWD_WAVE_UNITS] <= c[gart.CNT_BWD_ACTIVE]
    for k in GROUPS:
        assert rel_l2(gpu["grads"][k], ref["grads"][k]) <= 1e-6, k
    assert gart.CNT_BWD_WAVE_UNITS == 10


# Reduced-precision intermediate storage (Sec. 6 suggests fp16).  Each
# layout is checked against the oracle's model of it: the backward with L and
# T replaced by their stored values (the T-only layouts of the hybrid mode
# sum the colour behind a hit from the stored T of the later hits).
#
# The two sides' L and T differ by fp32 colour rounding (~1e-7 relative), so
# a stored value within that distance of a rounding boundary may land on the
# neighbouring code on one side only: a fraction p ~ 2e-7 |L| / q of the
# values (q the quantum: fp16 2^-11 |L|, fixed16 B / 2^16; p < 0.5% here).
# Such a value errs by a whole quantum where the model's own rounding errs by
# q / sqrt(12) on average, so the residual is about sqrt(12 p) < 0.25 of the
# storage effect itself, rel_l2(model, exact); in a small scene a single
# heavy hit can carry it, so the bar is 0.3 of the storage effect, and never
# below the full-precision 1e-4.  Per Gaussian the check is absolute: one
# quantum divided by 1 - alpha can be all of a small gradient, so the bar is
# |g_i - m_i| <= 1e-2 x the group's RMS (2^-11, one fp16 quantum of a unit
# colour, times the 1 / (1 - alpha) of alpha = 0.95).
STORAGE_MODEL = {("gather", "half"): "half", ("scatter", "half"): "half", ("hybrid", "half"): "t_half",
                 ("gather", "fixed16"): "fixed16", ("scatter", "fixed16"): "fixed16",
                 ("hybrid", "fixed16"): "t_log16"}
STORAGE_FLIP_FRAC = 0.3
STORAGE_ELEM_TOL = 1e-2


def _storage_grads(name, model):
    key = ("oracle_storage", name, model)
    if key not in _cache:
        sc = _cache[("scene", name)]
        _cache[key] = _cache[("oracle", name)][0].backward(sc.dl_dimage, storage=model)
    return _cache[key]


@pytest.mark.parametrize("mode,prec", sorted(STORAGE_MODEL))
@pytest.mark.parametrize("name", SCENES)
def test_backward_reduced_storage(name, mode, prec):
    sc, o, info, ren, grads, ref = _case(name, mode)
    gpu = run_gpu(sc, mode=mode, precision=prec)
    assert np.array_equal(gpu["image"], ref["image"])  # storage does not change the forward's result
    model = _storage_grads(name, STORAGE_MODEL[(mode, prec)])
    for k in GROUPS:
        e = rel_l2(gpu["grads"][k], model[k])
        assert e <= max(GRAD_TOL, STORAGE_FLIP_FRAC * rel_l2(model[k], grads[k])), (k, e)
        assert np.isfinite(gpu["grads"][k]).all(), k
        pe = max_abs_over_rms(gpu["grads"][k], model[k])
        assert pe <= STORAGE_ELEM_TOL, (k, pe)


@pytest.mark.parametrize("prec", ["half", "fixed16"])
@pytest.mark.parametrize("mode", ["gather", "hybrid"])
def test_reduced_storage_entries(mode, prec):
    """Stored entries decode to the oracle's (L, T) within the format's
    rounding: fp16 to 2^-11 relative; fixed16 L to half a step of
    color_step * 2^16 and T to 2^(1/8192) - 1 relative; plus 1e-6 for the
    fp32 colour evaluation behind the stored L."""
    import torch
    sc, o, info, ren, grads, _ = _case("small_reduced")
    gpu = run_gpu(sc, mode=mode, precision=prec, keep_frame=True)
    fr = gpu["frame"]
    ok = np.nonzero(ren["margin"] >= AMBIG)[0]
    pix = ok[ren["n_included"][ok] > 0][:20000]
    off, prim, LT, tau = o.records(pix, ren["n_included"][pix])
    idx = o.lt_index(sc.tile, prim, np.repeat(pix, np.diff(off)))
    L, T = fr.lt_entries_host(torch.from_numpy(idx).cuda())
    T, Tref = T.astype(np.float64), LT[:, 3]
    if prec == "half":
        assert np.all(np.abs(T - Tref) <= 2.0 ** -11 * Tref + 1e-7)
        if L is not None:
            assert np.all(np.abs(L - LT[:, :3]) <= 2.0 ** -11 * np.abs(LT[:, :3]) + 1e-6)
    else:
        assert np.all(np.abs(T - Tref) <= 8.6e-5 * Tref + 1e-7)
        if L is not None:
            assert np.all(np.abs(L - LT[:, :3]) <= 0.5 * fr.color_step * 65536 + 1e-6)
    assert (L is None) == (mode == "hybrid")


def test_backward_rejects_other_lt_format():
    """A frame rendered for one lt format cannot feed a backward that reads
    the other (INVALID_ARG, nothing launched)."""
    import torch
    from paper_2608_17298_amd import gart
    sc = make_scene("tiny")
    cam = gart.make_camera(sc.camera)
    g = gart.Gaussians.from_scene(sc)
    dl = torch.from_numpy(np.ascontiguousarray(sc.dl_dimage, dtype=np.float32)).cuda()
    for fwd, bwd in [("gather", "hybrid"), ("hybrid", "gather"), ("hybrid", "scatter")]:
        st = gart.make_settings(sc.tile, fwd)
        frame = gart.prepare(g, cam, st)
        image = torch.empty((cam.height, cam.width, 3), dtype=torch.float32, device="cuda")
        gart.gart_forward(g, cam, st, frame, image)
        with pytest.raises(gart.GartError, match="lt_format"):
            gart.gart_backward(g, cam, gart.make_settings(sc.tile, bwd), frame, dl, gart.empty_grads(g))
    torch.cuda.synchronize()


@pytest.mark.parametrize("name", ["random_sh3", "large_sh3", "large_sh3_tile16"])
def test_gather_deterministic(name):
    """Two gathers give bit-identical gradients, also where the reduction
    splits Gaussians over lane groups and flag chunks (large footprints)."""
    sc = _scene(name)
    a = run_gpu(sc, mode="gather")
    b = run_gpu(sc, mode="gather")
    for k in GROUPS:
        assert np.array_equal(a["grads"][k], b["grads"][k]), k


@pytest.mark.parametrize("tile", [8, 16])
def test_tile_sizes_agree(tile):
    sc, o, info, ren, grads, _ = _case("small_reduced")
    gpu = run_gpu(sc, tile=tile)
    ok = ren["margin"] >= AMBIG
    assert np.abs(gpu["image"].reshape(-1, 3) - ren["color"])[ok].max() <= PIX_TOL
    for k in GROUPS:
        assert rel_l2(gpu["grads"][k], grads[k]) <= GRAD_TOL, k


def test_counters_match_oracle():
    sc, o, info, ren, grads, gpu = _case("small_reduced")
    c = gpu["counters"]
    assert abs(int(c[0]) - int(ren["n_included"].sum())) <= 10
    assert c[3] == c[0]  # the backward visits exactly the composited hits


# ---------------------------------------------------------------------------
# Edge cases
# ---------------------------------------------------------------------------
def _mini(means, ls, logit, w=19, h=13, deg=0, tile=8):
    n = len(means)
    q = np.tile([1.0, 0.2, -0.1, 0.3], (n, 1))
    sh = np.zeros((n, (deg + 1) ** 2, 3))
    sh[:, 0, :] = dc_for_colour(0.6)
    dl = np.random.default_rng(0).standard_normal((h, w, 3))
    return custom_scene(means, ls, q, logit, sh, small_camera(w, h), tile=tile, dl_dimage=dl)


def test_empty_scene():
    sc = _mini(np.zeros((0, 3)), np.zeros((0, 3)), np.zeros(0))
    gpu = run_gpu(sc)
    assert gpu["pair_count"] == 0 and gpu["lt_entries"] == 0
    assert np.all(gpu["image"] == 0)
    assert all(v.size == 0 for v in gpu["grads"].values())


def test_all_culled():
    means = np.array([[0, 0, 0], [0.1, 0, 0], [0, 0, -9.0]])
    ls = np.full((3, 3), -2.0)
    logit = np.array([-8.0, -9.0, 2.0])  # two below alpha_min, one behind the camera
    sc = _mini(means, ls, logit)
    gpu = run_gpu(sc)
    assert gpu["pair_count"] == 0
    assert np.all(gpu["image"] == 0)
    assert all(np.all(v == 0) for v in gpu["grads"].values())


def test_one_pixel_image_and_camera_inside():
    means = np.array([[0, 0, -4.0], [0.0, 0.0, 0.0], [0.02, -0.01, 1.0]])
    ls = np.log(np.array([[0.6, 0.5, 0.7], [0.3, 0.3, 0.3], [0.2, 0.25, 0.3]]))
    logit = np.array([-1.0, 0.5, 1.5])
    for (w, h) in [(1, 1), (9, 17)]:
        sc = _mini(means, ls, logit, w=w, h=h, deg=1)
        o = oracle.OracleScene(sc)
        ren = o.render()
        gpu = run_gpu(sc)
        assert np.abs(gpu["image"].reshape(-1, 3) - ren["color"]).max() <= PIX_TOL
        g = o.backward(sc.dl_dimage)
        for k in GROUPS:
            assert rel_l2(gpu["grads"][k], g[k]) <= GRAD_TOL, (w, h, k)


def test_capacity_error_then_growth():
    import torch
    from paper_2608_17298_amd import gart
    sc = _scene("tiny")
    cam = gart.make_camera(sc.camera)
    st = gart.make_settings(sc.tile)
    g = gart.Gaussians.from_scene(sc)
    f = gart.Frame(g.n, g.sh_degree, cam, st, lt_capacity=10, pair_capacity=10)
    with pytest.raises(gart.GartCapacityError) as ei:
        gart.gart_bounds(g, cam, st, f)
    e = ei.value
    assert e.lt_entries == oracle.OracleScene(sc).lt_total() and e.pair_count > 10
    with pytest.raises(gart.GartError):  # a failed gart_bounds leaves the frame unusable
        gart.gart_build_tile_map(cam, st, f)
    f.grow(e.lt_entries, e.pair_count, 1.0)
    assert gart.gart_bounds(g, cam, st, f) == (e.lt_entries, e.pair_count)
    gart.gart_build_tile_map(cam, st, f)
    img = torch.empty((cam.height, cam.width, 3), device="cuda")
    gart.gart_forward(g, cam, st, f, img)


def test_invalid_args_on_device_path():
    import torch
    from paper_2608_17298_amd import gart
    sc = _scene("tiny")
    cam = gart.make_camera(sc.camera)
    g = gart.Gaussians.from_scene(sc)
    st = gart.make_settings(16)
    f = gart.prepare(g, cam, st)
    img = torch.empty((cam.height, cam.width, 3), device="cuda")
    with pytest.raises(gart.GartError):  # backward before forward
        gart.gart_backward(g, cam, st, f, img, gart.empty_grads(g))
    bad = gart.make_settings(16)
    bad.t_min = 0.0
    with pytest.raises(gart.GartError):
        gart.gart_forward(g, cam, bad, f, img)
