"""Pins for the oracle's tile-primitive lists and intermediate-buffer address.

Sec. 4.3: per-tile primitive lists (reverse tile mapping) and the address
idx(i,t,p) = O_prim(i) + O_tile(i,t) + O_pixel(i,t,p) (Eq. 16).

The lists are pinned to an O(tiles x N) overlap test; the address is pinned
by its defining properties: it is a bijection onto [0, sum A_i), primitive i
owns the block starting at the exclusive prefix sum of the areas, and inside
that block the order is (tile row, tile column, pixel row, pixel column).
"""
import numpy as np
import pytest

import oracle
from helpers import random_tiny_scene
from paper_2608_17298_amd.scenes import make_scene


def _brute_lists(rect, state, W, H, ts):
    ntx, nty = -(-W // ts), -(-H // ts)
    out = []
    for ty in range(nty):
        for tx in range(ntx):
            x0, x1, y0, y1 = tx * ts, min(W - 1, tx * ts + ts - 1), ty * ts, min(H - 1, ty * ts + ts - 1)
            hit = (state == 0) & (rect[:, 0] <= x1) & (rect[:, 2] >= x0) & (rect[:, 1] <= y1) & (rect[:, 3] >= y0)
            out.append(np.nonzero(hit)[0])
    return out


@pytest.mark.parametrize("name,kw,ts", [("tiny", {}, 16), ("tiny", {}, 8),
                                        ("small", dict(n=5000, width=100, height=75), 8)])
def test_tile_lists_brute(name, kw, ts):
    sc = make_scene(name, **kw)
    o = oracle.OracleScene(sc)
    info = o.prim_info()
    off, prim = oracle.tile_lists(info.rect, info.state, o.W, o.H, ts)
    ref = _brute_lists(info.rect, info.state, o.W, o.H, ts)
    assert len(off) == len(ref) + 1
    for t, r in enumerate(ref):
        assert np.array_equal(prim[off[t]:off[t + 1]], r)


def _all_rect_pixels(info, W):
    prims, pixels = [], []
    for i in np.nonzero(info.area > 0)[0]:
        x0, y0, x1, y1 = info.rect[i]
        ys, xs = np.mgrid[y0:y1 + 1, x0:x1 + 1]
        prims.append(np.full(xs.size, i))
        pixels.append((ys * W + xs).ravel())
    return np.concatenate(prims), np.concatenate(pixels)


@pytest.mark.parametrize("ts", [8, 16])
def test_lt_index_layout(ts):
    rng = np.random.default_rng(12)
    sc, params, _ = random_tiny_scene(rng, 30, 45, 37, 0, ls_mu=-1.6, ls_sd=0.5)
    o = oracle.OracleScene(sc, params=params)
    info = o.prim_info()
    W = o.W
    prims, pixels = _all_rect_pixels(info, W)
    idx = o.lt_index(ts, prims, pixels)
    total = int(info.area.sum())
    assert total == len(idx)
    assert np.array_equal(np.sort(idx), np.arange(total))          # bijection
    base = np.concatenate([[0], np.cumsum(info.area)])[:-1]
    px, py = pixels % W, pixels // W
    key = np.lexsort((px, py, px // ts, py // ts, prims))            # prim, tile row, tile col, row, col
    rank = np.empty_like(idx)
    rank[key] = np.arange(len(idx))
    assert np.array_equal(idx, rank)
    assert (idx >= base[prims]).all() and (idx < base[prims] + info.area[prims]).all()
    # outside the rectangle -> -1
    i = int(np.nonzero(info.area > 0)[0][0])
    x0, y0, x1, y1 = info.rect[i]
    outside = []
    if x1 + 1 < W:
        outside.append(y0 * W + x1 + 1)
    if y0 > 0:
        outside.append((y0 - 1) * W + x0)
    if outside:
        assert (o.lt_index(ts, np.full(len(outside), i), np.array(outside)) == -1).all()


def test_lt_index_tiny_workload_bijection():
    sc = make_scene("tiny")
    o = oracle.OracleScene(sc)
    info = o.prim_info()
    prims, pixels = _all_rect_pixels(info, o.W)
    idx = o.lt_index(16, prims, pixels)
    assert np.array_equal(np.sort(idx), np.arange(int(info.area.sum())))
