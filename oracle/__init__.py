"""fp64 CPU oracle -- TEST INFRASTRUCTURE ONLY.

The plain, slow, obviously-correct definition of what the GPU library
computes, used to check it.  Only the test-suite, ``__graft_entry__.smoke()``
and the CPU-baseline leg of ``bench.py`` may import this package; the GPU
library never does, and nothing here imports the GPU library.

Contents:
  * ``gart_oracle.cpp`` (built to ``_build/liboracle.so`` with g++/OpenMP):
    per-Gaussian quantities and bounds (Sec. 3.1-3.4, 4.2), the per-pixel
    ray trace and compositing (Sec. 3.2-3.3), the analytic pixel-centric
    gradient (Sec. 3.5), and the intermediate-buffer address (Sec. 4.3).
  * ``tile_lists``: per-tile primitive lists by plain enumeration of every
    (rectangle, tile) overlap (Sec. 4.3, reverse tile mapping).
  * ``train_ref``: the L1 loss gradient and the Adam step of the training
    loop around the path (numpy fp64).

Every function that has no independent pin says so in its docstring.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "gart_oracle.cpp")
_LIB_DIR = os.path.join(_HERE, "_build")
# GART_ORACLE_LIB names another build of this source to load instead (the
# mutation test loads copies with a planted mistake this way).
_LIB = os.environ.get("GART_ORACLE_LIB") or os.path.join(_LIB_DIR, "liboracle.so")

STATE_ACTIVE = 0
STATE_CULLED_OPACITY = 1
STATE_CULLED_BEHIND = 2
STATE_CULLED_OFFSCREEN = 3
STATE_CULLED_NONFINITE = 4

# Storage of (L, T) in the intermediate buffer, as the backward reads it back:
#   exact    L and T as composited
#   half     L and T rounded to float, then to the nearest fp16
#   t_half   T only (the colour behind a hit summed back to front from the
#            later hits with their stored T), T as in ``half``
#   fixed16  L in units of B / 2^16 (B = ``OracleScene.colour_bound``),
#            T = 2^(-q / 4096) with q = round(-log2(T) 4096)
#   t_log16  T only, coded as in ``fixed16``, colour behind as in ``t_half``
#   t_float  T only, rounded to float, colour behind as in ``t_half``
STORAGE_MODELS = {"exact": 0, "half": 1, "t_half": 2, "fixed16": 3, "t_log16": 4, "t_float": 5}


def storage_round(kind: str, x, unit: float = 1.0):
    """The rounding of a stored value: ``half`` (float, then fp16, ties to
    even), ``fixed16`` (L in units of ``unit``, saturating at 65535 units)
    or ``log16`` (the transmittance code of ``fixed16``)."""
    x = _c(x, np.float64).ravel()
    out = np.zeros_like(x)
    lib().orc_storage_round({"half": 1, "fixed16": 2, "log16": 3}[kind], x.shape[0], _ptr(x), _ptr(out),
                            float(unit))
    return out


def build(force: bool = True) -> str:
    """Compile the oracle with g++ (fp64, OpenMP, no fast-math)."""
    if not force and os.path.exists(_LIB):
        return _LIB
    os.makedirs(_LIB_DIR, exist_ok=True)
    tmp = _LIB + ".tmp"
    cmd = ["g++", "-O2", "-std=c++17", "-fopenmp", "-fPIC", "-shared", "-fno-fast-math",
           "-ffp-contract=off", _SRC, "-o", tmp]
    subprocess.run(cmd, check=True)
    os.replace(tmp, _LIB)
    return _LIB


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build()
        L = ctypes.CDLL(_LIB)
        P = ctypes.c_void_p
        i64, i32, f32 = ctypes.c_int64, ctypes.c_int32, ctypes.c_float
        L.orc_scene_new.restype = P
        L.orc_scene_new.argtypes = [i64, i32, P, P, P, P, P, i32, i32, P, P, P, ctypes.c_double,
                                    ctypes.c_double]
        L.orc_scene_free.argtypes = [P]
        L.orc_prim_info.argtypes = [P] * 8
        L.orc_sh_basis.argtypes = [i32, i64, P, P]
        L.orc_render.argtypes = [P, i64, P, i32, P, P, P, P, P, P]
        L.orc_bounds_raw.argtypes = [P, P]
        L.orc_ray_prim.argtypes = [P, i64, P, P, P, P, P, P, P]
        L.orc_camera_origin.argtypes = [P, P]
        L.orc_all_hits.argtypes = [P, i64, P, i32, i32, P, P, P]
        L.orc_records.argtypes = [P, i64, P, P, P, P, P]
        L.orc_backward.argtypes = [P, i64, P, P, P, P, P, P, P]
        L.orc_backward_stored.argtypes = [P, i64, P, P, P, P, P, P, P, i32]
        L.orc_storage_round.argtypes = [i32, i64, P, P, ctypes.c_double]
        L.orc_colour_bound.restype = ctypes.c_double
        L.orc_colour_bound.argtypes = [P]
        L.orc_lt_index.argtypes = [P, i32, i64, P, P, P]
        L.orc_num_threads.restype = i32
        _lib = L
    return _lib


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _c(a, dt):
    return np.ascontiguousarray(a, dtype=dt)


def num_threads() -> int:
    return int(lib().orc_num_threads())


def sh_basis(degree: int, dirs) -> np.ndarray:
    """Real SH basis (no Condon-Shortley phase), index l*l + l + m."""
    dirs = _c(dirs, np.float64).reshape(-1, 3)
    K = (degree + 1) ** 2
    Y = np.zeros((dirs.shape[0], K))
    lib().orc_sh_basis(degree, dirs.shape[0], _ptr(dirs), _ptr(Y))
    return Y


@dataclass
class PrimInfo:
    rect: np.ndarray    # [n,4] int32 x0,y0,x1,y1
    area: np.ndarray    # [n] int64
    state: np.ndarray   # [n] int32
    sigma: np.ndarray
    D2c: np.ndarray
    W: np.ndarray       # [n,3,3]
    og: np.ndarray      # [n,3]


class OracleScene:
    """Oracle view of one scene + camera + thresholds (all promoted to fp64)."""

    def __init__(self, scene, alpha_min: float | None = None, t_min: float | None = None, params=None):
        """``scene`` supplies camera, SH degree and (float32) parameters.

        ``params`` optionally overrides the parameters with float64 arrays
        (keys means, log_scales, quats, opacity_logits, sh), used by the
        finite-difference pins.  Thresholds default to the float32 values of
        1/255 and 1e-4, promoted to double.
        """
        self.scene = scene
        cam = scene.camera
        self.W, self.H = int(cam.width), int(cam.height)
        self.K = (scene.sh_degree + 1) ** 2
        self.n = scene.n
        am = float(np.float32(1.0 / 255.0) if alpha_min is None else alpha_min)
        tm = float(np.float32(1e-4) if t_min is None else t_min)
        src = dict(means=scene.means, log_scales=scene.log_scales, quats=scene.quats,
                   opacity_logits=scene.opacity_logits, sh=scene.sh)
        if params:
            src.update(params)
        self._keep = [_c(src["means"], np.float64), _c(src["log_scales"], np.float64),
                      _c(src["quats"], np.float64), _c(src["opacity_logits"], np.float64),
                      _c(src["sh"], np.float64),
                      np.array([cam.fx, cam.fy, cam.cx, cam.cy], np.float64),
                      _c(cam.R, np.float64).ravel(), _c(cam.t, np.float64)]
        m, ls, q, lg, sh, intr, R, t = self._keep
        self.h = lib().orc_scene_new(self.n, scene.sh_degree, _ptr(m), _ptr(ls), _ptr(q), _ptr(lg), _ptr(sh),
                                     self.W, self.H, _ptr(intr), _ptr(R), _ptr(t), am, tm)
        self._info = None

    def __del__(self):
        h = getattr(self, "h", None)
        if h:
            lib().orc_scene_free(h)
            self.h = None

    # -- per primitive ---------------------------------------------------
    def prim_info(self) -> PrimInfo:
        if self._info is None:
            n = self.n
            rect = np.zeros((n, 4), np.int32)
            area = np.zeros(n, np.int64)
            state = np.zeros(n, np.int32)
            sigma = np.zeros(n)
            D2c = np.zeros(n)
            W = np.zeros((n, 3, 3))
            og = np.zeros((n, 3))
            lib().orc_prim_info(self.h, _ptr(rect), _ptr(area), _ptr(state), _ptr(sigma), _ptr(D2c), _ptr(W), _ptr(og))
            self._info = PrimInfo(rect, area, state, sigma, D2c, W, og)
        return self._info

    # -- per pixel ---------------------------------------------------------
    def render(self, pixels=None, brute: bool = False):
        """Render the listed pixel indices (y*W+x), or the whole image."""
        if pixels is None:
            m, pix = self.W * self.H, None
        else:
            pix = _c(pixels, np.int64)
            m = pix.shape[0]
        color = np.zeros((m, 3))
        tau_end = np.zeros(m)
        id_end = np.zeros(m, np.int64)
        n_inc = np.zeros(m, np.int64)
        margin = np.zeros(m)
        T_final = np.zeros(m)
        lib().orc_render(self.h, m, _ptr(pix), int(brute), _ptr(color), _ptr(tau_end), _ptr(id_end),
                         _ptr(n_inc), _ptr(margin), _ptr(T_final))
        return dict(color=color, tau_end=tau_end, id_end=id_end, n_included=n_inc, margin=margin,
                    T_final=T_final)

    def bounds_raw(self):
        """Per primitive (Q_xx, Q_x4, Q_yy, Q_y4, Q_44) of the projected dual quadric."""
        out = np.zeros((self.n, 5))
        lib().orc_bounds_raw(self.h, _ptr(out))
        return out

    def ray_prim(self, pixels, prims):
        """tau_max, D^2 there, hit decision, alpha and unit ray direction per (pixel, prim)."""
        pix = _c(pixels, np.int64)
        pr = _c(prims, np.int64)
        m = pix.shape[0]
        tau, D2, alpha = np.zeros(m), np.zeros(m), np.zeros(m)
        hit = np.zeros(m, np.int32)
        d = np.zeros((m, 3))
        lib().orc_ray_prim(self.h, m, _ptr(pix), _ptr(pr), _ptr(tau), _ptr(D2), _ptr(hit), _ptr(alpha), _ptr(d))
        return dict(tau=tau, D2=D2, hit=hit.astype(bool), alpha=alpha, dir=d)

    def camera_origin(self):
        o = np.zeros(3)
        lib().orc_camera_origin(self.h, _ptr(o))
        return o

    def all_hits(self, pixels, brute: bool = False):
        """Every geometric hit (primitive ids, depth order) of each listed pixel, CSR."""
        pix = _c(pixels, np.int64)
        m = pix.shape[0]
        counts = np.zeros(m, np.int64)
        lib().orc_all_hits(self.h, m, _ptr(pix), int(brute), 1, _ptr(counts), None, None)
        off = np.zeros(m + 1, np.int64)
        np.cumsum(counts, out=off[1:])
        prims = np.zeros(int(off[-1]), np.int64)
        lib().orc_all_hits(self.h, m, _ptr(pix), int(brute), 0, None, _ptr(off), _ptr(prims))
        return off, prims

    def records(self, pixels, n_included):
        """Composited hits of each listed pixel in order: prim, (L.rgb, T) in front, tau."""
        pix = _c(pixels, np.int64)
        m = pix.shape[0]
        off = np.zeros(m + 1, np.int64)
        np.cumsum(_c(n_included, np.int64), out=off[1:])
        tot = int(off[-1])
        prim = np.zeros(tot, np.int64)
        LT = np.zeros((tot, 4))
        tau = np.zeros(tot)
        lib().orc_records(self.h, m, _ptr(pix), _ptr(off), _ptr(prim), _ptr(LT), _ptr(tau))
        return off, prim, LT, tau

    def backward(self, dl_dimage, pixels=None, storage="exact"):
        """Raw-parameter gradients of sum <dL/dC, C> over the listed pixels (all if None).

        ``storage`` names how the intermediate buffer keeps (L, T) (Sec. 6
        suggests fp16): the gradient is the plain one with L and T replaced
        by their stored values (``STORAGE_MODELS``)."""
        dl = _c(dl_dimage, np.float64).reshape(self.H, self.W, 3)
        if pixels is None:
            m, pix = 0, None
        else:
            pix = _c(pixels, np.int64)
            m = pix.shape[0]
        n, K = self.n, self.K
        g = dict(means=np.zeros((n, 3)), log_scales=np.zeros((n, 3)), quats=np.zeros((n, 4)),
                 logits=np.zeros(n), sh=np.zeros((n, K, 3)))
        lib().orc_backward_stored(self.h, m, _ptr(pix), _ptr(dl), _ptr(g["means"]), _ptr(g["log_scales"]),
                                  _ptr(g["quats"]), _ptr(g["logits"]), _ptr(g["sh"]), STORAGE_MODELS[storage])
        return g

    def colour_bound(self) -> float:
        """B of the ``fixed16`` storage model: the largest colour any visible
        Gaussian can give in any direction, raised by 2^-16."""
        return float(lib().orc_colour_bound(self.h))

    def lt_index(self, tile: int, prims, pixels):
        """idx(i,t,p) of Eq. 16 by enumeration; -1 outside the rectangle."""
        prims = _c(prims, np.int64)
        pixels = _c(pixels, np.int64)
        idx = np.zeros(prims.shape[0], np.int64)
        lib().orc_lt_index(self.h, int(tile), prims.shape[0], _ptr(prims), _ptr(pixels), _ptr(idx))
        return idx

    def lt_total(self) -> int:
        return int(self.prim_info().area.sum())


def tile_lists(rect, state, width: int, height: int, tile: int):
    """Per-tile primitive lists (Sec. 4.3, reverse tile mapping), ascending id.

    Plain enumeration: every active primitive contributes its index to every
    tile that its pixel rectangle meets.  Returns (offsets[n_tiles+1], prims).
    """
    ntx = (width + tile - 1) // tile
    nty = (height + tile - 1) // tile
    act = np.nonzero(state == STATE_ACTIVE)[0]
    r = rect[act].astype(np.int64)
    tx0, ty0, tx1, ty1 = r[:, 0] // tile, r[:, 1] // tile, r[:, 2] // tile, r[:, 3] // tile
    nx, ny = tx1 - tx0 + 1, ty1 - ty0 + 1
    cnt = nx * ny
    total = int(cnt.sum())
    owner = np.repeat(np.arange(act.shape[0]), cnt)
    start = np.zeros(act.shape[0] + 1, np.int64)
    np.cumsum(cnt, out=start[1:])
    k = np.arange(total, dtype=np.int64) - start[owner]
    tx = tx0[owner] + k % nx[owner]
    ty = ty0[owner] + k // nx[owner]
    key = ty * ntx + tx
    prim = act[owner]
    order = np.lexsort((prim, key))
    key, prim = key[order], prim[order]
    off = np.zeros(ntx * nty + 1, np.int64)
    np.cumsum(np.bincount(key, minlength=ntx * nty), out=off[1:])
    return off, prim
