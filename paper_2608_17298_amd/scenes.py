"""Seeded synthetic scenes shaped like the paper's training workloads.

This module only draws random numbers and lays them out; it contains none of
the renderer's arithmetic, so both the HIP path and the CPU oracle can consume
its output.  Every array is float32 and C-contiguous.

Scene parameters follow the Gaussian representation of Sec. 3.1 (mean,
rotation quaternion, per-axis scale, opacity, spherical-harmonic radiance).
The camera is a pinhole with OpenCV axes (x right, y down, z forward) and the
world-to-camera map x_c = R x_w + t.

The five named workloads stand in for the paper's real-scene benchmarks
(Sec. 5.1), which are not available here:

====  ======  ===  ===========  ====  ==================================
name   N      SH   W x H        tile  distribution
====  ======  ===  ===========  ====  ==================================
tiny   4096    0   128 x 128    16    means U[-1,1]^3, ls N(-3.5,.3)
small  100k    3   640 x 480     8    64 clusters (sd .3) in r<=3 ball
1m     1M      3   1237 x 822    8    70% ball r=2, 30% shell r=20
4m     4M      3   1600 x 1060   8    60% ball r=2, 40% shell r=20
stress 500k    3   1237 x 822    8    U[-2,2]^3, large low-opacity
====  ======  ===  ===========  ====  ==================================

The draw order is fixed (means, log-scales, quaternions, opacity logits, SH,
mean perturbation, upstream gradient) so that a scene is a pure function of
its name and seed.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 260817298

ALPHA_MIN = float(np.float32(1.0 / 255.0))
T_MIN = float(np.float32(1e-4))


@dataclass
class Camera:
    width: int
    height: int
    fx: float
    fy: float
    cx: float
    cy: float
    R: np.ndarray  # [3,3] float32, world -> camera rotation, row-major
    t: np.ndarray  # [3] float32

    def as_tuple(self):
        return (self.width, self.height, self.fx, self.fy, self.cx, self.cy,
                self.R.astype(np.float32).ravel(), self.t.astype(np.float32))


@dataclass
class Scene:
    name: str
    tile: int
    sh_degree: int
    camera: Camera
    means: np.ndarray          # [N,3]
    log_scales: np.ndarray     # [N,3]
    quats: np.ndarray          # [N,4]  (w, x, y, z)
    opacity_logits: np.ndarray # [N]
    sh: np.ndarray             # [N,K,3]
    means_perturbed: np.ndarray | None = None   # [N,3] target copy for an L1 upstream gradient
    dl_dimage: np.ndarray | None = None         # [H,W,3] drawn upstream gradient
    extra: dict = field(default_factory=dict)

    @property
    def n(self) -> int:
        return int(self.means.shape[0])

    @property
    def sh_k(self) -> int:
        return (self.sh_degree + 1) ** 2


WORKLOADS = {
    # name: (N, sh_degree, W, H, tile)
    "tiny": (4096, 0, 128, 128, 16),
    "small": (100_000, 3, 640, 480, 8),
    "1m": (1_000_000, 3, 1237, 822, 8),
    "4m": (4_000_000, 3, 1600, 1060, 8),
    "stress": (500_000, 3, 1237, 822, 8),
}
WORKLOAD_INDEX = {"tiny": 1, "small": 2, "1m": 3, "4m": 4, "stress": 5}


def pinhole_camera(width: int, height: int, fov_y_deg: float = 60.0,
                   distance: float = 4.0) -> Camera:
    """Camera at (0, 0, -distance) looking along +z at the origin (R = I).

    Focal length from the vertical field of view: f = (H/2) / tan(fov/2),
    square pixels, principal point at the image centre.
    """
    f = (height / 2.0) / math.tan(math.radians(fov_y_deg) / 2.0)
    return Camera(width=width, height=height, fx=float(np.float32(f)),
                  fy=float(np.float32(f)), cx=float(np.float32(width / 2.0)),
                  cy=float(np.float32(height / 2.0)),
                  R=np.eye(3, dtype=np.float32),
                  t=np.array([0.0, 0.0, distance], dtype=np.float32))


def orbit_camera(width: int, height: int, azimuth_deg: float, fov_y_deg: float = 60.0,
                 distance: float = 4.0) -> Camera:
    """The pinhole camera above, rotated about the world y axis through the
    origin by azimuth_deg: centre Ry(az) (0, 0, -distance), still looking at
    the origin (R = Ry(az)^T, t = (0, 0, distance))."""
    base = pinhole_camera(width, height, fov_y_deg, distance)
    a = math.radians(azimuth_deg)
    ry = np.array([[math.cos(a), 0.0, math.sin(a)], [0.0, 1.0, 0.0], [-math.sin(a), 0.0, math.cos(a)]])
    base.R = ry.T.astype(np.float32)
    return base


def _uniform_ball(rng, n, radius):
    v = rng.standard_normal((n, 3))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    r = radius * rng.random(n) ** (1.0 / 3.0)
    return v * r[:, None]


def _uniform_sphere(rng, n, radius):
    v = rng.standard_normal((n, 3))
    v /= np.linalg.norm(v, axis=1, keepdims=True)
    return v * radius


def _clusters(rng, n, n_clusters=64, radius=3.0, sd=0.3):
    centres = _uniform_ball(rng, n_clusters, radius)
    out = np.empty((n, 3))
    filled = 0
    while filled < n:
        m = n - filled
        idx = rng.integers(0, n_clusters, m)
        pts = centres[idx] + sd * rng.standard_normal((m, 3))
        keep = pts[np.linalg.norm(pts, axis=1) <= radius]
        out[filled:filled + len(keep)] = keep
        filled += len(keep)
    return out


def _fg_shell(rng, n, frac_fg):
    n_fg = int(round(frac_fg * n))
    fg = _uniform_ball(rng, n_fg, 2.0)
    bg = _uniform_sphere(rng, n - n_fg, 20.0)
    return np.concatenate([fg, bg], axis=0)


def _sh_coeffs(rng, n, degree, high_sd=0.05):
    k = (degree + 1) ** 2
    sh = np.zeros((n, k, 3))
    # DC: the colour map is c = 0.5 + Y00 * k00 + ..., Y00 = 1 / (2 sqrt(pi)),
    # so k00 = (u - 0.5) * 2 sqrt(pi) makes the DC colour term u ~ U(0,1).
    u = rng.random((n, 3))
    sh[:, 0, :] = (u - 0.5) * 2.0 * math.sqrt(math.pi)
    if k > 1:
        sh[:, 1:, :] = high_sd * rng.standard_normal((n, k - 1, 3))
    return sh


def make_scene(name: str, n: int | None = None, width: int | None = None,
               height: int | None = None, seed: int | None = None,
               upstream: str | None = None) -> Scene:
    """Build one of the named workloads.

    ``n``, ``width`` and ``height`` override the workload's size (same
    distributions) so tests can use a reduced copy that still spans several
    tiles with a ragged edge.  ``upstream`` selects the drawn upstream
    gradient: "normal" (N(0,1), the tiny workload's) or "sign" (independent
    +-1 values, the distribution of an L1 loss gradient).  The L1 gradient
    against a perturbed render itself needs a renderer and is formed by the
    caller from ``means_perturbed``.
    """
    N, deg, W, H, tile = WORKLOADS[name]
    N = N if n is None else int(n)
    W = W if width is None else int(width)
    H = H if height is None else int(height)
    seed = SEED_BASE + WORKLOAD_INDEX[name] if seed is None else seed
    rng = np.random.default_rng(seed)

    if name == "tiny":
        means = rng.uniform(-1.0, 1.0, (N, 3))
        ls = rng.normal(-3.5, 0.3, (N, 3))
    elif name == "small":
        means = _clusters(rng, N)
        ls = rng.normal(-4.0, 0.5, (N, 3))
    elif name == "1m":
        means = _fg_shell(rng, N, 0.7)
        ls = np.minimum(rng.normal(-4.5, 0.7, (N, 3)), -1.0)
    elif name == "4m":
        means = _fg_shell(rng, N, 0.6)
        ls = np.minimum(rng.normal(-5.0, 0.7, (N, 3)), -1.0)
    elif name == "stress":
        means = rng.uniform(-2.0, 2.0, (N, 3))
        ls = rng.normal(-2.0, 0.3, (N, 3))
    else:
        raise KeyError(name)

    q = rng.standard_normal((N, 4))
    q /= np.linalg.norm(q, axis=1, keepdims=True)

    logit_mu, logit_sd = {"tiny": (0.0, 1.0), "small": (0.0, 1.5), "1m": (-0.5, 2.0),
                          "4m": (-0.5, 2.0), "stress": (-3.0, 0.5)}[name]
    logits = rng.normal(logit_mu, logit_sd, N)

    sh = _sh_coeffs(rng, N, deg)

    perturbed = None
    if name != "tiny":
        perturbed = means + rng.normal(0.0, 0.01, (N, 3))

    if upstream is None:
        upstream = "normal" if name == "tiny" else "sign"
    if upstream == "normal":
        dl = rng.standard_normal((H, W, 3))
    elif upstream == "sign":
        dl = np.where(rng.random((H, W, 3)) < 0.5, -1.0, 1.0)
    else:
        raise ValueError(upstream)

    f32 = lambda a: np.ascontiguousarray(a, dtype=np.float32)
    return Scene(name=name, tile=tile, sh_degree=deg, camera=pinhole_camera(W, H),
                 means=f32(means), log_scales=f32(ls), quats=f32(q),
                 opacity_logits=f32(logits), sh=f32(sh),
                 means_perturbed=None if perturbed is None else f32(perturbed),
                 dl_dimage=f32(dl))


def custom_scene(means, log_scales, quats, opacity_logits, sh, camera: Camera,
                 tile: int = 8, dl_dimage=None, name: str = "custom") -> Scene:
    """Wrap hand-built arrays (used by the small analytic test scenes)."""
    f32 = lambda a: np.ascontiguousarray(np.asarray(a, dtype=np.float64), dtype=np.float32)
    sh = f32(sh)
    if sh.ndim != 3 or sh.shape[2] != 3:
        raise ValueError("sh must be [N, K, 3]")
    k = sh.shape[1]
    deg = int(round(math.sqrt(k))) - 1
    assert (deg + 1) ** 2 == k, "SH coefficient count must be a square"
    if dl_dimage is None:
        dl_dimage = np.ones((camera.height, camera.width, 3), np.float32)
    return Scene(name=name, tile=tile, sh_degree=deg, camera=camera,
                 means=f32(means).reshape(-1, 3), log_scales=f32(log_scales).reshape(-1, 3),
                 quats=f32(quats).reshape(-1, 4), opacity_logits=f32(opacity_logits).reshape(-1),
                 sh=sh, dl_dimage=f32(dl_dimage))
