"""Thin Python binding of the GART C ABI (``include/gart.h``).

Argument marshalling only: every step runs in the HIP kernels of
``_build/libgart.so``.  PyTorch provides device memory and the stream.  There
is no fallback: if the library is missing or no GPU is present, calls raise.

The four entry points keep their C names (``gart_bounds``,
``gart_build_tile_map``, ``gart_forward``, ``gart_backward``); ``Frame``
allocates the per-frame buffers the C ABI expects, growing the
intermediate buffer and pair list by a slack factor (the paper's lambda_s,
Sec. 4.2, Eq. 15) when ``gart_bounds`` reports a capacity shortfall.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass

import numpy as np
import torch

from . import build as _build

LIB_PATH = _build.LIB_PATH

GART_OK = 0
GART_ERR_INVALID_ARG = -1
GART_ERR_CAPACITY = -2
GART_ERR_HIP = -3
GART_ERR_UNSUPPORTED = -4

GATHER = 0
GATHER_ATOMIC = 1
SCATTER = 2
HYBRID = 3
GATHER_WAVE = 4
MODES = {"gather": GATHER, "gather_atomic": GATHER_ATOMIC, "scatter": SCATTER, "hybrid": HYBRID,
         "gather_wave": GATHER_WAVE}
LT_FULL, LT_T_ONLY, LT_HALF, LT_T_HALF, LT_FIXED16, LT_T_LOG16 = 0, 1, 2, 3, 4, 5
LT_PRECISION_FULL, LT_PRECISION_HALF, LT_PRECISION_FIXED16 = 0, 1, 2
PRECISIONS = {"full": LT_PRECISION_FULL, "half": LT_PRECISION_HALF, "fixed16": LT_PRECISION_FIXED16}

CNT_FWD_HITS, CNT_FWD_TESTS, CNT_FWD_RESCANS = 0, 1, 2
CNT_BWD_HITS, CNT_BWD_TESTS, CNT_BWD_ATOMICS, CNT_BWD_PAIRS, CNT_BWD_ACTIVE = 3, 4, 5, 6, 7
CNT_FWD_DROPS = 8
CNT_BWD_STEPS = 9
CNT_BWD_WAVE_UNITS = 10
NUM_COUNTERS = 16
EV_SORT, EV_FWD, EV_BWD, EV_REDUCE = 0, 2, 4, 6  # begin index; end = begin + 1
NUM_EVENTS = 8

_P = ctypes.c_void_p


class gart_camera(ctypes.Structure):
    _fields_ = [("width", ctypes.c_int32), ("height", ctypes.c_int32), ("fx", ctypes.c_float),
                ("fy", ctypes.c_float), ("cx", ctypes.c_float), ("cy", ctypes.c_float),
                ("R", ctypes.c_float * 9), ("t", ctypes.c_float * 3)]


class gart_gaussians(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int64), ("sh_degree", ctypes.c_int32), ("means", _P), ("log_scales", _P),
                ("quats", _P), ("opacity_logits", _P), ("sh", _P)]


class gart_settings(ctypes.Structure):
    _fields_ = [("alpha_min", ctypes.c_float), ("t_min", ctypes.c_float), ("tile", ctypes.c_int32),
                ("backward_mode", ctypes.c_int32), ("lt_precision", ctypes.c_int32)]


class gart_frame(ctypes.Structure):
    _fields_ = [("rect", _P), ("lt_offset", _P), ("prim_geom", _P), ("tile_count", _P),
                ("pair_offset", _P), ("pair_capacity", ctypes.c_int64), ("pair_tile", _P), ("pair_prim", _P),
                ("pair_key", _P), ("tile_range", _P), ("lt_capacity", ctypes.c_int64), ("lt", _P), ("pixel_state", _P), ("hit_list", _P),
                ("hit_list_capacity", ctypes.c_int64),
                ("scratch", _P), ("scratch_bytes", ctypes.c_size_t), ("counters", _P),
                ("events", _P * 8), ("n", ctypes.c_int64), ("sh_degree", ctypes.c_int32), ("tiles_x", ctypes.c_int32),
                ("tiles_y", ctypes.c_int32), ("lt_entries", ctypes.c_int64), ("pair_count", ctypes.c_int64),
                ("color_step", ctypes.c_double), ("stage", ctypes.c_int32),
                ("lt_format", ctypes.c_int32), ("width", ctypes.c_int32), ("height", ctypes.c_int32),
                ("tile", ctypes.c_int32), ("reserved", ctypes.c_int32)]


class GartError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__(f"{where}: {_status_name(status)}: {detail}")


class GartCapacityError(GartError):
    def __init__(self, where, detail, lt_entries, pair_count):
        super().__init__(GART_ERR_CAPACITY, where, detail)
        self.lt_entries = lt_entries
        self.pair_count = pair_count


_lib = None


def lib():
    """Load the built library (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"GART HIP library not built: {LIB_PATH} (run __graft_entry__.build())")
        L = ctypes.CDLL(LIB_PATH)
        L.gart_scratch_bytes.restype = ctypes.c_size_t
        L.gart_scratch_bytes.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int64, _P, _P]
        L.gart_lt_entry_bytes.restype = ctypes.c_int32
        L.gart_lt_entry_bytes.argtypes = [_P]
        L.gart_hit_list_slots.restype = ctypes.c_int64
        L.gart_hit_list_slots.argtypes = [ctypes.c_int64, _P, _P]
        L.gart_bounds.restype = ctypes.c_int
        L.gart_bounds.argtypes = [_P, _P, _P, _P, _P, _P, _P]
        L.gart_bounds_noalloc.restype = ctypes.c_int
        L.gart_bounds_noalloc.argtypes = [_P, _P, _P, _P, _P, _P, _P]
        L.gart_build_tile_map.restype = ctypes.c_int
        L.gart_build_tile_map.argtypes = [_P, _P, _P, _P]
        L.gart_forward.restype = ctypes.c_int
        L.gart_forward.argtypes = [_P, _P, _P, _P, _P, _P]
        L.gart_backward.restype = ctypes.c_int
        L.gart_backward.argtypes = [_P, _P, _P, _P, _P, _P, _P, _P, _P, _P, _P]
        L.gart_frame_status.restype = ctypes.c_int
        L.gart_frame_status.argtypes = [_P, _P, _P]
        L.gart_status_string.restype = ctypes.c_char_p
        L.gart_status_string.argtypes = [ctypes.c_int]
        L.gart_last_error.restype = ctypes.c_char_p
        L.gart_last_error.argtypes = []
        L.gart_l1_partials.restype = ctypes.c_int64
        L.gart_l1_partials.argtypes = [ctypes.c_int64]
        L.gart_l1_loss_grad.restype = ctypes.c_int
        L.gart_l1_loss_grad.argtypes = [_P, _P, ctypes.c_int64, _P, _P, _P, _P]
        L.gart_adam_step.restype = ctypes.c_int
        L.gart_adam_step.argtypes = [_P, _P, _P, _P, ctypes.c_int64, _P, ctypes.c_int64, _P]
        _lib = L
    return _lib


def _status_name(s: int) -> str:
    try:
        return lib().gart_status_string(s).decode()
    except Exception:  # library not loadable
        return str(s)


def _check(status: int, where: str):
    if status != GART_OK:
        raise GartError(status, where, lib().gart_last_error().decode())


def _ptr(t: torch.Tensor | None):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError("GART takes device tensors only")
    if not t.is_contiguous():
        raise ValueError("GART takes contiguous tensors only")
    return ctypes.c_void_p(t.data_ptr())


def _stream(stream):
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream)


# ---------------------------------------------------------------------------
# Marshalling helpers
# ---------------------------------------------------------------------------
def make_camera(cam) -> gart_camera:
    """From any object with width, height, fx, fy, cx, cy, R[3,3], t[3]."""
    c = gart_camera()
    c.width, c.height = int(cam.width), int(cam.height)
    c.fx, c.fy, c.cx, c.cy = float(cam.fx), float(cam.fy), float(cam.cx), float(cam.cy)
    R = [float(v) for v in np.asarray(cam.R, dtype=np.float32).ravel()]
    t = [float(v) for v in np.asarray(cam.t, dtype=np.float32).ravel()]
    c.R = (ctypes.c_float * 9)(*R)
    c.t = (ctypes.c_float * 3)(*t)
    return c


def make_settings(tile=8, backward_mode=GATHER, alpha_min=None, t_min=None, lt_precision=LT_PRECISION_FULL) -> gart_settings:
    s = gart_settings()
    s.alpha_min = float(1.0 / 255.0) if alpha_min is None else float(alpha_min)
    s.t_min = 1e-4 if t_min is None else float(t_min)
    s.tile = int(tile)
    s.backward_mode = MODES[backward_mode] if isinstance(backward_mode, str) else int(backward_mode)
    s.lt_precision = PRECISIONS[lt_precision] if isinstance(lt_precision, str) else int(lt_precision)
    return s


def gart_lt_entry_bytes(settings: gart_settings) -> int:
    """Bytes per intermediate-buffer entry that gart_forward writes for these settings."""
    n = int(lib().gart_lt_entry_bytes(ctypes.byref(settings)))
    if n <= 0:
        raise GartError(GART_ERR_INVALID_ARG, "gart_lt_entry_bytes", lib().gart_last_error().decode())
    return n


@dataclass
class Gaussians:
    """Device float32 parameter tensors (Sec. 3.1)."""
    means: torch.Tensor
    log_scales: torch.Tensor
    quats: torch.Tensor
    opacity_logits: torch.Tensor
    sh: torch.Tensor
    sh_degree: int

    @classmethod
    def from_scene(cls, scene, device="cuda"):
        f = lambda a: torch.from_numpy(a).to(device=device, dtype=torch.float32).contiguous()
        return cls(f(scene.means), f(scene.log_scales), f(scene.quats), f(scene.opacity_logits), f(scene.sh),
                   int(scene.sh_degree))

    @property
    def n(self):
        return int(self.means.shape[0])

    def c_struct(self) -> gart_gaussians:
        for t in (self.means, self.log_scales, self.quats, self.opacity_logits, self.sh):
            if t.dtype != torch.float32:
                raise ValueError("Gaussian parameters must be float32")
        g = gart_gaussians()
        g.n = self.n
        g.sh_degree = self.sh_degree
        g.means, g.log_scales, g.quats = _ptr(self.means), _ptr(self.log_scales), _ptr(self.quats)
        g.opacity_logits, g.sh = _ptr(self.opacity_logits), _ptr(self.sh)
        return g


def gart_hit_list_slots(pair_count, camera: gart_camera, settings: gart_settings) -> int:
    r = int(lib().gart_hit_list_slots(int(pair_count), ctypes.byref(camera), ctypes.byref(settings)))
    if r < 0:
        raise GartError(GART_ERR_INVALID_ARG, "gart_hit_list_slots", lib().gart_last_error().decode())
    return r


def gart_scratch_bytes(n, sh_degree, pair_capacity, camera: gart_camera, settings: gart_settings) -> int:
    return int(lib().gart_scratch_bytes(int(n), int(sh_degree), int(pair_capacity), ctypes.byref(camera),
                                        ctypes.byref(settings)))


class Frame:
    """Owns the device buffers of one gart_frame (all torch tensors)."""

    def __init__(self, n: int, sh_degree: int, camera: gart_camera, settings: gart_settings,
                 lt_capacity: int = 0, pair_capacity: int = 0, device="cuda", counters: bool = False):
        self.device = device
        self.n, self.sh_degree = int(n), int(sh_degree)
        self.camera, self.settings = camera, settings
        ts = settings.tile
        self.tiles_x = (camera.width + ts - 1) // ts
        self.tiles_y = (camera.height + ts - 1) // ts
        dev = dict(device=device)
        n1 = max(self.n, 1)
        self.rect = torch.empty((n1, 4), dtype=torch.int32, **dev)
        self.lt_offset = torch.empty(n1 + 1, dtype=torch.int64, **dev)
        self.prim_geom = torch.empty((n1, 16), dtype=torch.float64, **dev)
        self.tile_count = torch.empty(n1, dtype=torch.int32, **dev)
        self.pair_offset = torch.empty(n1 + 1, dtype=torch.int64, **dev)
        self.tile_range = torch.empty(self.tiles_x * self.tiles_y + 1, dtype=torch.int64, **dev)
        # gart_pixel_state, 32 bytes per pixel
        self.pixel_state = torch.empty((camera.height * camera.width, 4), dtype=torch.int64, **dev)
        self.counters = torch.zeros(NUM_COUNTERS, dtype=torch.int64, **dev) if counters else None
        self.c = gart_frame()
        self.events = [None] * NUM_EVENTS
        self.lt = self.pair_tile = self.pair_prim = self.pair_key = self.scratch = None
        self._alloc_lt(lt_capacity)
        self._alloc_pairs(pair_capacity)

    def _alloc_lt(self, cap):
        # entries of gart_lt_entry_bytes(settings) bytes, held as int16 words
        # (16 bytes: fixed-point L and float T; 4: float T; 8: fp16 L and T;
        # 2: fp16 T)
        words = gart_lt_entry_bytes(self.settings) // 2
        self.lt = torch.empty((max(int(cap), 1), words), dtype=torch.int16, device=self.device)
        self.lt_capacity = int(cap)

    def _alloc_pairs(self, cap):
        cap = int(cap)
        self.pair_tile = torch.empty(max(cap, 1), dtype=torch.int32, device=self.device)
        self.pair_prim = torch.empty(max(cap, 1), dtype=torch.int32, device=self.device)
        self.pair_key = torch.empty(max(cap, 1), dtype=torch.float32, device=self.device)
        # composited-hit lists (see gart_frame.hit_list)
        self.hit_list = torch.empty(max(gart_hit_list_slots(cap, self.camera, self.settings), 1), dtype=torch.int32,
                                    device=self.device)
        self.pair_capacity = cap
        # sized for every backward mode, so one frame serves all of them
        nbytes = 0
        for mode in (GATHER, GATHER_ATOMIC, SCATTER, HYBRID, GATHER_WAVE):
            st = gart_settings(self.settings.alpha_min, self.settings.t_min, self.settings.tile, mode,
                               self.settings.lt_precision)
            nbytes = max(nbytes, gart_scratch_bytes(self.n, self.sh_degree, cap, self.camera, st))
        self.scratch = torch.empty(nbytes, dtype=torch.uint8, device=self.device)

    def grow(self, lt_entries: int, pair_count: int, slack: float = 1.0):
        if lt_entries > self.lt_capacity:
            self.lt = None
            self._alloc_lt(int(lt_entries * slack) + 1)
        if pair_count > self.pair_capacity:
            self.pair_tile = self.pair_prim = self.pair_key = self.hit_list = self.scratch = None
            self._alloc_pairs(int(pair_count * slack) + 1)

    def c_struct(self) -> gart_frame:
        f = self.c
        f.rect, f.lt_offset, f.prim_geom = _ptr(self.rect), _ptr(self.lt_offset), _ptr(self.prim_geom)
        f.tile_count, f.pair_offset = _ptr(self.tile_count), _ptr(self.pair_offset)
        f.pair_capacity = self.pair_capacity
        f.pair_tile, f.pair_prim, f.tile_range = _ptr(self.pair_tile), _ptr(self.pair_prim), _ptr(self.tile_range)
        f.pair_key = _ptr(self.pair_key)
        f.lt_capacity = self.lt_capacity
        f.lt, f.pixel_state, f.hit_list = _ptr(self.lt), _ptr(self.pixel_state), _ptr(self.hit_list)
        f.hit_list_capacity = 0 if self.hit_list is None else self.hit_list.numel()
        f.scratch, f.scratch_bytes = _ptr(self.scratch), self.scratch.numel()
        f.counters = _ptr(self.counters)
        for k in range(NUM_EVENTS):
            f.events[k] = self.events[k]
        return f

    def set_events(self, handles):
        """Raw hipEvent_t handles (ints) the library records around its
        kernels (see GART_EV_* in gart.h); None entries are not recorded."""
        self.events = [None if h is None else int(h) for h in handles] + [None] * (NUM_EVENTS - len(handles))

    # host-side totals filled by the library
    @property
    def lt_entries(self):
        return int(self.c.lt_entries)

    @property
    def color_step(self) -> float:
        """Colour per fixed-point unit of the (L,T) entries and pixel colours."""
        return float(self.c.color_step)

    def lt_entries_host(self, index: torch.Tensor):
        """(L [m,3] float64, T [m] float32) of the listed (L,T) entries, on
        the host, decoded from the frame's lt_format; L is None for a T-only
        buffer (hybrid backward)."""
        raw = np.ascontiguousarray(self.lt[index].cpu().numpy())
        fmt = int(self.c.lt_format)
        if fmt == LT_T_ONLY:
            return None, raw.view(np.float32)[:, 0].copy()
        if fmt == LT_T_HALF:
            return None, raw.view(np.float16)[:, 0].astype(np.float32)
        if fmt == LT_HALF:
            h = raw.view(np.float16)
            return h[:, :3].astype(np.float64), h[:, 3].astype(np.float32)
        if fmt in (LT_FIXED16, LT_T_LOG16):
            u = raw.view(np.uint16).astype(np.float64)
            T = np.exp2(-u[:, -1] / 4096.0).astype(np.float32)
            return (None if fmt == LT_T_LOG16 else u[:, :3] * self.color_step * 65536.0), T
        w = raw.view(np.uint32)
        return w[:, :3].astype(np.float64) * self.color_step, w[:, 3].copy().view(np.float32)

    def pixel_state_host(self) -> dict:
        """gart_pixel_state fields of every pixel, on the host."""
        ps = self.pixel_state.cpu().numpy()
        w = ps.view(np.uint32)
        return dict(tau_end=ps[:, 0].copy().view(np.float64), id_end=w[:, 2].copy(), n_hits=w[:, 3].copy(),
                    color=w[:, 4:7].astype(np.float64) * self.color_step, t_final=w[:, 7].copy().view(np.float32))

    @property
    def pair_count(self):
        return int(self.c.pair_count)


# ---------------------------------------------------------------------------
# The four entry points (same names as the C ABI)
# ---------------------------------------------------------------------------
def gart_bounds(g: Gaussians, camera: gart_camera, settings: gart_settings, frame: Frame, stream=None):
    """Pre-processing (Sec. 4.2).  Returns (lt_entries, pair_count); raises
    GartCapacityError if the frame's buffers are too small."""
    gs = g.c_struct()
    fs = frame.c_struct()
    lt = ctypes.c_int64(0)
    pc = ctypes.c_int64(0)
    st = lib().gart_bounds(ctypes.byref(gs), ctypes.byref(camera), ctypes.byref(settings), ctypes.byref(fs),
                           ctypes.byref(lt), ctypes.byref(pc), _stream(stream))
    if st == GART_ERR_CAPACITY:
        raise GartCapacityError("gart_bounds", lib().gart_last_error().decode(), lt.value, pc.value)
    _check(st, "gart_bounds")
    return lt.value, pc.value


BOUNDS_NOALLOC_MAX_N = 1 << 25


def gart_bounds_noalloc(g: Gaussians, camera: gart_camera, settings: gart_settings, frame: Frame, stream=None):
    """gart_bounds with the library's static scratch instead of the frame's
    (for callers that cannot allocate).  Returns (lt_entries, pair_count);
    raises GartCapacityError if the frame's buffers are too small."""
    gs = g.c_struct()
    fs = frame.c_struct()
    lt = ctypes.c_int64(0)
    pc = ctypes.c_int64(0)
    st = lib().gart_bounds_noalloc(ctypes.byref(gs), ctypes.byref(camera), ctypes.byref(settings),
                                   ctypes.byref(fs), ctypes.byref(lt), ctypes.byref(pc), _stream(stream))
    if st == GART_ERR_CAPACITY:
        raise GartCapacityError("gart_bounds_noalloc", lib().gart_last_error().decode(), lt.value, pc.value)
    _check(st, "gart_bounds_noalloc")
    return lt.value, pc.value


FRAME_FORWARD_INCOMPLETE = 1
FRAME_HIT_LIST_FULL = 2


def gart_frame_status(frame: Frame, stream=None) -> int:
    """The frame status word (GART_FRAME_* bits) left by the last gart_forward;
    synchronises the stream."""
    fs = frame.c_struct()
    v = ctypes.c_uint32(0)
    _check(lib().gart_frame_status(ctypes.byref(fs), ctypes.byref(v), _stream(stream)), "gart_frame_status")
    return int(v.value)


def gart_build_tile_map(camera: gart_camera, settings: gart_settings, frame: Frame, stream=None):
    """Tile-primitive mapping (Sec. 4.3)."""
    fs = frame.c_struct()
    _check(lib().gart_build_tile_map(ctypes.byref(camera), ctypes.byref(settings), ctypes.byref(fs),
                                     _stream(stream)), "gart_build_tile_map")


def gart_forward(g: Gaussians, camera: gart_camera, settings: gart_settings, frame: Frame, image: torch.Tensor,
                 stream=None):
    """Forward trace (Sec. 3.2-3.3, 4.3); image is [H,W,3] float32."""
    if image.dtype != torch.float32 or image.shape != (camera.height, camera.width, 3):
        raise ValueError("image must be float32 [H,W,3]")
    if frame.lt.shape[1] * 2 < gart_lt_entry_bytes(settings):
        # lt_capacity counts entries of the size this call writes
        raise ValueError(f"frame's intermediate buffer has {frame.lt.shape[1] * 2}-byte entries; these settings "
                         f"write {gart_lt_entry_bytes(settings)}-byte entries (allocate the frame for them)")
    gs = g.c_struct()
    fs = frame.c_struct()
    _check(lib().gart_forward(ctypes.byref(gs), ctypes.byref(camera), ctypes.byref(settings), ctypes.byref(fs),
                              _ptr(image), _stream(stream)), "gart_forward")


def gart_backward(g: Gaussians, camera: gart_camera, settings: gart_settings, frame: Frame,
                  dl_dimage: torch.Tensor, grads: dict, stream=None):
    """Backward (Sec. 4.4); grads holds float32 device tensors means, log_scales,
    quats, logits, sh shaped like the parameters (overwritten)."""
    if dl_dimage.dtype != torch.float32 or dl_dimage.shape != (camera.height, camera.width, 3):
        raise ValueError("dl_dimage must be float32 [H,W,3]")
    gs = g.c_struct()
    fs = frame.c_struct()
    _check(lib().gart_backward(ctypes.byref(gs), ctypes.byref(camera), ctypes.byref(settings), ctypes.byref(fs),
                               _ptr(dl_dimage), _ptr(grads["means"]), _ptr(grads["log_scales"]),
                               _ptr(grads["quats"]), _ptr(grads["logits"]), _ptr(grads["sh"]),
                               _stream(stream)), "gart_backward")


class gart_adam(ctypes.Structure):
    _fields_ = [("lr", ctypes.c_float), ("beta1", ctypes.c_float), ("beta2", ctypes.c_float), ("eps", ctypes.c_float)]


def gart_l1_partials(n: int) -> int:
    return int(lib().gart_l1_partials(int(n)))


def gart_l1_loss_grad(image: torch.Tensor, target: torch.Tensor, dl_dimage: torch.Tensor,
                      loss: torch.Tensor | None = None, partial: torch.Tensor | None = None, stream=None):
    """dl_dimage = sign(image - target); loss (device fp64 [1]) = sum |image - target|."""
    for t in (image, target, dl_dimage):
        if t.dtype != torch.float32 or t.shape != image.shape:
            raise ValueError("image, target and dl_dimage must be float32 of one shape")
    if loss is not None and (loss.dtype != torch.float64 or partial is None or partial.dtype != torch.float64
                             or partial.numel() < gart_l1_partials(image.numel())):
        raise ValueError("loss needs a float64 scalar and float64 partials of gart_l1_partials(n)")
    _check(lib().gart_l1_loss_grad(_ptr(image), _ptr(target), image.numel(), _ptr(dl_dimage), _ptr(loss),
                                   _ptr(partial), _stream(stream)), "gart_l1_loss_grad")


def gart_adam_step(param: torch.Tensor, grad: torch.Tensor, m: torch.Tensor, v: torch.Tensor, h: gart_adam,
                   step: int, stream=None):
    """One Adam step in place on a float32 parameter tensor (m and v are its moment buffers)."""
    for t in (param, grad, m, v):
        if t.dtype != torch.float32 or t.shape != param.shape:
            raise ValueError("param, grad, m and v must be float32 of one shape")
    _check(lib().gart_adam_step(_ptr(param), _ptr(grad), _ptr(m), _ptr(v), param.numel(), ctypes.byref(h),
                                int(step), _stream(stream)), "gart_adam_step")


def empty_grads(g: Gaussians) -> dict:
    return dict(means=torch.empty_like(g.means), log_scales=torch.empty_like(g.log_scales),
                quats=torch.empty_like(g.quats), logits=torch.empty_like(g.opacity_logits),
                sh=torch.empty_like(g.sh))


def prepare(g: Gaussians, camera: gart_camera, settings: gart_settings, frame: Frame | None = None,
            slack: float = 1.1, counters: bool = False, stream=None) -> Frame:
    """gart_bounds with buffer growth, then gart_build_tile_map."""
    if frame is None:
        frame = Frame(g.n, g.sh_degree, camera, settings, counters=counters)
    try:
        gart_bounds(g, camera, settings, frame, stream)
    except GartCapacityError as e:
        frame.grow(e.lt_entries, e.pair_count, slack)
        gart_bounds(g, camera, settings, frame, stream)
    gart_build_tile_map(camera, settings, frame, stream)
    return frame
