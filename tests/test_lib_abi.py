"""CPU checks of the built C-ABI library: it loads without a GPU, exports
every function declared in include/gart.h, and rejects invalid arguments
before touching the device."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "gart.h")).read()
    src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
    return sorted(set(re.findall(r"\b(gart_[a-z_]+)\s*\(", src)))


@pytest.fixture(scope="module")
def lib():
    from paper_2608_17298_amd import gart
    return gart.lib()


def test_exports_every_declared_symbol(lib):
    names = _declared()
    assert {"gart_bounds", "gart_build_tile_map", "gart_forward", "gart_backward"} <= set(names)
    for n in names:
        assert hasattr(lib, n), n


def test_status_strings(lib):
    from paper_2608_17298_amd import gart
    for code, name in [(0, "GART_OK"), (-1, "GART_ERR_INVALID_ARG"), (-2, "GART_ERR_CAPACITY"),
                       (-3, "GART_ERR_HIP"), (-4, "GART_ERR_UNSUPPORTED")]:
        assert gart.lib().gart_status_string(code).decode() == name


def _structs(tile=8, mode=0, n=0, deg=0, w=16, h=16):
    from paper_2608_17298_amd import gart
    from helpers import small_camera
    cam = gart.make_camera(small_camera(w, h))
    st = gart.make_settings(tile, mode)
    g = gart.gart_gaussians()
    g.n, g.sh_degree = n, deg
    f = gart.gart_frame()
    return cam, st, g, f


@pytest.mark.parametrize("bad", ["tile", "mode", "precision", "alpha", "tmin", "width", "fx", "deg", "nptr", "frame"])
def test_invalid_arguments_rejected_on_host(lib, bad):
    cam, st, g, f = _structs()
    fp = ctypes.byref(f)
    if bad == "tile":
        st.tile = 12
    elif bad == "mode":
        st.backward_mode = 5
    elif bad == "precision":
        st.lt_precision = 2
    elif bad == "alpha":
        st.alpha_min = 0.0
    elif bad == "tmin":
        st.t_min = 1.5
    elif bad == "width":
        cam.width = 0
    elif bad == "fx":
        cam.fx = -1.0
    elif bad == "deg":
        g.sh_degree = 4
    elif bad == "nptr":
        g.n = 10  # non-zero count with null parameter pointers
    elif bad == "frame":
        fp = None
    r = lib.gart_bounds(ctypes.byref(g), ctypes.byref(cam), ctypes.byref(st), fp, None, None, None)
    expect = -4 if bad == "deg" else -1
    assert r == expect, (bad, r, lib.gart_last_error())
    assert lib.gart_last_error().decode() != ""


def test_call_order_enforced(lib):
    cam, st, g, f = _structs()
    assert lib.gart_build_tile_map(ctypes.byref(cam), ctypes.byref(st), ctypes.byref(f), None) == -1
    img = ctypes.c_float(0)
    assert lib.gart_forward(ctypes.byref(g), ctypes.byref(cam), ctypes.byref(st), ctypes.byref(f),
                            ctypes.byref(img), None) == -1


def test_scratch_bytes_monotone(lib):
    from paper_2608_17298_amd import gart
    cam, st, g, f = _structs()
    a = gart.gart_scratch_bytes(1000, 3, 10_000, cam, st)
    b = gart.gart_scratch_bytes(1000, 3, 100_000, cam, st)
    c = gart.gart_scratch_bytes(100_000, 3, 100_000, cam, st)
    assert 0 < a < b < c
    st.backward_mode = 1
    assert gart.gart_scratch_bytes(1000, 3, 100_000, cam, st) < b  # no per-pair rows needed
    st.backward_mode = 3
    assert gart.gart_scratch_bytes(1000, 3, 100_000, cam, st) == b  # the same per-pair rows


def test_ctypes_structs_match_header(tmp_path):
    """Every field of the ctypes mirrors sits at the offset the C compiler
    gives it from include/gart.h (and the struct sizes agree), so the
    binding passes the layout the library reads."""
    import subprocess
    from paper_2608_17298_amd import gart
    structs = [gart.gart_camera, gart.gart_gaussians, gart.gart_settings, gart.gart_frame, gart.gart_adam]
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "gart.h"', "int main(void) {"]
    for s in structs:
        lines.append(f'  printf("{s.__name__} size %zu\\n", sizeof({s.__name__}));')
        for f in s._fields_:
            lines.append(f'  printf("{s.__name__} {f[0]} %zu\\n", offsetof({s.__name__}, {f[0]}));')
    lines.append('  printf("gart_pixel_state size %zu\\n", sizeof(gart_pixel_state));')
    lines.append('  printf("gart_lt_entry size %zu\\n", sizeof(gart_lt_entry));')
    lines += ["  return 0;", "}"]
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-std=c11", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    got = {}
    for ln in subprocess.run([str(exe)], check=True, capture_output=True, text=True).stdout.splitlines():
        a, b, c = ln.split()
        got[(a, b)] = int(c)
    for s in structs:
        assert got[(s.__name__, "size")] == ctypes.sizeof(s), s.__name__
        for f in s._fields_:
            assert got[(s.__name__, f[0])] == getattr(s, f[0]).offset, (s.__name__, f[0])
    assert got[("gart_pixel_state", "size")] == 32 and got[("gart_lt_entry", "size")] == 16


def test_lt_entry_bytes(lib):
    """Entry size per (mode, precision): 16 / 4 (hybrid) bytes at full
    precision, 8 / 2 with fp16 storage; 0 for invalid settings."""
    from paper_2608_17298_amd import gart
    want = {("gather", "full"): 16, ("gather_atomic", "full"): 16, ("scatter", "full"): 16, ("hybrid", "full"): 4,
            ("gather", "half"): 8, ("gather_atomic", "half"): 8, ("scatter", "half"): 8, ("hybrid", "half"): 2}
    for (mode, prec), nb in want.items():
        assert gart.gart_lt_entry_bytes(gart.make_settings(8, mode, lt_precision=prec)) == nb, (mode, prec)
    st = gart.make_settings(8, "gather")
    st.lt_precision = 7
    assert lib.gart_lt_entry_bytes(ctypes.byref(st)) == 0
    assert lib.gart_lt_entry_bytes(None) == 0


@pytest.mark.parametrize("call", ["tile_map", "forward", "backward"])
@pytest.mark.parametrize("change", ["tile", "width", "height"])
def test_frame_geometry_checked_on_host(lib, call, change):
    """A frame sized by gart_bounds for one image and tile size is refused by
    later calls that describe another (the pixel state, tile ranges and hit
    lists are indexed with them): INVALID_ARG before anything is launched.
    The frame's stage is set by hand, so no GPU is involved."""
    cam, st, g, f = _structs(tile=8, w=16, h=16)
    f.stage = 3
    f.width, f.height, f.tile = 16, 16, 8
    f.tiles_x = f.tiles_y = 2
    f.lt_format = 0
    if change == "tile":
        st.tile = 16
    elif change == "width":
        cam.width = 17  # still two 8-pixel tile columns, but a wider pixel state
    else:
        cam.height = 15
    dl = ctypes.c_float(0)
    if call == "tile_map":
        r = lib.gart_build_tile_map(ctypes.byref(cam), ctypes.byref(st), ctypes.byref(f), None)
    elif call == "forward":
        r = lib.gart_forward(ctypes.byref(g), ctypes.byref(cam), ctypes.byref(st), ctypes.byref(f),
                             ctypes.byref(dl), None)
    else:
        r = lib.gart_backward(ctypes.byref(g), ctypes.byref(cam), ctypes.byref(st), ctypes.byref(f),
                              ctypes.byref(dl), None, None, None, None, None, None)
    assert r == -1, (call, change, lib.gart_last_error())
    msg = lib.gart_last_error().decode()
    assert "gart_bounds" in msg or "tile grid" in msg, msg


@pytest.mark.parametrize("call", ["forward", "backward"])
def test_hit_list_capacity_checked_on_host(lib, call):
    """hit_list needs tile^2 slots per pair: a frame whose hit_list_capacity
    is short of pair_count * tile^2 is refused with GART_ERR_CAPACITY before
    anything is launched (stage, pair count and pointers set by hand, no GPU)."""
    cam, st, g, f = _structs(tile=8, w=16, h=16)
    f.stage = 3
    f.width, f.height, f.tile = 16, 16, 8
    f.tiles_x = f.tiles_y = 2
    f.lt_format = 0
    f.pair_count = 5
    # pointers are never dereferenced: the check fails first
    f.hit_list = f.pixel_state = ctypes.c_void_p(256)
    f.hit_list_capacity = 5 * 64 - 1
    g.n = f.n = 0
    dl = ctypes.c_float(0)
    if call == "forward":
        r = lib.gart_forward(ctypes.byref(g), ctypes.byref(cam), ctypes.byref(st), ctypes.byref(f),
                             ctypes.byref(dl), None)
    else:
        r = lib.gart_backward(ctypes.byref(g), ctypes.byref(cam), ctypes.byref(st), ctypes.byref(f),
                              ctypes.byref(dl), None, None, None, None, None, None)
    assert r == -2, (call, lib.gart_last_error())
    assert "hit_list needs 320 slots (have 319)" in lib.gart_last_error().decode()


def test_hit_list_slots(lib):
    """gart_hit_list_slots: tile^2 slots per pair while the pairs are fewer
    than (tiles x k_max), then tiles x k_max rows, where k_max is the most
    hits a pixel can composite: the smallest k with (1 - alpha_min)^(k - 1)
    below t_min, plus a small guard; -1 for invalid arguments."""
    import math
    from paper_2608_17298_amd import gart
    cam, st, g, f = _structs(tile=8, w=57, h=43)  # 8 x 6 tiles
    n_tiles = 48
    a, t = float(st.alpha_min), float(st.t_min)  # float32 settings, read back as doubles
    k_lo = 1 + math.floor(math.log(t) / math.log(1 - a))  # hits a pixel can actually reach
    assert gart.gart_hit_list_slots(0, cam, st) == 0
    assert gart.gart_hit_list_slots(1000, cam, st) == 1000 * 64
    big = gart.gart_hit_list_slots(10 ** 9, cam, st)
    assert big % (64 * n_tiles) == 0
    k_max = big // (64 * n_tiles)
    assert k_lo <= k_max <= k_lo + 3, (k_lo, k_max)
    st16 = gart.make_settings(16, 0)  # 4 x 3 tiles of 256 pixels
    assert gart.gart_hit_list_slots(10 ** 9, cam, st16) == k_max * 256 * 12
    assert lib.gart_hit_list_slots(-1, ctypes.byref(cam), ctypes.byref(st)) == -1
    st.alpha_min = 0.0
    assert lib.gart_hit_list_slots(10, ctypes.byref(cam), ctypes.byref(st)) == -1


def test_frame_status_query_validated_on_host(lib):
    """gart_frame_status (the forward's GART_FRAME_* status word) refuses a
    NULL frame or output, and a frame the forward has not run on."""
    cam, st, g, f = _structs()
    v = ctypes.c_uint32(7)
    assert lib.gart_frame_status(None, ctypes.byref(v), None) == -1
    assert lib.gart_frame_status(ctypes.byref(f), None, None) == -1
    f.stage = 2
    assert lib.gart_frame_status(ctypes.byref(f), ctypes.byref(v), None) == -1
    assert "gart_forward" in lib.gart_last_error().decode()
    assert v.value == 7
