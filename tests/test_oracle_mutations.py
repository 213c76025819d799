"""Mutation check of the oracle's pins.

Each mutation below plants one plausible mistake in a copy of the oracle's
source (a flipped sign, a dropped term or factor, a transposed index, a wrong
threshold, rounding or walk index), builds the copy with the oracle's own
flags, and runs the oracle's CPU pins against it in a subprocess
(``GART_ORACLE_LIB`` points the ``oracle`` package at the copy).  Every
mutation must make at least one pin fail: a mutation that survives means the
pins cannot tell that part of the oracle from a wrong one.  The names say
which passage of the paper each mutated line follows.
"""
import os
import shutil
import subprocess
import sys
from concurrent.futures import ThreadPoolExecutor

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "gart_oracle.cpp")
PINS = ["test_oracle_camera.py", "test_oracle_geometry.py", "test_oracle_grad.py", "test_oracle_render.py",
        "test_oracle_sh.py", "test_oracle_storage.py", "test_oracle_tiles.py"]

# (name, exact source text, its replacement); each text occurs once in the source
MUTATIONS = [
    ("rotation of a quaternion: sign of an off-diagonal term (Sec. 3.1)",
     "R[1] = 2 * (x * y - w * z);", "R[1] = 2 * (x * y + w * z);"),
    ("pixel ray: focal lengths swapped (Eq. 3)",
     "double dc[3] = {(px + 0.5 - S.cx) / S.fx, (py + 0.5 - S.cy) / S.fy, 1.0};",
     "double dc[3] = {(px + 0.5 - S.cx) / S.fy, (py + 0.5 - S.cy) / S.fx, 1.0};"),
    ("pixel ray: camera rotation transposed (Eq. 3)",
     "d[k] = S.Rc[0 * 3 + k] * dc[0] + S.Rc[1 * 3 + k] * dc[1] + S.Rc[2 * 3 + k] * dc[2];",
     "d[k] = S.Rc[k * 3 + 0] * dc[0] + S.Rc[k * 3 + 1] * dc[1] + S.Rc[k * 3 + 2] * dc[2];"),
    ("hit test: response threshold moved (Eq. 8, alpha >= alpha_min)",
     "return tau > 0.0 && D2 <= P.D2c;", "return tau > 0.0 && D2 <= 0.9 * P.D2c;"),
    ("colour: the 0.5 offset of the SH colour dropped (Sec. 3.1)",
     "  double v = 0.5;\n  for (int k = 0; k < S.K; ++k) v += S.sh",
     "  double v = 0.0;\n  for (int k = 0; k < S.K; ++k) v += S.sh"),
    ("opacity: Gaussian falloff exp(-D2) instead of exp(-D2 / 2) (Eq. 5-6)",
     "double alpha = P.sigma * std::exp(-0.5 * H.D2);", "double alpha = P.sigma * std::exp(-H.D2);"),
    ("compositing: termination threshold halved (Eq. 7, T < T_min)",
     "if (T < S.t_min) {", "if (T < 0.5 * S.t_min) {"),
    ("gradient: sign of the colour-behind term of dL/dalpha (Sec. 3.5)",
     "dLdalpha += g[ch] * (Tst * c.c[ch] - behind[ch] / (1.0 - c.alpha));",
     "dLdalpha += g[ch] * (Tst * c.c[ch] + behind[ch] / (1.0 - c.alpha));"),
    ("gradient: transmittance dropped from dL/dc (Sec. 3.5)",
     "double dc = Tst * c.alpha * g[ch];", "double dc = c.alpha * g[ch];"),
    ("gradient: sign of dL/dmu (Sec. 3.5)",
     "atomic_add(&accMu[c.id * 3 + b], -v);", "atomic_add(&accMu[c.id * 3 + b], v);"),
    ("gradient: dL/dlog s taken from the transposed dL/dW (Sec. 3.5)",
     "v += dW[3 * k + j] * P.W[3 * k + j];", "v += dW[3 * j + k] * P.W[3 * j + k];"),
    ("gradient: sigmoid derivative dropped from dL/dlogit (Sec. 3.5)",
     "g_logits[i] = P.sigma * (1.0 - P.sigma) * accSig[i];", "g_logits[i] = P.sigma * accSig[i];"),
    ("SH basis: sine and cosine of the m < 0 functions swapped (Sec. 3.1)",
     "v = std::sqrt(2.0) * N * P * std::sin(am * phi);", "v = std::sqrt(2.0) * N * P * std::cos(am * phi);"),
    ("bounds: first covered column rounded down instead of up (Sec. 4.2)",
     "double a = std::ceil(p - h - 0.5 - e);", "double a = std::floor(p - h - 0.5 - e);"),
    ("fp16 storage: fixed-point L truncated instead of rounded (Sec. 6)",
     "return std::min(std::nearbyint(L / q), 65535.0) * q;", "return std::min(std::floor(L / q), 65535.0) * q;"),
    ("T-only storage: colour behind a hit includes the hit itself (Sec. 4.4 hybrid)",
     "behind[ch] = walk[3 * (k + 1) + ch];", "behind[ch] = walk[3 * k + ch];"),
]


def _build(src_text, out):
    with open(out + ".cpp", "w") as f:
        f.write(src_text)
    cmd = ["g++", "-O2", "-std=c++17", "-fopenmp", "-fPIC", "-shared", "-fno-fast-math", "-ffp-contract=off",
           out + ".cpp", "-o", out + ".so"]
    r = subprocess.run(cmd, capture_output=True, text=True)
    assert r.returncode == 0, r.stderr[-2000:]
    return out + ".so"


def _pins_fail(lib):
    env = dict(os.environ, GART_ORACLE_LIB=lib, OMP_NUM_THREADS="2", PYTHONPATH=ROOT)
    cmd = [sys.executable, "-m", "pytest", "-q", "-x", "-p", "no:cacheprovider", "-m", "not gpu",
           *[os.path.join(ROOT, "tests", p) for p in PINS]]
    r = subprocess.run(cmd, capture_output=True, text=True, env=env, cwd=ROOT, timeout=600)
    # exit status 1 with a failed test: a pin caught it (not a crash, a
    # collection error or an interrupted run)
    assert r.returncode in (0, 1) and ("failed" in r.stdout) == (r.returncode == 1), r.stdout[-1500:]
    return r.returncode == 1, r.stdout[-600:]


@pytest.mark.slow
@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_every_mutation_fails_a_pin(tmp_path):
    src = open(SRC).read()
    for name, old, new in MUTATIONS:
        assert src.count(old) == 1, name
    with ThreadPoolExecutor(8) as ex:
        libs = list(ex.map(lambda m: _build(src.replace(m[1][1], m[1][2]), str(tmp_path / f"m{m[0]}")),
                           enumerate(MUTATIONS)))
    with ThreadPoolExecutor(4) as ex:
        results = list(ex.map(_pins_fail, libs))
    survivors = [(MUTATIONS[i][0], out) for i, (failed, out) in enumerate(results) if not failed]
    assert not survivors, survivors


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_unmutated_copy_passes_the_pins(tmp_path):
    """The harness itself: an unchanged copy built the same way passes."""
    failed, out = _pins_fail(_build(open(SRC).read(), str(tmp_path / "same")))
    assert not failed, out
