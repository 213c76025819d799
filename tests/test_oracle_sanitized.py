"""The fp64 oracle built with AddressSanitizer and UndefinedBehaviorSanitizer
(g++, host code only) and driven through every C entry point the Python
wrapper uses (every storage model of the backward included), on a small
SH3 scene with a rotated camera, culled and
eye-plane-crossing Gaussians and terminating pixels: any out-of-bounds
access, use after free, leak of the scene or undefined behaviour (overflow,
misaligned or null access, bad shift) fails the run."""
import os
import shutil
import subprocess

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "gart_oracle.cpp")

DRIVER = r"""
#include <cmath>
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>
extern "C" {
void* orc_scene_new(int64_t, int32_t, const double*, const double*, const double*, const double*, const double*,
                    int32_t, int32_t, const double*, const double*, const double*, double, double);
void orc_scene_free(void*);
void orc_prim_info(void*, int32_t*, int64_t*, int32_t*, double*, double*, double*, double*);
void orc_sh_basis(int32_t, int64_t, const double*, double*);
void orc_render(void*, int64_t, const int64_t*, int32_t, double*, double*, int64_t*, int64_t*, double*, double*);
void orc_bounds_raw(void*, double*);
void orc_ray_prim(void*, int64_t, const int64_t*, const int64_t*, double*, double*, int32_t*, double*, double*);
void orc_camera_origin(void*, double*);
void orc_all_hits(void*, int64_t, const int64_t*, int32_t, int32_t, int64_t*, const int64_t*, int64_t*);
void orc_records(void*, int64_t, const int64_t*, const int64_t*, int64_t*, double*, double*);
void orc_backward(void*, int64_t, const int64_t*, const double*, double*, double*, double*, double*, double*);
void orc_lt_index(void*, int32_t, int64_t, const int64_t*, const int64_t*, int64_t*);
void orc_backward_stored(void*, int64_t, const int64_t*, const double*, double*, double*, double*, double*, double*,
                         int32_t);
void orc_storage_round(int32_t, int64_t, const double*, double*, double);
double orc_colour_bound(void*);
int32_t orc_num_threads();
}
static double u(unsigned& s) { s = s * 1664525u + 1013904223u; return (s >> 8) * (1.0 / 16777216.0); }
int main() {
  const int64_t n = 300; const int deg = 3, K = 16, W = 37, H = 29;
  unsigned seed = 12345u;
  std::vector<double> mu(3 * n), ls(3 * n), q(4 * n), lg(n), sh(3 * K * n);
  for (int64_t i = 0; i < n; ++i) {
    for (int k = 0; k < 3; ++k) { mu[3 * i + k] = 2.4 * u(seed) - 1.2; ls[3 * i + k] = -2.8 + 1.2 * u(seed); }
    for (int k = 0; k < 4; ++k) q[4 * i + k] = u(seed) - 0.5;
    lg[i] = 6.0 * u(seed) - 2.0;
    for (int k = 0; k < 3 * K; ++k) sh[3 * K * i + k] = (k < 3 ? 1.0 : 0.1) * (u(seed) - 0.5);
  }
  mu[0] = 0.0; mu[1] = 0.0; mu[2] = -4.0;      // contains the camera centre
  mu[3] = 0.4; mu[4] = 0.1; mu[5] = -3.9;      // crosses the eye plane
  lg[2] = -9.0;                                // below alpha_min
  mu[9] = 0.0; mu[10] = 0.0; mu[11] = -9.0;    // behind the camera
  q[16] = q[17] = q[18] = q[19] = 0.0;         // zero-norm quaternion
  mu[15] = NAN;                                // non-finite
  const double intr[4] = {36.0, 37.5, 18.25, 14.5};
  const double c = std::cos(0.4), s = std::sin(0.4);
  const double R[9] = {c, 0, s, 0, 1, 0, -s, 0, c};
  const double t[3] = {0.0, 0.0, 4.0};
  void* h = orc_scene_new(n, deg, mu.data(), ls.data(), q.data(), lg.data(), sh.data(), W, H, intr, R, t,
                          1.0 / 255.0, 1e-4);
  std::vector<int32_t> rect(4 * n), state(n); std::vector<int64_t> area(n);
  std::vector<double> sig(n), d2c(n), Wm(9 * n), og(3 * n), raw(5 * n);
  orc_prim_info(h, rect.data(), area.data(), state.data(), sig.data(), d2c.data(), Wm.data(), og.data());
  orc_bounds_raw(h, raw.data());
  const int64_t m = W * H;
  std::vector<int64_t> pix(m); for (int64_t p = 0; p < m; ++p) pix[p] = p;
  std::vector<double> col(3 * m), tend(m), marg(m), tfin(m); std::vector<int64_t> iend(m), ninc(m);
  for (int brute = 0; brute < 2; ++brute)
    orc_render(h, m, pix.data(), brute, col.data(), tend.data(), iend.data(), ninc.data(), marg.data(), tfin.data());
  orc_render(h, m, nullptr, 0, col.data(), tend.data(), iend.data(), ninc.data(), marg.data(), tfin.data());
  std::vector<int64_t> cnt(m), off(m + 1, 0);
  orc_all_hits(h, m, pix.data(), 1, 1, cnt.data(), nullptr, nullptr);
  for (int64_t p = 0; p < m; ++p) off[p + 1] = off[p] + cnt[p];
  std::vector<int64_t> prims(off[m] + 1);
  orc_all_hits(h, m, pix.data(), 1, 0, nullptr, off.data(), prims.data());
  std::vector<int64_t> roff(m + 1, 0); for (int64_t p = 0; p < m; ++p) roff[p + 1] = roff[p] + ninc[p];
  const int64_t tot = roff[m];
  std::vector<int64_t> rprim(tot + 1); std::vector<double> LT(4 * tot + 4), tau(tot + 1);
  orc_records(h, m, pix.data(), roff.data(), rprim.data(), LT.data(), tau.data());
  std::vector<int64_t> idx(tot + 1), owner(tot + 1);
  for (int64_t p = 0; p < m; ++p) for (int64_t k = roff[p]; k < roff[p + 1]; ++k) owner[k] = p;
  orc_lt_index(h, 8, tot, rprim.data(), owner.data(), idx.data());
  orc_lt_index(h, 16, tot, rprim.data(), owner.data(), idx.data());
  std::vector<int64_t> rp(64), rq(64); std::vector<double> ta(64), da(64), al(64), dir(192); std::vector<int32_t> hit(64);
  for (int k = 0; k < 64; ++k) { rp[k] = (k * 97) % m; rq[k] = (k * 31) % n; }
  orc_ray_prim(h, 64, rp.data(), rq.data(), ta.data(), da.data(), hit.data(), al.data(), dir.data());
  double o[3]; orc_camera_origin(h, o);
  std::vector<double> dl(3 * m); for (auto& v : dl) v = u(seed) - 0.5;
  std::vector<double> gm(3 * n), gs(3 * n), gq(4 * n), gl(n), gsh(3 * K * n);
  orc_backward(h, 0, nullptr, dl.data(), gm.data(), gs.data(), gq.data(), gl.data(), gsh.data());
  orc_backward(h, 200, pix.data() + 100, dl.data(), gm.data(), gs.data(), gq.data(), gl.data(), gsh.data());
  for (int model = 0; model <= 5; ++model)  // every storage model of the intermediate buffer
    orc_backward_stored(h, 0, nullptr, dl.data(), gm.data(), gs.data(), gq.data(), gl.data(), gsh.data(), model);
  const double bound = orc_colour_bound(h);
  std::vector<double> xs(64), rs(64);
  for (int k = 0; k < 64; ++k) xs[k] = k == 0 ? 0.0 : std::ldexp(u(seed), -(k % 30));
  for (int kind = 1; kind <= 3; ++kind) orc_storage_round(kind, 64, xs.data(), rs.data(), bound / 65536.0);
  std::vector<double> dirs(3 * 50), Y(16 * 50);
  for (auto& v : dirs) v = u(seed) - 0.5;
  orc_sh_basis(3, 50, dirs.data(), Y.data());
  orc_scene_free(h);
  long active = 0; for (int64_t i = 0; i < n; ++i) active += state[i] == 0;
  std::printf("ok active=%ld hits=%lld composited=%lld threads=%d\n", active, (long long)off[m], (long long)tot,
              orc_num_threads());
  return 0;
}
"""


@pytest.mark.skipif(shutil.which("g++") is None, reason="needs g++")
def test_oracle_under_address_and_ub_sanitizers(tmp_path):
    drv = tmp_path / "driver.cpp"
    drv.write_text(DRIVER)
    exe = tmp_path / "oracle_asan"
    flags = ["-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fopenmp", "-ffp-contract=off",
             "-fsanitize=address,undefined", "-fno-sanitize-recover=all"]
    subprocess.run(["g++", *flags, SRC, str(drv), "-o", str(exe)], check=True, capture_output=True, timeout=300)
    env = dict(os.environ, OMP_NUM_THREADS="4",
               ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:halt_on_error=1",
               UBSAN_OPTIONS="print_stacktrace=1:halt_on_error=1",
               LSAN_OPTIONS="suppressions=" + str(tmp_path / "lsan.supp"))
    (tmp_path / "lsan.supp").write_text("leak:libgomp\n")
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=300, env=env)
    assert r.returncode == 0, r.stderr[-4000:]
    assert "runtime error" not in r.stderr, r.stderr[-4000:]
    assert r.stdout.startswith("ok "), r.stdout
    active = int(r.stdout.split("active=")[1].split()[0])
    assert 200 < active < 300  # the planted culled Gaussians are culled, the rest not all
