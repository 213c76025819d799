// fp64 CPU oracle for ray-traced 3D Gaussian rendering and its gradient.
//
// TEST INFRASTRUCTURE ONLY.  This file is the plain, slow definition that the
// GPU library is checked against.  Only the test-suite, the smoke check and
// the benchmark's CPU-baseline leg may load it.  It shares no code, header,
// table or constant with the GPU library.
//
// What it computes (paper sections cited per function):
//   * per-Gaussian quantities: rotation from a quaternion, scales,
//     opacity, clamp radius, world->Gaussian map     (Sec. 3.1-3.4, Eq. 1-2, 9-10)
//   * conservative screen-space pixel rectangles from the projected quadric
//                                                     (Sec. 4.2, Eq. 11-14)
//   * per-pixel ray trace over every candidate: max-response point, hit test,
//     ordering by depth, front-to-back compositing   (Sec. 3.2-3.3, Eq. 3-8)
//   * the analytic per-pixel ("pixel-centric") gradient, scattered into
//     fp64 per-primitive accumulators, then the chain rule to the raw
//     parameters                                      (Sec. 3.5)
//   * the intermediate-buffer address idx(i,t,p) by plain enumeration
//                                                     (Sec. 4.3, Eq. 16)
//
// All arithmetic is double precision.  Inputs arrive as double (float32 scene
// values are promoted exactly by the caller; finite-difference pins perturb
// them in double).
// Readings where the paper is silent are documented next to the code that
// takes them.
#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdint>
#include <cstring>
#include <limits>
#include <vector>
#ifdef _OPENMP
#include <omp.h>
#endif

namespace {

constexpr double kPi = 3.14159265358979323846;
constexpr double kRectPad = 1e-4;  // pixels of slack on each rectangle edge

// ---------------------------------------------------------------------------
// Real spherical harmonics (degree <= 3) from the general definition:
//   Y_l^m = N_l^|m| P_l^|m|(cos th) * { sqrt2 cos(m phi)   m > 0
//                                      { 1                   m = 0
//                                      { sqrt2 sin(|m| phi)  m < 0
// with N_l^m = sqrt((2l+1)/(4 pi) (l-m)!/(l+m)!) and P_l^m the associated
// Legendre function WITHOUT the Condon-Shortley phase.  Index k = l*l + l + m.
// (Sec. 3.1: radiance is a spherical-harmonic function of the view direction.)
// ---------------------------------------------------------------------------
double factorial(int n) {
  double f = 1.0;
  for (int i = 2; i <= n; ++i) f *= i;
  return f;
}

// Associated Legendre P_l^m(x), m >= 0, no Condon-Shortley phase, by the
// standard upward recurrence in l.
double assoc_legendre(int l, int m, double x) {
  double pmm = 1.0;
  double somx2 = std::sqrt(std::max(0.0, (1.0 - x) * (1.0 + x)));
  double fact = 1.0;
  for (int i = 1; i <= m; ++i) {
    pmm *= fact * somx2;
    fact += 2.0;
  }
  if (l == m) return pmm;
  double pmmp1 = x * (2 * m + 1) * pmm;
  if (l == m + 1) return pmmp1;
  double pll = 0.0;
  for (int ll = m + 2; ll <= l; ++ll) {
    pll = ((2 * ll - 1) * x * pmmp1 - (ll + m - 1) * pmm) / (ll - m);
    pmm = pmmp1;
    pmmp1 = pll;
  }
  return pll;
}

void sh_basis(int degree, const double d[3], double* Y) {
  double ct = d[2];
  double phi = std::atan2(d[1], d[0]);
  for (int l = 0; l <= degree; ++l) {
    for (int m = -l; m <= l; ++m) {
      int am = m < 0 ? -m : m;
      double N = std::sqrt((2.0 * l + 1.0) / (4.0 * kPi) * factorial(l - am) / factorial(l + am));
      double P = assoc_legendre(l, am, ct);
      double v;
      if (m > 0)
        v = std::sqrt(2.0) * N * P * std::cos(m * phi);
      else if (m < 0)
        v = std::sqrt(2.0) * N * P * std::sin(am * phi);
      else
        v = N * P;
      Y[l * l + l + m] = v;
    }
  }
}

// Rotation matrix of a unit quaternion (w, x, y, z), row-major.
void quat_to_rot(const double q[4], double R[9]) {
  double w = q[0], x = q[1], y = q[2], z = q[3];
  R[0] = 1 - 2 * (y * y + z * z); R[1] = 2 * (x * y - w * z);     R[2] = 2 * (x * z + w * y);
  R[3] = 2 * (x * y + w * z);     R[4] = 1 - 2 * (x * x + z * z); R[5] = 2 * (y * z - w * x);
  R[6] = 2 * (x * z - w * y);     R[7] = 2 * (y * z + w * x);     R[8] = 1 - 2 * (x * x + y * y);
}

// dR/dq for the map above, dRdq[c][e] = d R[e] / d q[c].
void quat_to_rot_jacobian(const double q[4], double dRdq[4][9]) {
  double w = q[0], x = q[1], y = q[2], z = q[3];
  // d/dw
  double dw[9] = {0, -2 * z, 2 * y, 2 * z, 0, -2 * x, -2 * y, 2 * x, 0};
  // d/dx
  double dx[9] = {0, 2 * y, 2 * z, 2 * y, -4 * x, -2 * w, 2 * z, 2 * w, -4 * x};
  // d/dy
  double dy[9] = {-4 * y, 2 * x, 2 * w, 2 * x, 0, 2 * z, -2 * w, 2 * z, -4 * y};
  // d/dz
  double dz[9] = {-4 * z, -2 * w, 2 * x, 2 * w, -4 * z, 2 * y, 2 * x, 2 * y, 0};
  std::memcpy(dRdq[0], dw, sizeof dw);
  std::memcpy(dRdq[1], dx, sizeof dx);
  std::memcpy(dRdq[2], dy, sizeof dy);
  std::memcpy(dRdq[3], dz, sizeof dz);
}

enum PrimState : int32_t {
  kActive = 0,
  kCulledOpacity = 1,   // sigma <= alpha_min: clamp radius undefined (Eq. 10)
  kCulledBehind = 2,    // bounding ellipsoid wholly behind the camera
  kCulledOffscreen = 3, // no pixel column or row can meet the ellipsoid
  kCulledNonFinite = 4, // a parameter is NaN or infinite
};

struct Prim {
  int32_t state = kActive;
  double mu[3];
  double s[3];
  double qn[4];     // normalised quaternion
  double qnorm;
  double R[9];
  double W[9];      // world -> Gaussian space, W = S^-1 R^T (Eq. 5)
  double sigma;
  double D2c;       // squared clamp radius alpha_c^2 = 2 log(sigma / alpha_min)
  int32_t rect[4];  // x0, y0, x1, y1 inclusive
  int64_t area;
  double q44;       // <v, T'_4 . T'_4>: < 0 iff the eye plane misses the ellipsoid
  double Qx[2], Qy[2];  // (Q_aa, Q_a4) for a = x, y
};

struct Scene {
  int64_t n;
  int deg, K;
  int W, H;
  double fx, fy, cx, cy;
  double Rc[9], tc[3];
  double o[3];  // camera centre in world space
  double alpha_min, t_min;
  std::vector<Prim> prims;
  std::vector<double> sh;  // [n, K, 3]
  // Candidate buckets: the oracle's own 16x16-pixel grid, each bucket lists
  // (ascending) the primitives whose rectangle meets it.
  int bsz = 16, bnx = 0, bny = 0;
  std::vector<int64_t> bucket_off;
  std::vector<int64_t> bucket_prim;
};

// One axis of the pixel rectangle, from the 2x2 block of the projected dual
// quadric.  The plane through the camera containing image column coordinate
// u (clip-space plane X - u*w = 0) meets the ellipsoid iff
//       q(u) = Qaa - 2 u Qa4 + u^2 Q44 >= 0.
// Q44 < 0 (eye plane misses the ellipsoid): q >= 0 on [p-h, p+h] with
// p = Qa4/Q44, h = sqrt(p^2 - Qaa/Q44): this is Eq. 12-14.  Q44 >= 0 (the
// ellipsoid crosses the eye plane; the paper gives no bound there): the
// covered set is the complement of an open interval (or everything), and
// the rectangle is the hull of the covered pixel centres.  Returns false if
// no pixel centre is covered.
bool axis_range(double Qaa, double Qa4, double Q44, int npix, int32_t* lo, int32_t* hi) {
  const double e = kRectPad;
  if (Q44 < 0.0) {
    double p = Qa4 / Q44;
    double h2 = p * p - Qaa / Q44;
    double h = std::sqrt(std::max(0.0, h2));
    double a = std::ceil(p - h - 0.5 - e);
    double b = std::floor(p + h - 0.5 + e);
    a = std::max(a, 0.0);
    b = std::min(b, double(npix - 1));
    if (a > b) return false;
    *lo = int32_t(a);
    *hi = int32_t(b);
    return true;
  }
  // Q44 >= 0: solve q(u) = 0.
  if (Q44 == 0.0) {
    // q(u) = Qaa - 2 u Qa4, linear.
    if (Qa4 == 0.0) {
      if (Qaa >= 0.0) { *lo = 0; *hi = npix - 1; return true; }
      return false;
    }
    double r = Qaa / (2.0 * Qa4);
    if (Qa4 > 0.0) {  // covered for u <= r
      double b = std::min(std::floor(r - 0.5 + e), double(npix - 1));
      if (b < 0.0) return false;
      *lo = 0; *hi = int32_t(b); return true;
    }
    double a = std::max(std::ceil(r - 0.5 - e), 0.0);  // covered for u >= r
    if (a > npix - 1) return false;
    *lo = int32_t(a); *hi = npix - 1; return true;
  }
  double disc = Qa4 * Qa4 - Q44 * Qaa;
  if (disc <= 0.0) { *lo = 0; *hi = npix - 1; return true; }
  double sq = std::sqrt(disc);
  double u1 = (Qa4 - sq) / Q44, u2 = (Qa4 + sq) / Q44;  // covered: u <= u1 or u >= u2
  bool left = (u1 - 0.5 + e) >= 0.0;                   // some column x with x+.5 <= u1
  bool right = (u2 - 0.5 - e) <= double(npix - 1);     // some column with x+.5 >= u2
  if (!left && !right) return false;
  double a = left ? 0.0 : std::max(std::ceil(u2 - 0.5 - e), 0.0);
  double b = right ? double(npix - 1) : std::min(std::floor(u1 - 0.5 + e), double(npix - 1));
  if (a > b) return false;
  *lo = int32_t(a);
  *hi = int32_t(b);
  return true;
}

void prepare_prim(Scene& S, int64_t i, const double* means, const double* ls, const double* quats,
                  const double* logits, Prim& P) {
  bool finite = true;
  for (int k = 0; k < 3; ++k) {
    P.mu[k] = means[3 * i + k];
    double l = ls[3 * i + k];
    P.s[k] = std::exp(l);
    finite = finite && std::isfinite(P.mu[k]) && std::isfinite(l);
  }
  double qraw[4];
  double qq = 0;
  for (int k = 0; k < 4; ++k) {
    qraw[k] = quats[4 * i + k];
    finite = finite && std::isfinite(qraw[k]);
    qq += qraw[k] * qraw[k];
  }
  double lg = logits[i];
  finite = finite && std::isfinite(lg) && qq > 0.0;
  P.qnorm = std::sqrt(qq);
  for (int k = 0; k < 4; ++k) P.qn[k] = qraw[k] / (P.qnorm > 0 ? P.qnorm : 1.0);
  quat_to_rot(P.qn, P.R);
  for (int k = 0; k < 3; ++k)
    for (int j = 0; j < 3; ++j) P.W[3 * k + j] = P.R[3 * j + k] / P.s[k];  // (S^-1 R^T)_kj
  P.sigma = 1.0 / (1.0 + std::exp(-lg));
  P.area = 0;
  P.rect[0] = P.rect[1] = 0;
  P.rect[2] = P.rect[3] = -1;
  if (!finite) { P.state = kCulledNonFinite; P.D2c = 0; return; }
  if (!(P.sigma > S.alpha_min)) { P.state = kCulledOpacity; P.D2c = 0; return; }
  P.D2c = 2.0 * std::log(P.sigma / S.alpha_min);
  double ac = std::sqrt(P.D2c);

  // T maps the unit sphere to the clamped ellipsoid: [R S alpha_c | mu] (Eq. 9).
  double T[4][4] = {};
  for (int r = 0; r < 3; ++r) {
    for (int c = 0; c < 3; ++c) T[r][c] = P.R[3 * r + c] * P.s[c] * ac;
    T[r][3] = P.mu[r];
  }
  T[3][3] = 1.0;
  // VPM: world -> pixel-unit clip coordinates (X, Y, -, w) with X/w, Y/w the
  // continuous pixel coordinates and w the camera depth.  The third (depth)
  // row never enters the x/y bounds, so it is left zero.
  double V[4][4] = {};
  double E[4][4] = {};  // extrinsics [Rc tc; 0 1]
  for (int r = 0; r < 3; ++r) {
    for (int c = 0; c < 3; ++c) E[r][c] = S.Rc[3 * r + c];
    E[r][3] = S.tc[r];
  }
  E[3][3] = 1.0;
  double Kp[4][4] = {{S.fx, 0, S.cx, 0}, {0, S.fy, S.cy, 0}, {0, 0, 0, 0}, {0, 0, 1, 0}};
  for (int r = 0; r < 4; ++r)
    for (int c = 0; c < 4; ++c) {
      double acc = 0;
      for (int k = 0; k < 4; ++k) acc += Kp[r][k] * E[k][c];
      V[r][c] = acc;
    }
  double Tp[4][4];  // T' = VPM T (Eq. 11); rows are T'_1..T'_4
  for (int r = 0; r < 4; ++r)
    for (int c = 0; c < 4; ++c) {
      double acc = 0;
      for (int k = 0; k < 4; ++k) acc += V[r][k] * T[k][c];
      Tp[r][c] = acc;
    }
  // Dual-quadric entries <v, T'_a (.) T'_b>, v = (1,1,1,-1)  (Eq. 13-14).
  auto dq = [&](int a, int b) {
    return Tp[a][0] * Tp[b][0] + Tp[a][1] * Tp[b][1] + Tp[a][2] * Tp[b][2] - Tp[a][3] * Tp[b][3];
  };
  double s44 = dq(3, 3);
  P.q44 = s44;
  P.Qx[0] = dq(0, 0); P.Qx[1] = dq(0, 3);
  P.Qy[0] = dq(1, 1); P.Qy[1] = dq(1, 3);
  if (s44 < 0.0 && Tp[3][3] <= 0.0) { P.state = kCulledBehind; return; }
  int32_t x0, x1, y0, y1;
  bool okx = axis_range(dq(0, 0), dq(0, 3), s44, S.W, &x0, &x1);
  bool oky = axis_range(dq(1, 1), dq(1, 3), s44, S.H, &y0, &y1);
  if (!okx || !oky) { P.state = kCulledOffscreen; return; }
  P.rect[0] = x0; P.rect[1] = y0; P.rect[2] = x1; P.rect[3] = y1;
  P.area = int64_t(x1 - x0 + 1) * int64_t(y1 - y0 + 1);
  P.state = kActive;
}

void build_buckets(Scene& S) {
  S.bnx = (S.W + S.bsz - 1) / S.bsz;
  S.bny = (S.H + S.bsz - 1) / S.bsz;
  int64_t nb = int64_t(S.bnx) * S.bny;
  std::vector<int64_t> cnt(nb + 1, 0);
  for (int64_t i = 0; i < S.n; ++i) {
    const Prim& P = S.prims[i];
    if (P.state != kActive) continue;
    for (int by = P.rect[1] / S.bsz; by <= P.rect[3] / S.bsz; ++by)
      for (int bx = P.rect[0] / S.bsz; bx <= P.rect[2] / S.bsz; ++bx) cnt[int64_t(by) * S.bnx + bx + 1]++;
  }
  for (int64_t b = 0; b < nb; ++b) cnt[b + 1] += cnt[b];
  S.bucket_off = cnt;
  S.bucket_prim.assign(cnt[nb], 0);
  std::vector<int64_t> fill(cnt.begin(), cnt.end() - 1);
  for (int64_t i = 0; i < S.n; ++i) {  // ascending i -> each bucket ascending
    const Prim& P = S.prims[i];
    if (P.state != kActive) continue;
    for (int by = P.rect[1] / S.bsz; by <= P.rect[3] / S.bsz; ++by)
      for (int bx = P.rect[0] / S.bsz; bx <= P.rect[2] / S.bsz; ++bx)
        S.bucket_prim[fill[int64_t(by) * S.bnx + bx]++] = i;
  }
}

// Unit ray direction through the centre of pixel (px, py) (Eq. 3), in world
// space, and the camera centre.  Pixel centres sit at +0.5.
void pixel_ray(const Scene& S, int px, int py, double d[3]) {
  double dc[3] = {(px + 0.5 - S.cx) / S.fx, (py + 0.5 - S.cy) / S.fy, 1.0};
  for (int k = 0; k < 3; ++k) d[k] = S.Rc[0 * 3 + k] * dc[0] + S.Rc[1 * 3 + k] * dc[1] + S.Rc[2 * 3 + k] * dc[2];
  double nn = std::sqrt(d[0] * d[0] + d[1] * d[1] + d[2] * d[2]);
  for (int k = 0; k < 3; ++k) d[k] /= nn;
}

struct Hit {
  double tau;
  int64_t id;
  double D2;
  double xg[3];
};

// Max-response point of Gaussian P on the ray o + tau d (Eq. 4-5) and the
// hit test tau > 0 and D^2 <= D2c (equivalently alpha >= alpha_min, Eq. 8,
// 10).  Returns the raw margin quantities through the out parameters.
bool ray_gaussian(const Scene& S, const Prim& P, const double d[3], Hit* h) {
  double om[3] = {S.o[0] - P.mu[0], S.o[1] - P.mu[1], S.o[2] - P.mu[2]};
  double og[3], dg[3];
  for (int k = 0; k < 3; ++k) {
    og[k] = P.W[3 * k] * om[0] + P.W[3 * k + 1] * om[1] + P.W[3 * k + 2] * om[2];
    dg[k] = P.W[3 * k] * d[0] + P.W[3 * k + 1] * d[1] + P.W[3 * k + 2] * d[2];
  }
  double tau = -(og[0] * dg[0] + og[1] * dg[1] + og[2] * dg[2]) / (dg[0] * dg[0] + dg[1] * dg[1] + dg[2] * dg[2]);
  double xg[3] = {og[0] + tau * dg[0], og[1] + tau * dg[1], og[2] + tau * dg[2]};
  double D2 = xg[0] * xg[0] + xg[1] * xg[1] + xg[2] * xg[2];
  h->tau = tau;
  h->D2 = D2;
  h->xg[0] = xg[0]; h->xg[1] = xg[1]; h->xg[2] = xg[2];
  return tau > 0.0 && D2 <= P.D2c;
}

double colour_channel(const Scene& S, int64_t i, int ch, const double* Y, bool* unclamped) {
  double v = 0.5;
  for (int k = 0; k < S.K; ++k) v += S.sh[(i * S.K + k) * 3 + ch] * Y[k];
  *unclamped = v > 0.0;
  return v > 0.0 ? v : 0.0;
}

struct PixelResult {
  double C[3];
  double tau_end;
  int64_t id_end;
  int32_t terminated;
  int64_t n_included;
  double margin;
  double T_final;
};

struct Composited {
  int64_t id;
  double tau, D2, xg[3];
  double alpha, c[3], L[3], T;
  bool unclamped[3];
};

// Collect every hit of a pixel ray.  brute=1 ignores the rectangles and
// tests all primitives that can be hit (the plain definition); brute=0
// tests the primitives listed in the pixel's bucket whose rectangle contains
// the pixel.
void gather_hits(const Scene& S, int px, int py, const double d[3], int brute, std::vector<Hit>& hits,
                 double* margin) {
  hits.clear();
  auto test = [&](int64_t i) {
    const Prim& P = S.prims[i];
    Hit h;
    bool hit = ray_gaussian(S, P, d, &h);
    h.id = i;
    double mD = std::fabs(h.D2 - P.D2c) / P.D2c;
    if (mD < *margin) *margin = mD;
    if (hit) hits.push_back(h);
  };
  if (brute) {
    for (int64_t i = 0; i < S.n; ++i)
      if (S.prims[i].state == kActive || S.prims[i].state == kCulledBehind ||
          S.prims[i].state == kCulledOffscreen)
        test(i);
  } else {
    int64_t b = int64_t(py / S.bsz) * S.bnx + px / S.bsz;
    for (int64_t j = S.bucket_off[b]; j < S.bucket_off[b + 1]; ++j) {
      int64_t i = S.bucket_prim[j];
      const Prim& P = S.prims[i];
      if (px >= P.rect[0] && px <= P.rect[2] && py >= P.rect[1] && py <= P.rect[3]) test(i);
    }
  }
  // Depth order; equal depths broken by ascending primitive index.
  std::sort(hits.begin(), hits.end(), [](const Hit& a, const Hit& b) {
    return a.tau < b.tau || (a.tau == b.tau && a.id < b.id);
  });
}

// Front-to-back compositing of one pixel (Eq. 6-8) with termination once the
// transmittance drops below t_min (the hit that crosses is included).  The
// background is black.  Fills the composited list with the (L, T) state
// BEFORE each hit: L is the colour accumulated in front of the hit and T the
// transmittance in front of it (Eq. 7).
void render_pixel(const Scene& S, int px, int py, int brute, PixelResult* out, std::vector<Hit>& hits,
                  std::vector<Composited>* comp) {
  double d[3];
  pixel_ray(S, px, py, d);
  double margin = std::numeric_limits<double>::infinity();
  gather_hits(S, px, py, d, brute, hits, &margin);
  std::vector<double> Y(S.K);
  sh_basis(S.deg, d, Y.data());
  double T = 1.0, L[3] = {0, 0, 0};
  out->terminated = 0;
  out->tau_end = std::numeric_limits<double>::infinity();
  out->id_end = -1;
  out->n_included = 0;
  if (comp) comp->clear();
  for (size_t h = 0; h < hits.size(); ++h) {
    const Hit& H = hits[h];
    const Prim& P = S.prims[H.id];
    if (h + 1 < hits.size()) {
      double gap = std::fabs(hits[h + 1].tau - H.tau) / std::max(H.tau, 1e-300);
      if (gap < margin) margin = gap;
    }
    double tm = H.tau / std::sqrt((P.mu[0] - S.o[0]) * (P.mu[0] - S.o[0]) + (P.mu[1] - S.o[1]) * (P.mu[1] - S.o[1]) +
                                  (P.mu[2] - S.o[2]) * (P.mu[2] - S.o[2]));
    if (std::fabs(tm) < margin) margin = std::fabs(tm);
    double alpha = P.sigma * std::exp(-0.5 * H.D2);
    Composited c;
    c.id = H.id;
    c.tau = H.tau;
    c.D2 = H.D2;
    for (int k = 0; k < 3; ++k) c.xg[k] = H.xg[k];
    c.alpha = alpha;
    c.T = T;
    for (int ch = 0; ch < 3; ++ch) {
      c.L[ch] = L[ch];
      c.c[ch] = colour_channel(S, H.id, ch, Y.data(), &c.unclamped[ch]);
    }
    for (int ch = 0; ch < 3; ++ch) L[ch] += T * alpha * c.c[ch];
    T *= (1.0 - alpha);
    out->n_included++;
    if (comp) comp->push_back(c);
    double tmarg = std::fabs(T - S.t_min) / S.t_min;
    if (tmarg < margin) margin = tmarg;
    if (T < S.t_min) {
      out->terminated = 1;
      out->tau_end = H.tau;
      out->id_end = H.id;
      break;
    }
  }
  for (int ch = 0; ch < 3; ++ch) out->C[ch] = L[ch];
  out->margin = margin;
  out->T_final = T;
}

inline void atomic_add(double* p, double v) {
#pragma omp atomic
  *p += v;
}

}  // namespace

extern "C" {

// Build the oracle's scene: per-primitive quantities, rectangles and its own
// candidate buckets.  Camera: x_c = Rc x_w + tc, pinhole (fx, fy, cx, cy).
void* orc_scene_new(int64_t n, int32_t sh_degree, const double* means, const double* log_scales,
                    const double* quats, const double* logits, const double* sh, int32_t width, int32_t height,
                    const double* intrin /*fx fy cx cy*/, const double* Rc, const double* tc, double alpha_min,
                    double t_min) {
  Scene* S = new Scene();
  S->n = n;
  S->deg = sh_degree;
  S->K = (sh_degree + 1) * (sh_degree + 1);
  S->W = width;
  S->H = height;
  S->fx = intrin[0]; S->fy = intrin[1]; S->cx = intrin[2]; S->cy = intrin[3];
  for (int k = 0; k < 9; ++k) S->Rc[k] = Rc[k];
  for (int k = 0; k < 3; ++k) S->tc[k] = tc[k];
  for (int k = 0; k < 3; ++k)  // o = -Rc^T tc
    S->o[k] = -(S->Rc[0 * 3 + k] * S->tc[0] + S->Rc[1 * 3 + k] * S->tc[1] + S->Rc[2 * 3 + k] * S->tc[2]);
  S->alpha_min = alpha_min;
  S->t_min = t_min;
  S->prims.resize(n);
  S->sh.assign(sh, sh + n * S->K * 3);
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) prepare_prim(*S, i, means, log_scales, quats, logits, S->prims[i]);
  build_buckets(*S);
  return S;
}

void orc_scene_free(void* h) { delete static_cast<Scene*>(h); }

// Per-primitive outputs: rect [n,4], area [n], state [n], sigma [n], D2c [n],
// W [n,9], camera-relative Gaussian-space origin o_g = W (o - mu) [n,3].
void orc_prim_info(void* h, int32_t* rect, int64_t* area, int32_t* state, double* sigma, double* D2c, double* Wout,
                   double* og) {
  Scene& S = *static_cast<Scene*>(h);
  for (int64_t i = 0; i < S.n; ++i) {
    const Prim& P = S.prims[i];
    for (int k = 0; k < 4; ++k) rect[4 * i + k] = P.rect[k];
    area[i] = P.area;
    state[i] = P.state;
    sigma[i] = P.sigma;
    D2c[i] = P.D2c;
    for (int k = 0; k < 9; ++k) Wout[9 * i + k] = P.W[k];
    double om[3] = {S.o[0] - P.mu[0], S.o[1] - P.mu[1], S.o[2] - P.mu[2]};
    for (int k = 0; k < 3; ++k) og[3 * i + k] = P.W[3 * k] * om[0] + P.W[3 * k + 1] * om[1] + P.W[3 * k + 2] * om[2];
  }
}

// Real SH basis at a unit direction (exposed for the basis pins).
void orc_sh_basis(int32_t degree, int64_t m, const double* dirs, double* Y) {
  int K = (degree + 1) * (degree + 1);
  for (int64_t j = 0; j < m; ++j) sh_basis(degree, dirs + 3 * j, Y + K * j);
}

// Render the listed pixels (pix = y*W + x; null = all pixels in row-major
// order).  Outputs per listed pixel: colour [3], end marker (tau_end, id_end;
// +inf / -1 if the ray never terminated), number of composited hits, and the
// smallest decision margin met along the ray.
void orc_render(void* h, int64_t npix, const int64_t* pix, int32_t brute, double* color, double* tau_end,
                int64_t* id_end, int64_t* n_included, double* margin, double* T_final) {
  Scene& S = *static_cast<Scene*>(h);
  int64_t total = pix ? npix : int64_t(S.W) * S.H;
#pragma omp parallel
  {
    std::vector<Hit> hits;
#pragma omp for schedule(dynamic, 64)
    for (int64_t j = 0; j < total; ++j) {
      int64_t p = pix ? pix[j] : j;
      PixelResult r;
      render_pixel(S, int(p % S.W), int(p / S.W), brute, &r, hits, nullptr);
      for (int ch = 0; ch < 3; ++ch) color[3 * j + ch] = r.C[ch];
      tau_end[j] = r.tau_end;
      id_end[j] = r.id_end;
      n_included[j] = r.n_included;
      margin[j] = r.margin;
      T_final[j] = r.T_final;
    }
  }
}

// Per-pixel list of every geometric hit (unordered by depth is fine for the
// callers; emitted in depth order).  counts_only=1 fills counts[j];
// otherwise writes hit primitive ids at offsets[j]...
void orc_all_hits(void* h, int64_t npix, const int64_t* pix, int32_t brute, int32_t counts_only, int64_t* counts,
                  const int64_t* offsets, int64_t* prim_out) {
  Scene& S = *static_cast<Scene*>(h);
#pragma omp parallel
  {
    std::vector<Hit> hits;
#pragma omp for schedule(dynamic, 64)
    for (int64_t j = 0; j < npix; ++j) {
      int64_t p = pix[j];
      double d[3];
      pixel_ray(S, int(p % S.W), int(p / S.W), d);
      double margin = 1e300;
      gather_hits(S, int(p % S.W), int(p / S.W), d, brute, hits, &margin);
      if (counts_only) {
        counts[j] = int64_t(hits.size());
      } else {
        for (size_t k = 0; k < hits.size(); ++k) prim_out[offsets[j] + int64_t(k)] = hits[k].id;
      }
    }
  }
}

// Composited-hit records of the listed pixels, in compositing order:
// prim id and the (L.rgb, T) state in front of the hit.  offsets[j] is the
// first record slot of pixel j (from the counts of orc_render).
void orc_records(void* h, int64_t npix, const int64_t* pix, const int64_t* offsets, int64_t* rec_prim,
                 double* rec_LT, double* rec_tau) {
  Scene& S = *static_cast<Scene*>(h);
#pragma omp parallel
  {
    std::vector<Hit> hits;
    std::vector<Composited> comp;
#pragma omp for schedule(dynamic, 64)
    for (int64_t j = 0; j < npix; ++j) {
      int64_t p = pix[j];
      PixelResult r;
      render_pixel(S, int(p % S.W), int(p / S.W), 0, &r, hits, &comp);
      int64_t o = offsets[j];
      for (size_t k = 0; k < comp.size(); ++k) {
        rec_prim[o + k] = comp[k].id;
        rec_LT[4 * (o + k) + 0] = comp[k].L[0];
        rec_LT[4 * (o + k) + 1] = comp[k].L[1];
        rec_LT[4 * (o + k) + 2] = comp[k].L[2];
        rec_LT[4 * (o + k) + 3] = comp[k].T;
        rec_tau[o + k] = comp[k].tau;
      }
    }
  }
}

// Reduced-precision storage of the intermediate buffer (Sec. 6 suggests
// fp16).  The backward reads L and T back from the buffer, so the gradient a
// storage format yields is the plain gradient with L and T replaced by their
// stored values.  Models (each a reading of what the format keeps):
//   0  exact L and T (float T, fixed-point L are exact to ~1e-7)
//   1  L and T each rounded to float, then to the nearest fp16
//   2  T only (hybrid backward), rounded to float then fp16; the colour behind
//      a hit is summed from the later hits with their stored T
//   3  L in 16-bit fixed point with unit B / 2^16 (B = the frame's colour
//      bound), T as the code q = round(-log2(T) 4096), T = 2^(-q / 4096)
//   4  T only (hybrid backward) as the code of model 3, colour behind summed
//      as in model 2
//   5  T only (hybrid backward), T rounded to float, colour behind summed as
//      in model 2
// Rounds x (a float) to the nearest fp16, ties to even (normal and
// subnormal fp16 range; the values stored here are far below its maximum).
double round_half(double x) {
  const double f = double(float(x));
  const double a = std::fabs(f);
  if (a == 0.0) return f;
  double q;  // fp16 spacing at a
  if (a < std::ldexp(1.0, -14)) {
    q = std::ldexp(1.0, -24);
  } else {
    int e;
    std::frexp(a, &e);           // a = m 2^e, m in [0.5, 1)
    q = std::ldexp(1.0, e - 11);  // 11 significant bits
  }
  return std::nearbyint(f / q) * q;  // the default rounding mode is to nearest, ties to even
}

// L in model 3's fixed point with unit q (saturating at 65535 units).
double round_fixed16(double L, double q) { return std::min(std::nearbyint(L / q), 65535.0) * q; }

// T through the 16-bit logarithmic code of model 3.
double round_log16(double T) {
  const double q = std::min(std::nearbyint(-std::log2(double(float(T))) * 4096.0), 65535.0);
  return std::exp2(-q / 4096.0);
}

// The frame's colour bound B (model 3): over every visible Gaussian and
// channel, 1/2 + sum_l sqrt((2l + 1) / (4 pi)) |sh_l| (the largest |colour|
// any direction can give, by Cauchy-Schwarz and the SH addition theorem),
// raised by 2^-16.
double colour_bound(const Scene& S) {
  double B = 0.0;
  for (int64_t i = 0; i < S.n; ++i) {
    if (S.prims[i].state != kActive) continue;
    for (int ch = 0; ch < 3; ++ch) {
      double v = 0.5;
      for (int l = 0; l <= S.deg; ++l) {
        double ss = 0.0;
        for (int m = -l; m <= l; ++m) {
          const double k = S.sh[(i * S.K + l * l + l + m) * 3 + ch];
          ss += k * k;
        }
        v += std::sqrt(ss * (2.0 * l + 1.0) / (4.0 * kPi));
      }
      B = std::max(B, v);
    }
  }
  return (B > 0.0 ? B : 1.0) * (1.0 + std::ldexp(1.0, -16));
}

// Gradient of L = sum_p <dL/dC_p, C_p> over the listed pixels (null = all),
// with respect to the raw parameters: means, log-scales, the unnormalised
// quaternion, opacity logits and SH coefficients.  Outputs are overwritten.
//
// Per composited hit i of a pixel (pixel-centric, Sec. 3.5), with g = dL/dC,
// S_i = colour composited behind hit i:
//   dL/dc_i      = T_i alpha_i g            (zero on a clamped channel)
//   dL/dalpha_i  = <g, T_i c_i - S_i / (1 - alpha_i)>
//   dL/dsigma_i += dL/dalpha_i * rho_i
//   dL/dD2       = -alpha_i / 2 * dL/dalpha_i
// and, since D2 is minimal over tau at tau_max (so dD2/dtau = 0 there),
//   dD2/do_g = 2 x_g,  dD2/dd_g = 2 tau x_g,
//   dL/dW  += dL/do_g (o - mu)^T + dL/dd_g d^T,   dL/dmu += -W^T dL/do_g.
// Per primitive: W = S^-1 R^T gives dL/dlog s_k = -sum_j dW_kj W_kj and
// dL/dR_jk = dW_kj / s_k; the quaternion gradient goes through R(q/|q|).
void orc_backward_stored(void* h, int64_t npix, const int64_t* pix, const double* dl_dimage, double* g_means,
                         double* g_log_scales, double* g_quats, double* g_logits, double* g_sh, int32_t model) {
  Scene& S = *static_cast<Scene*>(h);
  const double lq = model == 3 ? colour_bound(S) * std::ldexp(1.0, -16) : 1.0;  // model 3 unit of L
  const int64_t n = S.n;
  const int K = S.K;
  std::vector<double> accW(n * 9, 0.0), accMu(n * 3, 0.0), accSig(n, 0.0), accSh(n * K * 3, 0.0);
  int64_t total = pix ? npix : int64_t(S.W) * S.H;
#pragma omp parallel
  {
    std::vector<Hit> hits;
    std::vector<Composited> comp;
    std::vector<double> Y(K);
#pragma omp for schedule(dynamic, 64)
    for (int64_t j = 0; j < total; ++j) {
      int64_t p = pix ? pix[j] : j;
      int px = int(p % S.W), py = int(p / S.W);
      PixelResult r;
      render_pixel(S, px, py, 0, &r, hits, &comp);
      if (comp.empty()) continue;
      double d[3];
      pixel_ray(S, px, py, d);
      sh_basis(S.deg, d, Y.data());
      double g[3] = {dl_dimage[3 * p], dl_dimage[3 * p + 1], dl_dimage[3 * p + 2]};
      // stored T of each hit and, for the T-only models, the colour behind
      // each hit summed from the later hits (back to front)
      const size_t nc = comp.size();
      std::vector<double> Ts(nc), walk(3 * (nc + 1), 0.0);
      for (size_t k = 0; k < nc; ++k) {
        const double T = comp[k].T;
        Ts[k] = (model == 1 || model == 2) ? round_half(T)
                : (model == 3 || model == 4) ? round_log16(T)
                : model == 5                 ? double(float(T))
                                             : T;
      }
      for (size_t k = nc; k-- > 0;)
        for (int ch = 0; ch < 3; ++ch)
          walk[3 * k + ch] = walk[3 * (k + 1) + ch] + Ts[k] * comp[k].alpha * comp[k].c[ch];
      for (size_t k = 0; k < nc; ++k) {
        const Composited& c = comp[k];
        const Prim& P = S.prims[c.id];
        const double Tst = Ts[k];
        double behind[3], dLdalpha = 0.0;
        for (int ch = 0; ch < 3; ++ch) {
          if (model == 2 || model == 4 || model == 5) {
            behind[ch] = walk[3 * (k + 1) + ch];
          } else {
            double L = c.L[ch];
            if (model == 1) L = round_half(L);
            if (model == 3) L = round_fixed16(L, lq);
            behind[ch] = r.C[ch] - L - Tst * c.alpha * c.c[ch];
          }
          dLdalpha += g[ch] * (Tst * c.c[ch] - behind[ch] / (1.0 - c.alpha));
        }
        for (int ch = 0; ch < 3; ++ch) {
          if (!c.unclamped[ch]) continue;
          double dc = Tst * c.alpha * g[ch];
          for (int k = 0; k < K; ++k) atomic_add(&accSh[(c.id * K + k) * 3 + ch], dc * Y[k]);
        }
        double rho = std::exp(-0.5 * c.D2);
        atomic_add(&accSig[c.id], dLdalpha * rho);
        double dLdD2 = -0.5 * c.alpha * dLdalpha;
        double dog[3], ddg[3];
        for (int k = 0; k < 3; ++k) {
          dog[k] = dLdD2 * 2.0 * c.xg[k];
          ddg[k] = dLdD2 * 2.0 * c.tau * c.xg[k];
        }
        double om[3] = {S.o[0] - P.mu[0], S.o[1] - P.mu[1], S.o[2] - P.mu[2]};
        for (int a = 0; a < 3; ++a)
          for (int b = 0; b < 3; ++b) atomic_add(&accW[c.id * 9 + 3 * a + b], dog[a] * om[b] + ddg[a] * d[b]);
        for (int b = 0; b < 3; ++b) {
          double v = 0;
          for (int a = 0; a < 3; ++a) v += P.W[3 * a + b] * dog[a];
          atomic_add(&accMu[c.id * 3 + b], -v);
        }
      }
    }
  }
#pragma omp parallel for schedule(static)
  for (int64_t i = 0; i < n; ++i) {
    const Prim& P = S.prims[i];
    if (P.state != kActive) {
      // A culled Gaussian (R2; non-finite parameters) meets no ray, so every
      // gradient of it is zero; the chain rule is not evaluated through
      // parameters that may be non-finite.
      for (int k = 0; k < 3; ++k) g_means[3 * i + k] = g_log_scales[3 * i + k] = 0.0;
      for (int k = 0; k < 4; ++k) g_quats[4 * i + k] = 0.0;
      g_logits[i] = 0.0;
      for (int k = 0; k < K * 3; ++k) g_sh[i * K * 3 + k] = 0.0;
      continue;
    }
    const double* dW = &accW[9 * i];
    for (int k = 0; k < 3; ++k) g_means[3 * i + k] = accMu[3 * i + k];
    for (int k = 0; k < 3; ++k) {
      double v = 0;
      for (int j = 0; j < 3; ++j) v += dW[3 * k + j] * P.W[3 * k + j];
      g_log_scales[3 * i + k] = -v;
    }
    double dR[9];
    for (int jj = 0; jj < 3; ++jj)
      for (int k = 0; k < 3; ++k) dR[3 * jj + k] = dW[3 * k + jj] / P.s[k];
    double dRdq[4][9];
    quat_to_rot_jacobian(P.qn, dRdq);
    double dqn[4];
    for (int c = 0; c < 4; ++c) {
      double v = 0;
      for (int e = 0; e < 9; ++e) v += dRdq[c][e] * dR[e];
      dqn[c] = v;
    }
    double proj = 0;
    for (int c = 0; c < 4; ++c) proj += P.qn[c] * dqn[c];
    for (int c = 0; c < 4; ++c) g_quats[4 * i + c] = (dqn[c] - P.qn[c] * proj) / P.qnorm;
    g_logits[i] = P.sigma * (1.0 - P.sigma) * accSig[i];
    for (int k = 0; k < K * 3; ++k) g_sh[i * K * 3 + k] = accSh[i * K * 3 + k];
  }
}

void orc_backward(void* h, int64_t npix, const int64_t* pix, const double* dl_dimage, double* g_means,
                  double* g_log_scales, double* g_quats, double* g_logits, double* g_sh) {
  orc_backward_stored(h, npix, pix, dl_dimage, g_means, g_log_scales, g_quats, g_logits, g_sh, 0);
}

// A stored value's rounding applied to m values (for the pins): kind 1 the
// fp16 of model 1, 2 model 3's L with unit q, 3 model 3's T.
void orc_storage_round(int32_t kind, int64_t m, const double* x, double* out, double q) {
  for (int64_t k = 0; k < m; ++k)
    out[k] = kind == 1 ? round_half(x[k]) : kind == 2 ? round_fixed16(x[k], q) : round_log16(x[k]);
}

// The colour bound B of model 3.
double orc_colour_bound(void* h) { return colour_bound(*static_cast<Scene*>(h)); }

// Intermediate-buffer address idx(i, t, p) = O_prim(i) + O_tile(i, t) +
// O_pixel(i, t, p) (Eq. 16, Sec. 4.3), by plain counting:
//   O_prim  = sum of the rectangle areas of primitives 0..i-1;
//   O_tile  = pixels of rect_i inside the tiles that precede tile t, tiles of
//             the rectangle's tile range taken in row-major order;
//   O_pixel = row-major rank of pixel p among the pixels of rect_i inside t.
// Returns -1 for a pixel outside the primitive's rectangle.
void orc_lt_index(void* h, int32_t tile, int64_t m, const int64_t* prim, const int64_t* pixel, int64_t* idx) {
  Scene& S = *static_cast<Scene*>(h);
  std::vector<int64_t> base(S.n + 1, 0);
  for (int64_t i = 0; i < S.n; ++i) base[i + 1] = base[i] + S.prims[i].area;
#pragma omp parallel for schedule(dynamic, 256)
  for (int64_t j = 0; j < m; ++j) {
    int64_t i = prim[j];
    const Prim& P = S.prims[i];
    int px = int(pixel[j] % S.W), py = int(pixel[j] / S.W);
    if (P.area == 0 || px < P.rect[0] || px > P.rect[2] || py < P.rect[1] || py > P.rect[3]) {
      idx[j] = -1;
      continue;
    }
    int ttx = px / tile, tty = py / tile;
    int64_t before = 0;
    // Tiles of the rectangle's range in row-major order, up to tile (ttx, tty).
    for (int ty = P.rect[1] / tile; ty <= P.rect[3] / tile; ++ty) {
      for (int tx = P.rect[0] / tile; tx <= P.rect[2] / tile; ++tx) {
        int xa = std::max(P.rect[0], tx * tile), xb = std::min(P.rect[2], tx * tile + tile - 1);
        int ya = std::max(P.rect[1], ty * tile), yb = std::min(P.rect[3], ty * tile + tile - 1);
        if (tx == ttx && ty == tty) {
          // Row-major rank inside this tile's part of the rectangle.
          int64_t rank = 0;
          for (int y = ya; y <= yb; ++y)
            for (int x = xa; x <= xb; ++x) {
              if (x == px && y == py) goto found;
              ++rank;
            }
        found:
          idx[j] = base[i] + before + rank;
          goto next;
        }
        before += int64_t(xb - xa + 1) * int64_t(yb - ya + 1);
      }
    }
    idx[j] = -1;
  next:;
  }
}

// Raw projected-bound quantities per primitive: (Q_xx, Q_x4, Q_yy, Q_y4, Q_44).
// For an ellipsoid in front of the eye plane the centre and half-width of the
// screen interval are p = Q_a4 / Q_44, h = sqrt(p^2 - Q_aa / Q_44) (Eq. 12-14).
void orc_bounds_raw(void* h, double* out) {
  Scene& S = *static_cast<Scene*>(h);
  for (int64_t i = 0; i < S.n; ++i) {
    const Prim& P = S.prims[i];
    out[5 * i + 0] = P.Qx[0];
    out[5 * i + 1] = P.Qx[1];
    out[5 * i + 2] = P.Qy[0];
    out[5 * i + 3] = P.Qy[1];
    out[5 * i + 4] = P.q44;
  }
}

// Ray/primitive queries: for each (pixel, prim) the max-response depth tau,
// the squared normalised distance D2 there, the hit decision and alpha.
void orc_ray_prim(void* h, int64_t m, const int64_t* pixel, const int64_t* prim, double* tau, double* D2,
                  int32_t* hit, double* alpha, double* dir) {
  Scene& S = *static_cast<Scene*>(h);
  for (int64_t j = 0; j < m; ++j) {
    int64_t p = pixel[j];
    double d[3];
    pixel_ray(S, int(p % S.W), int(p / S.W), d);
    const Prim& P = S.prims[prim[j]];
    Hit hh;
    hit[j] = ray_gaussian(S, P, d, &hh) && P.state != kCulledOpacity && P.state != kCulledNonFinite;
    tau[j] = hh.tau;
    D2[j] = hh.D2;
    alpha[j] = P.sigma * std::exp(-0.5 * hh.D2);
    for (int k = 0; k < 3; ++k) dir[3 * j + k] = d[k];
  }
}

void orc_camera_origin(void* h, double* o) {
  Scene& S = *static_cast<Scene*>(h);
  for (int k = 0; k < 3; ++k) o[k] = S.o[k];
}

int32_t orc_num_threads() {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

}  // extern "C"
