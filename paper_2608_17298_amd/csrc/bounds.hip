// Per-Gaussian pre-processing and the tile-primitive map.
//
// bounds_kernel: one thread per Gaussian, fp64.  Rotation from the
// normalised quaternion, scales, opacity, clamp radius alpha_c (Sec. 3.4,
// Eq. 9-10), the world-to-Gaussian map W = S^-1 R^T and o_g = W (o - mu)
// (Eq. 5, "w2g" pre-computation of Sec. 5.3), and the conservative pixel
// rectangle from the projected dual quadric (Sec. 4.2, Eq. 11-14).
//
// Tile map (Sec. 4.3, reverse tile mapping): pairs are emitted in order of
// a per-Gaussian depth lower bound so that, after the stable sort by tile
// id, every tile's list is ordered front to back.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "ops.h"

namespace gart {
namespace {

constexpr double kRectPad = 1e-4;  // pixels added on each side of a rectangle

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Pixel index range [lo, hi] covered on one image axis.  The plane through
// the camera containing the pixel line u (clip-space X - u w = 0) meets the
// ellipsoid iff q(u) = Qaa - 2 u Qa4 + u^2 Q44 >= 0.  With Q44 < 0 (the eye
// plane misses the ellipsoid) that is u in [p - h, p + h], p = Qa4 / Q44,
// h = sqrt(p^2 - Qaa / Q44) (Eq. 12-14).  With Q44 >= 0 the ellipsoid crosses
// the eye plane: the covered set is u <= u1 or u >= u2 (or all u), and the
// range is the hull of the covered pixel centres.
__device__ bool axis_cover(double Qaa, double Qa4, double Q44, int npix, int* lo, int* hi) {
  const double e = kRectPad;
  const double last = double(npix - 1);
  double a, b;
  if (Q44 < 0.0) {
    const double p = Qa4 / Q44;
    const double h = sqrt(fmax(0.0, p * p - Qaa / Q44));
    a = fmax(ceil(p - h - 0.5 - e), 0.0);
    b = fmin(floor(p + h - 0.5 + e), last);
  } else if (Q44 == 0.0) {
    if (Qa4 == 0.0) {
      if (!(Qaa >= 0.0)) return false;
      a = 0.0;
      b = last;
    } else {
      const double r = Qaa / (2.0 * Qa4);
      if (Qa4 > 0.0) {
        a = 0.0;
        b = fmin(floor(r - 0.5 + e), last);
      } else {
        a = fmax(ceil(r - 0.5 - e), 0.0);
        b = last;
      }
    }
  } else {
    const double disc = Qa4 * Qa4 - Q44 * Qaa;
    if (disc <= 0.0) {
      a = 0.0;
      b = last;
    } else {
      const double sq = sqrt(disc);
      const double u1 = (Qa4 - sq) / Q44, u2 = (Qa4 + sq) / Q44;
      const bool left = (u1 - 0.5 + e) >= 0.0;
      const bool right = (u2 - 0.5 - e) <= last;
      if (!left && !right) return false;
      a = left ? 0.0 : fmax(ceil(u2 - 0.5 - e), 0.0);
      b = right ? last : fmin(floor(u1 - 0.5 + e), last);
    }
  }
  if (a > b) return false;
  *lo = int(a);
  *hi = int(b);
  return true;
}

template <int K>
__global__ __launch_bounds__(kBoundsBlock) void bounds_kernel(BoundsArgs A) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  uint32_t my_tiles = 0;
  float my_cb = 0.0f;
  if (i < A.n) {
    const CamParams& c = A.cam;
    float mf[3], lf[3], qf[4];
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      mf[k] = A.means[3 * i + k];
      lf[k] = A.log_scales[3 * i + k];
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) qf[k] = A.quats[4 * i + k];
    const float lg = A.logits[i];
    bool ok = isfinite(lg);
#pragma unroll
    for (int k = 0; k < 3; ++k) ok = ok && isfinite(mf[k]) && isfinite(lf[k]);
#pragma unroll
    for (int k = 0; k < 4; ++k) ok = ok && isfinite(qf[k]);
    const double qw = qf[0], qx = qf[1], qy = qf[2], qz = qf[3];
    const double qq = qw * qw + qx * qx + qy * qy + qz * qz;
    ok = ok && qq > 0.0;
    const double sigma = 1.0 / (1.0 + exp(-double(lg)));
    ok = ok && sigma > A.alpha_min;

    double* G = A.geom + kGeomStride * i;
    int rx0 = 0, ry0 = 0, rx1 = -1, ry1 = -1;

    if (ok) {
      const double inv = 1.0 / sqrt(qq);
      const double w = qw * inv, x = qx * inv, y = qy * inv, z = qz * inv;
      // R(q), row-major
      const double R[9] = {1.0 - 2.0 * (y * y + z * z), 2.0 * (x * y - w * z), 2.0 * (x * z + w * y),
                           2.0 * (x * y + w * z), 1.0 - 2.0 * (x * x + z * z), 2.0 * (y * z - w * x),
                           2.0 * (x * z - w * y), 2.0 * (y * z + w * x), 1.0 - 2.0 * (x * x + y * y)};
      const double s[3] = {exp(double(lf[0])), exp(double(lf[1])), exp(double(lf[2]))};
      const double mu[3] = {mf[0], mf[1], mf[2]};
      const double D2c = 2.0 * log(sigma / A.alpha_min);
      const double ac = sqrt(D2c);

      // Projected transform rows T'_a = V_a [R S alpha_c | mu] for the X, Y
      // and w rows of the pixel-clip matrix, and the dual-quadric entries
      // <v, T'_a . T'_b>, v = (1, 1, 1, -1).
      double Tp[3][4];
      const double* V[3] = {c.V0, c.V1, c.V3};
#pragma unroll
      for (int a = 0; a < 3; ++a) {
#pragma unroll
        for (int k = 0; k < 3; ++k)
          Tp[a][k] = (V[a][0] * R[k] + V[a][1] * R[3 + k] + V[a][2] * R[6 + k]) * (s[k] * ac);
        Tp[a][3] = V[a][0] * mu[0] + V[a][1] * mu[1] + V[a][2] * mu[2] + V[a][3];
      }
      auto Q = [&](int a, int b) {
        return Tp[a][0] * Tp[b][0] + Tp[a][1] * Tp[b][1] + Tp[a][2] * Tp[b][2] - Tp[a][3] * Tp[b][3];
      };
      const double Q44 = Q(2, 2);
      const bool behind = Q44 < 0.0 && Tp[2][3] <= 0.0;
      bool vis = !behind;
      if (vis) vis = axis_cover(Q(0, 0), Q(0, 2), Q44, c.W, &rx0, &rx1);
      if (vis) vis = axis_cover(Q(1, 1), Q(1, 2), Q44, c.H, &ry0, &ry1);
      if (vis) {
        // W = S^-1 R^T, o_g = W (o - mu)
        const double om[3] = {c.o[0] - mu[0], c.o[1] - mu[1], c.o[2] - mu[2]};
#pragma unroll
        for (int k = 0; k < 3; ++k) {
          const double is = 1.0 / s[k];
          const double w0 = R[k] * is, w1 = R[3 + k] * is, w2 = R[6 + k] * is;
          G[kGeoW + 3 * k + 0] = w0;
          G[kGeoW + 3 * k + 1] = w1;
          G[kGeoW + 3 * k + 2] = w2;
          G[kGeoOg + k] = w0 * om[0] + w1 * om[1] + w2 * om[2];
        }
        G[kGeoD2c] = D2c;
        G[kGeoSigma] = sigma;
        G[kGeoOneMinusSigma] = 1.0 / (1.0 + exp(double(lg)));  // 1 - sigma without cancellation
        // Lower bound on the depth tau of any hit.  The max-response point
        // x = o + tau d lies in the clamped ellipsoid, hence within r =
        // alpha_c max(s) of mu, so tau >= |mu - o| - r.  Tighter: x is the
        // midpoint of the ray's chord, so y = x - mu lies on the diametral
        // plane conjugate to d (y^T Sigma^-1 d = 0) with y^T Sigma^-1 y <=
        // alpha_c^2, which gives |y.d| <= alpha_c sqrt(d^T Sigma d -
        // 1/(d^T Sigma^-1 d)); and (mu - o).d >= sqrt(|mu-o|^2 - r^2) since
        // the ray passes within r of mu.  Over directions d within the angle
        // th = asin(r/|mu-o|) of u = (mu - o)/|mu - o|:
        //   |S R^T d| <= |S R^T u| + s_max th,  |S^-1 R^T d| <= |S^-1 R^T u| + th / s_min.
        const double dist = sqrt(om[0] * om[0] + om[1] * om[1] + om[2] * om[2]);
        const double smax = fmax(s[0], fmax(s[1], s[2])), smin = fmin(s[0], fmin(s[1], s[2]));
        const double r = ac * smax;
        double lo = dist - r;
        if (dist > r) {
          const double th = asin(r / dist);
          double a1 = 0.0, a2 = 0.0;
#pragma unroll
          for (int k = 0; k < 3; ++k) {
            const double ck = -(R[k] * om[0] + R[3 + k] * om[1] + R[6 + k] * om[2]) / dist;  // (R^T u)_k
            a1 += ck * ck * s[k] * s[k];
            a2 += ck * ck / (s[k] * s[k]);
          }
          const double p = sqrt(a1) + smax * th, q = sqrt(a2) + th / smin;
          const double hb = sqrt(fmax(0.0, p * p - 1.0 / (q * q)));
          lo = fmax(lo, sqrt(dist * dist - r * r) - ac * hb);
        }
        lo -= 1e-12 * (dist + r);
        G[kGeoKey] = lo > 0.0 ? lo : 0.0;
        const int ts = A.tile;
        my_tiles = uint32_t(rx1 / ts - rx0 / ts + 1) * uint32_t(ry1 / ts - ry0 / ts + 1);
      } else {
        rx0 = ry0 = 0;
        rx1 = ry1 = -1;
      }
    }
    if (my_tiles == 0) {
#pragma unroll
      for (int k = 0; k < kGeomStride; ++k) G[k] = 0.0;
      G[kGeoD2c] = -1.0;  // no ray can pass the hit test
      G[kGeoKey] = double(__int_as_float(0x7f800000));
      rx0 = ry0 = 0;
      rx1 = ry1 = -1;
    }
    A.rect[4 * i + 0] = rx0;
    A.rect[4 * i + 1] = ry0;
    A.rect[4 * i + 2] = rx1;
    A.rect[4 * i + 3] = ry1;
    A.area[i] = my_tiles ? int64_t(rx1 - rx0 + 1) * int64_t(ry1 - ry0 + 1) : 0;
    A.tile_count[i] = my_tiles;
    if (my_tiles) {
      // Colour bound over all directions: per band l, |sum_m sh_lm Y_lm| <=
      // |sh_l| sqrt((2l+1)/(4 pi)) (Cauchy-Schwarz and the addition theorem).
      // fp32 with a margin of 2^-16 (far above the rounding of this sum and
      // of the forward's fp32 colour); the fixed-point conversion saturates
      // in any case.
      // all 3K coefficients are loaded before use (wide loads, each line
      // fetched once)
      const float* sp = A.sh + int64_t(3 * K) * i;
      float c[3 * K];
#pragma unroll
      for (int k = 0; k < 3 * K; ++k) c[k] = sp[k];
      float ss[4][3] = {};
      constexpr int kBand[16] = {0, 1, 1, 1, 2, 2, 2, 2, 2, 3, 3, 3, 3, 3, 3, 3};
#pragma unroll
      for (int k = 0; k < K; ++k)
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) ss[kBand[k]][ch] = fmaf(c[3 * k + ch], c[3 * k + ch], ss[kBand[k]][ch]);
      float cb = 0.0f;
#pragma unroll
      for (int ch = 0; ch < 3; ++ch) {
        float v = 0.5f;
#pragma unroll
        for (int l = 0; l < 4; ++l) v += sqrtf(ss[l][ch] * (float(2 * l + 1) * 0.07957747154594767f));
        cb = fmaxf(cb, v);
      }
      my_cb = cb * (1.0f + 1.0f / 65536.0f);
      if (!(my_cb >= 0.0f && my_cb < 1e30f)) my_cb = 1e30f;  // non-finite SH: saturate
    }
  }
  // block sum of tile counts and max of colour bounds -> one partial per block
  __shared__ unsigned long long s_t[kBoundsBlock / 64];
  __shared__ float s_cb[kBoundsBlock / 64];
  unsigned long long t = my_tiles;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    t += __shfl_xor(t, off);
    my_cb = fmaxf(my_cb, __shfl_xor(my_cb, off));
  }
  if (__lane_id() == 0) {
    s_t[threadIdx.x / 64] = t;
    s_cb[threadIdx.x / 64] = my_cb;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < kBoundsBlock / 64; ++w) {
      t += s_t[w];
      my_cb = fmaxf(my_cb, s_cb[w]);
    }
    A.block_partial[2 * blockIdx.x] = t;
    A.block_partial[2 * blockIdx.x + 1] = __float_as_uint(my_cb);
  }
}

__global__ __launch_bounds__(256) void bounds_totals_kernel(const unsigned long long* __restrict__ part, int64_t nb,
                                                            const int64_t* __restrict__ area_total,
                                                            unsigned long long* __restrict__ totals) {
  __shared__ unsigned long long s_t[4];
  __shared__ float s_cb[4];
  unsigned long long t = 0;
  float cb = 0.0f;
  for (int64_t b = threadIdx.x; b < nb; b += 256) {
    t += part[2 * b];
    cb = fmaxf(cb, __uint_as_float(uint32_t(part[2 * b + 1])));
  }
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) {
    t += __shfl_xor(t, off);
    cb = fmaxf(cb, __shfl_xor(cb, off));
  }
  if (__lane_id() == 0) {
    s_t[threadIdx.x / 64] = t;
    s_cb[threadIdx.x / 64] = cb;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    for (int w = 1; w < 4; ++w) {
      t += s_t[w];
      cb = fmaxf(cb, s_cb[w]);
    }
    totals[0] = static_cast<unsigned long long>(*area_total);
    totals[1] = t;
    totals[2] = __float_as_uint(cb);
  }
}

// Depth bound <-> `bits`-bit code: the float at or below the bound, cut to
// the 32 binary exponents of [2^-12, 2^20) (5 bits) and the leading
// bits - 5 mantissa bits.  The code is monotone in the bound (the bits of a
// positive float are), saturates above 2^20, is 0 below 2^-12 and for fewer
// than 6 bits, and its value (code 0 stands for 0) never exceeds the bound.
__device__ __forceinline__ uint32_t depth_code(double x, int bits) {
  if (bits < 6) return 0u;
  const float f = __double2float_rd(x);
  if (!(f >= 0x1p-12f)) return 0u;
  const int m = bits - 5;
  const uint32_t u = __float_as_uint(f);
  const uint32_t e = (u >> 23) - (127u - 12u);
  if (e >= 32u) return (1u << bits) - 1u;
  return (e << m) | ((u & 0x7fffffu) >> (23 - m));
}
__device__ __forceinline__ float depth_code_value(uint32_t c, int bits) {
  if (c == 0 || bits < 6) return 0.0f;
  const int m = bits - 5;
  return __uint_as_float((((c >> m) + 127u - 12u) << 23) | ((c & ((1u << m) - 1u)) << (23 - m)));
}

// One block emits the pairs of 256 consecutive Gaussians (index order); its
// threads stride over the block's pair slots and find their Gaussian by
// binary search over first slots held in LDS.  Each pair gets a lower bound on
// the depth tau (Eq. 3) of its Gaussian's max-response point (Eq. 4-5) along
// the pixel-centre rays of its tile that lie in the Gaussian's rectangle,
// measured relative to the tile: the key is min over those rays q of
// tau_q / s_q with s_q = |R^T u_q| / (c . u_q), where u_q = (a, b, 1) is the
// camera ray of pixel q, a = (x + 1/2 - cx)/fx, b = (y + 1/2 - cy)/fy, and c
// is the unit direction through the tile's centre (tile_axis).  s_q exceeds 1
// by under 2e-5 on an 8x8 tile, and each kernel scales a key by its own
// pixel's s to bound that pixel's tau.  tau_q / s_q is the depth along c of
// the max-response point: with u' = u / (c . u), tau / s = N(u') / D(u'),
// N(u) = -o_g . P u, D(u) = |P u|^2, P = W R^T (the world ray R^T u has
// length |R^T u|, which cancels).  The pixel rectangle maps to a convex quadrilateral
// of u' whose vertices are its four corner rays; N is linear and D a convex
// quadratic on it, so for t >= 0 N - t D is concave and its minimum lies at a
// vertex: the smallest N / D over the four corners is the exact minimum over
// the tile's rays.  The key is that minimum less 1e-12 relative (the forward
// evaluates tau another way), and at least the Gaussian's own bound on tau
// divided by the largest corner s; a hit needs tau > 0.
constexpr int kEmitGaussians = 256;

__global__ __launch_bounds__(256) void emit_pairs_kernel(TileMapArgs A) {
  __shared__ uint32_t s_base[kEmitGaussians + 1];  // first pair slot, relative to the block's first
  __shared__ int32_t s_tile[kEmitGaussians][3];     // first tile column, first tile row, tile columns
  __shared__ double s_q[kEmitGaussians][10];  // M (m00 m01 m02 m11 m12 m22), n (3), the Gaussian's bound
  const int64_t i0 = int64_t(blockIdx.x) * kEmitGaussians;
  const int nr = int(std::min<int64_t>(kEmitGaussians, A.n - i0));
  const int ts = A.tile;
  const int64_t first = A.pair_offset[i0];
  for (int k = threadIdx.x; k <= nr; k += blockDim.x) s_base[k] = uint32_t(A.pair_offset[i0 + k] - first);
  for (int k = threadIdx.x; k < nr; k += blockDim.x) {
    const int64_t i = i0 + k;
    if (A.tile_count[i] == 0) continue;
    const int tx0 = A.rect[4 * i] / ts;
    s_tile[k][0] = tx0;
    s_tile[k][1] = A.rect[4 * i + 1] / ts;
    s_tile[k][2] = A.rect[4 * i + 2] / ts - tx0 + 1;
    const double* G = A.geom + int64_t(kGeomStride) * i;
    // P = W Rt maps (a, b, 1) to d_g = W d (Rt: camera -> world)
    double P[9];
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
      for (int c = 0; c < 3; ++c)
        P[3 * r + c] = fma(G[kGeoW + 3 * r], A.cam.Rt[c],
                           fma(G[kGeoW + 3 * r + 1], A.cam.Rt[3 + c], G[kGeoW + 3 * r + 2] * A.cam.Rt[6 + c]));
    auto m = [&](int a, int b) { return fma(P[a], P[b], fma(P[3 + a], P[3 + b], P[6 + a] * P[6 + b])); };
    s_q[k][0] = m(0, 0);
    s_q[k][1] = m(0, 1);
    s_q[k][2] = m(0, 2);
    s_q[k][3] = m(1, 1);
    s_q[k][4] = m(1, 2);
    s_q[k][5] = m(2, 2);
    // n = P^T W (mu - o) = -P^T o_g
#pragma unroll
    for (int a = 0; a < 3; ++a)
      s_q[k][6 + a] = -fma(P[a], G[kGeoOg], fma(P[3 + a], G[kGeoOg + 1], P[6 + a] * G[kGeoOg + 2]));
    s_q[k][9] = G[kGeoKey];
  }
  __syncthreads();
  const uint32_t count = s_base[nr];
  for (uint32_t jr = threadIdx.x; jr < count; jr += blockDim.x) {
    int lo = 0, hi = nr - 1;  // largest k with s_base[k] <= jr
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (s_base[mid] <= jr) lo = mid; else hi = mid - 1;
    }
    const int k = lo;
    const uint32_t q = jr - s_base[k];
    const uint32_t ntx = uint32_t(s_tile[k][2]);
    const uint32_t row = q / ntx;
    const int tx = s_tile[k][0] + int(q - row * ntx), ty = s_tile[k][1] + int(row);
    const int64_t j = first + jr;
    // corners of the pixel-centre rectangle of rect cap tile, depths along
    // the tile's axis c (camera coordinates by the reciprocal focal lengths:
    // within an ulp of the pixel rays' quotients, inside the margin below)
    const int32_t* rc = A.rect + 4 * (i0 + k);
    const double ax[2] = {(double(max(rc[0], tx * ts)) + 0.5 - A.cam.cx) * A.cam.ifx,
                          (double(min(rc[2], tx * ts + ts - 1)) + 0.5 - A.cam.cx) * A.cam.ifx};
    const double by[2] = {(double(max(rc[1], ty * ts)) + 0.5 - A.cam.cy) * A.cam.ify,
                          (double(min(rc[3], ty * ts + ts - 1)) + 0.5 - A.cam.cy) * A.cam.ify};
    double cax[3];
    tile_axis(A.cam, tx, ty, ts, cax);
    const double* Q = s_q[k];
    // The corner with the smallest N (c . u) / D and the one with the
    // largest s = |R^T u| / (c . u) are chosen by cross-multiplied
    // comparisons (D, c . u > 0), so that one division (and one square root)
    // per pair forms each value; a choice off by rounding moves the value by
    // about 1e-16 relative, inside the 1e-12 margin below.
    double kn = 0.0, kd = 1.0, sw = 0.0, sc = 1.0;  // kmin = kn / kd, smax^2 = sw / sc^2
#pragma unroll
    for (int corner = 0; corner < 4; ++corner) {
      const double a = ax[corner & 1], b = by[corner >> 1];
      const double N = fma(Q[6], a, fma(Q[7], b, Q[8]));
      const double D = fma(a, fma(Q[0], a, 2.0 * fma(Q[1], b, Q[2])), fma(b, fma(Q[3], b, 2.0 * Q[4]), Q[5]));
      const double cu = fma(cax[0], a, fma(cax[1], b, cax[2]));  // c . u
      const double nc = N * cu;
      if (corner == 0 || nc * kd < kn * D) {
        kn = nc;
        kd = D;
      }
      double w2 = 0.0;  // |R^T u|^2
#pragma unroll
      for (int r = 0; r < 3; ++r) {
        const double wr = fma(A.cam.Rt[3 * r], a, fma(A.cam.Rt[3 * r + 1], b, A.cam.Rt[3 * r + 2]));
        w2 = fma(wr, wr, w2);
      }
      if (corner == 0 || w2 * (sc * sc) > sw * (cu * cu)) {
        sw = w2;
        sc = cu;
      }
    }
    const double kmin = kn / kd;
    const double tk = kmin > 0.0 ? kmin - 1e-12 * kmin : 0.0;
    const double own = Q[9] * sc / sqrt(sw) * (1.0 - 1e-12);
    const double bound = fmax(own, tk);
    A.keys[j] = (uint32_t(ty * A.tiles_x + tx) << A.key_bits) | depth_code(bound, A.key_bits);
    A.vals[j] = uint32_t(i0 + k);
  }
}

// One thread per sorted pair j, plus one for the end: splits the combined key
// into the tile id and the decoded depth bound, and sets tile_range[t] = j for
// every tile t after the previous pair's tile up to this pair's.
__global__ void finish_pairs_kernel(TileMapArgs A, const uint32_t* __restrict__ sorted, int64_t n_tiles) {
  const int64_t j = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  const int64_t m = A.pair_count;
  if (j > m) return;
  const int64_t prev = (j == 0) ? -1 : int64_t(sorted[j - 1] >> A.key_bits);
  int64_t cur = n_tiles;
  if (j < m) {
    const uint32_t key = sorted[j];
    cur = int64_t(key >> A.key_bits);
    A.keys[j] = uint32_t(cur);
    A.pair_key[j] = depth_code_value(key & ((1u << A.key_bits) - 1u), A.key_bits);
  }
  for (int64_t t = prev + 1; t <= cur && t <= n_tiles; ++t) A.tile_range[t] = j;
}

__global__ void hit_rows_kernel(const int64_t* __restrict__ tile_range, int64_t n_tiles, int64_t cap,
                                int64_t* __restrict__ rows) {
  const int64_t t = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (t < n_tiles) rows[t] = min(tile_range[t + 1] - tile_range[t], cap);
}

}  // namespace

hipError_t launch_hit_rows(const int64_t* tile_range, int64_t n_tiles, int64_t cap, int64_t* rows, hipStream_t s) {
  if (n_tiles <= 0) return hipSuccess;
  hit_rows_kernel<<<ceil_div(n_tiles, 256), 256, 0, s>>>(tile_range, n_tiles, cap, rows);
  return hipGetLastError();
}

hipError_t launch_bounds(const BoundsArgs& a, hipStream_t s) {
  if (a.n <= 0) return hipSuccess;
  const int64_t nb = ceil_div(a.n, kBoundsBlock);
  switch (a.K) {
    case 1: bounds_kernel<1><<<nb, kBoundsBlock, 0, s>>>(a); break;
    case 4: bounds_kernel<4><<<nb, kBoundsBlock, 0, s>>>(a); break;
    case 9: bounds_kernel<9><<<nb, kBoundsBlock, 0, s>>>(a); break;
    case 16: bounds_kernel<16><<<nb, kBoundsBlock, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

hipError_t launch_bounds_totals(const unsigned long long* block_partial, int64_t n_blocks, const int64_t* area_total,
                                unsigned long long* totals, hipStream_t s) {
  bounds_totals_kernel<<<1, 256, 0, s>>>(block_partial, n_blocks, area_total, totals);
  return hipGetLastError();
}

hipError_t launch_emit_pairs(const TileMapArgs& a, hipStream_t s) {
  if (a.n <= 0 || a.pair_count <= 0) return hipSuccess;
  emit_pairs_kernel<<<ceil_div(a.n, kEmitGaussians), 256, 0, s>>>(a);
  return hipGetLastError();
}

hipError_t launch_finish_pairs(const TileMapArgs& a, const uint32_t* sorted_keys, int64_t n_tiles, hipStream_t s) {
  finish_pairs_kernel<<<ceil_div(a.pair_count + 1, 256), 256, 0, s>>>(a, sorted_keys, n_tiles);
  return hipGetLastError();
}

}  // namespace gart
