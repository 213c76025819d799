// Device-side building blocks shared by the GART kernels (gfx950, wave64).
//
// Every routine that decides a discrete outcome (ray direction, hit test,
// depth) is written once here and used unchanged by the forward trace and
// by both backward variants, so the backward re-derives exactly the hits the
// forward composited.  The library is compiled with -ffp-contract=off;
// fused multiply-adds appear only where written explicitly.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "../../include/gart.h"

namespace gart {

constexpr int kGeomStride = 16;  // doubles per Gaussian in prim_geom
// prim_geom layout (double): [0..8] W = S^-1 R^T row-major, [9..11] o_g =
// W (o - mu), [12] squared clamp radius D2c, [13] opacity sigma, [14] lower
// bound on the depth tau of any hit, [15] 1 - sigma = sigmoid(-logit)
// (so that 1 - alpha keeps its precision for nearly opaque Gaussians).
constexpr int kGeoW = 0, kGeoOg = 9, kGeoD2c = 12, kGeoSigma = 13, kGeoKey = 14, kGeoOneMinusSigma = 15;

constexpr uint32_t kNoPrim = 0xffffffffu;

// Camera constants, computed on the host in double from the float inputs.
struct CamParams {
  double o[3];        // camera centre in world space, o = -R^T t
  double Rt[9];       // R^T row-major (camera -> world rotation)
  double fx, fy, cx, cy;
  double ifx, ify;    // 1 / fx, 1 / fy (for bounds only; pixel rays divide)
  double V0[4], V1[4], V3[4];  // rows of the world -> pixel-clip matrix (X, Y, w)
  int32_t W, H;
};

// Gradient values accumulated per Gaussian before the chain rule:
// [0..2] sum 2u x_g, [3..8] sum 2u x_g x_g^T (xx, yy, zz, xy, xz, yz),
// [9] dL/dsigma, [10..10+3K) dL/dsh.  Rows are padded to a multiple of 4.
__host__ __device__ constexpr int acc_width(int K) { return 10 + 3 * K; }
// Row stride of the per-pair partial sums: whole 128-byte lines (16 floats
// at SH degree 0), so that a row's write and its read in the reduction touch
// no partly used line (stride 60 -> 64 floats at degree 3: gather and
// reduction each a few per cent faster).
__host__ __device__ constexpr int acc_stride(int K) {
  return acc_width(K) <= 16 ? 16 : (acc_width(K) + 31) / 32 * 32;
}

// Unit world-space ray direction through the centre of pixel (px, py).
__device__ __forceinline__ void pixel_ray(const CamParams& c, int px, int py, double d[3]) {
  const double a = (double(px) + 0.5 - c.cx) / c.fx;
  const double b = (double(py) + 0.5 - c.cy) / c.fy;
  double v[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) v[k] = fma(c.Rt[3 * k], a, fma(c.Rt[3 * k + 1], b, c.Rt[3 * k + 2]));
  const double inv = 1.0 / sqrt(fma(v[0], v[0], fma(v[1], v[1], v[2] * v[2])));
#pragma unroll
  for (int k = 0; k < 3; ++k) d[k] = v[k] * inv;
}

// Unit camera-space direction c through the centre of tile (tx, ty) (its
// pixel coordinates ((tx + 1/2) ts, (ty + 1/2) ts)).  The tile's list keys are
// depths measured along c.
__device__ __forceinline__ void tile_axis(const CamParams& cam, int tx, int ty, int ts, double c[3]) {
  const double a = (double(tx * ts) + 0.5 * ts - cam.cx) * cam.ifx;
  const double b = (double(ty * ts) + 0.5 * ts - cam.cy) * cam.ify;
  const double inv = 1.0 / sqrt(fma(a, a, fma(b, b, 1.0)));
  c[0] = a * inv;
  c[1] = b * inv;
  c[2] = inv;
}

// Scale s = |R^T u| / (c . u) of the camera ray u = (a, b, 1) of pixel
// (px, py) against its tile's axis c (|R^T u| is the length of the world ray
// vector the trace normalises, so the identity below holds for any rotation
// matrix as given), lowered by 2^-40 against rounding: a list key k bounds
// the depth of a hit on this pixel's ray by tau >= k s.
__device__ __forceinline__ double key_scale(const CamParams& cam, const double c[3], int px, int py) {
  const double a = (double(px) + 0.5 - cam.cx) / cam.fx;
  const double b = (double(py) + 0.5 - cam.cy) / cam.fy;
  double w2 = 0.0;
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    const double wk = fma(cam.Rt[3 * k], a, fma(cam.Rt[3 * k + 1], b, cam.Rt[3 * k + 2]));
    w2 = fma(wk, wk, w2);
  }
  return sqrt(w2) / fma(c[0], a, fma(c[1], b, c[2])) * (1.0 - 0x1p-40);
}

// Max-response point of a Gaussian on the ray o + tau d (Eq. 4-5) in the
// Gaussian's normalised frame: d_g = W d, tau = -<o_g, d_g> / <d_g, d_g>,
// x_g = o_g + tau d_g, D2 = |x_g|^2.  Returns the hit decision tau > 0 and
// D2 <= D2c (alpha >= alpha_min).
__device__ __forceinline__ bool ray_hit(const double W[9], const double og[3], double D2c, const double d[3],
                                        double* tau_out, double* D2_out, double xg[3]) {
  double dg[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) dg[k] = fma(W[3 * k], d[0], fma(W[3 * k + 1], d[1], W[3 * k + 2] * d[2]));
  const double num = fma(og[0], dg[0], fma(og[1], dg[1], og[2] * dg[2]));
  const double den = fma(dg[0], dg[0], fma(dg[1], dg[1], dg[2] * dg[2]));
  const double tau = -num / den;
#pragma unroll
  for (int k = 0; k < 3; ++k) xg[k] = fma(tau, dg[k], og[k]);
  const double D2 = fma(xg[0], xg[0], fma(xg[1], xg[1], xg[2] * xg[2]));
  *tau_out = tau;
  *D2_out = D2;
  return tau > 0.0 && D2 <= D2c;
}

// Closest-approach point x_g and D^2 there for a ray already known to hit,
// for gradient evaluation only (never for a decision): tau uses the hardware
// reciprocal refined by two Newton steps instead of a correctly rounded
// division.
__device__ __forceinline__ void hit_point(const double W[9], const double og[3], const double d[3], double* D2_out,
                                          double xg[3]) {
  double dg[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) dg[k] = fma(W[3 * k], d[0], fma(W[3 * k + 1], d[1], W[3 * k + 2] * d[2]));
  const double num = fma(og[0], dg[0], fma(og[1], dg[1], og[2] * dg[2]));
  const double den = fma(dg[0], dg[0], fma(dg[1], dg[1], dg[2] * dg[2]));
  double r = __builtin_amdgcn_rcp(den);
  r = fma(r, fma(-den, r, 1.0), r);
  r = fma(r, fma(-den, r, 1.0), r);
  const double tau = -num * r;
#pragma unroll
  for (int k = 0; k < 3; ++k) xg[k] = fma(tau, dg[k], og[k]);
  *D2_out = fma(xg[0], xg[0], fma(xg[1], xg[1], xg[2] * xg[2]));
}

// 1 - alpha for alpha = sigma rho, rho = exp(-x), x = D2 / 2, formed as
// (1 - sigma) + sigma (1 - rho) from the Gaussian's own 1 - sigma, so that
// it keeps its relative precision when alpha is close to 1 (1 - rho comes
// from its Taylor series below x = 1/4, error under 2e-9 relative; above,
// 1 - rho > 0.22 and the plain difference is exact to rounding).  Only
// feeds gradients.
__device__ __forceinline__ float one_minus_alpha(float sigma, float one_minus_sigma, float x, float rho) {
  float t = fmaf(-x, 1.0f / 7.0f, 1.0f);
  t = fmaf(-x * (1.0f / 6.0f), t, 1.0f);
  t = fmaf(-x * (1.0f / 5.0f), t, 1.0f);
  t = fmaf(-x * (1.0f / 4.0f), t, 1.0f);
  t = fmaf(-x * (1.0f / 3.0f), t, 1.0f);
  t = fmaf(-x * 0.5f, t, 1.0f);
  const float om_rho = x < 0.25f ? x * t : 1.0f - rho;
  return fmaf(sigma, om_rho, one_minus_sigma);
}

// 1 / (1 - alpha) for the colour-behind term S / (1 - alpha) of dL/dalpha;
// 0 for a fully opaque hit (alpha = 1), which nothing behind can reach.
__device__ __forceinline__ float inv_one_minus_alpha(float oma) {
  return oma > 0.0f ? __builtin_amdgcn_rcpf(oma) : 0.0f;
}

// (tau, id) lexicographic order used to composite hits.
__device__ __forceinline__ bool key_less(double t1, uint32_t i1, double t2, uint32_t i2) {
  return t1 < t2 || (t1 == t2 && i1 < i2);
}

// Real spherical harmonics without Condon-Shortley phase, index l*l + l + m,
// as polynomials of the unit direction (x, y, z).
template <int K>
__device__ __forceinline__ void sh_basis(float x, float y, float z, float Y[K]) {
  Y[0] = 0.28209479177387814f;
  if constexpr (K > 1) {
    Y[1] = 0.4886025119029199f * y;
    Y[2] = 0.4886025119029199f * z;
    Y[3] = 0.4886025119029199f * x;
  }
  if constexpr (K > 4) {
    const float xx = x * x, yy = y * y, zz = z * z;
    Y[4] = 1.0925484305920792f * x * y;
    Y[5] = 1.0925484305920792f * y * z;
    Y[6] = 0.31539156525252005f * (3.0f * zz - 1.0f);
    Y[7] = 1.0925484305920792f * x * z;
    Y[8] = 0.5462742152960396f * (xx - yy);
    if constexpr (K > 9) {
      Y[9] = 0.5900435899266435f * y * (3.0f * xx - yy);
      Y[10] = 2.890611442640554f * x * y * z;
      Y[11] = 0.4570457994644658f * y * (5.0f * zz - 1.0f);
      Y[12] = 0.3731763325901154f * z * (5.0f * zz - 3.0f);
      Y[13] = 0.4570457994644658f * x * (5.0f * zz - 1.0f);
      Y[14] = 1.445305721320277f * z * (xx - yy);
      Y[15] = 0.5900435899266435f * x * (xx - 3.0f * yy);
    }
  }
}

// Offset of pixel (px, py) inside the block of Gaussian i's intermediate
// buffer entries, relative to O_prim(i) (Eq. 16): O_tile + O_pixel with the
// rectangle's tiles in row-major order and pixels row-major inside a tile.
__device__ __forceinline__ int64_t lt_local_index(int x0, int y0, int x1, int y1, int ts, int px, int py) {
  const int tx = px / ts, ty = py / ts;
  const int ya = max(y0, ty * ts), yb = min(y1, ty * ts + ts - 1);
  const int xa = max(x0, tx * ts), xb = min(x1, tx * ts + ts - 1);
  const int64_t o_tile = int64_t(x1 - x0 + 1) * (ya - y0) + int64_t(yb - ya + 1) * (xa - x0);
  const int64_t o_pix = int64_t(py - ya) * (xb - xa + 1) + (px - xa);
  return o_tile + o_pix;
}

// Block index -> tile index.  Blocks reach the 8 XCDs round-robin; each
// XCD receives patches of 4x2 neighbouring tiles (which share Gaussians in
// its L2), and consecutive patches go to different XCDs, so that every XCD
// gets a share of the dense and of the sparse parts of the image.  tiles_x
// is the tile grid width.  A bijection of [0, n).
__device__ __forceinline__ int xcd_tile(int b, int n, int tiles_x) {
  // blocks 64a + r, r = 8 q + x (XCD x): patch slot 8 x + q of group a
  int i = b;
  if (b < (n / 64) * 64) {
    const int r = b % 64;
    i = (b - r) + 8 * (r % 8) + r / 8;
  }
  // order tiles in bands of two tile rows, column by column inside a band,
  // so that 8 consecutive indices form a 4x2 patch
  const int band = i / (2 * tiles_x), k = i % (2 * tiles_x);
  const int tiles_y_full = (n / tiles_x) & ~1;  // rows covered by complete bands
  if (2 * band >= tiles_y_full) return i;       // last, single-row band: row-major
  return (2 * band + k % 2) * tiles_x + k / 2;
}

__device__ __forceinline__ unsigned lane_id() { return __lane_id(); }

// Non-negative colour -> the frame's fixed point (round to nearest,
// saturating at 2^32 - 1; the colour bound keeps composited colours below).
__device__ __forceinline__ uint32_t color_fixed(double v, double inv_step) {
  return uint32_t(fmin(rint(v * inv_step), 4294967295.0));
}

// fp16 storage of intermediate-buffer values: float rounded to the nearest
// fp16 (hardware conversion), and back.
__device__ __forceinline__ uint32_t half_bits(float x) {
  return __builtin_bit_cast(uint16_t, static_cast<_Float16>(x));
}
__device__ __forceinline__ float half_value(uint32_t bits) {
  return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(bits & 0xffffu)));
}

// 16-bit logarithmic code of a transmittance T in (0, 1]: 4096 codes per
// octave, q = round(-log2(T) * 4096) (saturating), T = 2^(-q / 4096); the
// relative error is at most 2^(1/8192) - 1 = 8.5e-5 (hardware log2 / exp2).
__device__ __forceinline__ uint32_t t_log16(float T) {
  return uint32_t(fminf(rintf(-__builtin_amdgcn_logf(T) * 4096.0f), 65535.0f));
}
__device__ __forceinline__ float t_from_log16(uint32_t q) {
  return __builtin_amdgcn_exp2f(float(q & 0xffffu) * (-1.0f / 4096.0f));
}

// Loads intermediate-buffer entry e in layout FMT (gart_lt_format) into a
// uint4 container: FULL as stored; T_ONLY, T_HALF and T_LOG16 with the T
// bits in .w; HALF and FIXED16 with their two words in .x (L.r | L.g << 16)
// and .y (L.b | T << 16).
template <int FMT>
__device__ __forceinline__ uint4 lt_load(const uint4* lt, int64_t e) {
  if constexpr (FMT == GART_LT_FULL) {
    return lt[e];
  } else if constexpr (FMT == GART_LT_T_ONLY) {
    return make_uint4(0u, 0u, 0u, reinterpret_cast<const uint32_t*>(lt)[e]);
  } else if constexpr (FMT == GART_LT_HALF || FMT == GART_LT_FIXED16) {
    const uint2 v = reinterpret_cast<const uint2*>(lt)[e];
    return make_uint4(v.x, v.y, 0u, 0u);
  } else {
    return make_uint4(0u, 0u, 0u, uint32_t(reinterpret_cast<const uint16_t*>(lt)[e]));
  }
}

// Transmittance in front of the hit, from a loaded entry.
template <int FMT>
__device__ __forceinline__ float lt_T(uint4 v) {
  if constexpr (FMT == GART_LT_FULL || FMT == GART_LT_T_ONLY) return __uint_as_float(v.w);
  else if constexpr (FMT == GART_LT_HALF) return half_value(v.y >> 16);
  else if constexpr (FMT == GART_LT_T_HALF) return half_value(v.w);
  else if constexpr (FMT == GART_LT_FIXED16) return t_from_log16(v.y >> 16);
  else return t_from_log16(v.w);
}

// C - L of channel ch (final colour minus the colour in front of the hit),
// from the pixel's fixed-point C and a loaded FULL, HALF or FIXED16 entry.
// FULL and FIXED16: an exact integer difference in units of step (the 16-bit
// L is in units of step * 2^16), then one rounding; HALF: C minus the fp16 L
// in fp64 (one fused rounding of the exact C and L), then to float, so that
// deep hits, where L is close to C, keep the stored L's precision.
template <int FMT>
__device__ __forceinline__ float lt_c_minus_l(uint4 v, const uint32_t Cq[3], int ch, float step) {
  if constexpr (FMT == GART_LT_FULL) {
    const uint32_t Lq = ch == 0 ? v.x : (ch == 1 ? v.y : v.z);
    return __uint2float_rn(Cq[ch] - Lq) * step;
  } else {
    const uint32_t hb = ch == 0 ? v.x : (ch == 1 ? (v.x >> 16) : v.y);
    if constexpr (FMT == GART_LT_FIXED16)
      return float(int64_t(Cq[ch]) - int64_t(hb & 0xffffu) * 65536) * step;
    else
      return float(fma(double(Cq[ch]), double(step), -double(half_value(hb))));
  }
}

// Adds a per-lane count to a device counter with one atomic per wave.  Must
// be called with the whole wave active.
__device__ __forceinline__ void count_add(uint64_t* ctr, uint32_t v) {
  if (ctr == nullptr) return;
  unsigned long long s = v;
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off);
  if (lane_id() == 0 && s) atomicAdd(reinterpret_cast<unsigned long long*>(ctr), static_cast<unsigned long long>(s));
}

}  // namespace gart
