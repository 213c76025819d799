// Backward pass (Sec. 4.4): primitive-centric gather over (tile, primitive)
// pairs, and the pixel-centric scatter control (Sec. 3.5).
//
// Per composited hit of Gaussian i at a pixel with upstream gradient g,
// colour in front L, transmittance in front T (read from the intermediate
// buffer), final pixel colour C and colour behind S = C - L - T a c (C and
// L are in the frame's fixed point, so C - L is an exact integer difference
// and S keeps its precision for hits deep behind the front):
//   dL/dc      = T a g              (zero on a clamped channel)
//   dL/da      = <g, T c - S / (1 - a)>
//   dL/dsigma += dL/da rho,   dL/dsh_k += dL/dc Y_k
// and with 2u = -a dL/da, since D2 is stationary in tau at the maximum
// response, dL/do_g = 2u x_g and dL/dd_g = 2u tau x_g.  Summed over hits this
// gives dL/dW = B S R^T with B = sum 2u x_g x_g^T and dL/dmu = -W^T sum 2u x_g,
// so each Gaussian only needs the 10 + 3K sums
//   [sum 2u x_g (3), B (6, symmetric), dL/dsigma (1), dL/dsh (3K)]
// which the chain-rule kernel turns into raw-parameter gradients:
//   dL/dmu = -R S^-1 sum 2u x_g,  dL/dlog s_k = -B_kk,
//   dL/dR = R S B S^-1 -> quaternion through the normalisation,
//   dL/dlogit = sigma (1 - sigma) dL/dsigma.
#include <hip/hip_runtime.h>

#include <algorithm>

#include "ops.h"

namespace gart {
namespace {

constexpr int kRow = 20;  // doubles per staged Gaussian (same layout as the forward)

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Adds the gradient contribution of one composited hit to acc (accumulator
// layout), with explicit fused multiply-adds.
template <int K, int FMT>
__device__ __forceinline__ void hit_grad_acc(double D2, const double xg[3], double sigma, float one_minus_sigma,
                                             const float sh[3 * K], const float Y[K], const uint32_t Cq[3],
                                             const float g[3], uint4 lt, float step, float acc[acc_width(K)]) {
  // exp(-D2 / 2) as 2^(-D2 log2(e) / 2) on the hardware exp2 (about 1 ulp)
  const float rho = __builtin_amdgcn_exp2f(float(-0.72134752044448170368 * D2));
  const float a = float(sigma) * rho;
  float c[3];
  bool pos[3];
#pragma unroll
  for (int ch = 0; ch < 3; ++ch) {
    float v = 0.5f;
#pragma unroll
    for (int k = 0; k < K; ++k) v = fmaf(sh[3 * k + ch], Y[k], v);
    pos[ch] = v > 0.0f;
    c[ch] = pos[ch] ? v : 0.0f;
  }
  const float T = lt_T<FMT>(lt);
  const float ta = T * a;
  const float inv = inv_one_minus_alpha(one_minus_alpha(float(sigma), one_minus_sigma, float(0.5 * D2), rho));
  float dlda = 0.0f;
  float dc[3];
#pragma unroll
  for (int ch = 0; ch < 3; ++ch) {
    const float S = fmaf(-ta, c[ch], lt_c_minus_l<FMT>(lt, Cq, ch, step));  // colour behind the hit
    dlda = fmaf(g[ch], fmaf(T, c[ch], -S * inv), dlda);
    dc[ch] = pos[ch] ? ta * g[ch] : 0.0f;
  }
  const float u2 = -a * dlda;
  const float x = float(xg[0]), y = float(xg[1]), z = float(xg[2]);
  const float ux = u2 * x, uy = u2 * y, uz = u2 * z;
  acc[0] += ux;
  acc[1] += uy;
  acc[2] += uz;
  acc[3] = fmaf(ux, x, acc[3]);
  acc[4] = fmaf(uy, y, acc[4]);
  acc[5] = fmaf(uz, z, acc[5]);
  acc[6] = fmaf(ux, y, acc[6]);
  acc[7] = fmaf(ux, z, acc[7]);
  acc[8] = fmaf(uy, z, acc[8]);
  acc[9] = fmaf(dlda, rho, acc[9]);
#pragma unroll
  for (int k = 0; k < K; ++k)
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) acc[10 + 3 * k + ch] = fmaf(dc[ch], Y[k], acc[10 + 3 * k + ch]);
}

// SH part of one composited hit (hybrid mode): dL/dc = T a g on unclamped
// channels, dL/dsh_k += dL/dc Y_k; the geometric sums come from the pixel
// pass.  Same rounding as hit_grad_acc.
template <int K>
__device__ __forceinline__ void hit_sh_acc(double D2, double sigma, const float sh[3 * K], const float Y[K],
                                           const float g[3], float T, float acc[acc_width(K)]) {
  const float rho = __builtin_amdgcn_exp2f(float(-0.72134752044448170368 * D2));
  const float a = float(sigma) * rho;
  const float ta = T * a;
#pragma unroll
  for (int ch = 0; ch < 3; ++ch) {
    float v = 0.5f;
#pragma unroll
    for (int k = 0; k < K; ++k) v = fmaf(sh[3 * k + ch], Y[k], v);
    const float dc = v > 0.0f ? ta * g[ch] : 0.0f;
#pragma unroll
    for (int k = 0; k < K; ++k) acc[10 + 3 * k + ch] = fmaf(dc, Y[k], acc[10 + 3 * k + ch]);
  }
}

// Sums v[0..31] over the 64 lanes of a wave; afterwards lanes l and l + 32
// hold the total of value l (l < 32).  After one plain step across the two
// half-waves, each halving step keeps half of the remaining values and adds
// the partner lane's copy of them (63 cross-lane moves for 32 values,
// against 32 x 6 for a plain reduction of each).
__device__ __forceinline__ float wave_sum32_transposed(float* v) {
  const int lane = __lane_id();
#pragma unroll
  for (int j = 0; j < 32; ++j) v[j] += __shfl_xor(v[j], 32);
#pragma unroll
  for (int half = 16; half >= 1; half >>= 1) {
    const bool hi = lane & half;
#pragma unroll
    for (int j = 0; j < half; ++j) {
      const float keep = hi ? v[half + j] : v[j];
      const float send = hi ? v[j] : v[half + j];
      v[j] = keep + __shfl_xor(send, half);
    }
  }
  return v[0];
}

// ---------------------------------------------------------------------------
// Gather: one workgroup per tile.  The tile's pixels form G = TILE^2 / 64
// groups of 64 pixels (whole rows, one wave each); the unit of work is a
// (pair, group): the composited hits of one Gaussian in one group.  Per tile:
//  1. Per-pixel state (ray direction, SH basis, final colour and upstream
//     gradient) is staged in LDS.
//  2. The tile's pairs, up to one past the largest list position the forward
//     composited in the tile, are taken in LDS passes of up to kUnits units.  Each
//     pixel walks the list of its composited hits that the forward recorded
//     and sets its bit in the 64-bit mask of the unit it belongs to (LDS
//     atomics).  Units without a composited hit are dropped, the rest are
//     dealt to lanes in order of hit count, so the lanes of a round run
//     loops of similar length.
//  3. Each lane accumulates the gradient of one unit's hits in registers
//     (a unit with more than kSplit hits is shared by two lanes, whose sums
//     are then added across lanes) and writes one partial row (or adds it
//     atomically).
// ---------------------------------------------------------------------------
constexpr int kUnits = 512;  // units per LDS pass
constexpr int kBatch = 8;    // composited hits whose (L,T) loads are issued together
#ifndef GART_WAVE_MIN
#define GART_WAVE_MIN 48
#endif
constexpr int kWaveMin = GART_WAVE_MIN;  // hits from which a unit is evaluated by its whole wave (mode GATHER_WAVE)

// Lane pairs: a unit with more than kSplit composited hits is shared by two
// adjacent lanes.  Lane j of the pair takes the unit's hits of rank j mod 2
// (ranks in row-major pixel order), and the pair's partial sums are added
// across the two lanes before the first writes the row.  A round's time is
// its largest per-lane hit count, so sharing the largest units evens the
// lanes of a round.  (Groups of four lanes above 16 hits were slower: the
// second cross-lane sum cost more than the shorter rounds saved.)
#ifndef GART_SPLIT
#define GART_SPLIT 6
#endif
constexpr int kSplit = GART_SPLIT;
static_assert(0 < kSplit && kSplit < 64, "split threshold");

// Inclusive prefix parity: bit b of the result is the parity of bits 0..b of x.
__device__ __forceinline__ uint64_t prefix_parity(uint64_t x) {
  x ^= x << 1;
  x ^= x << 2;
  x ^= x << 4;
  x ^= x << 8;
  x ^= x << 16;
  x ^= x << 32;
  return x;
}

// The set bits of m whose rank (0 = lowest set bit) is even (j = 0) or odd.
__device__ __forceinline__ uint64_t rank_half(uint64_t m, int j) {
  const uint64_t p = prefix_parity(m);  // 1 at even ranks
  return j ? (m & ~p) : (m & p);
}

// Value of the lane whose index differs in bit 0 (a DPP quad permutation,
// which needs every lane of the wave active).
__device__ __forceinline__ float pair_swap(float v) {
  return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0xb1, 0xf, 0xf, false));
}

// Per-pixel ray direction in LDS, padded to 32 bytes.
struct __align__(16) RayRec {
  double d[3];
  double pad;
};

// Deals the units of a pass by bucket (0 first; 0xff = dropped): counting
// sort into s_order.  s_hist holds the bucket counts on entry and is zero on
// return.  Returns the number of units kept.  Called by the whole block.
template <int NT>
__device__ __forceinline__ int deal_units(int nu, const uint8_t* s_bucket, uint32_t* s_hist, uint16_t* s_order,
                                          uint32_t* s_total, int dense_min = 65, uint32_t* s_dense = nullptr,
                                          uint32_t* s_split = nullptr) {
  __syncthreads();  // buckets and counts complete
  if (threadIdx.x < 64) {
    const uint32_t c = s_hist[threadIdx.x];
    uint32_t inc = c;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t u = __shfl_up(inc, off);
      if (__lane_id() >= unsigned(off)) inc += u;
    }
    s_hist[threadIdx.x] = inc - c;
    if (threadIdx.x == 63) *s_total = inc;
    // bucket b holds the units with 64 - b hits: those with >= dense_min
    // hits are buckets 0 .. 64 - dense_min, the first entries of the order
    if (s_dense && int(threadIdx.x) == 64 - dense_min) *s_dense = inc;
    // units with more than kSplit hits: buckets below 64 - kSplit, the first
    // entries of the order
    if (s_split && threadIdx.x == 64 - kSplit) *s_split = inc - c;
  }
  __syncthreads();
  for (int u = threadIdx.x; u < nu; u += NT) {
    const uint8_t b = s_bucket[u];
    if (b != 0xff) s_order[atomicAdd(&s_hist[b], 1u)] = uint16_t(u);
  }
  __syncthreads();
  const int kept = int(*s_total);
  if (threadIdx.x < 64) s_hist[threadIdx.x] = 0;
  __syncthreads();
  return kept;
}

template <int TILE, int K, bool ATOMIC, bool HYBRID, int FMT, bool WAVE = false>
__global__ __launch_bounds__(TILE* TILE, 2) void gather_kernel(BackwardArgs A) {
  // HYBRID: the intermediate buffer holds T only (FMT T_ONLY or T_HALF) and
  // the unit accumulates only the SH sums (the pixel pass adds the others).
  // WAVE: units with at least kWaveMin hits are evaluated by their whole wave
  // (one lane per pixel, then a cross-lane sum) before the others are dealt
  // to single lanes.
  constexpr int NT = TILE * TILE;
  constexpr int G = NT / 64;      // pixel groups (waves) per tile
  constexpr int R = 64 / TILE;    // tile rows per group
  constexpr int kPairs = kUnits / G;
  constexpr int AW = acc_width(K), AS = acc_stride(K);
  constexpr int KP = (K + 3) & ~3;  // SH basis row padded to 16 bytes
  static_assert(NT % 64 == 0 && (TILE == 8 || TILE == 16), "tile of 8 or 16");

  __shared__ RayRec s_ray[NT];
  __shared__ __align__(16) float s_Y[NT][KP];
  __shared__ __align__(16) float s_cg[NT][8];  // C.rgb (fixed-point bits), g.rgb
  __shared__ uint32_t s_hist[64];
  __shared__ uint32_t s_total;
  __shared__ uint32_t s_dense;
  __shared__ uint32_t s_split;
  __shared__ uint64_t s_mask[kUnits];
  __shared__ uint32_t s_id[kPairs];
  __shared__ uint8_t s_bucket[kUnits];
  __shared__ uint16_t s_order[kUnits];

  const int n_tiles = A.tiles_x * A.tiles_y;
  const int tile = xcd_tile(blockIdx.x, n_tiles, A.tiles_x);
  const int tx = tile % A.tiles_x, ty = tile / A.tiles_x;
  const int ox = tx * TILE, oy = ty * TILE;
  const int tid = threadIdx.x;
  uint32_t my_hits = 0;  // composited hits of this thread's pixel
  {
    const int px = ox + tid % TILE, py = oy + tid / TILE;
    const bool valid = px < A.cam.W && py < A.cam.H;
    double d[3];
    pixel_ray(A.cam, valid ? px : 0, valid ? py : 0, d);
    float Y[K];
    sh_basis<K>(float(d[0]), float(d[1]), float(d[2]), Y);
#pragma unroll
    for (int k = 0; k < KP; ++k) s_Y[tid][k] = k < K ? Y[k] : 0.0f;
    uint32_t cq[3] = {0, 0, 0};
    float gg[3] = {0, 0, 0};
    if (valid) {
      const int64_t p = int64_t(py) * A.cam.W + px;
#pragma unroll
      for (int ch = 0; ch < 3; ++ch) {
        gg[ch] = A.dl_dimage[3 * p + ch];
        cq[ch] = A.pixel_state[p].color_fixed[ch];
      }
      my_hits = A.pixel_state[p].n_hits;
    }
    RayRec rr;
    rr.d[0] = d[0];
    rr.d[1] = d[1];
    rr.d[2] = d[2];
    rr.pad = 0.0;
    s_ray[tid] = rr;
    *reinterpret_cast<uint4*>(&s_cg[tid][0]) = make_uint4(cq[0], cq[1], cq[2], __float_as_uint(gg[0]));
    *reinterpret_cast<float4*>(&s_cg[tid][4]) = make_float4(gg[1], gg[2], 0.0f, 0.0f);
  }
  __syncthreads();

  // Composited hits lie in the first tile_visit[tile] positions of the tile's
  // list (the forward records one past the largest position it composited).
  const int64_t beg = A.tile_range[tile], end = A.tile_range[tile + 1];
  const int64_t vend = min(end, beg + int64_t(A.tile_visit[tile]));

  uint32_t n_pairs = 0, n_hits = 0, n_atom = 0, n_active = 0, n_wave = 0;
  for (int64_t c0 = beg; c0 < vend; c0 += kPairs) {
    const int nc = int(min<int64_t>(kPairs, vend - c0));
    const int nu = nc * G;
    for (int u = tid; u < nu; u += NT) s_mask[u] = 0;
    for (int q = tid; q < nc; q += NT) {
      s_id[q] = A.pair_prim[c0 + q];
      ++n_pairs;
    }
    if (tid < 64) s_hist[tid] = 0;
    __syncthreads();
    // This pixel's composited hits whose pair lies in the pass (list loads
    // issued eight at a time).
    {
      const uint32_t lo = uint32_t(c0 - beg);
      const uint32_t* hl = A.hit_list + int64_t(NT) * A.hl_off[tile] + tid;
      const uint64_t bit = 1ull << (tid % 64);
      uint32_t k = 0;
      for (; k + 8 <= my_hits; k += 8) {
        uint32_t q[8];
#pragma unroll
        for (int t = 0; t < 8; ++t) q[t] = hl[int64_t(NT) * (k + t)] - lo;
#pragma unroll
        for (int t = 0; t < 8; ++t)
          if (q[t] < uint32_t(nc)) atomicOr(&s_mask[q[t] * G + tid / 64], bit);
      }
      for (; k < my_hits; ++k) {
        const uint32_t q = hl[int64_t(NT) * k] - lo;
        if (q < uint32_t(nc)) atomicOr(&s_mask[q * G + tid / 64], bit);
      }
    }
    __syncthreads();
    for (int u = tid; u < nu; u += NT) {
      const int c = __popcll(s_mask[u]);
      s_bucket[u] = c ? uint8_t(64 - c) : uint8_t(0xff);
      if (c) atomicAdd(&s_hist[64 - c], 1u);
    }
    const int nu2 = deal_units<NT>(nu, s_bucket, s_hist, s_order, &s_total, WAVE ? kWaveMin : 65, &s_dense,
                                   WAVE ? nullptr : &s_split);

    int o0 = 0;
    if constexpr (WAVE) {
      // Dense units, whole wave per unit: the wave of group g takes the dense
      // units of its group; lane l is pixel l of the group.
      const int nd = int(s_dense), wv = tid / 64, lane = tid % 64;
      for (int o = 0; o < nd; ++o) {
        const int u = __builtin_amdgcn_readfirstlane(int(s_order[o]));
        if (u % G != wv) continue;
        const uint32_t i = __builtin_amdgcn_readfirstlane(s_id[u / G]);
        const bool has = (s_mask[u] >> lane) & 1ull;
        const int4 r = *reinterpret_cast<const int4*>(A.rect + 4 * int64_t(i));
        float v[64];
#pragma unroll
        for (int e = 0; e < 64; ++e) v[e] = 0.0f;
        if (has) {
          const double* Gm = A.geom + int64_t(kGeomStride) * i;
          double W[9], og[3];
#pragma unroll
          for (int k = 0; k < 9; ++k) W[k] = Gm[k];
#pragma unroll
          for (int k = 0; k < 3; ++k) og[k] = Gm[kGeoOg + k];
          const double sigma = Gm[kGeoSigma];
          const float oms = float(Gm[kGeoOneMinusSigma]);
          float sh[3 * K];
          const float* shp = A.sh + int64_t(i) * (3 * K);
#pragma unroll
          for (int k = 0; k < 3 * K; ++k) sh[k] = shp[k];
          const int px = ox + tid % TILE, py = oy + tid / TILE;
          const uint4 lt = lt_load<FMT>(A.lt, A.lt_offset[i] + lt_local_index(r.x, r.y, r.z, r.w, TILE, px, py));
          double D2, xg[3];
          hit_point(W, og, s_ray[tid].d, &D2, xg);
          float Y[KP];
#pragma unroll
          for (int kk = 0; kk < KP; kk += 4) {
            const float4 y4 = *reinterpret_cast<const float4*>(&s_Y[tid][kk]);
            Y[kk] = y4.x;
            Y[kk + 1] = y4.y;
            Y[kk + 2] = y4.z;
            Y[kk + 3] = y4.w;
          }
          const uint4 c4 = *reinterpret_cast<const uint4*>(&s_cg[tid][0]);
          const float4 g4 = *reinterpret_cast<const float4*>(&s_cg[tid][4]);
          const uint32_t Cq[3] = {c4.x, c4.y, c4.z};
          const float gr[3] = {__uint_as_float(c4.w), g4.x, g4.y};
          hit_grad_acc<K, FMT>(D2, xg, sigma, oms, sh, Y, Cq, gr, lt, A.color_step, v);  // v[0 .. AW)
          ++n_hits;
        }
        // lane e < 32: sum of value e; lane e >= 32: sum of value e
        const float lo = wave_sum32_transposed(v);
        const float hi = wave_sum32_transposed(v + 32);
        const float total = lane < 32 ? lo : hi;
        const int tx0 = r.x / TILE, ty0 = r.y / TILE, tx1 = r.z / TILE;
        const int64_t row = (A.pair_offset[i] + int64_t(ty - ty0) * (tx1 - tx0 + 1) + (tx - tx0)) * G + u % G;
        if (lane < AS) A.rows[row * AS + lane] = lane < AW ? total : 0.0f;
        if (lane == 0) {
          A.row_flag[row] = 1;
          ++n_active;
          ++n_wave;
        }
      }
      o0 = nd;
    }

    // Slots: 2 per unit of the first n2 in the order (the shared units), 1 per
    // remaining unit; pairs start at even slots.  Rounds are block-uniform so
    // that every lane of a wave reaches the cross-lane sums.
    const int n2 = WAVE ? 0 : int(s_split);
    const int nslots = 2 * n2 + (nu2 - o0 - n2);
    for (int sb = 0; sb < nslots; sb += NT) {
      const int slot = sb + tid;
      const bool live = slot < nslots;
      const bool paired = slot < 2 * n2;
      const int j = paired ? (slot & 1) : 0;
      const int o = live ? o0 + (paired ? slot >> 1 : slot - n2) : o0;
      const int u = s_order[o], g = u % G;
      const uint32_t i = s_id[u / G];
      const double* Gm = A.geom + int64_t(kGeomStride) * i;
      double W[9], og[3];
#pragma unroll
      for (int k = 0; k < 9; ++k) W[k] = Gm[k];
#pragma unroll
      for (int k = 0; k < 3; ++k) og[k] = Gm[kGeoOg + k];
      const double sigma = Gm[kGeoSigma];
      const float oms = float(Gm[kGeoOneMinusSigma]);
      const int4 r = *reinterpret_cast<const int4*>(A.rect + 4 * int64_t(i));
      float sh[3 * K];
      const float* shp = A.sh + int64_t(i) * (3 * K);
#pragma unroll
      for (int k = 0; k < 3 * K; ++k) sh[k] = shp[k];
      const int xa = max(r.x, ox), xb = min(r.z, ox + TILE - 1);
      const int ya = max(r.y, oy);
      const int w = xb - xa + 1;
      // (L,T) index of pixel b of the group: O_prim + O_tile + row-major
      // offset inside rect cap tile (Eq. 16).
      const int64_t base = A.lt_offset[i] + lt_local_index(r.x, r.y, r.z, r.w, TILE, xa, ya) +
                           int64_t(oy + g * R - ya) * w + (ox - xa);
      auto lt_at = [&](int b) { return lt_load<FMT>(A.lt, base + int64_t(b / TILE) * w + (b % TILE)); };
      float acc[AW];
#pragma unroll
      for (int v = 0; v < AW; ++v) acc[v] = 0.0f;
      // Composited hits in row-major order, in batches of kBatch: the batch's
      // (L,T) loads are all issued before its first hit is evaluated, so one
      // memory latency is paid per batch (no load is pending across
      // iterations, which would make the compiler wait for it early).
      uint64_t m = !live ? 0ull : paired ? rank_half(s_mask[u], j) : s_mask[u];
      while (m) {
        int bb[kBatch];
        uint4 lv[kBatch];
#pragma unroll
        for (int t = 0; t < kBatch; ++t) {
          bb[t] = m ? __builtin_ctzll(m) : -1;
          if (m) {
            m &= m - 1;
            lv[t] = lt_at(bb[t]);
          } else {
            lv[t] = make_uint4(0, 0, 0, 0);
          }
        }
#pragma unroll
        for (int t = 0; t < kBatch; ++t) {
          if (bb[t] < 0) break;
          const int lp = g * 64 + bb[t];
          double D2, xg[3];
          hit_point(W, og, s_ray[lp].d, &D2, xg);
          ++n_hits;
          float Y[KP];
#pragma unroll
          for (int kk = 0; kk < KP; kk += 4) {
            const float4 y4 = *reinterpret_cast<const float4*>(&s_Y[lp][kk]);
            Y[kk] = y4.x;
            Y[kk + 1] = y4.y;
            Y[kk + 2] = y4.z;
            Y[kk + 3] = y4.w;
          }
          const uint4 c4 = *reinterpret_cast<const uint4*>(&s_cg[lp][0]);
          const float4 g4 = *reinterpret_cast<const float4*>(&s_cg[lp][4]);
          const uint32_t Cq[3] = {c4.x, c4.y, c4.z};
          const float gr[3] = {__uint_as_float(c4.w), g4.x, g4.y};
          if constexpr (HYBRID)
            hit_sh_acc<K>(D2, sigma, sh, Y, gr, lt_T<FMT>(lv[t]), acc);
          else
            hit_grad_acc<K, FMT>(D2, xg, sigma, oms, sh, Y, Cq, gr, lv[t], A.color_step, acc);
        }
      }
      // Partial sums of a pair, added across its two lanes (skipped by waves
      // without pairs; lanes on their own keep theirs).
      if (__ballot(paired)) {
#pragma unroll
        for (int v = 0; v < AW; ++v) {
          const float t = pair_swap(acc[v]);
          acc[v] += paired ? t : 0.0f;
        }
      }
      if (!live || j != 0) continue;
      ++n_active;
      if constexpr (ATOMIC) {
        float* dst = A.acc + int64_t(i) * AS;
#pragma unroll
        for (int v = 0; v < AW; ++v) unsafeAtomicAdd(dst + v, acc[v]);
        n_atom += AW;
      } else {
        const int tx0 = r.x / TILE, ty0 = r.y / TILE, tx1 = r.z / TILE;
        const int64_t row = (A.pair_offset[i] + int64_t(ty - ty0) * (tx1 - tx0 + 1) + (tx - tx0)) * G + g;
        float4* dst = reinterpret_cast<float4*>(A.rows + row * AS);
#pragma unroll
        for (int v = 0; v < AS; v += 4) {
          float4 q4;
          q4.x = v + 0 < AW ? acc[v + 0] : 0.0f;
          q4.y = v + 1 < AW ? acc[v + 1] : 0.0f;
          q4.z = v + 2 < AW ? acc[v + 2] : 0.0f;
          q4.w = v + 3 < AW ? acc[v + 3] : 0.0f;
          dst[v / 4] = q4;
        }
        A.row_flag[row] = 1;
      }
    }
    __syncthreads();  // the pass's LDS arrays are rewritten by the next pass
  }
  if (A.counters) {
    count_add(A.counters + GART_CNT_BWD_PAIRS, n_pairs);
    count_add(A.counters + GART_CNT_BWD_ACTIVE, n_active);
    count_add(A.counters + GART_CNT_BWD_HITS, n_hits);
    count_add(A.counters + GART_CNT_BWD_ATOMICS, n_atom);
    if constexpr (WAVE) count_add(A.counters + GART_CNT_BWD_WAVE_UNITS, n_wave);
  }
}

// ---------------------------------------------------------------------------
// Hybrid pixel pass: each lane (pixel) walks its own composited hits back to
// front (the forward's hit list), forming the colour behind each hit, S, from
// the walk in fp64 (the intermediate buffer holds T only, so S cannot come
// from C - L), and adds the hit's 10 geometric terms (2u x_g, 2u x_g x_g^T,
// dL/dsigma) into LDS accumulators of its (list position, pixel group) with
// LDS float atomics.  The tile's list is covered in windows of kWin
// positions; each window is walked once more (S needs every hit behind), and
// its nonzero accumulators are written into the (pair, group) rows that the
// SH gather filled (zeros there).
// ---------------------------------------------------------------------------
template <int TILE>
struct HybridWindow {
  static constexpr int G = TILE * TILE / 64;
  static constexpr int kWin = TILE == 8 ? 384 : 128;  // list positions per window
};

template <int TILE, int K, int FMT>
__global__ __launch_bounds__(TILE* TILE) void hybrid_pixel_kernel(BackwardArgs A) {
  constexpr int NT = TILE * TILE;
  constexpr int G = HybridWindow<TILE>::G, kWin = HybridWindow<TILE>::kWin;
  constexpr int AS = acc_stride(K);
  __shared__ float s_acc[kWin * G][10];
  __shared__ int s_maxpos[G];

  const int n_tiles = A.tiles_x * A.tiles_y;
  const int tile = xcd_tile(blockIdx.x, n_tiles, A.tiles_x);
  const int tx = tile % A.tiles_x, ty = tile / A.tiles_x;
  const int tid = threadIdx.x, grp = tid / 64;
  const int px = tx * TILE + tid % TILE, py = ty * TILE + tid / TILE;
  const bool valid = px < A.cam.W && py < A.cam.H;
  double d[3];
  pixel_ray(A.cam, valid ? px : 0, valid ? py : 0, d);
  float Y[K];
  sh_basis<K>(float(d[0]), float(d[1]), float(d[2]), Y);
  float g[3] = {0.0f, 0.0f, 0.0f};
  int nh = 0;
  if (valid) {
    const int64_t p = int64_t(py) * A.cam.W + px;
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) g[ch] = A.dl_dimage[3 * p + ch];
    nh = int(A.pixel_state[p].n_hits);
  }
  const int64_t beg = A.tile_range[tile];
  const uint32_t* hl = A.hit_list + int64_t(NT) * A.hl_off[tile] + tid;
  uint32_t n_walk = 0;

  for (int w0 = 0;; w0 += kWin) {
    for (int u = tid; u < kWin * G; u += NT) {
#pragma unroll
      for (int v = 0; v < 10; ++v) s_acc[u][v] = 0.0f;
    }
    __syncthreads();
    double S[3] = {0.0, 0.0, 0.0};  // colour behind the current hit
    int maxpos = -1;
    for (int k = nh - 1; k >= 0; --k) {
      const int pos = int(hl[int64_t(NT) * k]);
      maxpos = max(maxpos, pos);
      const uint32_t i = A.pair_prim[beg + pos];
      const double* Gm = A.geom + int64_t(kGeomStride) * i;
      double W[9], og[3];
#pragma unroll
      for (int e = 0; e < 9; ++e) W[e] = Gm[e];
#pragma unroll
      for (int e = 0; e < 3; ++e) og[e] = Gm[kGeoOg + e];
      const double sigma = Gm[kGeoSigma];
      const float oms = float(Gm[kGeoOneMinusSigma]);
      const int4 r = *reinterpret_cast<const int4*>(A.rect + 4 * int64_t(i));
      const float T = lt_T<FMT>(lt_load<FMT>(A.lt, A.lt_offset[i] + lt_local_index(r.x, r.y, r.z, r.w, TILE, px, py)));
      double D2, xg[3];
      hit_point(W, og, d, &D2, xg);
      const float rho = __builtin_amdgcn_exp2f(float(-0.72134752044448170368 * D2));
      const float a = float(sigma) * rho;
      const float* shp = A.sh + int64_t(i) * (3 * K);
      float c[3];
#pragma unroll
      for (int ch = 0; ch < 3; ++ch) {
        float cv = 0.5f;
#pragma unroll
        for (int kk = 0; kk < K; ++kk) cv = fmaf(shp[3 * kk + ch], Y[kk], cv);
        c[ch] = cv > 0.0f ? cv : 0.0f;
      }
      if (pos >= w0 && pos < w0 + kWin) {
        const float inv = inv_one_minus_alpha(one_minus_alpha(float(sigma), oms, float(0.5 * D2), rho));
        float dlda = 0.0f;
#pragma unroll
        for (int ch = 0; ch < 3; ++ch) dlda = fmaf(g[ch], fmaf(T, c[ch], -float(S[ch]) * inv), dlda);
        const float u2 = -a * dlda;
        const float x = float(xg[0]), y = float(xg[1]), z = float(xg[2]);
        const float ux = u2 * x, uy = u2 * y, uz = u2 * z;
        float* acc = s_acc[(pos - w0) * G + grp];
        atomicAdd(acc + 0, ux);
        atomicAdd(acc + 1, uy);
        atomicAdd(acc + 2, uz);
        atomicAdd(acc + 3, ux * x);
        atomicAdd(acc + 4, uy * y);
        atomicAdd(acc + 5, uz * z);
        atomicAdd(acc + 6, ux * y);
        atomicAdd(acc + 7, ux * z);
        atomicAdd(acc + 8, uy * z);
        atomicAdd(acc + 9, dlda * rho);
      }
      const double wt = double(T) * double(a);
#pragma unroll
      for (int ch = 0; ch < 3; ++ch) S[ch] = fma(wt, double(c[ch]), S[ch]);
      ++n_walk;
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) maxpos = max(maxpos, __shfl_xor(maxpos, off));
    if (tid % 64 == 0) s_maxpos[grp] = maxpos;
    __syncthreads();
    // write the window's nonzero accumulators into their rows (a unit whose
    // sums are all zero keeps the zeros the SH gather wrote; a position with
    // no hit in this group has no row to write and stays zero)
    for (int u = tid; u < kWin * G; u += NT) {
      bool nz = false;
#pragma unroll
      for (int v = 0; v < 10; ++v) nz |= s_acc[u][v] != 0.0f;
      if (!nz) continue;
      const uint32_t i = A.pair_prim[beg + w0 + u / G];
      const int4 r = *reinterpret_cast<const int4*>(A.rect + 4 * int64_t(i));
      const int tx0 = r.x / TILE, ty0 = r.y / TILE, tx1 = r.z / TILE;
      const int64_t row = (A.pair_offset[i] + int64_t(ty - ty0) * (tx1 - tx0 + 1) + (tx - tx0)) * G + u % G;
      float4* dst = reinterpret_cast<float4*>(A.rows + row * AS);
      const float* v = s_acc[u];
      dst[0] = make_float4(v[0], v[1], v[2], v[3]);
      dst[1] = make_float4(v[4], v[5], v[6], v[7]);
      reinterpret_cast<float2*>(dst + 2)[0] = make_float2(v[8], v[9]);
    }
    int mp = s_maxpos[0];
#pragma unroll
    for (int w = 1; w < G; ++w) mp = max(mp, s_maxpos[w]);
    if (mp < w0 + kWin) break;
    __syncthreads();  // the window's LDS arrays are cleared by the next window
  }
  if (A.counters) count_add(A.counters + GART_CNT_BWD_STEPS, n_walk);
}

// ---------------------------------------------------------------------------
// Scatter control: one lane per pixel walks the tile's list front to back
// and adds every composited hit's gradient with float atomics.
// ---------------------------------------------------------------------------
template <int TILE, int K, int FMT>
__global__ __launch_bounds__(TILE* TILE) void scatter_kernel(BackwardArgs A) {
  constexpr int NT = TILE * TILE;
  constexpr int AW = acc_width(K), AS = acc_stride(K);
  constexpr double kInf = __builtin_huge_val();
  __shared__ __align__(16) double s_row[NT * kRow];

  const int n_tiles = A.tiles_x * A.tiles_y;
  const int tile = xcd_tile(blockIdx.x, n_tiles, A.tiles_x);
  const int tx = tile % A.tiles_x, ty = tile / A.tiles_x;
  const int tid = threadIdx.x;
  const int px = tx * TILE + tid % TILE, py = ty * TILE + tid / TILE;
  const bool valid = px < A.cam.W && py < A.cam.H;

  double d[3];
  pixel_ray(A.cam, valid ? px : 0, valid ? py : 0, d);
  double cax[3];
  tile_axis(A.cam, tx, ty, TILE, cax);
  const double kscale = key_scale(A.cam, cax, valid ? px : 0, valid ? py : 0);  // key -> depth bound on this ray
  float Y[K];
  sh_basis<K>(float(d[0]), float(d[1]), float(d[2]), Y);
  uint32_t Cq[3] = {0, 0, 0};
  float g[3] = {0, 0, 0};
  double tend = -kInf;
  uint32_t iend = 0;
  if (valid) {
    const int64_t p = int64_t(py) * A.cam.W + px;
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) g[ch] = A.dl_dimage[3 * p + ch];
    const gart_pixel_state st = A.pixel_state[p];
    tend = st.tau_end;
    iend = st.id_end;
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) Cq[ch] = st.color_fixed[ch];
  }
  bool done = !valid;
  uint32_t n_hits = 0, n_tests = 0, n_atom = 0;
  const int64_t beg = A.tile_range[tile], end = A.tile_range[tile + 1];
  for (int64_t base = beg; base < end; base += NT) {
    const int nb = int(min<int64_t>(NT, end - base));
    if (tid < nb) {
      const uint32_t id = A.pair_prim[base + tid];
      const double* G = A.geom + int64_t(kGeomStride) * id;
      double* row = s_row + tid * kRow;
#pragma unroll
      for (int k = 0; k < 14; ++k) row[k] = G[k];
      row[14] = double(A.pair_key[base + tid]);
      row[15] = __longlong_as_double(A.lt_offset[id]);
      const int4 r = *reinterpret_cast<const int4*>(A.rect + 4 * int64_t(id));
      int* ri = reinterpret_cast<int*>(row + 16);
      ri[0] = r.x;
      ri[1] = r.y;
      ri[2] = r.z;
      ri[3] = r.w;
      reinterpret_cast<uint32_t*>(row + 18)[0] = id;
      row[19] = G[kGeoOneMinusSigma];
    }
    __syncthreads();
    if (!done) {
      for (int c = 0; c < nb; ++c) {
        const double* row = s_row + c * kRow;
        if (row[14] * kscale > tend) {  // every remaining Gaussian lies behind this ray's end
          done = true;
          break;
        }
        const int4 r = *reinterpret_cast<const int4*>(row + 16);
        if (px < r.x || px > r.z || py < r.y || py > r.w) continue;
        ++n_tests;
        double W[9], og[3];
#pragma unroll
        for (int k = 0; k < 9; ++k) W[k] = row[k];
#pragma unroll
        for (int k = 0; k < 3; ++k) og[k] = row[9 + k];
        double tau, D2, xg[3];
        const uint32_t id = reinterpret_cast<const uint32_t*>(row + 18)[0];
        if (!ray_hit(W, og, row[12], d, &tau, &D2, xg)) continue;
        if (key_less(tend, iend, tau, id)) continue;
        ++n_hits;
        const int64_t li = __double_as_longlong(row[15]) + lt_local_index(r.x, r.y, r.z, r.w, TILE, px, py);
        const uint4 lt = lt_load<FMT>(A.lt, li);
        float sh[3 * K];
        const float* shp = A.sh + int64_t(id) * (3 * K);
#pragma unroll
        for (int k = 0; k < 3 * K; ++k) sh[k] = shp[k];
        float h[AW];
#pragma unroll
        for (int v = 0; v < AW; ++v) h[v] = 0.0f;
        hit_grad_acc<K, FMT>(D2, xg, row[13], float(row[19]), sh, Y, Cq, g, lt, A.color_step, h);
        float* dst = A.acc + int64_t(id) * AS;
#pragma unroll
        for (int v = 0; v < AW; ++v) unsafeAtomicAdd(dst + v, h[v]);
        n_atom += AW;
      }
    }
    if (!__syncthreads_or(!done)) break;
  }
  if (A.counters) {
    count_add(A.counters + GART_CNT_BWD_HITS, n_hits);
    count_add(A.counters + GART_CNT_BWD_TESTS, n_tests);
    count_add(A.counters + GART_CNT_BWD_ATOMICS, n_atom);
  }
}

// ---------------------------------------------------------------------------
// Per-Gaussian reduction of the pair rows (gather mode) or read of the
// atomic accumulators, then the chain rule to the raw parameters.  A block
// serves 64 Gaussians, whose rows form one contiguous range (pairs are in
// emission order, Gaussian by Gaussian, rows_per_pair pixel groups each).
//
// Row sums: the block reads the range's row flags in coalesced chunks, lists
// a chunk's active rows in row order, and gives each of its sixteen lane
// groups an equal contiguous share of the list (lane q of a group owns
// float4 q of a row).  A group sums its share in order.  A Gaussian whose
// rows in the chunk all lie in one share is added to its LDS row directly;
// one cut by share boundaries is added there by its first share, and the
// partials of the following shares are added afterwards in share order.
// Every order depends on the flags alone, so the sums are deterministic, and
// a Gaussian with a thousand tiles is spread over the block instead of
// serialising one lane group.
//
// Chain rule: one Gaussian per lane of the first wave.  SH gradients: all
// threads, coalesced.
// ---------------------------------------------------------------------------
#ifndef GART_REDUCE_CHUNK
#define GART_REDUCE_CHUNK 1024
#endif
constexpr int kReduceLanes = 16;  // lanes per row: 16 float4 hold the widest row (64 floats)
constexpr int kReduceBlock = 256;
constexpr int kReduceGaussians = 64;
constexpr int kReduceChunk = GART_REDUCE_CHUNK;  // row flags listed per pass
static_assert(kReduceChunk % kReduceBlock == 0 && kReduceChunk <= 65536, "chunk of whole block strides");

__device__ const uint8_t g_zero_flag = 0;  // read in place of a row flag past the range

// The block's Gaussian (0 .. nb-1) whose pair range holds `pair`: the last
// one whose first pair is <= pair (empty ranges before it are skipped).
__device__ __forceinline__ int gaussian_of(const int64_t* po, int nb, int64_t pair) {
  int lo = 0, hi = nb - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (po[mid] <= pair)
      lo = mid;
    else
      hi = mid - 1;
  }
  return lo;
}

template <int AS>
__device__ __forceinline__ void sum_rows(const BackwardArgs& A, int64_t i0, int nb, float (*s_acc)[AS]) {
  constexpr int NQ = AS / 4, GROUPS = kReduceBlock / kReduceLanes;
  constexpr int NC = (NQ + kReduceLanes - 1) / kReduceLanes;  // float4 columns per lane
  constexpr int J = kReduceChunk / kReduceBlock;             // flags per thread per chunk
  constexpr int W = kReduceBlock / 64;
  __shared__ int64_t s_po[kReduceGaussians + 1];
  __shared__ uint32_t s_list[kReduceChunk];
  __shared__ uint32_t s_cnt[J * W];
  __shared__ __align__(16) float s_part[GROUPS][AS];  // head partial of each share
  __shared__ int s_head_id[GROUPS], s_tail_id[GROUPS];
  const int tid = threadIdx.x, lane = tid % 64, w = tid / 64;
  const int grp = tid / kReduceLanes, q = tid % kReduceLanes;
  const float4 zero4 = make_float4(0.0f, 0.0f, 0.0f, 0.0f);

  if (tid <= nb) s_po[tid] = A.pair_offset[i0 + tid];
  for (int e = tid; e < kReduceGaussians * NQ; e += kReduceBlock)
    reinterpret_cast<float4*>(&s_acc[0][0])[e] = zero4;
  __syncthreads();
  const int rsh = __ffs(int(A.rows_per_pair)) - 1;  // rows_per_pair is 1 or 4
  const int64_t R0 = s_po[0] << rsh, R1 = s_po[nb] << rsh;
  const float4* rows = reinterpret_cast<const float4*>(A.rows);

  for (int64_t cb = R0; cb < R1; cb += kReduceChunk) {
    // flags of the chunk, every load issued before any is used
    uint32_t f[J];
#pragma unroll
    for (int j = 0; j < J; ++j) {
      const int64_t r = cb + j * kReduceBlock + tid;
      f[j] = *(r < R1 ? A.row_flag + r : &g_zero_flag);
    }
    uint64_t bal[J];
#pragma unroll
    for (int j = 0; j < J; ++j) bal[j] = __ballot(f[j] != 0u);
    if (lane == 0)
#pragma unroll
      for (int j = 0; j < J; ++j) s_cnt[j * W + w] = uint32_t(__popcll(bal[j]));
    __syncthreads();
    // the list of active rows (offsets from cb), in row order: (j, wave, lane)
    uint32_t base[J], total = 0;
#pragma unroll
    for (int j = 0; j < J; ++j)
#pragma unroll
      for (int v = 0; v < W; ++v) {
        const uint32_t c = s_cnt[j * W + v];
        if (v == w) base[j] = total;
        total += c;
      }
    // entry: Gaussian slot << 16 | row offset in the chunk
#pragma unroll
    for (int j = 0; j < J; ++j)
      if (f[j] != 0u) {
        const uint32_t rel = uint32_t(j * kReduceBlock + tid);
        s_list[base[j] + __builtin_amdgcn_mbcnt_hi(uint32_t(bal[j] >> 32), __builtin_amdgcn_mbcnt_lo(uint32_t(bal[j]), 0u))] =
            uint32_t(gaussian_of(s_po, nb, (cb + rel) >> rsh)) << 16 | rel;
      }
    const int L = int(total);
    __syncthreads();

    // this group's share [sb, se) of the list
    const int sb = grp * L / GROUPS, se = (grp + 1) * L / GROUPS;
    auto gl_at = [&](int e) { return int(s_list[e] >> 16); };
    int gfirst = -1, glast = -1;
    bool head_cut = false, tail_cut = false;
    if (sb < se) {
      gfirst = gl_at(sb);
      glast = gl_at(se - 1);
      head_cut = sb > 0 && gl_at(sb - 1) == gfirst;
      tail_cut = se < L && gl_at(se) == glast;
    }
    if (q == 0) s_head_id[grp] = s_tail_id[grp] = -1;
    float4 acc[NC];
    int cur = -1;
    auto flush = [&]() {
      // a Gaussian continued from the previous share keeps its partial apart;
      // any other goes to its LDS row (a tail-cut one first of all its shares)
      const bool head = cur == gfirst && head_cut;
#pragma unroll
      for (int c = 0; c < NC; ++c) {
        const int col = q + c * kReduceLanes;
        if (col >= NQ) continue;
        if (head) {
          reinterpret_cast<float4*>(s_part[grp])[col] = acc[c];
        } else {
          float4* d = reinterpret_cast<float4*>(s_acc[cur]) + col;
          float4 t = *d;
          t.x += acc[c].x;
          t.y += acc[c].y;
          t.z += acc[c].z;
          t.w += acc[c].w;
          *d = t;
        }
      }
      if (q == 0) {
        if (head)
          s_head_id[grp] = cur;
        else if (cur == glast && tail_cut)
          s_tail_id[grp] = cur;
      }
    };
    for (int e = sb; e < se; e += 4) {
      int gu[4];
      int64_t ru[4];
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        const bool ok = e + u < se;
        const uint32_t x = ok ? s_list[e + u] : 0u;
        ru[u] = cb + (x & 0xffffu);
        gu[u] = ok ? int(x >> 16) : -1;
      }
      float4 v[4][NC];
#pragma unroll
      for (int u = 0; u < 4; ++u)
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          const int col = q + c * kReduceLanes;
          v[u][c] = (gu[u] >= 0 && col < NQ) ? rows[ru[u] * NQ + col] : zero4;
        }
#pragma unroll
      for (int u = 0; u < 4; ++u) {
        if (gu[u] < 0) break;
        if (gu[u] != cur) {
          if (cur >= 0) flush();
          cur = gu[u];
#pragma unroll
          for (int c = 0; c < NC; ++c) acc[c] = v[u][c];
        } else {
#pragma unroll
          for (int c = 0; c < NC; ++c) {
            acc[c].x += v[u][c].x;
            acc[c].y += v[u][c].y;
            acc[c].z += v[u][c].z;
            acc[c].w += v[u][c].w;
          }
        }
      }
    }
    if (cur >= 0) flush();
    __syncthreads();

    // A cut Gaussian's first share added its part to the LDS row and named
    // it as its tail; that share's group adds the head partials of the
    // following shares, in share order (the shares holding one Gaussian are
    // consecutive).
    {
      const int gl = s_tail_id[grp];
      if (gl >= 0) {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
          const int col = q + c * kReduceLanes;
          if (col >= NQ) continue;
          float4* d = reinterpret_cast<float4*>(s_acc[gl]) + col;
          float4 a = *d;
          for (int g = grp + 1; g < GROUPS; ++g) {
            if (s_head_id[g] != gl) continue;
            const float4 p = reinterpret_cast<const float4*>(s_part[g])[col];
            a.x += p.x;
            a.y += p.y;
            a.z += p.z;
            a.w += p.w;
          }
          *d = a;
        }
      }
    }
    __syncthreads();
  }
}

// Six waves per SIMD: 80 VGPRs, and six blocks' LDS (25 KB each) fit a CU.
template <int K, bool ROWS>
__global__ __launch_bounds__(kReduceBlock) __attribute__((amdgpu_waves_per_eu(6))) void reduce_chain_kernel(BackwardArgs A) {
  constexpr int AS = acc_stride(K), NQ = AS / 4;
  __shared__ __align__(16) float s_acc[kReduceGaussians][AS];
  const int64_t i0 = int64_t(blockIdx.x) * kReduceGaussians;
  const int nb = int(min<int64_t>(kReduceGaussians, A.n - i0));

  // The chain rule's own inputs (thread t < 64 serves Gaussian i0 + t), read
  // now so that their latency overlaps the row sums.
  float cq[4] = {1.0f, 0.0f, 0.0f, 0.0f}, cls[3] = {0.0f, 0.0f, 0.0f}, clg = 0.0f;
  uint32_t ctc = 0;
  if (int(threadIdx.x) < nb) {
    const int64_t ic = i0 + threadIdx.x;
#pragma unroll
    for (int k = 0; k < 4; ++k) cq[k] = A.quats[4 * ic + k];
#pragma unroll
    for (int k = 0; k < 3; ++k) cls[k] = A.log_scales[3 * ic + k];
    clg = A.logits[ic];
    ctc = A.tile_count[ic];
  }
  if constexpr (ROWS) {
    sum_rows<AS>(A, i0, nb, s_acc);
  } else {
    // the atomic modes' accumulators (zeroed before the backward), coalesced
    for (int e = threadIdx.x; e < kReduceGaussians * NQ; e += kReduceBlock)
      reinterpret_cast<float4*>(&s_acc[0][0])[e] =
          e < nb * NQ ? reinterpret_cast<const float4*>(A.acc)[i0 * NQ + e] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    __syncthreads();
  }

  for (int e = threadIdx.x; e < nb * 3 * K; e += kReduceBlock) {
    const int gl = e / (3 * K), v = e % (3 * K);
    A.g_sh[(i0 + gl) * 3 * K + v] = s_acc[gl][10 + v];
  }
  if (int(threadIdx.x) >= nb) return;
  const int64_t i = i0 + threadIdx.x;
  const float* acc = s_acc[threadIdx.x];
  float* gm = A.g_means + 3 * i;
  float* gs = A.g_log_scales + 3 * i;
  float* gq = A.g_quats + 4 * i;
  if (ctc == 0) {  // culled: no ray can reach it (its sums are zero)
    for (int k = 0; k < 3; ++k) gm[k] = gs[k] = 0.0f;
    for (int k = 0; k < 4; ++k) gq[k] = 0.0f;
    A.g_logits[i] = 0.0f;
    return;
  }
  const double qw0 = cq[0], qx0 = cq[1], qy0 = cq[2], qz0 = cq[3];
  const double inv_qn = 1.0 / sqrt(qw0 * qw0 + qx0 * qx0 + qy0 * qy0 + qz0 * qz0);
  const double w = qw0 * inv_qn, x = qx0 * inv_qn, y = qy0 * inv_qn, z = qz0 * inv_qn;
  const double R[3][3] = {{1.0 - 2.0 * (y * y + z * z), 2.0 * (x * y - w * z), 2.0 * (x * z + w * y)},
                          {2.0 * (x * y + w * z), 1.0 - 2.0 * (x * x + z * z), 2.0 * (y * z - w * x)},
                          {2.0 * (x * z - w * y), 2.0 * (y * z + w * x), 1.0 - 2.0 * (x * x + y * y)}};
  double s[3], is[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    s[k] = exp(double(cls[k]));
    is[k] = 1.0 / s[k];
  }
  const double go[3] = {acc[0], acc[1], acc[2]};
  const double B[3][3] = {{acc[3], acc[6], acc[7]}, {acc[6], acc[4], acc[8]}, {acc[7], acc[8], acc[5]}};
  // dL/dmu = -R S^-1 go
#pragma unroll
  for (int j = 0; j < 3; ++j)
    gm[j] = float(-(R[j][0] * go[0] * is[0] + R[j][1] * go[1] * is[1] + R[j][2] * go[2] * is[2]));
  // dL/dlog s_k = -B_kk
#pragma unroll
  for (int k = 0; k < 3; ++k) gs[k] = float(-B[k][k]);
  // dL/dR = R S B S^-1
  double GR[3][3];
#pragma unroll
  for (int j = 0; j < 3; ++j)
#pragma unroll
    for (int k = 0; k < 3; ++k)
      GR[j][k] = (R[j][0] * s[0] * B[0][k] + R[j][1] * s[1] * B[1][k] + R[j][2] * s[2] * B[2][k]) * is[k];
  // dL/d(unit quaternion), then through q / |q|
  double dq[4];
  dq[0] = 2.0 * (z * (GR[1][0] - GR[0][1]) + y * (GR[0][2] - GR[2][0]) + x * (GR[2][1] - GR[1][2]));
  dq[1] = 2.0 * (y * (GR[0][1] + GR[1][0]) + z * (GR[0][2] + GR[2][0]) + w * (GR[2][1] - GR[1][2])) -
          4.0 * x * (GR[1][1] + GR[2][2]);
  dq[2] = 2.0 * (x * (GR[0][1] + GR[1][0]) + w * (GR[0][2] - GR[2][0]) + z * (GR[1][2] + GR[2][1])) -
          4.0 * y * (GR[0][0] + GR[2][2]);
  dq[3] = 2.0 * (w * (GR[1][0] - GR[0][1]) + x * (GR[0][2] + GR[2][0]) + y * (GR[1][2] + GR[2][1])) -
          4.0 * z * (GR[0][0] + GR[1][1]);
  const double proj = w * dq[0] + x * dq[1] + y * dq[2] + z * dq[3];
  const double qv[4] = {w, x, y, z};
#pragma unroll
  for (int k = 0; k < 4; ++k) gq[k] = float((dq[k] - qv[k] * proj) * inv_qn);
  const double sig = 1.0 / (1.0 + exp(-double(clg)));  // as in the bounds kernel
  A.g_logits[i] = float(sig * (1.0 - sig) * double(acc[9]));
}

template <int TILE, int K>
hipError_t launch_tk(const BackwardArgs& args, hipStream_t s) {
  constexpr int AS = acc_stride(K);
  BackwardArgs a = args;
  a.rows_per_pair = TILE * TILE / 64;
  const int n_tiles = a.tiles_x * a.tiles_y;
  hipError_t e = hipSuccess;
  const bool hybrid = a.mode == GART_BACKWARD_HYBRID;
  const bool rows = a.mode == GART_BACKWARD_GATHER || a.mode == GART_BACKWARD_GATHER_WAVE || hybrid;
  if (rows && (e = fill_u8(a.row_flag, 0, a.pair_count * a.rows_per_pair, s)) != hipSuccess) return e;
  if (!rows && (e = fill_f32(a.acc, 0.0f, a.n * AS, s)) != hipSuccess) return e;
  if ((e = record(a.ev[0], s)) != hipSuccess) return e;
  if (n_tiles > 0) {
    switch (a.mode) {
      case GART_BACKWARD_GATHER:
        switch (a.lt_format) {
          case GART_LT_FULL: gather_kernel<TILE, K, false, false, GART_LT_FULL><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
          case GART_LT_HALF: gather_kernel<TILE, K, false, false, GART_LT_HALF><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
          case GART_LT_FIXED16: gather_kernel<TILE, K, false, false, GART_LT_FIXED16><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
          default: return hipErrorInvalidValue;
        }
        break;
      case GART_BACKWARD_GATHER_WAVE:
        switch (a.lt_format) {
          case GART_LT_FULL: gather_kernel<TILE, K, false, false, GART_LT_FULL, true><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
          case GART_LT_HALF: gather_kernel<TILE, K, false, false, GART_LT_HALF, true><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
          case GART_LT_FIXED16: gather_kernel<TILE, K, false, false, GART_LT_FIXED16, true><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
          default: return hipErrorInvalidValue;
        }
        break;
      case GART_BACKWARD_GATHER_ATOMIC:
        switch (a.lt_format) {
          case GART_LT_FULL: gather_kernel<TILE, K, true, false, GART_LT_FULL><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
          case GART_LT_HALF: gather_kernel<TILE, K, true, false, GART_LT_HALF><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
          case GART_LT_FIXED16: gather_kernel<TILE, K, true, false, GART_LT_FIXED16><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
          default: return hipErrorInvalidValue;
        }
        break;
      case GART_BACKWARD_SCATTER:
        switch (a.lt_format) {
          case GART_LT_FULL: scatter_kernel<TILE, K, GART_LT_FULL><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
          case GART_LT_HALF: scatter_kernel<TILE, K, GART_LT_HALF><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
          case GART_LT_FIXED16: scatter_kernel<TILE, K, GART_LT_FIXED16><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
          default: return hipErrorInvalidValue;
        }
        break;
      case GART_BACKWARD_HYBRID:
        switch (a.lt_format) {
          case GART_LT_T_ONLY:
            gather_kernel<TILE, K, false, true, GART_LT_T_ONLY><<<n_tiles, TILE * TILE, 0, s>>>(a);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            hybrid_pixel_kernel<TILE, K, GART_LT_T_ONLY><<<n_tiles, TILE * TILE, 0, s>>>(a);
            break;
          case GART_LT_T_HALF:
            gather_kernel<TILE, K, false, true, GART_LT_T_HALF><<<n_tiles, TILE * TILE, 0, s>>>(a);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            hybrid_pixel_kernel<TILE, K, GART_LT_T_HALF><<<n_tiles, TILE * TILE, 0, s>>>(a);
            break;
          case GART_LT_T_LOG16:
            gather_kernel<TILE, K, false, true, GART_LT_T_LOG16><<<n_tiles, TILE * TILE, 0, s>>>(a);
            if ((e = hipGetLastError()) != hipSuccess) return e;
            hybrid_pixel_kernel<TILE, K, GART_LT_T_LOG16><<<n_tiles, TILE * TILE, 0, s>>>(a);
            break;
          default: return hipErrorInvalidValue;
        }
        break;
      default: return hipErrorInvalidValue;
    }
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  if ((e = record(a.ev[1], s)) != hipSuccess) return e;
  if ((e = record(a.ev[2], s)) != hipSuccess) return e;
  if (a.n > 0) {
    const int64_t blocks = ceil_div(a.n, kReduceGaussians);
    if (rows)
      reduce_chain_kernel<K, true><<<blocks, kReduceBlock, 0, s>>>(a);
    else
      reduce_chain_kernel<K, false><<<blocks, kReduceBlock, 0, s>>>(a);
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return record(a.ev[3], s);
}

template <int TILE>
hipError_t launch_t(const BackwardArgs& a, hipStream_t s) {
  switch (a.sh_k) {
    case 1: return launch_tk<TILE, 1>(a, s);
    case 4: return launch_tk<TILE, 4>(a, s);
    case 9: return launch_tk<TILE, 9>(a, s);
    case 16: return launch_tk<TILE, 16>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_backward(const BackwardArgs& a, hipStream_t s) {
  return a.tile == 16 ? launch_t<16>(a, s) : launch_t<8>(a, s);
}

}  // namespace gart
