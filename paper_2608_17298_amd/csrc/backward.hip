// Backward pass (Sec. 4.4): primitive-centric gather over (tile, primitive)
// pairs, and the pixel-centric scatter control (Sec. 3.5).
//
// Per composited hit of Gaussian i at a pixel with upstream gradient g,
// colour in front L, transmittance in front T (read from the intermediate
// buffer), final pixel colour C and colour behind S = C - L - T a c:
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

// Gradient contribution of one composited hit, in the accumulator layout.
template <int K>
__device__ __forceinline__ void hit_grad(double D2, const double xg[3], double sigma, const float sh[3 * K],
                                         const float Y[K], const float C[3], const float g[3], float4 lt,
                                         float out[acc_width(K)]) {
  const float rho = expf(float(-0.5 * D2));
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
  const float T = lt.w;
  const float Lc[3] = {lt.x, lt.y, lt.z};
  const float ta = T * a;
  const float inv = 1.0f / (1.0f - a);
  float dlda = 0.0f;
  float dc[3];
#pragma unroll
  for (int ch = 0; ch < 3; ++ch) {
    const float S = C[ch] - Lc[ch] - ta * c[ch];
    dlda = fmaf(g[ch], T * c[ch] - S * inv, dlda);
    dc[ch] = pos[ch] ? ta * g[ch] : 0.0f;
  }
  const float u2 = -a * dlda;
  const float x = float(xg[0]), y = float(xg[1]), z = float(xg[2]);
  out[0] = u2 * x;
  out[1] = u2 * y;
  out[2] = u2 * z;
  out[3] = u2 * x * x;
  out[4] = u2 * y * y;
  out[5] = u2 * z * z;
  out[6] = u2 * x * y;
  out[7] = u2 * x * z;
  out[8] = u2 * y * z;
  out[9] = dlda * rho;
#pragma unroll
  for (int k = 0; k < K; ++k)
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) out[10 + 3 * k + ch] = dc[ch] * Y[k];
}

// ---------------------------------------------------------------------------
// Gather: one workgroup per tile; lane j owns pairs j, j+NT, ... of the
// tile's list (ordered by depth lower bound).  Per pixel state is staged in
// LDS once per tile.
// ---------------------------------------------------------------------------
template <int TILE, int K, bool ATOMIC>
__global__ __launch_bounds__(TILE* TILE) void gather_kernel(BackwardArgs A) {
  constexpr int NT = TILE * TILE;
  constexpr int AW = acc_width(K), AS = acc_stride(K);
  constexpr double kInf = __builtin_huge_val();

  __shared__ double s_d[3][NT];
  __shared__ float s_Y[K][NT];
  __shared__ float s_C[3][NT];
  __shared__ float s_g[3][NT];
  __shared__ double s_tend[NT];
  __shared__ uint32_t s_iend[NT];
  __shared__ double s_wmax[NT / 64];

  const int n_tiles = A.tiles_x * A.tiles_y;
  const int tile = xcd_tile(blockIdx.x, n_tiles);
  const int tx = tile % A.tiles_x, ty = tile / A.tiles_x;
  const int ox = tx * TILE, oy = ty * TILE;
  const int tid = threadIdx.x;

  {
    const int px = ox + tid % TILE, py = oy + tid / TILE;
    const bool valid = px < A.cam.W && py < A.cam.H;
    double d[3];
    pixel_ray(A.cam, valid ? px : 0, valid ? py : 0, d);
    float Y[K];
    sh_basis<K>(float(d[0]), float(d[1]), float(d[2]), Y);
#pragma unroll
    for (int k = 0; k < 3; ++k) s_d[k][tid] = d[k];
#pragma unroll
    for (int k = 0; k < K; ++k) s_Y[k][tid] = Y[k];
    double tend = -kInf;
    uint32_t iend = 0;
    if (valid) {
      const int64_t p = int64_t(py) * A.cam.W + px;
#pragma unroll
      for (int ch = 0; ch < 3; ++ch) {
        s_C[ch][tid] = A.image[3 * p + ch];
        s_g[ch][tid] = A.dl_dimage[3 * p + ch];
      }
      const gart_pixel_state st = A.pixel_state[p];
      tend = st.tau_end;
      iend = st.id_end;
    } else {
#pragma unroll
      for (int ch = 0; ch < 3; ++ch) s_C[ch][tid] = s_g[ch][tid] = 0.0f;
    }
    s_tend[tid] = tend;
    s_iend[tid] = iend;
    double m = tend;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) m = fmax(m, __shfl_xor(m, off));
    if (__lane_id() == 0) s_wmax[tid / 64] = m;
  }
  __syncthreads();
  double tmax = s_wmax[0];
#pragma unroll
  for (int w = 1; w < NT / 64; ++w) tmax = fmax(tmax, s_wmax[w]);

  const int64_t beg = A.tile_range[tile], end = A.tile_range[tile + 1];
  uint32_t n_pairs = 0, n_hits = 0, n_tests = 0, n_atom = 0, n_active = 0;
  for (int64_t j = beg + tid; j < end; j += NT) {
    const uint32_t i = A.pair_prim[j];
    const double* G = A.geom + int64_t(kGeomStride) * i;
    if (G[kGeoKey] > tmax) break;  // this and every later pair lie behind every ray's end
    ++n_pairs;
    double W[9], og[3];
#pragma unroll
    for (int k = 0; k < 9; ++k) W[k] = G[k];
#pragma unroll
    for (int k = 0; k < 3; ++k) og[k] = G[kGeoOg + k];
    const double D2c = G[kGeoD2c], sigma = G[kGeoSigma];
    const int4 r = *reinterpret_cast<const int4*>(A.rect + 4 * int64_t(i));
    float sh[3 * K];
    const float* shp = A.sh + int64_t(i) * (3 * K);
#pragma unroll
    for (int k = 0; k < 3 * K; ++k) sh[k] = shp[k];
    const int xa = max(r.x, ox), xb = min(r.z, ox + TILE - 1);
    const int ya = max(r.y, oy), yb = min(r.w, oy + TILE - 1);
    int64_t idx = A.lt_offset[i] + lt_local_index(r.x, r.y, r.z, r.w, TILE, xa, ya);
    float acc[AW];
#pragma unroll
    for (int v = 0; v < AW; ++v) acc[v] = 0.0f;
    bool any = false;
    for (int y = ya; y <= yb; ++y) {
      for (int x = xa; x <= xb; ++x, ++idx) {
        const int lp = (y - oy) * TILE + (x - ox);
        const double d[3] = {s_d[0][lp], s_d[1][lp], s_d[2][lp]};
        double tau, D2, xg[3];
        ++n_tests;
        if (!ray_hit(W, og, D2c, d, &tau, &D2, xg)) continue;
        if (key_less(s_tend[lp], s_iend[lp], tau, i)) continue;  // behind the ray's last composited hit
        ++n_hits;
        any = true;
        const float4 lt = A.lt[idx];
        float Y[K];
#pragma unroll
        for (int k = 0; k < K; ++k) Y[k] = s_Y[k][lp];
        const float C[3] = {s_C[0][lp], s_C[1][lp], s_C[2][lp]};
        const float g[3] = {s_g[0][lp], s_g[1][lp], s_g[2][lp]};
        float h[AW];
        hit_grad<K>(D2, xg, sigma, sh, Y, C, g, lt, h);
#pragma unroll
        for (int v = 0; v < AW; ++v) acc[v] += h[v];
      }
    }
    if (!any) continue;
    ++n_active;
    if constexpr (ATOMIC) {
      float* dst = A.acc + int64_t(i) * AS;
#pragma unroll
      for (int v = 0; v < AW; ++v) unsafeAtomicAdd(dst + v, acc[v]);
      n_atom += AW;
    } else {
      const int tx0 = r.x / TILE, ty0 = r.y / TILE, tx1 = r.z / TILE;
      const int64_t row = A.pair_offset[i] + int64_t(ty - ty0) * (tx1 - tx0 + 1) + (tx - tx0);
      float4* dst = reinterpret_cast<float4*>(A.rows + row * AS);
#pragma unroll
      for (int v = 0; v < AS; v += 4) {
        float4 q;
        q.x = v + 0 < AW ? acc[v + 0] : 0.0f;
        q.y = v + 1 < AW ? acc[v + 1] : 0.0f;
        q.z = v + 2 < AW ? acc[v + 2] : 0.0f;
        q.w = v + 3 < AW ? acc[v + 3] : 0.0f;
        dst[v / 4] = q;
      }
      A.row_flag[row] = 1;
    }
  }
  if (A.counters) {
    count_add(A.counters + GART_CNT_BWD_PAIRS, n_pairs);
    count_add(A.counters + GART_CNT_BWD_ACTIVE, n_active);
    count_add(A.counters + GART_CNT_BWD_HITS, n_hits);
    count_add(A.counters + GART_CNT_BWD_TESTS, n_tests);
    count_add(A.counters + GART_CNT_BWD_ATOMICS, n_atom);
  }
}

// ---------------------------------------------------------------------------
// Scatter control: one lane per pixel walks the tile's list front to back
// and adds every composited hit's gradient with float atomics.
// ---------------------------------------------------------------------------
template <int TILE, int K>
__global__ __launch_bounds__(TILE* TILE) void scatter_kernel(BackwardArgs A) {
  constexpr int NT = TILE * TILE;
  constexpr int AW = acc_width(K), AS = acc_stride(K);
  constexpr double kInf = __builtin_huge_val();
  __shared__ __align__(16) double s_row[NT * kRow];

  const int n_tiles = A.tiles_x * A.tiles_y;
  const int tile = xcd_tile(blockIdx.x, n_tiles);
  const int tx = tile % A.tiles_x, ty = tile / A.tiles_x;
  const int tid = threadIdx.x;
  const int px = tx * TILE + tid % TILE, py = ty * TILE + tid / TILE;
  const bool valid = px < A.cam.W && py < A.cam.H;

  double d[3];
  pixel_ray(A.cam, valid ? px : 0, valid ? py : 0, d);
  float Y[K];
  sh_basis<K>(float(d[0]), float(d[1]), float(d[2]), Y);
  float C[3] = {0, 0, 0}, g[3] = {0, 0, 0};
  double tend = -kInf;
  uint32_t iend = 0;
  if (valid) {
    const int64_t p = int64_t(py) * A.cam.W + px;
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) {
      C[ch] = A.image[3 * p + ch];
      g[ch] = A.dl_dimage[3 * p + ch];
    }
    const gart_pixel_state st = A.pixel_state[p];
    tend = st.tau_end;
    iend = st.id_end;
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
      for (int k = 0; k < 15; ++k) row[k] = G[k];
      row[15] = __longlong_as_double(A.lt_offset[id]);
      const int4 r = *reinterpret_cast<const int4*>(A.rect + 4 * int64_t(id));
      int* ri = reinterpret_cast<int*>(row + 16);
      ri[0] = r.x;
      ri[1] = r.y;
      ri[2] = r.z;
      ri[3] = r.w;
      reinterpret_cast<uint32_t*>(row + 18)[0] = id;
    }
    __syncthreads();
    if (!done) {
      for (int c = 0; c < nb; ++c) {
        const double* row = s_row + c * kRow;
        if (row[14] > tend) {  // every remaining Gaussian lies behind this ray's end
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
        const float4 lt = A.lt[li];
        float sh[3 * K];
        const float* shp = A.sh + int64_t(id) * (3 * K);
#pragma unroll
        for (int k = 0; k < 3 * K; ++k) sh[k] = shp[k];
        float h[AW];
        hit_grad<K>(D2, xg, row[13], sh, Y, C, g, lt, h);
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
// serves 64 Gaussians.  Reduction: sixteen lanes per Gaussian, lane q reads
// float4 q of each active row (rows are contiguous in emission order), 16
// row flags are read at once and up to four rows are loaded per step.
// Chain rule: one Gaussian per lane of the first wave.  SH gradients: all
// threads, coalesced.
// ---------------------------------------------------------------------------
constexpr int kReduceLanes = 16;
constexpr int kReduceBlock = 256;
constexpr int kReduceGaussians = 64;

template <int K, bool ROWS>
__global__ __launch_bounds__(kReduceBlock) void reduce_chain_kernel(BackwardArgs A) {
  constexpr int AS = acc_stride(K), NQ = AS / 4;
  constexpr int GROUPS = kReduceBlock / kReduceLanes;
  static_assert(NQ <= kReduceLanes, "accumulator row wider than a lane group");
  __shared__ __align__(16) float s_acc[kReduceGaussians][AS];
  const int64_t i0 = int64_t(blockIdx.x) * kReduceGaussians;
  const int grp = threadIdx.x / kReduceLanes, q = threadIdx.x % kReduceLanes;
  const int shift = (threadIdx.x % 64) / kReduceLanes * kReduceLanes;

  for (int gl = grp; gl < kReduceGaussians; gl += GROUPS) {
    const int64_t i = i0 + gl;
    const bool live = i < A.n;
    const uint32_t tc = live ? A.tile_count[i] : 0u;
    float4 a = make_float4(0.0f, 0.0f, 0.0f, 0.0f);
    if constexpr (ROWS) {
      const float4* rows = reinterpret_cast<const float4*>(A.rows);
      const int64_t r0 = live ? A.pair_offset[i] : 0, r1 = r0 + tc;
      for (int64_t rb = r0; rb < r1; rb += kReduceLanes) {
        const int64_t rq = rb + q;
        const bool act = rq < r1 && A.row_flag[rq] != 0;
        uint32_t m = uint32_t(__ballot(act) >> shift) & 0xffffu;
        while (m) {
          int k[4];
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            k[u] = m ? __ffs(m) - 1 : -1;
            m &= m ? m - 1 : 0u;
          }
          float4 v[4];
#pragma unroll
          for (int u = 0; u < 4; ++u)
            v[u] = (k[u] >= 0 && q < NQ) ? rows[(rb + k[u]) * NQ + q] : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
          for (int u = 0; u < 4; ++u) {
            a.x += v[u].x;
            a.y += v[u].y;
            a.z += v[u].z;
            a.w += v[u].w;
          }
        }
      }
    } else if (live && tc && q < NQ) {
      a = reinterpret_cast<const float4*>(A.acc)[i * NQ + q];
    }
    if (q < NQ) reinterpret_cast<float4*>(s_acc[gl])[q] = a;
  }
  __syncthreads();

  const int nb = int(min<int64_t>(kReduceGaussians, A.n - i0));
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
  if (A.tile_count[i] == 0) {  // culled: no ray can reach it (its sums are zero)
    for (int k = 0; k < 3; ++k) gm[k] = gs[k] = 0.0f;
    for (int k = 0; k < 4; ++k) gq[k] = 0.0f;
    A.g_logits[i] = 0.0f;
    return;
  }
  const double qw0 = A.quats[4 * i], qx0 = A.quats[4 * i + 1], qy0 = A.quats[4 * i + 2], qz0 = A.quats[4 * i + 3];
  const double inv_qn = 1.0 / sqrt(qw0 * qw0 + qx0 * qx0 + qy0 * qy0 + qz0 * qz0);
  const double w = qw0 * inv_qn, x = qx0 * inv_qn, y = qy0 * inv_qn, z = qz0 * inv_qn;
  const double R[3][3] = {{1.0 - 2.0 * (y * y + z * z), 2.0 * (x * y - w * z), 2.0 * (x * z + w * y)},
                          {2.0 * (x * y + w * z), 1.0 - 2.0 * (x * x + z * z), 2.0 * (y * z - w * x)},
                          {2.0 * (x * z - w * y), 2.0 * (y * z + w * x), 1.0 - 2.0 * (x * x + y * y)}};
  double s[3], is[3];
#pragma unroll
  for (int k = 0; k < 3; ++k) {
    s[k] = exp(double(A.log_scales[3 * i + k]));
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
  const double sig = A.geom[int64_t(kGeomStride) * i + kGeoSigma];
  A.g_logits[i] = float(sig * (1.0 - sig) * double(acc[9]));
}

template <int TILE, int K>
hipError_t launch_tk(const BackwardArgs& a, hipStream_t s) {
  constexpr int AS = acc_stride(K);
  const int n_tiles = a.tiles_x * a.tiles_y;
  hipError_t e = hipSuccess;
  const bool rows = a.mode == GART_BACKWARD_GATHER;
  e = rows ? fill_u8(a.row_flag, 0, a.pair_count, s) : fill_f32(a.acc, 0.0f, a.n * AS, s);
  if (e != hipSuccess) return e;
  if ((e = record(a.ev[0], s)) != hipSuccess) return e;
  if (n_tiles > 0) {
    if (rows)
      gather_kernel<TILE, K, false><<<n_tiles, TILE * TILE, 0, s>>>(a);
    else if (a.mode == GART_BACKWARD_GATHER_ATOMIC)
      gather_kernel<TILE, K, true><<<n_tiles, TILE * TILE, 0, s>>>(a);
    else
      scatter_kernel<TILE, K><<<n_tiles, TILE * TILE, 0, s>>>(a);
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
