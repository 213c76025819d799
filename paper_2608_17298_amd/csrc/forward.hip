// Forward software trace (Sec. 3.2-3.3, Eq. 3-8) writing the (L, T)
// intermediate buffer in primitive-major order (Sec. 4.3, Eq. 16).
//
// One workgroup per tile, one lane per pixel.  The tile's Gaussian list is
// ordered by a conservative lower bound on the depth at which each Gaussian
// can be hit, so a lane can stream it front to back with a small sorted hit
// buffer held in registers: a buffered hit is final -- and is composited --
// as soon as its depth is below the lower bound of the next Gaussian in the
// list.  The result is exactly the (tau, index) order.  If the buffer
// overflows, the largest hits are dropped and the lane later rescans the
// list from the first Gaussian it dropped, skipping hits already
// composited; compositing stops once the transmittance falls below t_min.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>

#include "ops.h"

namespace gart {
namespace {

#ifndef GART_FWD_KB
#define GART_FWD_KB 14
#endif
#ifndef GART_FWD_FLUSH
#define GART_FWD_FLUSH 16
#endif
#ifndef GART_FWD_BATCH
#define GART_FWD_BATCH 256
#endif
// Minimum waves per SIMD asked of the register allocator (default: none).
#ifdef GART_FWD_WAVES
#define GART_FWD_LAUNCH_BOUNDS(n) __launch_bounds__(n, GART_FWD_WAVES)
#else
#define GART_FWD_LAUNCH_BOUNDS(n) __launch_bounds__(n)
#endif

constexpr int kRow = 20;  // doubles per staged Gaussian in LDS
// Each rescan composites at least one hit per rescanning lane, so the pass
// count is bounded by the hits of a tile; this cap only guards against a
// defect turning into a hang.
constexpr int kMaxPasses = 1 << 20;
// row: [0..8] W, [9..11] o_g, [12] D2c, [13] sigma, [14] depth key,
// [15] O_prim (int64 bits), [16..17] rect (4 x int32), [18] index (uint32)

template <int TILE, int K, int FMT>
__global__ GART_FWD_LAUNCH_BOUNDS(TILE* TILE) void forward_kernel(ForwardArgs A) {
  constexpr int NT = TILE * TILE;
  constexpr int KB = GART_FWD_KB;  // per-lane hit buffer (registers)
  constexpr int kFlushEvery = GART_FWD_FLUSH;
  constexpr int NB = GART_FWD_BATCH < NT ? GART_FWD_BATCH : NT;  // candidates staged per batch
  constexpr double kInf = __builtin_huge_val();

  constexpr int KP = (K + 3) & ~3;  // SH basis row padded to 16 bytes
  __shared__ __align__(16) double s_row[NB * kRow];
  __shared__ __align__(16) float s_Y[NT][KP];  // SH basis of each pixel's ray
  __shared__ float s_key[NB + 1];
  __shared__ unsigned s_restart;

  const int n_tiles = A.tiles_x * A.tiles_y;
  const int tile = xcd_tile(blockIdx.x, n_tiles, A.tiles_x);
  const int tx = tile % A.tiles_x, ty = tile / A.tiles_x;
  const int tid = threadIdx.x;
  const int px = tx * TILE + tid % TILE, py = ty * TILE + tid / TILE;
  const bool valid = px < A.cam.W && py < A.cam.H;

  double d[3];
  pixel_ray(A.cam, valid ? px : 0, valid ? py : 0, d);
  {
    float Y[K];
    sh_basis<K>(float(d[0]), float(d[1]), float(d[2]), Y);
#pragma unroll
    for (int k = 0; k < KP; ++k) s_Y[tid][k] = k < K ? Y[k] : 0.0f;
  }

  const int64_t beg = A.tile_range[tile], end = A.tile_range[tile + 1];

  double T = 1.0, L0 = 0.0, L1 = 0.0, L2 = 0.0;
  bool done = !valid;     // terminated (or no pixel)
  bool finished = false;  // every hit composited
  bool stalled = false;   // must wait for a rescan
  uint32_t n_hits = 0, n_tests = 0, n_drops = 0;
  double last_tau = -kInf;
  uint32_t last_id = 0;
  double end_tau = kInf;
  uint32_t end_id = kNoPrim;

  // Hit buffer: depth, alpha, tile-list position and Gaussian index of each
  // pending hit, sorted by (depth, index); the (L,T) address is recomputed
  // from the Gaussian's rectangle when the hit is composited, which keeps an
  // entry at six registers.
  double bt[KB], ba[KB];
  uint32_t bc[KB], bid[KB];
  int cnt = 0;
  double e_tau = kInf;  // smallest dropped hit (all buffered hits are smaller)
  uint32_t e_id = kNoPrim;
  uint32_t jr = UINT_MAX;  // first list position holding a dropped hit
  // A rescan starts the wave at the smallest jr of its lanes; a lane skips
  // the positions before its own jr (from): every hit there was composited
  // in an earlier pass.
  uint32_t from = 0;
#pragma unroll
  for (int s = 0; s < KB; ++s) {
    bt[s] = kInf;
    ba[s] = 0.0;
    bc[s] = 0;
    bid[s] = kNoPrim;
  }

  auto drop = [&](double t, uint32_t id, uint32_t c) {
    ++n_drops;
    if (key_less(t, id, e_tau, e_id)) {
      e_tau = t;
      e_id = id;
    }
    jr = min(jr, c);
  };

  auto composite_front = [&]() {
    const double a = ba[0];
    const uint32_t id = bid[0];
    const float* shp = A.sh + int64_t(id) * (3 * K);
    const int4 rr = *reinterpret_cast<const int4*>(A.rect + 4 * int64_t(id));
    const int64_t lt_base = A.lt_offset[id] + lt_local_index(rr.x, rr.y, rr.z, rr.w, TILE, px, py);
    float c[3] = {0.5f, 0.5f, 0.5f};
#pragma unroll
    for (int k = 0; k < KP; k += 4) {
      const float4 y4 = *reinterpret_cast<const float4*>(&s_Y[tid][k]);
      const float yk[4] = {y4.x, y4.y, y4.z, y4.w};
#pragma unroll
      for (int u = 0; u < 4; ++u)
        if (k + u < K)
#pragma unroll
          for (int ch = 0; ch < 3; ++ch) c[ch] = fmaf(shp[3 * (k + u) + ch], yk[u], c[ch]);
    }
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) c[ch] = fmaxf(c[ch], 0.0f);
    // k-th composited hit of this pixel -> its list position (read by the
    // gather backward)
    A.hit_list[int64_t(NT) * (beg + n_hits) + tid] = bc[0];
    const int64_t e = lt_base;
    if constexpr (FMT == GART_LT_FULL) {
      A.lt[e] = make_uint4(color_fixed(L0, A.inv_color_step), color_fixed(L1, A.inv_color_step),
                           color_fixed(L2, A.inv_color_step), __float_as_uint(float(T)));
    } else if constexpr (FMT == GART_LT_T_ONLY) {
      reinterpret_cast<float*>(A.lt)[e] = float(T);
    } else if constexpr (FMT == GART_LT_HALF) {
      reinterpret_cast<uint2*>(A.lt)[e] = make_uint2(half_bits(float(L0)) | (half_bits(float(L1)) << 16),
                                                     half_bits(float(L2)) | (half_bits(float(T)) << 16));
    } else if constexpr (FMT == GART_LT_FIXED16) {
      const double inv16 = A.inv_color_step * (1.0 / 65536.0);
      reinterpret_cast<uint2*>(A.lt)[e] = make_uint2(
          min(color_fixed(L0, inv16), 65535u) | (min(color_fixed(L1, inv16), 65535u) << 16),
          min(color_fixed(L2, inv16), 65535u) | (t_log16(float(T)) << 16));
    } else if constexpr (FMT == GART_LT_T_LOG16) {
      reinterpret_cast<uint16_t*>(A.lt)[e] = uint16_t(t_log16(float(T)));
    } else {
      reinterpret_cast<uint16_t*>(A.lt)[e] = uint16_t(half_bits(float(T)));
    }
    const double w = T * a;
    L0 = fma(w, double(c[0]), L0);
    L1 = fma(w, double(c[1]), L1);
    L2 = fma(w, double(c[2]), L2);
    T = T * (1.0 - a);
    ++n_hits;
    last_tau = bt[0];
    last_id = id;
    if (T < A.t_min) {
      done = true;
      end_tau = bt[0];
      end_id = id;
    }
#pragma unroll
    for (int s = 0; s + 1 < KB; ++s) {
      bt[s] = bt[s + 1];
      ba[s] = ba[s + 1];
      bc[s] = bc[s + 1];
      bid[s] = bid[s + 1];
    }
    bt[KB - 1] = kInf;  // unused slots hold depth +inf
    --cnt;
  };

  uint32_t restart = 0;
  int passes = 0;
  for (;;) {
    for (int64_t base = beg + restart; base < end; base += NB) {
      const int nb = int(min<int64_t>(NB, end - base));
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
        s_key[tid] = A.pair_key[base + tid];
      }
      if (tid == 0) {
        const int64_t nx = base + nb;
        s_key[nb] = (nx < end) ? A.pair_key[nx] : __int_as_float(0x7f800000);
      }
      __syncthreads();
      if (!done && !finished && !stalled) {
        for (int c = 0; c < nb; ++c) {
          // The candidate's whole staged row is read at once (one LDS round
          // trip; every lane reads the same address), then the rectangle
          // decides which lanes test it.
          const double* row = s_row + c * kRow;
          const int4 r = *reinterpret_cast<const int4*>(row + 16);
          double W[9], og[3];
#pragma unroll
          for (int k = 0; k < 9; ++k) W[k] = row[k];
#pragma unroll
          for (int k = 0; k < 3; ++k) og[k] = row[9 + k];
          double D2c = row[12], sig = row[13];
          uint32_t id = reinterpret_cast<const uint32_t*>(row + 18)[0];
          // materialise the row here, so that the compiler does not sink its
          // reads into the branch (a second LDS round trip per candidate)
#pragma unroll
          for (int k = 0; k < 9; ++k) asm volatile("" : "+v"(W[k]));
#pragma unroll
          for (int k = 0; k < 3; ++k) asm volatile("" : "+v"(og[k]));
          asm volatile("" : "+v"(D2c), "+v"(sig), "+v"(id));
          const bool inside = (uint32_t(base - beg) + uint32_t(c) >= from) & (px >= r.x) & (px <= r.z) &
                              (py >= r.y) & (py <= r.w);
          if (inside) {
            ++n_tests;
            double tau, D2, xg[3];
            if (ray_hit(W, og, D2c, d, &tau, &D2, xg) && key_less(last_tau, last_id, tau, id)) {
              const uint32_t cpos = uint32_t(base - beg) + uint32_t(c);
              if (!key_less(tau, id, e_tau, e_id)) {
                drop(tau, id, cpos);
              } else {
                bool ins = true;
                if (cnt == KB) {
                  if (!key_less(tau, id, bt[KB - 1], bid[KB - 1])) {
                    drop(tau, id, cpos);
                    ins = false;
                  } else {
                    drop(bt[KB - 1], bid[KB - 1], bc[KB - 1]);
                    cnt = KB - 1;
                  }
                }
                if (ins) {
                  const double a = sig * exp(-0.5 * D2);
                  // Position = entries with a smaller (depth, index) key.
                  // Unused slots hold depth +inf, so a strict depth count
                  // needs no occupancy test; equal depths (rare) also count
                  // the entries of smaller index.  Shift and placement are
                  // selects, not branches.
                  int pos = 0;
                  bool tie = false;
#pragma unroll
                  for (int s = 0; s < KB; ++s) {
                    pos += bt[s] < tau ? 1 : 0;
                    tie = tie || bt[s] == tau;
                  }
                  if (tie) {
#pragma unroll
                    for (int s = 0; s < KB; ++s) pos += (bt[s] == tau && bid[s] < id) ? 1 : 0;
                  }
#pragma unroll
                  for (int s = KB - 1; s >= 1; --s) {
                    const bool sh = s > pos, pl = s == pos;
                    bt[s] = sh ? bt[s - 1] : (pl ? tau : bt[s]);
                    ba[s] = sh ? ba[s - 1] : (pl ? a : ba[s]);
                    bc[s] = sh ? bc[s - 1] : (pl ? cpos : bc[s]);
                    bid[s] = sh ? bid[s - 1] : (pl ? id : bid[s]);
                  }
                  if (pos == 0) {
                    bt[0] = tau;
                    ba[0] = a;
                    bc[0] = cpos;
                    bid[0] = id;
                  }
                  ++cnt;
                }
              }
            }
          }
          // Composite the final hits every kFlushEvery Gaussians, at the end
          // of a batch, and whenever a lane's buffer is full -- for every
          // lane of the wave at once, so that each compositing step serves
          // more lanes.
          if (__ballot((c + 1) % kFlushEvery == 0 || c + 1 == nb || cnt == KB) != 0) {
            const double nk = double(s_key[c + 1]);
            while (cnt > 0 && bt[0] < nk && !done) composite_front();
            if (done) break;
            if (e_tau < kInf && nk > e_tau) {
              stalled = true;
              break;
            }
          }
        }
      }
      const bool busy = !done && !finished && !stalled;
      if (!__syncthreads_or(busy)) break;
    }
    // End of pass: every buffered hit is below the smallest dropped one and
    // no unscanned Gaussian can precede it.
    while (cnt > 0 && !done) composite_front();
    const bool need = !done && !finished && e_tau < kInf;
    if (!done && !need) finished = true;
    if (tid == 0) s_restart = UINT_MAX;
    __syncthreads();
    if (need) atomicMin(&s_restart, jr);
    __syncthreads();
    const unsigned rs = s_restart;
    __syncthreads();
    if (rs == UINT_MAX) break;
    if (passes >= kMaxPasses) {  // never expected: reported, not hidden
      if (tid == 0) atomicOr(A.status, unsigned(GART_FRAME_FORWARD_INCOMPLETE));
      break;
    }
    restart = rs;
    ++passes;
    if (need) {
      from = jr;
      e_tau = kInf;
      e_id = kNoPrim;
      jr = UINT_MAX;
      stalled = false;
      cnt = 0;
    }
  }

  if (valid) {
    const int64_t p = int64_t(py) * A.cam.W + px;
    A.image[3 * p + 0] = float(L0);
    A.image[3 * p + 1] = float(L1);
    A.image[3 * p + 2] = float(L2);
    gart_pixel_state st;
    st.tau_end = end_tau;
    st.id_end = end_id;
    st.n_hits = n_hits;
    st.color_fixed[0] = color_fixed(L0, A.inv_color_step);
    st.color_fixed[1] = color_fixed(L1, A.inv_color_step);
    st.color_fixed[2] = color_fixed(L2, A.inv_color_step);
    st.t_final = float(T);
    A.pixel_state[p] = st;
  }
  if (A.counters) {
    count_add(A.counters + GART_CNT_FWD_HITS, n_hits);
    count_add(A.counters + GART_CNT_FWD_TESTS, n_tests);
    count_add(A.counters + GART_CNT_FWD_DROPS, n_drops);
    if (tid == 0 && passes)
      atomicAdd(reinterpret_cast<unsigned long long*>(A.counters + GART_CNT_FWD_RESCANS), (unsigned long long)passes);
  }
}

template <int TILE, int K>
hipError_t launch_t(const ForwardArgs& a, hipStream_t s) {
  const int n_tiles = a.tiles_x * a.tiles_y;
  hipError_t e = record(a.ev_begin, s);
  if (e != hipSuccess) return e;
  switch (a.lt_format) {
    case GART_LT_FULL: forward_kernel<TILE, K, GART_LT_FULL><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
    case GART_LT_T_ONLY: forward_kernel<TILE, K, GART_LT_T_ONLY><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
    case GART_LT_HALF: forward_kernel<TILE, K, GART_LT_HALF><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
    case GART_LT_T_HALF: forward_kernel<TILE, K, GART_LT_T_HALF><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
    case GART_LT_FIXED16: forward_kernel<TILE, K, GART_LT_FIXED16><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
    case GART_LT_T_LOG16: forward_kernel<TILE, K, GART_LT_T_LOG16><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  if ((e = hipGetLastError()) != hipSuccess) return e;
  return record(a.ev_end, s);
}

template <int TILE>
hipError_t launch_k(const ForwardArgs& a, hipStream_t s) {
  switch (a.sh_k) {
    case 1: return launch_t<TILE, 1>(a, s);
    case 4: return launch_t<TILE, 4>(a, s);
    case 9: return launch_t<TILE, 9>(a, s);
    case 16: return launch_t<TILE, 16>(a, s);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace

hipError_t launch_forward(const ForwardArgs& a, hipStream_t s) {
  if (a.tiles_x * a.tiles_y <= 0) return hipSuccess;
  return a.tile == 16 ? launch_k<16>(a, s) : launch_k<8>(a, s);
}

}  // namespace gart
