// Forward software trace (Sec. 3.2-3.3, Eq. 3-8) writing the (L, T)
// intermediate buffer in primitive-major order (Sec. 4.3, Eq. 16).
//
// One workgroup per tile, one lane per pixel.  The tile's Gaussian list is
// ordered by a lower bound on the depth at which each Gaussian can be hit by
// a pixel ray of the tile, so a lane can stream it front to back with a small
// sorted buffer of pending hits: a buffered hit is final -- and is composited
// -- as soon as its depth is below the bound of the next Gaussian in the list.
// The result is exactly the (tau, index) order.  The buffer is a ring of KB
// entries per lane in LDS, laid out [slot][lane], so the lanes of a wave
// touch consecutive words whatever slot each is at (no bank conflicts); a new
// hit is inserted from the tail, which with tight bounds is nearly always an
// append.  If a ring overflows, its largest hits are dropped and the lane
// later rescans the list from the first Gaussian it dropped, skipping hits
// already composited; compositing stops once the transmittance falls below
// t_min.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <climits>

#include "ops.h"

namespace gart {
namespace {

#ifndef GART_FWD_FLUSH
#define GART_FWD_FLUSH 8
#endif
#ifndef GART_FWD_BATCH
#define GART_FWD_BATCH 16
#endif

constexpr int kRow = 20;  // doubles per staged Gaussian in LDS
// row: [0..8] W, [9..11] o_g, [12] D2c, [13] sigma, [14] depth key,
// [15] O_prim (int64 bits), [16..17] rect (4 x int32), [18] index (uint32)

// Each rescan composites at least one hit per rescanning lane, so the pass
// count is bounded by the hits of a tile; this cap only guards against a
// defect turning into a hang, and is reported in the frame status if reached.
constexpr int kMaxPasses = 1 << 20;

// Minimum 64-thread workgroups per CU asked of the register allocator (default: none).
#ifdef GART_FWD_MINBLOCKS
#define GART_FWD_LAUNCH_BOUNDS(n) __launch_bounds__(n) __attribute__((amdgpu_waves_per_eu(GART_FWD_MINBLOCKS / 4)))
#else
#define GART_FWD_LAUNCH_BOUNDS(n) __launch_bounds__(n)
#endif

template <int TILE, int K, int FMT, int KB>
__global__ GART_FWD_LAUNCH_BOUNDS(TILE* TILE) void forward_kernel(ForwardArgs A) {
  constexpr int NT = TILE * TILE;
  constexpr int kFlushEvery = GART_FWD_FLUSH;
  constexpr int NB = GART_FWD_BATCH < NT ? GART_FWD_BATCH : NT;  // candidates staged per batch
  constexpr double kInf = __builtin_huge_val();
  static_assert(KB >= 2 && (KB & (KB - 1)) == 0, "ring of a power-of-two size");

  __shared__ __align__(16) double s_row[NB * kRow];
  __shared__ float s_key[NB + 1];
  __shared__ unsigned s_restart;
  // pending hits of each lane: depth rounded up to a float, alpha, and
  // (list position, Gaussian index) -- 20 bytes; the exact depth is
  // recomputed on the rare paths that need it.  Large rings keep the list
  // position only (16 bytes, the index is read from the list when needed):
  // the LDS saved raises occupancy where the ring is what limits it.
  constexpr bool kPosOnly = KB >= 16;
  __shared__ float s_btf[KB][NT];
  __shared__ double s_balpha[KB][NT];
  __shared__ uint32_t s_bpos[KB][NT];
  __shared__ uint32_t s_bid[kPosOnly ? 1 : KB][kPosOnly ? 1 : NT];

  const int n_tiles = A.tiles_x * A.tiles_y;
  const int tile = xcd_tile(blockIdx.x, n_tiles, A.tiles_x);
  const int tx = tile % A.tiles_x, ty = tile / A.tiles_x;
  const int tid = threadIdx.x;
  const int px = tx * TILE + tid % TILE, py = ty * TILE + tid / TILE;
  const bool valid = px < A.cam.W && py < A.cam.H;

  double d[3];
  pixel_ray(A.cam, valid ? px : 0, valid ? py : 0, d);
  // the tile's list keys are depths along the tile's axis; key k bounds the
  // depth of a hit on this pixel's ray by k * kscale
  double cax[3];
  tile_axis(A.cam, tx, ty, TILE, cax);
  const double kscale = key_scale(A.cam, cax, valid ? px : 0, valid ? py : 0);
  float Y[K];  // SH basis of this pixel's ray
  sh_basis<K>(float(d[0]), float(d[1]), float(d[2]), Y);

  const int64_t beg = A.tile_range[tile], end = A.tile_range[tile + 1];
  const int64_t hl_beg = A.hl_off[tile];  // this tile's first hit_list row
  // its rows (>= 1 if the tile has pairs); a hit beyond them, which the
  // bound on hits per pixel excludes, would overwrite the last row and is
  // reported in the frame status after the trace
  const uint32_t hl_last = uint32_t(max<int64_t>(A.hl_off[tile + 1] - hl_beg, 1) - 1);
  // Gaussian index of ring entry s
  auto entry_id = [&](int s) -> uint32_t {
    if constexpr (kPosOnly) return A.pair_prim[beg + s_bpos[s][tid]];
    else return s_bid[s][tid];
  };

  double T = 1.0, L0 = 0.0, L1 = 0.0, L2 = 0.0;
  bool done = !valid;     // terminated (or no pixel)
  bool finished = false;  // every hit composited
  bool stalled = false;   // must wait for a rescan
  uint32_t n_hits = 0, n_tests = 0, n_drops = 0;
  uint32_t visited = 0;  // one past the largest list position composited
  double last_tau = -kInf;
  uint32_t last_id = 0;
  double end_tau = kInf;
  uint32_t end_id = kNoPrim;

  int head = 0, cnt = 0;  // ring: entries head, head + 1, ... (mod KB), sorted by (depth, index)
  double e_tau = kInf;    // lower bound on the depths of dropped hits (every buffered hit is smaller)
  // The ring's head entry (depth bound, alpha, list position, index) and the
  // tail's depth bound are kept in registers: a plain append and each
  // compositing step then need no LDS round trip to find them.
  float head_tf = __int_as_float(0x7f800000);  // +inf if empty
  double head_a = 0.0;
  uint32_t head_pos = 0, head_id = 0;
  float tail_tf = 0.0f;                        // valid while cnt > 0
  uint32_t jr = UINT_MAX;  // first list position holding a dropped hit
  // A rescan starts the wave at the smallest jr of its lanes; a lane skips
  // the positions before its own jr (from): every hit there was composited
  // in an earlier pass.
  uint32_t from = 0;

  // A dropped hit at list position c whose depth is at least t_lb.
  auto drop = [&](double t_lb, uint32_t c) {
    ++n_drops;
    e_tau = fmin(e_tau, t_lb);
    jr = min(jr, c);
  };

  // Exact depth of Gaussian id's max-response point on this lane's ray (the
  // same evaluation as the trace's).
  auto exact_tau = [&](uint32_t id) {
    const double* G = A.geom + int64_t(kGeomStride) * id;
    double W[9], og[3];
#pragma unroll
    for (int k = 0; k < 9; ++k) W[k] = G[kGeoW + k];
#pragma unroll
    for (int k = 0; k < 3; ++k) og[k] = G[kGeoOg + k];
    double tau, D2, xg[3];
    ray_hit(W, og, G[kGeoD2c], d, &tau, &D2, xg);
    return tau;
  };

  // Inserts a hit smaller than every dropped one into a ring with room:
  // larger entries move up one slot, from the tail.
  // (tau, id) < entry s of the ring in (depth, index) order, tu = tau
  // rounded up to a float: rounding up is monotone, so unequal floats decide;
  // a tie of the floats is decided on the entry's exact depth
  auto before_entry = [&](double tau, float tu, uint32_t id, int s) {
    const float st = s_btf[s][tid];
    if (tu != st) return tu < st;
    const uint32_t sid = entry_id(s);
    return key_less(tau, id, exact_tau(sid), sid);
  };

  // Inserts a hit smaller than every dropped one into a ring with room:
  // larger entries move up one slot, from the tail.
  auto insert = [&](double tau, float tu, uint32_t id, uint32_t cpos, double a) {
    int j = cnt;
    if (cnt > 0 && !(tu > tail_tf)) {  // not above the tail: find the place from the tail down
      while (j > 0) {
        const int s = (head + j - 1) & (KB - 1);
        if (!before_entry(tau, tu, id, s)) break;
        const int t = (s + 1) & (KB - 1);
        s_btf[t][tid] = s_btf[s][tid];
        s_balpha[t][tid] = s_balpha[s][tid];
        s_bpos[t][tid] = s_bpos[s][tid];
        if constexpr (!kPosOnly) s_bid[t][tid] = s_bid[s][tid];
        --j;
      }
    }
    const int t = (head + j) & (KB - 1);
    s_btf[t][tid] = tu;
    s_balpha[t][tid] = a;
    s_bpos[t][tid] = cpos;
    if constexpr (!kPosOnly) s_bid[t][tid] = id;
    if (j == cnt) tail_tf = tu;
    if (j == 0) {
      head_tf = tu;
      head_a = a;
      head_pos = cpos;
      head_id = id;
    }
    ++cnt;
  };

  auto composite_front = [&]() {
    const double a = head_a;
    const uint32_t cpos = head_pos, id = head_id;
    visited = max(visited, cpos + 1u);
    const float* shp = A.sh + int64_t(id) * (3 * K);
    const int4 rr = *reinterpret_cast<const int4*>(A.rect + 4 * int64_t(id));
    const int64_t e = A.lt_offset[id] + lt_local_index(rr.x, rr.y, rr.z, rr.w, TILE, px, py);
    float c[3] = {0.5f, 0.5f, 0.5f};
#pragma unroll
    for (int k = 0; k < K; ++k)
#pragma unroll
      for (int ch = 0; ch < 3; ++ch) c[ch] = fmaf(shp[3 * k + ch], Y[k], c[ch]);
#pragma unroll
    for (int ch = 0; ch < 3; ++ch) c[ch] = fmaxf(c[ch], 0.0f);
    // k-th composited hit of this pixel -> its list position (read by the
    // gather backward)
    A.hit_list[int64_t(NT) * (hl_beg + min(n_hits, hl_last)) + tid] = cpos;
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
    last_id = id;
    if (T < A.t_min) {  // terminated; its exact depth is found after the trace
      done = true;
      end_id = id;
    }
    head = (head + 1) & (KB - 1);
    --cnt;
    if (cnt > 0) {
      head_tf = s_btf[head][tid];
      head_a = s_balpha[head][tid];
      head_pos = s_bpos[head][tid];
      head_id = entry_id(head);
    } else {
      head_tf = __int_as_float(0x7f800000);
    }
  };

  uint32_t restart = 0;
  int passes = 0;  // rescans so far

  // One staged candidate: geometry row, rectangle and index.
  struct Cand {
    double W[9], og[3], D2c, sig;
    int4 r;
    uint32_t id;
  };
  auto load_cand = [&](int c) {
    const double* row = s_row + c * kRow;
    Cand cd;
#pragma unroll
    for (int k = 0; k < 9; ++k) cd.W[k] = row[k];
#pragma unroll
    for (int k = 0; k < 3; ++k) cd.og[k] = row[9 + k];
    cd.D2c = row[12];
    cd.sig = row[13];
    cd.r = *reinterpret_cast<const int4*>(row + 16);
    cd.id = reinterpret_cast<const uint32_t*>(row + 18)[0];
    return cd;
  };

  // Tests candidate c of the batch starting at list position base against
  // this lane's ray, buffers a hit, and at the flush points composites the
  // hits that are final.  Returns true when the lane leaves the batch
  // (terminated, or stalled until a rescan).
  auto visit = [&](const Cand& cd, int c, int nb, int64_t base) -> bool {
    const uint32_t cpos = uint32_t(base - beg) + uint32_t(c);
    const bool inside = (cpos >= from) & (px >= cd.r.x) & (px <= cd.r.z) & (py >= cd.r.y) & (py <= cd.r.w);
    if (inside) {
      ++n_tests;
      double tau, D2, xg[3];
      const uint32_t id = cd.id;
      // in a rescan, hits up to the last composited one were composited before
      if (ray_hit(cd.W, cd.og, cd.D2c, d, &tau, &D2, xg) && (passes == 0 || key_less(last_tau, last_id, tau, id))) {
        if (!(tau < e_tau)) {
          drop(tau, cpos);
        } else {
          const float tu = __double2float_ru(tau);
          bool ins = true;
          if (cnt == KB) {  // full: the larger of the new hit and the tail is dropped
            const int s = (head + KB - 1) & (KB - 1);
            if (!before_entry(tau, tu, id, s)) {
              drop(tau, cpos);
              ins = false;
            } else {
              // the tail's depth is above the float below its rounded-up bound
              const float tf = s_btf[s][tid];  // > 0 (a hit has tau > 0)
              drop(double(__uint_as_float(__float_as_uint(tf) - 1u)), s_bpos[s][tid]);
              cnt = KB - 1;
              tail_tf = s_btf[(head + KB - 2) & (KB - 1)][tid];
            }
          }
          if (ins) insert(tau, tu, id, cpos, cd.sig * exp(-0.5 * D2));
        }
      }
    }
    // Composite the final hits every kFlushEvery Gaussians, at the end of a
    // batch, and whenever a lane's ring is full -- for every lane of the wave
    // at once, so that each compositing step serves more lanes.
    if (__ballot((c + 1) % kFlushEvery == 0 || c + 1 == nb || cnt == KB) != 0) {
      const double nk = double(s_key[c + 1]) * kscale;
      while (cnt > 0 && !done && double(head_tf) < nk) composite_front();
      if (done) return true;
      if (e_tau < kInf && nk > e_tau) {
        stalled = true;
        return true;
      }
    }
    return false;
  };

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
          Cand cd = load_cand(c);
          // materialise the row here, so that the compiler does not sink its
          // reads into the branch (a second LDS round trip per candidate)
#pragma unroll
          for (int k = 0; k < 9; ++k) asm volatile("" : "+v"(cd.W[k]));
#pragma unroll
          for (int k = 0; k < 3; ++k) asm volatile("" : "+v"(cd.og[k]));
          asm volatile("" : "+v"(cd.D2c), "+v"(cd.sig), "+v"(cd.id));
          if (visit(cd, c, nb, base)) break;
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
      jr = UINT_MAX;
      stalled = false;
      cnt = 0;
      head = 0;
      head_tf = __int_as_float(0x7f800000);
      last_tau = n_hits ? exact_tau(last_id) : -kInf;  // for the skip test of the rescan
    }
  }

  // the tile's visited prefix for the backward: the block's largest
  __shared__ uint32_t s_visited;
  if (tid == 0) s_visited = 0;
  __syncthreads();
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) visited = max(visited, uint32_t(__shfl_xor(int(visited), off)));
  if (lane_id() == 0) atomicMax(&s_visited, visited);
  __syncthreads();
  if (tid == 0) A.tile_visit[tile] = s_visited;
  if (end_id != kNoPrim) end_tau = exact_tau(end_id);
  if (__ballot(n_hits > hl_last + 1u) != 0 && lane_id() == 0) atomicOr(A.status, unsigned(GART_FRAME_HIT_LIST_FULL));
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

// Ring sizes: deep frames (long tile lists, many pending hits per ray) get
// the larger ring; it costs occupancy (LDS), so others get the smaller.
#ifndef GART_FWD_RING_SMALL
#define GART_FWD_RING_SMALL 8
#endif
#ifndef GART_FWD_RING_LARGE
#define GART_FWD_RING_LARGE 16
#endif
constexpr int64_t kDeepListPairs = 2048;  // mean pairs per tile from which a frame counts as deep

template <int TILE, int K, int KB>
hipError_t launch_ring(const ForwardArgs& a, hipStream_t s) {
  const int n_tiles = a.tiles_x * a.tiles_y;
  switch (a.lt_format) {
    case GART_LT_FULL: forward_kernel<TILE, K, GART_LT_FULL, KB><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
    case GART_LT_T_ONLY: forward_kernel<TILE, K, GART_LT_T_ONLY, KB><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
    case GART_LT_HALF: forward_kernel<TILE, K, GART_LT_HALF, KB><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
    case GART_LT_T_HALF: forward_kernel<TILE, K, GART_LT_T_HALF, KB><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
    case GART_LT_FIXED16: forward_kernel<TILE, K, GART_LT_FIXED16, KB><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
    case GART_LT_T_LOG16: forward_kernel<TILE, K, GART_LT_T_LOG16, KB><<<n_tiles, TILE * TILE, 0, s>>>(a); break;
    default: return hipErrorInvalidValue;
  }
  return hipGetLastError();
}

template <int TILE, int K>
hipError_t launch_t(const ForwardArgs& a, hipStream_t s) {
  hipError_t e = record(a.ev_begin, s);
  if (e != hipSuccess) return e;
  const int64_t n_tiles = int64_t(a.tiles_x) * a.tiles_y;
  const bool deep = a.pair_count > kDeepListPairs * n_tiles;
  // 16x16 tiles hold four waves' rings per workgroup: at most 16 entries each
  constexpr int kLarge = TILE == 8 ? GART_FWD_RING_LARGE : (GART_FWD_RING_LARGE < 16 ? GART_FWD_RING_LARGE : 16);
  e = deep ? launch_ring<TILE, K, kLarge>(a, s) : launch_ring<TILE, K, GART_FWD_RING_SMALL>(a, s);
  if (e != hipSuccess) return e;
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
