// Host-side launchers shared between the library's translation units.
// Every launcher enqueues on `s` and returns the first HIP error it sees.
#pragma once

#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "common.h"

namespace gart {

// ---- scan.hip / sort ------------------------------------------------------
// Exclusive prefix sum of n values (in may equal out).  If total is not
// null, the sum of all n values is stored at *total (device).  tmp must hold
// scan_tmp_bytes(n) bytes.
size_t scan_tmp_bytes(int64_t n);
hipError_t scan_exclusive_i64(const int64_t* in, int64_t* out, int64_t n, int64_t* total, void* tmp, hipStream_t s);
hipError_t scan_exclusive_u32(const uint32_t* in, uint32_t* out, int64_t n, uint32_t* total, void* tmp, hipStream_t s);
// The same with 32-bit inputs and 64-bit sums (in and out are distinct).
hipError_t scan_exclusive_u32_i64(const uint32_t* in, int64_t* out, int64_t n, int64_t* total, void* tmp,
                                  hipStream_t s);

// Stable LSD radix sort of (key, value) pairs on key bits [0, bits), 8 bits
// per pass.  The sorted pairs end in (keys, vals); (keys_alt, vals_alt) are
// scratch of the same length.  tmp must hold radix_tmp_bytes(m) bytes.
size_t radix_tmp_bytes(int64_t m);
hipError_t radix_sort_u32(uint32_t* keys, uint32_t* vals, uint32_t* keys_alt, uint32_t* vals_alt, int64_t m, int bits,
                          void* tmp, hipStream_t s);

// Records an optional event (no-op for NULL).
inline hipError_t record(void* ev, hipStream_t s) {
  return ev ? hipEventRecord(static_cast<hipEvent_t>(ev), s) : hipSuccess;
}

// Simple fills and gathers.
hipError_t fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s);
hipError_t fill_f32(float* p, float v, int64_t n, hipStream_t s);
hipError_t fill_u8(uint8_t* p, uint8_t v, int64_t n, hipStream_t s);
hipError_t iota_u32(uint32_t* p, int64_t n, hipStream_t s);

// ---- bounds.hip ----------------------------------------------------------
struct BoundsArgs {
  const float* means;
  const float* log_scales;
  const float* quats;
  const float* logits;
  const float* sh;          // [n, K, 3]
  int32_t K;
  int64_t n;
  CamParams cam;
  double alpha_min;
  int32_t tile;
  int32_t* rect;
  int64_t* area;            // [n] rectangle areas (scanned later into O_prim)
  double* geom;
  uint32_t* tile_count;
  // per block of kBoundsBlock Gaussians: [2b] sum of tile counts, [2b+1]
  // max colour bound (float bits); reduced by launch_bounds_totals
  unsigned long long* block_partial;
};
constexpr int kBoundsBlock = 256;
hipError_t launch_bounds(const BoundsArgs& a, hipStream_t s);
// totals[0] = *area_total, totals[1] = sum of the pair partials, totals[2] =
// max of the colour partials (float bits; 0 if no visible Gaussian)
hipError_t launch_bounds_totals(const unsigned long long* block_partial, int64_t n_blocks, const int64_t* area_total,
                                unsigned long long* totals, hipStream_t s);

struct TileMapArgs {
  int64_t n;
  int32_t tile, tiles_x, tiles_y;
  CamParams cam;
  const int32_t* rect;
  const uint32_t* tile_count;
  const double* geom;       // [n, 16] per-Gaussian geometry (W, o_g, per-Gaussian depth bound)
  int64_t* pair_offset;     // [n+1] first pair slot of each Gaussian (tile counts, scanned in place)
  uint32_t* keys;           // [P] (tile << key_bits) | depth code of each emitted pair
  uint32_t* vals;           // [P] emitted Gaussian indices
  float* pair_key;          // [P] camera-depth bound of each sorted pair (decoded code)
  int32_t key_bits;         // bits of the depth code in keys
  int64_t pair_count;
  int64_t* tile_range;      // [n_tiles+1]
};
hipError_t launch_emit_pairs(const TileMapArgs& a, hipStream_t s);
// From the sorted combined keys (a buffer other than a.keys): a.keys[j] = tile
// id, a.pair_key[j] = decoded depth bound, and a.tile_range[t] = first pair
// whose tile id is >= t, for t in [0, n_tiles].
hipError_t launch_finish_pairs(const TileMapArgs& a, const uint32_t* sorted_keys, int64_t n_tiles, hipStream_t s);
// rows[t] = min(tile_range[t+1] - tile_range[t], cap): the hit_list rows of
// tile t (a pixel composites at most one hit per pair and at most cap hits)
hipError_t launch_hit_rows(const int64_t* tile_range, int64_t n_tiles, int64_t cap, int64_t* rows, hipStream_t s);

// ---- forward.hip -------------------------------------------------------
struct ForwardArgs {
  CamParams cam;
  int32_t tile, tiles_x, tiles_y, sh_k;
  double t_min;
  const int64_t* tile_range;
  const uint32_t* pair_prim;
  const float* pair_key;     // [pairs] camera-depth lower bound of each pair (ascending in a tile list)
  const double* geom;
  const int32_t* rect;
  const int64_t* lt_offset;
  const float* sh;
  uint4* lt;                // entries in the layout lt_format names
  int lt_format;            // gart_lt_format
  double inv_color_step;    // fixed-point units per unit of colour
  float* image;
  gart_pixel_state* pixel_state;
  uint32_t* hit_list;       // list position of each pixel's k-th composited hit, at row hl_off[tile] + k
  const int64_t* hl_off;    // [n_tiles+1] first hit_list row of each tile (tile^2 slots per row)
  uint32_t* tile_visit;     // [n_tiles] one past the largest list position composited in the tile
  uint32_t* status;         // frame status word (GART_FRAME_* bits), cleared before the launch
  int64_t pair_count;       // pairs in the tile lists (sizes the per-lane pending-hit rings)
  uint64_t* counters;
  void* ev_begin;  // optional hipEvent_t recorded around the kernel
  void* ev_end;
};
hipError_t launch_forward(const ForwardArgs& a, hipStream_t s);

// ---- backward.hip ------------------------------------------------------
struct BackwardArgs {
  CamParams cam;
  int32_t tile, tiles_x, tiles_y, sh_k, mode;
  int64_t n;
  const int64_t* tile_range;
  const uint32_t* pair_prim;
  const float* pair_key;     // [pairs] camera-depth lower bound of each pair (ascending in a tile list)
  const double* geom;
  const int32_t* rect;
  const int64_t* lt_offset;
  const int64_t* pair_offset;
  const uint32_t* tile_count;
  const float* sh;
  const uint4* lt;          // entries in the layout lt_format names
  int lt_format;            // gart_lt_format
  float color_step;         // colour per fixed-point unit (a power of two times a float)
  const float* dl_dimage;
  const gart_pixel_state* pixel_state;
  const uint32_t* hit_list;  // list position of each pixel's k-th composited hit, at row hl_off[tile] + k
  const int64_t* hl_off;     // [n_tiles+1] first hit_list row of each tile (tile^2 slots per row)
  const uint32_t* tile_visit;  // [n_tiles] one past the largest list position composited (forward)
  // gradient accumulation
  float* acc;          // [n, acc_stride] per-Gaussian accumulators (atomic modes)
  float* rows;         // [P * rows_per_pair, acc_stride] partial rows (gather mode)
  uint8_t* row_flag;   // [P * rows_per_pair] 1 if the row was written
  int64_t pair_count;
  int32_t rows_per_pair;  // 64-pixel groups per tile (set by the launcher)
  // raw inputs and outputs
  const float* logits;
  const float* log_scales;
  const float* quats;
  float* g_means;
  float* g_log_scales;
  float* g_quats;
  float* g_logits;
  float* g_sh;
  uint64_t* counters;
  void* ev[4];  // optional hipEvent_t: main kernel begin/end, reduction begin/end
};
hipError_t launch_backward(const BackwardArgs& a, hipStream_t s);

// ---- train.hip -----------------------------------------------------------
constexpr int kL1Block = 256;
constexpr int kL1Items = 4096;  // image floats per block (and per loss partial)
int64_t l1_partials(int64_t n);
// dl = sign(image - target); if loss != NULL, *loss = sum |image - target|
// (fp64, deterministic) using partial[l1_partials(n)]
hipError_t launch_l1_grad(const float* image, const float* target, int64_t n, float* dl, double* partial,
                          double* loss, hipStream_t s);

struct AdamArgs {
  float lr, b1, b2, eps;
  float one_minus_b1, one_minus_b2;
  float inv_c1, inv_c2;  // 1 / (1 - b1^t), 1 / (1 - b2^t)
};
hipError_t launch_adam(float* p, const float* g, float* m, float* v, int64_t n, const AdamArgs& h, hipStream_t s);

}  // namespace gart
