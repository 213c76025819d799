/*
 * gart.h -- C ABI of the 3DGART hot path on MI355X (gfx950).
 *
 * Ray-traced 3D Gaussian rendering (Sec. 3.1-3.3) with the primitive-centric
 * backward pass (Sec. 4): conservative screen-space bounds and the
 * intermediate-buffer pre-allocation (Sec. 4.2), the tile-primitive mapping
 * (Sec. 4.3), a software forward trace that fills the (L, T) intermediate
 * buffer, and a backward in which one GPU lane owns one (tile, primitive)
 * pair (Sec. 4.4).
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 *  - Every pointer is a DEVICE pointer unless the comment says "host".
 *    All device memory is owned and allocated by the caller; the library
 *    never allocates, frees or keeps device memory, and keeps no state
 *    between calls other than what the caller's gart_frame holds.
 *  - Work is enqueued on `stream` (a hipStream_t; NULL = the default
 *    stream) and is asynchronous, except for the single documented
 *    device->host copy in gart_bounds.
 *  - Arguments are validated before anything is launched; an invalid
 *    argument returns GART_ERR_INVALID_ARG and launches nothing.  A failing
 *    HIP call returns GART_ERR_HIP.  Kernels never read or write outside
 *    the sizes the caller declares.
 *  - One gart_frame is used by one stream at a time.  Calls on the same
 *    frame from different streams race.
 *  - gart_build_tile_map, gart_forward, gart_backward and the training
 *    calls only enqueue kernels (buffers are cleared by kernels, not by
 *    memset), so they may be captured in a HIP graph and replayed while the
 *    frame's sizes (N, pair count) stay the ones the capture saw.
 *    gart_bounds synchronises the host and cannot be captured.
 *  - Scene: N Gaussians with mean mu, rotation from a quaternion q = (w, x,
 *    y, z) (any non-zero norm; normalised internally), per-axis scale
 *    s = exp(log_scale), opacity sigma = 1 / (1 + exp(-logit)) and RGB
 *    radiance given by real spherical harmonics of degree 0..3 evaluated at
 *    the unit ray direction (Sec. 3.1): colour = max(0, 0.5 + sum_k
 *    sh[k] Y_k(d)), with Y_l^m the real harmonics without Condon-Shortley
 *    phase, k = l*l + l + m.
 *  - Camera: pinhole, OpenCV axes, world-to-camera x_c = R x_w + t.  Pixel
 *    (x, y) is traced through its centre (x + 0.5, y + 0.5).
 *  - A ray hits a Gaussian iff its max-response point (Eq. 4-5) lies in
 *    front of the camera (tau > 0) and inside the clamped ellipsoid of
 *    radius alpha_c = sqrt(2 log(sigma / alpha_min)) (Eq. 9-10), i.e. iff
 *    alpha = sigma rho >= alpha_min (Eq. 8).  Hits are composited front to
 *    back in (tau, index) order (Eq. 6-7) until the transmittance falls
 *    below t_min; the hit that crosses is included.  No cap on hits.
 *    Background is black.
 */
#ifndef GART_H_
#define GART_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  GART_OK = 0,
  GART_ERR_INVALID_ARG = -1, /* bad size, pointer, enum value or call order */
  GART_ERR_CAPACITY = -2,    /* frame buffers too small; required sizes returned */
  GART_ERR_HIP = -3,         /* a HIP runtime call failed */
  GART_ERR_UNSUPPORTED = -4  /* valid but not implemented (e.g. SH degree > 3) */
} gart_status;

typedef enum {
  GART_BACKWARD_GATHER = 0,        /* (tile, prim) pairs -> per-pair rows -> one reduction per primitive */
  GART_BACKWARD_GATHER_ATOMIC = 1, /* (tile, prim) pairs -> one atomic update per pair (Sec. 4.4 as printed) */
  GART_BACKWARD_SCATTER = 2,       /* pixel-centric control: one atomic update per composited hit (Sec. 3.5) */
  GART_BACKWARD_HYBRID = 3,        /* Sec. 4.4 "Hybrid approach": SH sums gathered per pair, the other 10 sums
                                      scattered per hit from a back-to-front walk; lt holds T only (4 B) */
  GART_BACKWARD_GATHER_WAVE = 4    /* GATHER, with units of >= 48 hits evaluated by a whole wave, one lane per
                                      pixel (Sec. 4.4, a warp per primitive) */
} gart_backward_mode;

/* Layout of gart_frame.lt, chosen by gart_forward from settings->backward_mode
 * and settings->lt_precision (see gart_lt_entry_bytes). */
typedef enum {
  GART_LT_FULL = 0,   /* gart_lt_entry (16 bytes): fixed-point L and float T */
  GART_LT_T_ONLY = 1, /* float T (4 bytes) per entry, entry e at ((float*)lt)[e] (hybrid backward) */
  GART_LT_HALF = 2,   /* fp16 L.r, L.g, L.b, T (8 bytes, in that order; Sec. 6 fp16 storage) */
  GART_LT_T_HALF = 3, /* fp16 T (2 bytes) per entry (hybrid backward with fp16 storage) */
  GART_LT_FIXED16 = 4,/* uint16 L.r, L.g, L.b in units of color_step * 2^16, then uint16 T code
                         q = round(-log2(T) * 4096), T = 2^(-q / 4096) (8 bytes) */
  GART_LT_T_LOG16 = 5 /* uint16 T code as in GART_LT_FIXED16 (2 bytes; hybrid backward) */
} gart_lt_format;

typedef enum {
  GART_LT_PRECISION_FULL = 0, /* 16-byte (L,T) entries, or 4-byte T with the hybrid backward */
  GART_LT_PRECISION_HALF = 1, /* fp16 entries: 8 bytes, or 2 bytes with the hybrid backward;
                                 values are rounded to float, then to the nearest fp16 */
  GART_LT_PRECISION_FIXED16 = 2 /* 16-bit fixed-point L and log-coded T: 8 bytes, or 2 bytes with
                                   the hybrid backward; needs t_min >= 2^-15 (T of every composited
                                   hit is at least t_min, so its code fits 16 bits) */
} gart_lt_precision;

/* Pinhole camera.  Host struct, passed by pointer. */
typedef struct {
  int32_t width, height;   /* image size in pixels, both >= 1 */
  float fx, fy, cx, cy;    /* intrinsics in pixels; fx, fy > 0 */
  float R[9];              /* world -> camera rotation, row-major */
  float t[3];              /* world -> camera translation */
} gart_camera;

/* Gaussian parameters (Sec. 3.1).  Host struct holding device pointers to
 * float32 arrays, structure-of-arrays, C-contiguous. */
typedef struct {
  int64_t n;                 /* number of Gaussians, 0 <= n < 2^31 */
  int32_t sh_degree;         /* 0..3; K = (sh_degree + 1)^2 */
  const float* means;        /* [n,3] */
  const float* log_scales;   /* [n,3] */
  const float* quats;        /* [n,4] (w, x, y, z) */
  const float* opacity_logits; /* [n] */
  const float* sh;           /* [n,K,3] */
} gart_gaussians;

typedef struct {
  float alpha_min;        /* response cut-off, 1/255 in the paper (Sec. 3.4); in (0, 1) */
  float t_min;            /* stop a ray once its transmittance drops below this; in (0, 1) */
  int32_t tile;           /* tile edge in pixels: 8 or 16 (Sec. 4.4 uses 8) */
  int32_t backward_mode;  /* gart_backward_mode */
  int32_t lt_precision;   /* gart_lt_precision */
} gart_settings;

/* Per-pixel state the forward leaves for the backward (32 bytes): the depth
 * and index of the last composited hit if the ray terminated (T < t_min),
 * else tau_end = +inf and id_end = 0xffffffff; a hit (tau, i) of this pixel
 * was composited iff (tau, i) <= (tau_end, id_end) lexicographically.
 * color_fixed is the final pixel colour C (Eq. 1) in the fixed point of
 * gart_lt_entry, so that the colour behind a hit, C - L - T a c, is formed
 * from an exact integer difference C - L. */
typedef struct {
  double tau_end;
  uint32_t id_end;
  uint32_t n_hits;          /* composited hits of the pixel */
  uint32_t color_fixed[3];  /* round(C / gart_frame.color_step) per channel */
  float t_final;            /* transmittance left after the last composited hit */
} gart_pixel_state;

/* One intermediate-buffer entry (Sec. 4.3, 16 bytes): the colour
 * accumulated in front of a composited hit, L, as unsigned fixed point
 * (L = L_fixed * gart_frame.color_step, rounded to nearest; every composited
 * colour lies below 2^32 color_step), and the transmittance T in front of
 * the hit. */
typedef struct {
  uint32_t L_fixed[3];
  float T;
} gart_lt_entry;

/* Per-frame buffers.  Host struct; the caller allocates every device array
 * (sizes in the comments; "cap" = the capacity fields) and the library
 * fills them.  Fields marked [out] are written by the library. */
typedef struct {
  /* written by gart_bounds */
  int32_t* rect;          /* [n,4] inclusive pixel rectangle x0,y0,x1,y1; x0 > x1 if culled */
  int64_t* lt_offset;     /* [n+1] O_prim: exclusive prefix sum of rectangle areas; [n] = total */
  double* prim_geom;      /* [n,16] per-Gaussian fp64 precompute (opaque layout) */
  uint32_t* tile_count;   /* [n] tiles overlapped by the rectangle */
  /* written by gart_build_tile_map */
  int64_t* pair_offset;   /* [n+1] first pair slot of each Gaussian in emission order */
  int64_t pair_capacity;  /* number of (tile, prim) pair slots allocated */
  uint32_t* pair_tile;    /* [pair_capacity] tile id of each pair, sorted ascending */
  uint32_t* pair_prim;    /* [pair_capacity] Gaussian index of each pair */
  float* pair_key;        /* [pair_capacity] lower bound on tau_q / s_q over the pixel-centre rays q of
                             the pair's tile inside the Gaussian's rectangle, where tau_q is the depth
                             (Eq. 3) of the Gaussian's maximum-response point (Eq. 4-5) on ray q,
                             s_q = |R^T u_q| / (c . u_q), u_q = ((x + 1/2 - cx)/fx, (y + 1/2 - cy)/fy, 1),
                             and c is the unit camera-space direction through the tile centre
                             (pixel ((tx + 1/2) tile, (ty + 1/2) tile)): the depth measured along c
                             (s_q - 1 < 2e-5 on 8x8 tiles); each tile's list is sorted ascending by
                             it, then by Gaussian index */
  int64_t* tile_range;    /* [n_tiles+1] pairs of tile t are [tile_range[t], tile_range[t+1]) */
  /* written by gart_forward, read by gart_backward */
  int64_t lt_capacity;    /* number of intermediate entries allocated, each of
                             gart_lt_entry_bytes(settings) bytes */
  gart_lt_entry* lt;      /* [lt_capacity] (L, T) in front of each composited hit, in the layout
                             frame->lt_format names (see gart_lt_format) */
  gart_pixel_state* pixel_state; /* [height*width] per-pixel end marker (see gart_pixel_state) */
  uint32_t* hit_list;     /* [hit_list_capacity] composited hits of each pixel, front to back:
                             for tile t with pairs [b, e) (tile_range), the k-th composited hit of
                             pixel q of the tile (row-major) is list position (pair - b), stored at
                             hit_list[tile^2 * (o_t + k) + q]; tile t owns rows [o_t, o_t + r_t)
                             with r_t = min(e - b, k_max), k_max the most hits a pixel can
                             composite (see gart_hit_list_slots), o_t their running sum (kept in
                             the frame's scratch) */
  int64_t hit_list_capacity; /* number of uint32 slots allocated for hit_list; gart_forward and
                             gart_backward return GART_ERR_CAPACITY if it is below
                             gart_hit_list_slots(pair_count, ...) */
  /* scratch for sorting and gradient accumulation, size from gart_scratch_bytes */
  void* scratch;
  size_t scratch_bytes;
  /* optional device counters (NULL = not counted), uint64[GART_NUM_COUNTERS] */
  uint64_t* counters;
  /* optional hipEvent_t handles (NULL = not recorded), see GART_EV_*: the
   * library records each on `stream` immediately before / after the named
   * kernel, so a caller can time single kernels on the library's stream */
  void* events[8];
  /* [out] host-side totals and call-order state, filled by the library */
  int64_t n;              /* Gaussians seen by gart_bounds */
  int32_t sh_degree;
  int32_t tiles_x, tiles_y;
  int64_t lt_entries;     /* sum of rectangle areas (Eq. 15 without slack) */
  int64_t pair_count;     /* number of (tile, prim) pairs */
  double color_step;      /* colour per fixed-point unit of lt and pixel_state (see gart_lt_entry):
                             a bound on every Gaussian's colour, divided by 2^32 */
  int32_t stage;          /* 0 none, 1 bounds, 2 tile map, 3 forward */
  int32_t lt_format;      /* gart_lt_format written by the last gart_forward */
  int32_t width, height;  /* camera image size gart_bounds sized the frame for; later calls on
                             the frame must pass a camera of this size (else INVALID_ARG) */
  int32_t tile;           /* settings->tile gart_bounds used; later calls must use the same */
  int32_t reserved;       /* set to 0 */
} gart_frame;

enum {
  GART_CNT_FWD_HITS = 0,      /* composited hits written by the forward */
  GART_CNT_FWD_TESTS = 1,     /* (pixel, Gaussian) ray tests in the forward */
  GART_CNT_FWD_RESCANS = 2,   /* forward rescans of a tile list (hit-buffer overflow) */
  GART_CNT_BWD_HITS = 3,      /* composited hits visited by the backward */
  GART_CNT_BWD_TESTS = 4,     /* (pixel, Gaussian) ray tests in the backward (scatter mode) */
  GART_CNT_BWD_ATOMICS = 5,   /* float atomic adds issued by the backward */
  GART_CNT_BWD_PAIRS = 6,     /* (tile, prim) pairs visited by the backward */
  GART_CNT_BWD_ACTIVE = 7,    /* (pair, 64-pixel group) units with a composited hit (gather) */
  GART_CNT_FWD_DROPS = 8,     /* forward hits dropped from a full hit buffer (found again by a rescan) */
  GART_CNT_BWD_STEPS = 9,     /* hits walked by the hybrid pixel pass (composited hits, once per window
                                 of list positions that the tile needs) */
  GART_CNT_BWD_WAVE_UNITS = 10, /* units evaluated by a whole wave (GATHER_WAVE) */
  GART_NUM_COUNTERS = 16
};

/* Bits of the frame status word (see gart_frame_status). */
enum {
  GART_FRAME_STATUS_OK = 0,
  GART_FRAME_FORWARD_INCOMPLETE = 1, /* the forward stopped tracing a tile at its safety limit on list
                                       passes: image, intermediate buffer, hit_list and pixel_state of
                                       that tile are incomplete (a library defect; never expected) */
  GART_FRAME_HIT_LIST_FULL = 2       /* a pixel composited more hits than its tile's hit_list rows
                                       (see gart_hit_list_slots); its last row holds the last such hit
                                       and the backward misses the others (a library defect; never
                                       expected) */
};

enum {
  GART_EV_SORT_BEGIN = 0,   /* radix sort of the (tile, prim) pairs (all passes) */
  GART_EV_SORT_END = 1,
  GART_EV_FWD_BEGIN = 2,    /* forward trace kernel */
  GART_EV_FWD_END = 3,
  GART_EV_BWD_BEGIN = 4,    /* backward main kernel (gather or scatter) */
  GART_EV_BWD_END = 5,
  GART_EV_REDUCE_BEGIN = 6, /* per-Gaussian reduction and chain rule */
  GART_EV_REDUCE_END = 7,
  GART_NUM_EVENTS = 8
};

/* Slots (uint32) that frame->hit_list needs for pair_count (tile, Gaussian)
 * pairs on this camera and settings: tile^2 per row, min(pairs, tiles x
 * k_max) rows, where k_max = floor(ln t_min / ln(1 - alpha_min)) + 3 bounds
 * the hits one pixel composites: every composited hit has alpha >= alpha_min
 * (Sec. 3.4, Eq. 10) and compositing stops after the first hit that takes T
 * below t_min (Sec. 5.2).  Returns -1 on invalid arguments (message from
 * gart_last_error). */
int64_t gart_hit_list_slots(int64_t pair_count, const gart_camera* camera, const gart_settings* settings);

/* Bytes per intermediate-buffer entry that gart_forward writes for these
 * settings: 16 (GART_LT_FULL), 4 (GART_LT_T_ONLY), 8 (GART_LT_HALF,
 * GART_LT_FIXED16) or 2 (GART_LT_T_HALF, GART_LT_T_LOG16); 0 for invalid
 * settings.  lt must hold lt_capacity such
 * entries (Sec. 4.3 Eq. 15; Sec. 4.4 hybrid approach; Sec. 6 fp16). */
int32_t gart_lt_entry_bytes(const gart_settings* settings);

/* Bytes of scratch a frame needs for n Gaussians of the given SH degree and
 * pair_capacity pair slots (all backward modes covered).  Pure host
 * function. */
size_t gart_scratch_bytes(int64_t n, int32_t sh_degree, int64_t pair_capacity, const gart_camera* camera,
                          const gart_settings* settings);

/* Pre-processing (Sec. 4.2, Eq. 9-15; Sec. 5.3 "pre-processing").
 * Per Gaussian: normalised rotation, scales, opacity, clamp radius, the
 * world-to-Gaussian map W = S^-1 R^T and o_g = W (o - mu) (Eq. 5), and the
 * conservative pixel rectangle from the projected dual quadric
 * T' = VPM T (Eq. 11-14).  For an ellipsoid that crosses the camera's eye
 * plane (where Eq. 12-14 do not apply) the rectangle is the hull of the
 * pixel columns / rows whose plane through the camera meets the ellipsoid.
 * Culled (rect x0 > x1, area 0): sigma <= alpha_min, ellipsoid behind the
 * camera, no pixel centre covered, non-finite parameters.
 * Then O_prim = exclusive prefix sum of the areas (Sec. 4.3 "primitive
 * offset").  Also a bound on the colour of every visible Gaussian in any
 * direction, 1/2 + sum_l sqrt((2l+1)/(4 pi)) |sh_l| per channel (Cauchy-
 * Schwarz with the addition theorem of spherical harmonics), which fixes
 * the frame's colour step = bound / 2^32.  Writes rect, lt_offset,
 * prim_geom, tile_count and frame->n, sh_degree, tiles_x, tiles_y,
 * lt_entries, pair_count, color_step, stage.
 * Synchronises `stream` once to copy the totals to the host:
 * *lt_entries_host = sum A_i (Eq. 15 with lambda_s = 1), *pair_count_host =
 * number of (tile, prim) pairs.  Either host pointer may be NULL.
 * Returns GART_ERR_CAPACITY (after filling the totals) if they exceed
 * frame->lt_capacity or frame->pair_capacity; the caller may grow the
 * buffers (the paper's slack factor lambda_s) and call again. */
gart_status gart_bounds(const gart_gaussians* g, const gart_camera* camera, const gart_settings* settings,
                        gart_frame* frame, int64_t* lt_entries_host, int64_t* pair_count_host, void* stream);

/* Largest n gart_bounds_noalloc serves (2^25 Gaussians). */
#define GART_BOUNDS_NOALLOC_MAX_N (INT64_C(1) << 25)

/* gart_bounds for callers that cannot allocate device memory (code under
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same computation and outputs as gart_bounds, bit for bit, but the step's
 * scratch (block partial sums, prefix-sum temporaries and the totals) is a
 * 4 MiB array the library holds as a static device variable, one copy per
 * GPU, kept until the process ends.  frame->scratch is neither read nor
 * written and may be NULL (the later calls still need it).  Calls no
 * hipMalloc, hipFree or other allocating routine; synchronises `stream`
 * once, as gart_bounds does.
 * Every call on one GPU shares that GPU's copy of the array: calls that
 * overlap in time on one GPU (from several streams or threads) race and
 * must be serialised by the caller.  Nothing in the array needs to start at
 * zero (each call writes every word it reads first).
 * Errors: as gart_bounds; INVALID_ARG (nothing launched) if
 * g->n > GART_BOUNDS_NOALLOC_MAX_N. */
gart_status gart_bounds_noalloc(const gart_gaussians* g, const gart_camera* camera, const gart_settings* settings,
                                gart_frame* frame, int64_t* lt_entries_host, int64_t* pair_count_host,
                                void* stream);

/* Tile-primitive mapping (Sec. 4.3 "reverse tile mapping").
 * Emits one (tile, Gaussian) pair per tile that a rectangle overlaps and
 * radix-sorts the pairs by tile id, then builds tile_range (the tile offset
 * table).  Within one tile, pairs are ordered by pair_key (see gart_frame),
 * the smallest depth along the tile's centre direction of the Gaussian's
 * maximum-response points over the tile's pixel rays (attained at a corner
 * of the pixel rectangle; less 1e-12 relative), rounded down to a float with
 * min(24, 32 - tile id bits) - 5 mantissa bits (0 below 2^-12, saturating
 * below 2^20), then by index; the set of Gaussians per tile is exactly the
 * set of rectangles meeting the tile.
 * Requires gart_bounds on the same frame first (else INVALID_ARG). */
gart_status gart_build_tile_map(const gart_camera* camera, const gart_settings* settings, gart_frame* frame,
                                void* stream);

/* Forward trace (Sec. 3.2-3.3, Eq. 3-8; Sec. 4.3 "LT buffer access").
 * One workgroup per tile, one lane per pixel.  Each ray tests the
 * Gaussians of its tile list whose rectangle contains the pixel, orders the
 * hits by (tau, index), composites them front to back and, for every
 * composited hit of Gaussian i at pixel p in tile t, writes
 * lt[idx(i,t,p)] = (L.rgb, T) -- the colour accumulated and the
 * transmittance in front of the hit, L in the frame's fixed point -- with idx(i,t,p) = O_prim(i) +
 * O_tile(i,t) + O_pixel(i,t,p) (Eq. 16): tiles of the rectangle in
 * row-major order, pixels row-major inside each tile.  Entries for
 * pixels that are not composited hits are left untouched.  With
 * settings->backward_mode == HYBRID only T is written (float per entry,
 * frame->lt_format = GART_LT_T_ONLY, 4 bytes per entry suffice); otherwise
 * frame->lt_format = GART_LT_FULL (16 bytes per entry).  hit_list
 * records the pair of every composited hit per pixel (entries past a
 * pixel's n_hits are left untouched), so that the gather backward reads
 * which hits to visit instead of re-testing rays.
 * image: [height,width,3] float32, written for every pixel.
 * pixel_state (end marker, final colour in fixed point, final
 * transmittance) is written for every pixel.
 * Requires gart_build_tile_map first (else INVALID_ARG). */
gart_status gart_forward(const gart_gaussians* g, const gart_camera* camera, const gart_settings* settings,
                         gart_frame* frame, float* image, void* stream);

/* Backward (Sec. 4.4).  Gradient of L = sum_p <dL_dimage[p], C[p]> with
 * respect to the raw parameters, OVERWRITING g_means [n,3],
 * g_log_scales [n,3], g_quats [n,4] (w.r.t. the unnormalised input
 * quaternion), g_logits [n] and g_sh [n,K,3].
 * settings->backward_mode:
 *   GATHER: one workgroup per tile; each lane owns a (pair, 64-pixel
 *     group) unit of the tile list, walks the unit's composited hits (from
 *     hit_list), reads (L,T) from the intermediate buffer and accumulates
 *     the Gaussian's gradient in registers; each unit writes one partial
 *     row and a per-Gaussian reduction sums its rows and applies the chain
 *     rule.  Deterministic.
 *   GATHER_ATOMIC: as GATHER, but each unit adds its partial into
 *     per-Gaussian accumulators with one atomic update per value.
 *   SCATTER: the pixel-centric control (Sec. 3.5): one lane per pixel, one
 *     atomic add per gradient value per composited hit.
 *   GATHER_WAVE: as GATHER, but a unit with at least 48 composited hits is
 *     evaluated by its whole wave, one lane per pixel, and its 10 + 3K sums
 *     are formed by a cross-lane reduction (Sec. 4.4 discusses a warp per
 *     primitive).  Deterministic.
 *   HYBRID (Sec. 4.4, hybrid approach): the SH sums (3K) are gathered per
 *     unit into rows as in GATHER; a second kernel walks each pixel's
 *     composited hits back to front (hit_list), forms the colour behind
 *     each hit from that walk and adds the other 10 terms into per-tile LDS
 *     accumulators (LDS atomics, so the summation order varies from run to
 *     run), written into the same rows.  Needs a frame rendered with the same mode (lt_format
 *     GART_LT_T_ONLY); the other modes need GART_LT_FULL (else INVALID_ARG).
 * Except in HYBRID, the colour in front of and behind each hit comes from
 * the frame's lt and pixel_state (the forward's image is not read); dL_dimage is
 * [height,width,3] float32.  Requires gart_forward first (else
 * INVALID_ARG). */
gart_status gart_backward(const gart_gaussians* g, const gart_camera* camera, const gart_settings* settings,
                          const gart_frame* frame, const float* dL_dimage, float* g_means,
                          float* g_log_scales, float* g_quats, float* g_logits, float* g_sh, void* stream);

/* ---- Training step around the path (multi-view synthetic training) ----
 * The paper trains with the usual 3DGS recipe; these two calls close the
 * loop: the L1 photometric loss supplies the backward's upstream gradient
 * and Adam updates each parameter group from the gradients gart_backward
 * writes. */

/* Adam hyper-parameters of one parameter group (host struct). */
typedef struct {
  float lr;     /* step size, > 0 */
  float beta1;  /* first-moment decay, in [0, 1) */
  float beta2;  /* second-moment decay, in [0, 1) */
  float eps;    /* added to sqrt(v_hat), >= 0 */
} gart_adam;

/* Number of fp64 partial sums gart_l1_loss_grad needs for n image floats. */
int64_t gart_l1_partials(int64_t n);

/* L1 loss against a target image: dL_dimage[k] = sign(image[k] - target[k])
 * (0 where equal) for k < n (n = height*width*3; all device float32 arrays of
 * n elements, dL_dimage may not alias the inputs).  If loss is non-NULL it
 * receives sum_k |image[k] - target[k]| (device fp64 scalar), summed in a fixed
 * order (deterministic) through partial (device fp64[gart_l1_partials(n)],
 * caller-owned scratch; may be NULL when loss is NULL).  Asynchronous on
 * stream.  INVALID_ARG for NULL arrays (when n > 0) or n < 0. */
gart_status gart_l1_loss_grad(const float* image, const float* target, int64_t n, float* dL_dimage, double* loss,
                              double* partial, void* stream);

/* One Adam step (Kingma and Ba) on n float32 parameters in place, with the
 * moment buffers m and v (device float32[n], zero before the first step):
 *   m = b1 m + (1-b1) g;  v = b2 v + (1-b2) g^2;
 *   param -= lr (m / (1 - b1^t)) / (sqrt(v / (1 - b2^t)) + eps)
 * with t = step >= 1.  Asynchronous on stream.  INVALID_ARG for NULL arrays
 * (when n > 0), n < 0, step < 1 or hyper-parameters outside the ranges above. */
gart_status gart_adam_step(float* param, const float* grad, float* m, float* v, int64_t n, const gart_adam* h,
                           int64_t step, void* stream);

/* Frame status word: the GART_FRAME_* bits the kernels of the last
 * gart_forward on this frame raised (0 = the forward traced every ray to
 * completion).  The word lives in the frame's scratch; gart_forward clears
 * it before tracing.  Copies it to *flags_host after synchronising stream.
 * INVALID_ARG if frame or flags_host is NULL, or if gart_forward has not
 * run on the frame. */
gart_status gart_frame_status(const gart_frame* frame, uint32_t* flags_host, void* stream);

/* Human-readable name of a status code (static string). */
const char* gart_status_string(gart_status status);

/* Last error detail of the calling thread (static thread-local string;
 * empty if none). */
const char* gart_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* GART_H_ */
