// C ABI entry points (include/gart.h): argument validation, scratch layout
// and the launch sequence of each step.  No device memory is allocated here.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <mutex>

#include "../../include/gart.h"
#include "ops.h"

using namespace gart;

// Scratch of gart_bounds_noalloc (see gart.h): 4 MiB per GPU.
static __device__ __align__(256) unsigned char scratch[size_t(4) << 20];

namespace {

thread_local char g_err[512] = "";

gart_status fail(gart_status s, const char* fmt, ...) {
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(g_err, sizeof g_err, fmt, ap);
  va_end(ap);
  return s;
}

#define GART_HIP(expr)                                                                   \
  do {                                                                                   \
    const hipError_t e_ = (expr);                                                        \
    if (e_ != hipSuccess) return fail(GART_ERR_HIP, "%s: %s", #expr, hipGetErrorString(e_)); \
  } while (0)

#define GART_REQUIRE(cond, ...)                                   \
  do {                                                            \
    if (!(cond)) return fail(GART_ERR_INVALID_ARG, __VA_ARGS__); \
  } while (0)

size_t align_up(size_t v) { return (v + 255) & ~size_t(255); }

struct Layout {
  size_t pair_key_alt, pair_val_alt, radix_tmp, scan_tmp, totals, partials, status, hl_off, tile_visit, acc, rows,
      row_flag, total;
};

Layout make_layout(int64_t n, int K, int64_t pair_cap, int mode, int tile, int64_t n_tiles) {
  Layout L{};
  size_t off = 0;
  auto take = [&](size_t bytes) {
    const size_t o = off;
    off += align_up(bytes);
    return o;
  };
  const int64_t nn = std::max<int64_t>(n, 1), pc = std::max<int64_t>(pair_cap, 1);
  L.pair_key_alt = take(pc * 4);
  L.pair_val_alt = take(pc * 4);
  L.radix_tmp = take(radix_tmp_bytes(std::max(nn, pc)));
  const int64_t nt = std::max<int64_t>(n_tiles, 1);
  L.scan_tmp = take(scan_tmp_bytes(std::max(nn, nt) + 1));
  L.totals = take(64);
  L.partials = take(size_t((nn + kBoundsBlock - 1) / kBoundsBlock) * 16);
  L.status = take(4);
  L.hl_off = take(size_t(nt + 1) * 8);  // first hit_list row of each tile
  L.tile_visit = take(size_t(nt) * 4);  // the forward's visited prefix of each tile's list
  const size_t AS = size_t(acc_stride(K));
  const bool rows = mode == GART_BACKWARD_GATHER || mode == GART_BACKWARD_GATHER_WAVE || mode == GART_BACKWARD_HYBRID;
  L.acc = take(rows ? 4 : size_t(nn) * AS * 4);
  const size_t rpp = size_t(tile) * size_t(tile) / 64;  // partial rows per pair (64-pixel groups)
  L.rows = take(rows ? size_t(pc) * rpp * AS * 4 : 4);
  L.row_flag = take(rows ? size_t(pc) * rpp : 4);
  L.total = off;
  return L;
}

template <typename T>
T* at(void* base, size_t off) {
  return reinterpret_cast<T*>(static_cast<char*>(base) + off);
}

bool finite_f(float v) { return std::isfinite(v); }

gart_status check_camera(const gart_camera* c) {
  GART_REQUIRE(c != nullptr, "camera is NULL");
  GART_REQUIRE(c->width >= 1 && c->height >= 1, "image size %dx%d", c->width, c->height);
  GART_REQUIRE(int64_t(c->width) * c->height < (int64_t(1) << 31), "image too large");
  GART_REQUIRE(finite_f(c->fx) && finite_f(c->fy) && c->fx > 0 && c->fy > 0, "focal lengths must be > 0");
  GART_REQUIRE(finite_f(c->cx) && finite_f(c->cy), "principal point not finite");
  for (int k = 0; k < 9; ++k) GART_REQUIRE(finite_f(c->R[k]), "camera R not finite");
  for (int k = 0; k < 3; ++k) GART_REQUIRE(finite_f(c->t[k]), "camera t not finite");
  return GART_OK;
}

gart_status check_settings(const gart_settings* s) {
  GART_REQUIRE(s != nullptr, "settings is NULL");
  GART_REQUIRE(s->alpha_min > 0.0f && s->alpha_min < 1.0f, "alpha_min must be in (0,1)");
  GART_REQUIRE(s->t_min > 0.0f && s->t_min < 1.0f, "t_min must be in (0,1)");
  GART_REQUIRE(s->tile == 8 || s->tile == 16, "tile must be 8 or 16");
  GART_REQUIRE(s->backward_mode >= 0 && s->backward_mode <= 4, "unknown backward_mode %d", s->backward_mode);
  GART_REQUIRE(s->lt_precision >= GART_LT_PRECISION_FULL && s->lt_precision <= GART_LT_PRECISION_FIXED16,
               "unknown lt_precision %d", s->lt_precision);
  GART_REQUIRE(s->lt_precision != GART_LT_PRECISION_FIXED16 || s->t_min >= 0x1p-15f,
               "lt_precision FIXED16 needs t_min >= 2^-15 (T codes are 16 bits)");
  return GART_OK;
}

int lt_format_for(const gart_settings* s) {
  const bool hybrid = s->backward_mode == GART_BACKWARD_HYBRID;
  if (s->lt_precision == GART_LT_PRECISION_HALF) return hybrid ? GART_LT_T_HALF : GART_LT_HALF;
  if (s->lt_precision == GART_LT_PRECISION_FIXED16) return hybrid ? GART_LT_T_LOG16 : GART_LT_FIXED16;
  return hybrid ? GART_LT_T_ONLY : GART_LT_FULL;
}

gart_status check_gaussians(const gart_gaussians* g) {
  GART_REQUIRE(g != nullptr, "gaussians is NULL");
  GART_REQUIRE(g->n >= 0 && g->n < (int64_t(1) << 31) - 1, "n out of range");
  if (g->sh_degree > 3) return fail(GART_ERR_UNSUPPORTED, "sh_degree %d > 3", g->sh_degree);
  GART_REQUIRE(g->sh_degree >= 0, "sh_degree < 0");
  if (g->n > 0)
    GART_REQUIRE(g->means && g->log_scales && g->quats && g->opacity_logits && g->sh, "null parameter pointer");
  return GART_OK;
}

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

CamParams make_cam(const gart_camera* c) {
  CamParams p{};
  double R[9], t[3];
  for (int k = 0; k < 9; ++k) R[k] = c->R[k];
  for (int k = 0; k < 3; ++k) t[k] = c->t[k];
  for (int j = 0; j < 3; ++j)
    for (int k = 0; k < 3; ++k) p.Rt[3 * j + k] = R[3 * k + j];
  for (int k = 0; k < 3; ++k) p.o[k] = -(R[k] * t[0] + R[3 + k] * t[1] + R[6 + k] * t[2]);
  p.fx = c->fx;
  p.fy = c->fy;
  p.ifx = 1.0 / p.fx;
  p.ify = 1.0 / p.fy;
  p.cx = c->cx;
  p.cy = c->cy;
  for (int k = 0; k < 3; ++k) {
    p.V0[k] = p.fx * R[k] + p.cx * R[6 + k];
    p.V1[k] = p.fy * R[3 + k] + p.cy * R[6 + k];
    p.V3[k] = R[6 + k];
  }
  p.V0[3] = p.fx * t[0] + p.cx * t[2];
  p.V1[3] = p.fy * t[1] + p.cy * t[2];
  p.V3[3] = t[2];
  p.W = c->width;
  p.H = c->height;
  return p;
}

int tiles_along(int pixels, int tile) { return (pixels + tile - 1) / tile; }

// Later calls on a frame must describe the image and tiles gart_bounds sized
// it for: the pixel state, the tile ranges and the hit lists are indexed with
// them.
gart_status check_frame_geometry(const gart_frame* f, const gart_camera* c, const gart_settings* s) {
  GART_REQUIRE(c->width == f->width && c->height == f->height,
               "camera is %dx%d but gart_bounds sized the frame for %dx%d", c->width, c->height, f->width,
               f->height);
  GART_REQUIRE(s->tile == f->tile, "settings tile %d differs from the %d gart_bounds used", s->tile, f->tile);
  GART_REQUIRE(f->tiles_x == tiles_along(c->width, s->tile) && f->tiles_y == tiles_along(c->height, s->tile),
               "frame tile grid %dx%d does not match the camera", f->tiles_x, f->tiles_y);
  return GART_OK;
}

// Composited hits one pixel can have: each has alpha >= alpha_min (the hit
// criterion) and compositing stops after the first hit that takes T below
// t_min, so before the last hit T >= t_min while T <= (1 - alpha_min)^(k-1):
// k <= 1 + ln(t_min) / ln(1 - alpha_min).  alpha_min is lowered by 1e-9
// relative and 2 added against the rounding of alpha and of the products.
int64_t hit_rows_cap(const gart_settings* st) {
  const double a = double(st->alpha_min), t = double(st->t_min);
  if (!(a > 0.0 && a < 1.0 && t > 0.0 && t < 1.0)) return INT64_MAX;
  const double k = std::floor(std::log(t) / std::log1p(-a * (1.0 - 1e-9))) + 3.0;
  return k < 1e15 ? int64_t(k) : INT64_MAX;
}

// hit_list slots a frame needs: tile^2 per row, each tile's rows its list
// length capped at hit_rows_cap.
int64_t hit_list_slots(int64_t pair_count, int64_t n_tiles, int tile, const gart_settings* st) {
  const int64_t cap = hit_rows_cap(st);
  const int64_t rows = (cap == INT64_MAX || n_tiles > pair_count / cap) ? pair_count : n_tiles * cap;
  return std::min(pair_count, rows) * int64_t(tile) * tile;
}

gart_status check_hit_list_capacity(const gart_frame* f, const gart_settings* st) {
  const int64_t need = hit_list_slots(f->pair_count, int64_t(f->tiles_x) * f->tiles_y, f->tile, st);
  if (need > f->hit_list_capacity)
    return fail(GART_ERR_CAPACITY, "hit_list needs %lld slots (have %lld)", (long long)need,
                (long long)f->hit_list_capacity);
  return GART_OK;
}

// Scratch regions of the bounds step, wherever they live (the frame's
// scratch, or the library's static array).
struct BoundsScratch {
  void* scan_tmp;                 // area prefix-sum temporaries
  unsigned long long* totals;     // 3 words: (L,T) entries, pairs, colour bound bits
  unsigned long long* partials;   // 2 words per block of kBoundsBlock Gaussians
};

gart_status check_bounds_args(const gart_gaussians* g, const gart_camera* camera, const gart_settings* settings,
                              const gart_frame* f) {
  gart_status st;
  if ((st = check_gaussians(g)) != GART_OK) return st;
  if ((st = check_camera(camera)) != GART_OK) return st;
  if ((st = check_settings(settings)) != GART_OK) return st;
  GART_REQUIRE(f != nullptr, "frame is NULL");
  GART_REQUIRE(f->lt_offset != nullptr, "frame lt_offset is NULL");
  if (g->n > 0) GART_REQUIRE(f->rect && f->prim_geom && f->tile_count, "frame per-Gaussian buffer is NULL");
  GART_REQUIRE(f->rect == nullptr || aligned16(f->rect), "rect must be 16-byte aligned");
  return GART_OK;
}

// Per-Gaussian bounds, the area prefix sum and the totals, then the one host
// synchronisation (arguments already checked).
gart_status run_bounds(const gart_gaussians* g, const gart_camera* camera, const gart_settings* settings,
                       gart_frame* f, int64_t* lt_entries_host, int64_t* pair_count_host, hipStream_t s,
                       const BoundsScratch& S) {
  const int64_t n = g->n;
  const int K = (g->sh_degree + 1) * (g->sh_degree + 1);
  f->stage = 0;
  BoundsArgs A{};
  A.means = g->means;
  A.log_scales = g->log_scales;
  A.quats = g->quats;
  A.logits = g->opacity_logits;
  A.sh = g->sh;
  A.K = K;
  A.n = n;
  A.cam = make_cam(camera);
  A.alpha_min = settings->alpha_min;
  A.tile = settings->tile;
  A.rect = f->rect;
  A.area = f->lt_offset;
  A.geom = f->prim_geom;
  A.tile_count = f->tile_count;
  A.block_partial = S.partials;
  GART_HIP(launch_bounds(A, s));
  GART_HIP(scan_exclusive_i64(f->lt_offset, f->lt_offset, n, f->lt_offset + n, S.scan_tmp, s));
  GART_HIP(launch_bounds_totals(A.block_partial, (n + kBoundsBlock - 1) / kBoundsBlock, f->lt_offset + n, S.totals,
                                s));
  unsigned long long tot[3] = {0, 0, 0};  // (L,T) entries, pairs, colour bound bits
  GART_HIP(hipMemcpyAsync(tot, S.totals, sizeof tot, hipMemcpyDeviceToHost, s));
  GART_HIP(hipStreamSynchronize(s));
  const int64_t host[2] = {int64_t(tot[0]), int64_t(tot[1])};
  float cb;
  const uint32_t cb_bits = uint32_t(tot[2]);
  std::memcpy(&cb, &cb_bits, sizeof cb);
  f->color_step = double(cb > 0.0f ? cb : 1.0f) / 4294967296.0;

  f->n = n;
  f->sh_degree = g->sh_degree;
  f->tiles_x = tiles_along(camera->width, settings->tile);
  f->tiles_y = tiles_along(camera->height, settings->tile);
  f->width = camera->width;
  f->height = camera->height;
  f->tile = settings->tile;
  f->reserved = 0;
  f->lt_entries = host[0];
  f->pair_count = host[1];
  if (lt_entries_host) *lt_entries_host = host[0];
  if (pair_count_host) *pair_count_host = host[1];
  if (host[0] > f->lt_capacity || host[1] > f->pair_capacity)
    return fail(GART_ERR_CAPACITY, "need lt %lld (have %lld), pairs %lld (have %lld)", (long long)host[0],
                (long long)f->lt_capacity, (long long)host[1], (long long)f->pair_capacity);
  if (host[1] >= (int64_t(1) << 32)) return fail(GART_ERR_UNSUPPORTED, "more than 2^32 tile pairs");
  f->stage = 1;
  return GART_OK;
}

// ---- allocation-free bounds (gart_bounds_noalloc) ----
// The scratch of the bounds step held by the library itself, one copy per
// GPU for the life of the process, so that callers that cannot allocate
// device memory need not bring any.  Host code never uses the array's name
// as an address: each device's address comes from hipGetSymbolAddress.
struct StaticLayout {
  size_t scan_tmp, totals, partials, total;
};

StaticLayout static_layout(int64_t n) {
  StaticLayout L{};
  const int64_t nn = std::max<int64_t>(n, 1);
  L.scan_tmp = 0;
  L.totals = align_up(scan_tmp_bytes(nn + 1));
  L.partials = L.totals + align_up(64);
  L.total = L.partials + align_up(size_t((nn + kBoundsBlock - 1) / kBoundsBlock) * 16);
  return L;
}

constexpr int kMaxDevices = 64;
std::mutex g_static_mu;
void* g_static_ptr[kMaxDevices] = {};

// Device address of this GPU's copy of the static scratch, looked up once per
// device with that device current.
hipError_t static_scratch_ptr(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return e;
  if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
  std::lock_guard<std::mutex> lock(g_static_mu);
  if (g_static_ptr[dev] == nullptr) {
    void* p = nullptr;
    if ((e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch))) != hipSuccess) return e;
    if (p == nullptr) return hipErrorInvalidSymbol;
    g_static_ptr[dev] = p;
  }
  *out = g_static_ptr[dev];
  return hipSuccess;
}

}  // namespace

extern "C" {

int64_t gart_l1_partials(int64_t n) { return n > 0 ? l1_partials(n) : 1; }

gart_status gart_l1_loss_grad(const float* image, const float* target, int64_t n, float* dL_dimage, double* loss,
                              double* partial, void* stream) {
  g_err[0] = 0;
  GART_REQUIRE(n >= 0, "n < 0");
  GART_REQUIRE(n == 0 || (image && target && dL_dimage), "image/target/dL_dimage is NULL");
  GART_REQUIRE(loss == nullptr || partial != nullptr, "loss requested without partial scratch");
  GART_REQUIRE(n == 0 || (dL_dimage != image && dL_dimage != target), "dL_dimage aliases an input");
  GART_HIP(launch_l1_grad(image, target, n, dL_dimage, partial, loss, static_cast<hipStream_t>(stream)));
  return GART_OK;
}

gart_status gart_adam_step(float* param, const float* grad, float* m, float* v, int64_t n, const gart_adam* h,
                           int64_t step, void* stream) {
  g_err[0] = 0;
  GART_REQUIRE(h != nullptr, "hyper-parameters are NULL");
  GART_REQUIRE(n >= 0 && step >= 1, "n < 0 or step < 1");
  GART_REQUIRE(n == 0 || (param && grad && m && v), "param/grad/m/v is NULL");
  GART_REQUIRE(std::isfinite(h->lr) && h->lr > 0.0f, "lr must be > 0");
  GART_REQUIRE(h->beta1 >= 0.0f && h->beta1 < 1.0f && h->beta2 >= 0.0f && h->beta2 < 1.0f, "betas outside [0, 1)");
  GART_REQUIRE(std::isfinite(h->eps) && h->eps >= 0.0f, "eps must be >= 0");
  AdamArgs a;
  a.lr = h->lr;
  a.b1 = h->beta1;
  a.b2 = h->beta2;
  a.eps = h->eps;
  a.one_minus_b1 = float(1.0 - double(h->beta1));
  a.one_minus_b2 = float(1.0 - double(h->beta2));
  a.inv_c1 = float(1.0 / (1.0 - std::pow(double(h->beta1), double(step))));
  a.inv_c2 = float(1.0 / (1.0 - std::pow(double(h->beta2), double(step))));
  GART_HIP(launch_adam(param, grad, m, v, n, a, static_cast<hipStream_t>(stream)));
  return GART_OK;
}

const char* gart_status_string(gart_status s) {
  switch (s) {
    case GART_OK: return "GART_OK";
    case GART_ERR_INVALID_ARG: return "GART_ERR_INVALID_ARG";
    case GART_ERR_CAPACITY: return "GART_ERR_CAPACITY";
    case GART_ERR_HIP: return "GART_ERR_HIP";
    case GART_ERR_UNSUPPORTED: return "GART_ERR_UNSUPPORTED";
  }
  return "unknown gart_status";
}

const char* gart_last_error(void) { return g_err; }

gart_status gart_frame_status(const gart_frame* f, uint32_t* flags_host, void* stream) {
  g_err[0] = 0;
  GART_REQUIRE(f != nullptr && flags_host != nullptr, "frame/flags_host is NULL");
  GART_REQUIRE(f->stage >= 3, "gart_forward has not run on this frame");
  const int K = (f->sh_degree + 1) * (f->sh_degree + 1);
  // the status word's offset does not depend on the backward mode
  const Layout L = make_layout(f->n, K, f->pair_capacity, GART_BACKWARD_GATHER, f->tile,
                               int64_t(f->tiles_x) * f->tiles_y);
  GART_REQUIRE(f->scratch != nullptr && f->scratch_bytes >= L.status + 4, "frame scratch is too small");
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint32_t v = 0;
  GART_HIP(hipMemcpyAsync(&v, at<uint32_t>(f->scratch, L.status), sizeof v, hipMemcpyDeviceToHost, s));
  GART_HIP(hipStreamSynchronize(s));
  *flags_host = v;
  return GART_OK;
}

int64_t gart_hit_list_slots(int64_t pair_count, const gart_camera* camera, const gart_settings* settings) {
  g_err[0] = 0;
  if (check_camera(camera) != GART_OK || check_settings(settings) != GART_OK) return -1;
  if (pair_count < 0) {
    fail(GART_ERR_INVALID_ARG, "pair_count %lld < 0", (long long)pair_count);
    return -1;
  }
  const int64_t n_tiles =
      int64_t(tiles_along(camera->width, settings->tile)) * tiles_along(camera->height, settings->tile);
  return hit_list_slots(pair_count, n_tiles, settings->tile, settings);
}

int32_t gart_lt_entry_bytes(const gart_settings* settings) {
  g_err[0] = 0;
  if (check_settings(settings) != GART_OK) return 0;
  static const int32_t bytes[6] = {16, 4, 8, 2, 8, 2};
  return bytes[lt_format_for(settings)];
}

size_t gart_scratch_bytes(int64_t n, int32_t sh_degree, int64_t pair_capacity, const gart_camera* camera,
                          const gart_settings* settings) {
  const int deg = std::min(std::max(sh_degree, 0), 3);
  const int mode = settings ? settings->backward_mode : GART_BACKWARD_GATHER;
  const int tile = settings && settings->tile == 16 ? 16 : 8;
  const int64_t n_tiles = camera && camera->width > 0 && camera->height > 0
                              ? int64_t(tiles_along(camera->width, tile)) * tiles_along(camera->height, tile)
                              : 1;
  return make_layout(std::max<int64_t>(n, 0), (deg + 1) * (deg + 1), std::max<int64_t>(pair_capacity, 0), mode, tile,
                     n_tiles)
      .total;
}

gart_status gart_bounds(const gart_gaussians* g, const gart_camera* camera, const gart_settings* settings,
                        gart_frame* f, int64_t* lt_entries_host, int64_t* pair_count_host, void* stream) {
  g_err[0] = 0;
  gart_status st;
  if ((st = check_bounds_args(g, camera, settings, f)) != GART_OK) return st;
  const int64_t n = g->n;
  const int K = (g->sh_degree + 1) * (g->sh_degree + 1);
  GART_REQUIRE(f->scratch != nullptr, "frame scratch is NULL");
  const Layout L = make_layout(n, K, f->pair_capacity, settings->backward_mode, settings->tile,
                               int64_t(tiles_along(camera->width, settings->tile)) *
                                   tiles_along(camera->height, settings->tile));
  GART_REQUIRE(f->scratch_bytes >= L.total, "scratch_bytes %zu < required %zu", f->scratch_bytes, L.total);
  BoundsScratch S;
  S.scan_tmp = at<void>(f->scratch, L.scan_tmp);
  S.totals = at<unsigned long long>(f->scratch, L.totals);
  S.partials = at<unsigned long long>(f->scratch, L.partials);
  return run_bounds(g, camera, settings, f, lt_entries_host, pair_count_host, static_cast<hipStream_t>(stream), S);
}

gart_status gart_bounds_noalloc(const gart_gaussians* g, const gart_camera* camera, const gart_settings* settings,
                                gart_frame* f, int64_t* lt_entries_host, int64_t* pair_count_host, void* stream) {
  g_err[0] = 0;
  gart_status st;
  if ((st = check_bounds_args(g, camera, settings, f)) != GART_OK) return st;
  GART_REQUIRE(g->n <= GART_BOUNDS_NOALLOC_MAX_N,
               "n = %lld exceeds the %lld Gaussians the library's static scratch serves (use gart_bounds)",
               (long long)g->n, (long long)GART_BOUNDS_NOALLOC_MAX_N);
  const StaticLayout SL = static_layout(g->n);
  GART_REQUIRE(SL.total <= sizeof(scratch), "static scratch of %zu bytes < required %zu", sizeof(scratch), SL.total);
  char* base = nullptr;
  GART_HIP(static_scratch_ptr(reinterpret_cast<void**>(&base)));
  BoundsScratch S;
  S.scan_tmp = base + SL.scan_tmp;
  S.totals = reinterpret_cast<unsigned long long*>(base + SL.totals);
  S.partials = reinterpret_cast<unsigned long long*>(base + SL.partials);
  return run_bounds(g, camera, settings, f, lt_entries_host, pair_count_host, static_cast<hipStream_t>(stream), S);
}

gart_status gart_build_tile_map(const gart_camera* camera, const gart_settings* settings, gart_frame* f,
                                void* stream) {
  g_err[0] = 0;
  gart_status st;
  if ((st = check_camera(camera)) != GART_OK) return st;
  if ((st = check_settings(settings)) != GART_OK) return st;
  GART_REQUIRE(f != nullptr, "frame is NULL");
  GART_REQUIRE(f->stage >= 1, "gart_bounds must succeed on this frame first");
  if ((st = check_frame_geometry(f, camera, settings)) != GART_OK) return st;
  const int64_t n = f->n, P = f->pair_count;
  const int64_t n_tiles = int64_t(f->tiles_x) * f->tiles_y;
  GART_REQUIRE(f->pair_offset && f->tile_range, "frame pair_offset/tile_range is NULL");
  GART_REQUIRE(P <= f->pair_capacity, "pair capacity");
  if (P > 0) GART_REQUIRE(f->pair_tile && f->pair_prim && f->pair_key, "frame pair buffers are NULL");
  const int K = (f->sh_degree + 1) * (f->sh_degree + 1);
  const Layout L = make_layout(n, K, f->pair_capacity, settings->backward_mode, settings->tile, n_tiles);
  GART_REQUIRE(f->scratch_bytes >= L.total, "scratch_bytes %zu < required %zu", f->scratch_bytes, L.total);
  hipStream_t s = static_cast<hipStream_t>(stream);

  TileMapArgs T{};
  T.n = n;
  T.tile = settings->tile;
  T.tiles_x = f->tiles_x;
  T.tiles_y = f->tiles_y;
  T.cam = make_cam(camera);
  T.rect = f->rect;
  T.tile_count = f->tile_count;
  T.geom = f->prim_geom;
  T.pair_offset = f->pair_offset;
  // Emission and the sort keep the combined keys in scratch; the last step
  // splits them into pair_tile and pair_key.
  uint32_t* sorted_keys = at<uint32_t>(f->scratch, L.pair_key_alt);
  T.keys = sorted_keys;
  T.vals = f->pair_prim;
  T.pair_key = f->pair_key;
  T.pair_count = P;
  T.tile_range = f->tile_range;
  // Pair slots per Gaussian in index order, then one key per pair: tile id in
  // the high bits, the pair's depth-bound code below; a stable sort by that
  // key orders each tile's list by depth bound, then by Gaussian index.
  int tile_bits = 1;
  while ((int64_t(1) << tile_bits) < n_tiles) ++tile_bits;
  T.key_bits = std::min(24, 32 - tile_bits);
  GART_HIP(scan_exclusive_u32_i64(f->tile_count, f->pair_offset, n, f->pair_offset + n,
                                  at<void>(f->scratch, L.scan_tmp), s));
  GART_HIP(launch_emit_pairs(T, s));
  GART_HIP(record(f->events[GART_EV_SORT_BEGIN], s));
  GART_HIP(radix_sort_u32(sorted_keys, f->pair_prim, f->pair_tile, at<uint32_t>(f->scratch, L.pair_val_alt), P,
                          tile_bits + T.key_bits, at<void>(f->scratch, L.radix_tmp), s));
  GART_HIP(record(f->events[GART_EV_SORT_END], s));
  T.keys = f->pair_tile;
  GART_HIP(launch_finish_pairs(T, sorted_keys, n_tiles, s));
  // hit_list rows of each tile: its list length, at most the hits a pixel can
  // composite; offsets by an exclusive scan
  int64_t* hl_off = at<int64_t>(f->scratch, L.hl_off);
  GART_HIP(launch_hit_rows(f->tile_range, n_tiles, hit_rows_cap(settings), hl_off, s));
  GART_HIP(scan_exclusive_i64(hl_off, hl_off, n_tiles, hl_off + n_tiles, at<void>(f->scratch, L.scan_tmp), s));
  f->stage = 2;
  return GART_OK;
}

gart_status gart_forward(const gart_gaussians* g, const gart_camera* camera, const gart_settings* settings,
                         gart_frame* f, float* image, void* stream) {
  g_err[0] = 0;
  gart_status st;
  if ((st = check_gaussians(g)) != GART_OK) return st;
  if ((st = check_camera(camera)) != GART_OK) return st;
  if ((st = check_settings(settings)) != GART_OK) return st;
  GART_REQUIRE(f != nullptr, "frame is NULL");
  GART_REQUIRE(f->stage >= 2, "gart_build_tile_map must succeed on this frame first");
  if ((st = check_frame_geometry(f, camera, settings)) != GART_OK) return st;
  GART_REQUIRE(g->n == f->n && g->sh_degree == f->sh_degree, "gaussians differ from gart_bounds");
  GART_REQUIRE(image != nullptr && f->pixel_state != nullptr, "image/pixel_state is NULL");
  GART_REQUIRE(f->lt_entries <= f->lt_capacity, "lt capacity");
  GART_REQUIRE(f->lt_entries == 0 || (f->lt != nullptr && aligned16(f->lt)), "lt must be non-NULL, 16-byte aligned");
  GART_REQUIRE(f->pair_count == 0 || f->hit_list != nullptr, "hit_list is NULL");
  if ((st = check_hit_list_capacity(f, settings)) != GART_OK) return st;
  const int Kf = (f->sh_degree + 1) * (f->sh_degree + 1);
  const Layout Lf = make_layout(f->n, Kf, f->pair_capacity, settings->backward_mode, settings->tile,
                                int64_t(f->tiles_x) * f->tiles_y);
  GART_REQUIRE(f->scratch != nullptr && f->scratch_bytes >= Lf.total, "scratch_bytes %zu < required %zu",
               f->scratch_bytes, Lf.total);
  hipStream_t s = static_cast<hipStream_t>(stream);
  ForwardArgs A{};
  A.cam = make_cam(camera);
  A.tile = settings->tile;
  A.tiles_x = f->tiles_x;
  A.tiles_y = f->tiles_y;
  A.sh_k = (g->sh_degree + 1) * (g->sh_degree + 1);
  A.t_min = settings->t_min;
  A.tile_range = f->tile_range;
  A.pair_prim = f->pair_prim;
  A.pair_key = f->pair_key;
  A.geom = f->prim_geom;
  A.rect = f->rect;
  A.lt_offset = f->lt_offset;
  A.sh = g->sh;
  A.lt = reinterpret_cast<uint4*>(f->lt);
  A.lt_format = lt_format_for(settings);
  A.inv_color_step = 1.0 / f->color_step;
  A.image = image;
  A.pixel_state = f->pixel_state;
  A.hit_list = f->hit_list;
  A.hl_off = at<int64_t>(f->scratch, Lf.hl_off);
  A.tile_visit = at<uint32_t>(f->scratch, Lf.tile_visit);
  A.counters = f->counters;
  A.ev_begin = f->events[GART_EV_FWD_BEGIN];
  A.ev_end = f->events[GART_EV_FWD_END];
  A.status = at<uint32_t>(f->scratch, Lf.status);
  A.pair_count = f->pair_count;
  GART_HIP(fill_u32(A.status, 0u, 1, s));
  GART_HIP(launch_forward(A, s));
  f->lt_format = A.lt_format;
  f->stage = 3;
  return GART_OK;
}

gart_status gart_backward(const gart_gaussians* g, const gart_camera* camera, const gart_settings* settings,
                          const gart_frame* f, const float* dL_dimage, float* g_means,
                          float* g_log_scales, float* g_quats, float* g_logits, float* g_sh, void* stream) {
  g_err[0] = 0;
  gart_status st;
  if ((st = check_gaussians(g)) != GART_OK) return st;
  if ((st = check_camera(camera)) != GART_OK) return st;
  if ((st = check_settings(settings)) != GART_OK) return st;
  GART_REQUIRE(f != nullptr, "frame is NULL");
  GART_REQUIRE(f->stage >= 3, "gart_forward must succeed on this frame first");
  if ((st = check_frame_geometry(f, camera, settings)) != GART_OK) return st;
  GART_REQUIRE(g->n == f->n && g->sh_degree == f->sh_degree, "gaussians differ from gart_bounds");
  GART_REQUIRE(dL_dimage != nullptr, "dL_dimage is NULL");
  GART_REQUIRE(f->pair_count == 0 || f->hit_list != nullptr, "hit_list is NULL");
  if ((st = check_hit_list_capacity(f, settings)) != GART_OK) return st;
  GART_REQUIRE(f->lt_format == lt_format_for(settings),
               "frame lt_format %d does not match backward mode %d / lt_precision %d (render with the same settings)",
               f->lt_format, settings->backward_mode, settings->lt_precision);
  if (g->n > 0) GART_REQUIRE(g_means && g_log_scales && g_quats && g_logits && g_sh, "gradient pointer is NULL");
  const int K = (g->sh_degree + 1) * (g->sh_degree + 1);
  const Layout L = make_layout(f->n, K, f->pair_capacity, settings->backward_mode, settings->tile,
                               int64_t(f->tiles_x) * f->tiles_y);
  GART_REQUIRE(f->scratch_bytes >= L.total, "scratch_bytes %zu < required %zu (backward mode %d)", f->scratch_bytes,
               L.total, settings->backward_mode);
  GART_REQUIRE(aligned16(f->scratch), "scratch must be 16-byte aligned");
  hipStream_t s = static_cast<hipStream_t>(stream);
  BackwardArgs A{};
  A.cam = make_cam(camera);
  A.tile = settings->tile;
  A.tiles_x = f->tiles_x;
  A.tiles_y = f->tiles_y;
  A.sh_k = K;
  A.mode = settings->backward_mode;
  A.n = f->n;
  A.tile_range = f->tile_range;
  A.pair_prim = f->pair_prim;
  A.pair_key = f->pair_key;
  A.geom = f->prim_geom;
  A.rect = f->rect;
  A.lt_offset = f->lt_offset;
  A.pair_offset = f->pair_offset;
  A.tile_count = f->tile_count;
  A.sh = g->sh;
  A.lt = reinterpret_cast<const uint4*>(f->lt);
  A.lt_format = f->lt_format;
  A.color_step = float(f->color_step);
  A.dl_dimage = dL_dimage;
  A.pixel_state = f->pixel_state;
  A.hit_list = f->hit_list;
  A.hl_off = at<int64_t>(f->scratch, L.hl_off);
  A.tile_visit = at<uint32_t>(f->scratch, L.tile_visit);
  A.acc = at<float>(f->scratch, L.acc);
  A.rows = at<float>(f->scratch, L.rows);
  A.row_flag = at<uint8_t>(f->scratch, L.row_flag);
  A.pair_count = f->pair_count;
  A.logits = g->opacity_logits;
  A.log_scales = g->log_scales;
  A.quats = g->quats;
  A.g_means = g_means;
  A.g_log_scales = g_log_scales;
  A.g_quats = g_quats;
  A.g_logits = g_logits;
  A.g_sh = g_sh;
  A.counters = f->counters;
  for (int k = 0; k < 4; ++k) A.ev[k] = f->events[GART_EV_BWD_BEGIN + k];
  GART_HIP(launch_backward(A, s));
  return GART_OK;
}

}  // extern "C"
