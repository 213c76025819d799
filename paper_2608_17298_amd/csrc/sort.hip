// Device-wide exclusive scans and a stable LSD radix sort for wave64.  A scan
// is reduce-then-scan: block sums, then a down-sweep whose blocks add up the
// sums before them (or, past 2048 blocks, a scan of the sums first).
//
// Used for the primitive offset table (prefix sum of footprints, Sec. 4.3),
// the pair offsets, and the radix sort of (tile, primitive) pairs by tile id
// (Sec. 4.3, reverse tile mapping).
#include <hip/hip_runtime.h>

#include <algorithm>

#include "ops.h"

namespace gart {
namespace {

constexpr int kScanThreads = 256;
constexpr int kScanItems = 8;
constexpr int kScanTile = kScanThreads * kScanItems;

constexpr int kSortThreads = 256;
#ifndef GART_SORT_ITEMS
#define GART_SORT_ITEMS 16
#endif
constexpr int kSortItems = GART_SORT_ITEMS;  // keys per thread and radix pass
constexpr int kSortTile = kSortThreads * kSortItems;
constexpr int kWaves = kSortThreads / 64;

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Inclusive scan across one wave64 with shuffles.
template <typename T>
__device__ __forceinline__ T wave_inclusive(T v) {
  const unsigned lane = __lane_id();
#pragma unroll
  for (int off = 1; off < 64; off <<= 1) {
    T u = __shfl_up(v, off);
    if (lane >= unsigned(off)) v += u;
  }
  return v;
}

// Exclusive scan across a 256-thread block; *block_total receives the sum.
template <typename T>
__device__ __forceinline__ T block_exclusive(T v, T* block_total) {
  __shared__ T wsum[kScanThreads / 64];
  const int wave = threadIdx.x / 64;
  const T inc = wave_inclusive(v);
  if (__lane_id() == 63) wsum[wave] = inc;
  __syncthreads();
  T before = 0, total = 0;
#pragma unroll
  for (int w = 0; w < kScanThreads / 64; ++w) {
    if (w < wave) before += wsum[w];
    total += wsum[w];
  }
  __syncthreads();
  *block_total = total;
  return before + inc - v;
}

template <typename Tin, typename T>
__global__ __launch_bounds__(kScanThreads) void scan_reduce_kernel(const Tin* __restrict__ in, int64_t n,
                                                                   T* __restrict__ sums) {
  const int64_t base = int64_t(blockIdx.x) * kScanTile + int64_t(threadIdx.x) * kScanItems;
  T s = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k)
    if (base + k < n) s += T(in[base + k]);
  T total;
  block_exclusive(s, &total);
  if (threadIdx.x == 0) sums[blockIdx.x] = total;
}

// Block offsets come either scanned (block_offset[b]) or as raw block sums,
// which each block adds up for the blocks before it.
template <typename Tin, typename T>
__global__ __launch_bounds__(kScanThreads) void scan_down_kernel(const Tin* in, T* out, int64_t n,
                                                                 const T* __restrict__ block_offset,
                                                                 T* __restrict__ total_out,
                                                                 const T* __restrict__ block_sums) {
  const int64_t base = int64_t(blockIdx.x) * kScanTile + int64_t(threadIdx.x) * kScanItems;
  T v[kScanItems];
  T s = 0;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    v[k] = (base + k < n) ? T(in[base + k]) : T(0);
    s += v[k];
  }
  T off = block_offset ? block_offset[blockIdx.x] : T(0);
  if (block_sums) {
    T part = 0;
    for (int k = threadIdx.x; k < int(blockIdx.x); k += kScanThreads) part += block_sums[k];
    block_exclusive(part, &off);
  }
  T total;
  T run = block_exclusive(s, &total);
  run += off;
#pragma unroll
  for (int k = 0; k < kScanItems; ++k) {
    if (base + k < n) out[base + k] = run;
    run += v[k];
  }
  if (total_out && blockIdx.x == gridDim.x - 1 && threadIdx.x == 0) *total_out = off + total;
}

template <typename Tin, typename T>
hipError_t scan_impl(const Tin* in, T* out, int64_t n, T* total, char* tmp, hipStream_t s) {
  const int64_t nb = std::max<int64_t>(1, ceil_div(n, kScanTile));
  if (nb == 1) {
    scan_down_kernel<Tin, T><<<1, kScanThreads, 0, s>>>(in, out, n, nullptr, total, nullptr);
    return hipGetLastError();
  }
  T* sums = reinterpret_cast<T*>(tmp);
  char* rest = tmp + ((nb * sizeof(T) + 255) & ~size_t(255));
  scan_reduce_kernel<Tin, T><<<nb, kScanThreads, 0, s>>>(in, n, sums);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (nb <= kScanTile) {  // few enough block sums for each block to add up its predecessors
    scan_down_kernel<Tin, T><<<nb, kScanThreads, 0, s>>>(in, out, n, nullptr, total, sums);
    return hipGetLastError();
  }
  e = scan_impl<T, T>(sums, sums, nb, nullptr, rest, s);
  if (e != hipSuccess) return e;
  scan_down_kernel<Tin, T><<<nb, kScanThreads, 0, s>>>(in, out, n, sums, total, nullptr);
  return hipGetLastError();
}

// ---------------------------------------------------------------------------
// Radix sort, 8-bit digits.  Pass = per-block digit histogram (digit-major
// layout), exclusive scan of the histogram, stable scatter.  In the scatter
// each wave owns a contiguous quarter of the block's keys and ranks them on
// its own, 64 at a time: wave64 ballots find the peers holding the same digit
// and a per-wave running count per digit in LDS carries the rank across
// rounds, so the rounds need no block barrier.  One block-wide scan then turns
// the per-wave counts into offsets; the block's keys are staged in LDS in
// digit order and written out as contiguous runs per digit.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(kSortThreads) void radix_hist_kernel(const uint32_t* __restrict__ keys, int64_t m,
                                                                  int shift, uint32_t* __restrict__ counts,
                                                                  int nblocks) {
  __shared__ uint32_t h[256];
  h[threadIdx.x] = 0;
  __syncthreads();
  const int64_t base = int64_t(blockIdx.x) * kSortTile;
  uint32_t kv[kSortItems];
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const int64_t j = base + int64_t(r) * kSortThreads + threadIdx.x;
    kv[r] = j < m ? keys[j] : 0u;
  }
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const int64_t j = base + int64_t(r) * kSortThreads + threadIdx.x;
    if (j < m) atomicAdd(&h[(kv[r] >> shift) & 255u], 1u);
  }
  __syncthreads();
  counts[int64_t(threadIdx.x) * nblocks + blockIdx.x] = h[threadIdx.x];
}

__global__ __launch_bounds__(kSortThreads) void radix_scatter_kernel(
    const uint32_t* __restrict__ kin, const uint32_t* __restrict__ vin, uint32_t* __restrict__ kout,
    uint32_t* __restrict__ vout, int64_t m, int shift, const uint32_t* __restrict__ offsets, int nblocks) {
  __shared__ uint32_t s_keys[kSortTile];
  __shared__ uint32_t s_vals[kSortTile];
  __shared__ uint32_t s_wave[kWaves][256];  // per-wave digit counts, later per-wave digit bases
  __shared__ uint32_t s_start[256];
  __shared__ uint32_t s_gofs[256];
  __shared__ uint32_t s_wsum[kWaves];

  const int tid = threadIdx.x;
  const int wave = tid / 64;
  const unsigned lane = __lane_id();
  const uint64_t lt_mask = (lane == 0) ? 0ull : (~0ull >> (64 - lane));

#pragma unroll
  for (int w = 0; w < kWaves; ++w) s_wave[w][tid] = 0;
  s_gofs[tid] = offsets[int64_t(tid) * nblocks + blockIdx.x];
  __syncthreads();

  // Keys [wbase, wbase + 64 * kSortItems) belong to this wave, so block order
  // is wave, round, lane: the order of the input.
  const int64_t wbase = int64_t(blockIdx.x) * kSortTile + int64_t(wave) * (64 * kSortItems);
  uint32_t myk[kSortItems], myv[kSortItems], myr[kSortItems];
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const int64_t j = wbase + int64_t(r) * 64 + lane;
    myk[r] = j < m ? kin[j] : 0u;
    myv[r] = j < m ? vin[j] : 0u;
  }
  // The running counts are read and updated by different lanes of one wave;
  // LDS executes a wave's accesses in issue order, and volatile keeps the
  // compiler from reordering or caching them.
  volatile uint32_t* wcount = s_wave[wave];
#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    const bool valid = wbase + int64_t(r) * 64 + lane < m;
    const uint32_t d = (myk[r] >> shift) & 255u;
    uint64_t peers = __ballot(valid);
#pragma unroll
    for (int b = 0; b < 8; ++b) {
      const bool bit = (d >> b) & 1u;
      const uint64_t bal = __ballot(bit);
      peers &= bit ? bal : ~bal;
    }
    const uint32_t below = __popcll(peers & lt_mask);
    const uint32_t before = wcount[d];
    myr[r] = before + below;
    if (valid && below == 0) wcount[d] = before + uint32_t(__popcll(peers));
  }
  __syncthreads();

  // Digit tid: block-exclusive start over digits, then each wave's base.
  {
    uint32_t c[kWaves], total = 0;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      c[w] = s_wave[w][tid];
      total += c[w];
    }
    uint32_t inc = total;
#pragma unroll
    for (int off = 1; off < 64; off <<= 1) {
      const uint32_t u = __shfl_up(inc, off);
      if (lane >= unsigned(off)) inc += u;
    }
    if (lane == 63) s_wsum[wave] = inc;
    __syncthreads();
    uint32_t before = 0;
    for (int w = 0; w < wave; ++w) before += s_wsum[w];
    uint32_t run = before + inc - total;
    s_start[tid] = run;
#pragma unroll
    for (int w = 0; w < kWaves; ++w) {
      s_wave[w][tid] = run;
      run += c[w];
    }
  }
  __syncthreads();

#pragma unroll
  for (int r = 0; r < kSortItems; ++r) {
    if (wbase + int64_t(r) * 64 + lane < m) {
      const uint32_t d = (myk[r] >> shift) & 255u;
      const uint32_t pos = s_wave[wave][d] + myr[r];
      s_keys[pos] = myk[r];
      s_vals[pos] = myv[r];
    }
  }
  __syncthreads();

  const int64_t base = int64_t(blockIdx.x) * kSortTile;
  const int cnt = int(std::min<int64_t>(kSortTile, m - base));
  for (int q = tid; q < cnt; q += kSortThreads) {
    const uint32_t k = s_keys[q];
    const uint32_t d = (k >> shift) & 255u;
    const int64_t g = int64_t(s_gofs[d]) + (q - int(s_start[d]));
    kout[g] = k;
    vout[g] = s_vals[q];
  }
}

__global__ void copy_pairs_kernel(const uint32_t* __restrict__ ka, const uint32_t* __restrict__ va,
                                  uint32_t* __restrict__ kb, uint32_t* __restrict__ vb, int64_t m) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < m) {
    kb[i] = ka[i];
    vb[i] = va[i];
  }
}

template <typename T>
__global__ void fill_kernel(T* __restrict__ p, T v, int64_t n) {
  const int64_t stride = int64_t(gridDim.x) * blockDim.x;
  for (int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x; i < n; i += stride) p[i] = v;
}

__global__ void iota_kernel(uint32_t* __restrict__ p, int64_t n) {
  const int64_t i = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
  if (i < n) p[i] = uint32_t(i);
}

template <typename T>
hipError_t fill_any(T* p, T v, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  const int64_t blocks = std::min<int64_t>(ceil_div(n, 256), 4096);
  fill_kernel<T><<<blocks, 256, 0, s>>>(p, v, n);
  return hipGetLastError();
}

}  // namespace

size_t scan_tmp_bytes(int64_t n) {
  size_t total = 0;
  int64_t nb = ceil_div(std::max<int64_t>(n, 1), kScanTile);
  while (nb > 1) {
    total += ((nb * sizeof(int64_t) + 255) & ~size_t(255));
    nb = ceil_div(nb, kScanTile);
  }
  return total + 256;
}

hipError_t scan_exclusive_i64(const int64_t* in, int64_t* out, int64_t n, int64_t* total, void* tmp, hipStream_t s) {
  return scan_impl<int64_t, int64_t>(in, out, n, total, static_cast<char*>(tmp), s);
}

hipError_t scan_exclusive_u32_i64(const uint32_t* in, int64_t* out, int64_t n, int64_t* total, void* tmp,
                                  hipStream_t s) {
  return scan_impl<uint32_t, int64_t>(in, out, n, total, static_cast<char*>(tmp), s);
}

hipError_t scan_exclusive_u32(const uint32_t* in, uint32_t* out, int64_t n, uint32_t* total, void* tmp,
                              hipStream_t s) {
  return scan_impl<uint32_t, uint32_t>(in, out, n, total, static_cast<char*>(tmp), s);
}

size_t radix_tmp_bytes(int64_t m) {
  const int64_t nb = std::max<int64_t>(1, ceil_div(m, kSortTile));
  const size_t counts = ((size_t(nb) * 256 * sizeof(uint32_t) + 255) & ~size_t(255));
  return counts + scan_tmp_bytes(nb * 256);
}

hipError_t radix_sort_u32(uint32_t* keys, uint32_t* vals, uint32_t* keys_alt, uint32_t* vals_alt, int64_t m, int bits,
                          void* tmp, hipStream_t s) {
  if (m <= 1 || bits <= 0) return hipSuccess;
  const int64_t nb = ceil_div(m, kSortTile);
  uint32_t* counts = static_cast<uint32_t*>(tmp);
  char* scan_tmp = static_cast<char*>(tmp) + ((size_t(nb) * 256 * sizeof(uint32_t) + 255) & ~size_t(255));
  uint32_t *ka = keys, *va = vals, *kb = keys_alt, *vb = vals_alt;
  int passes = 0;
  for (int shift = 0; shift < bits; shift += 8, ++passes) {
    radix_hist_kernel<<<nb, kSortThreads, 0, s>>>(ka, m, shift, counts, int(nb));
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    e = scan_exclusive_u32(counts, counts, nb * 256, nullptr, scan_tmp, s);
    if (e != hipSuccess) return e;
    radix_scatter_kernel<<<nb, kSortThreads, 0, s>>>(ka, va, kb, vb, m, shift, counts, int(nb));
    e = hipGetLastError();
    if (e != hipSuccess) return e;
    std::swap(ka, kb);
    std::swap(va, vb);
  }
  if (ka != keys) {
    copy_pairs_kernel<<<ceil_div(m, 256), 256, 0, s>>>(ka, va, keys, vals, m);
    return hipGetLastError();
  }
  return hipSuccess;
}

hipError_t fill_u32(uint32_t* p, uint32_t v, int64_t n, hipStream_t s) { return fill_any<uint32_t>(p, v, n, s); }
hipError_t fill_f32(float* p, float v, int64_t n, hipStream_t s) { return fill_any<float>(p, v, n, s); }
hipError_t fill_u8(uint8_t* p, uint8_t v, int64_t n, hipStream_t s) { return fill_any<uint8_t>(p, v, n, s); }

hipError_t iota_u32(uint32_t* p, int64_t n, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  iota_kernel<<<ceil_div(n, 256), 256, 0, s>>>(p, n);
  return hipGetLastError();
}

}  // namespace gart
