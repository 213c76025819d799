// Training-step kernels around the render/backward path: the L1 photometric
// loss and its gradient (the upstream gradient dL/dC of the backward), and
// the Adam update of one parameter group.
//
// L1: loss = sum_k |C_k - C*_k| over the image's floats, dL/dC_k =
// sign(C_k - C*_k) (0 where equal).  The loss sum is deterministic: fixed
// per-block partial sums in fp64, then one block sums the partials.
//
// Adam (Kingma and Ba): m <- b1 m + (1 - b1) g, v <- b2 v + (1 - b2) g^2,
// p <- p - lr (m / c1) / (sqrt(v / c2) + eps) with the bias corrections
// c1 = 1 - b1^t, c2 = 1 - b2^t of step t (computed on the host in fp64).
#include <hip/hip_runtime.h>

#include "ops.h"

namespace gart {
namespace {

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

__global__ __launch_bounds__(kL1Block) void l1_grad_kernel(const float* __restrict__ image,
                                                           const float* __restrict__ target, int64_t n,
                                                           float* __restrict__ dl, double* __restrict__ partial) {
  __shared__ double s_sum[kL1Block / 64];
  double acc = 0.0;
  const int64_t b0 = int64_t(blockIdx.x) * kL1Items;
  // each thread: kL1Items / kL1Block consecutive strided elements
  for (int64_t k = b0 + threadIdx.x; k < min(n, b0 + kL1Items); k += kL1Block) {
    const float d = image[k] - target[k];
    dl[k] = d > 0.0f ? 1.0f : (d < 0.0f ? -1.0f : 0.0f);
    acc += fabs(double(image[k]) - double(target[k]));
  }
  if (partial) {
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
    if (__lane_id() == 0) s_sum[threadIdx.x / 64] = acc;
    __syncthreads();
    if (threadIdx.x == 0) {
      double t = 0.0;
      for (int w = 0; w < kL1Block / 64; ++w) t += s_sum[w];
      partial[blockIdx.x] = t;
    }
  }
}

__global__ __launch_bounds__(256) void sum_partials_kernel(const double* __restrict__ partial, int64_t nb,
                                                           double* __restrict__ out) {
  __shared__ double s_sum[4];
  double acc = 0.0;
  for (int64_t b = threadIdx.x; b < nb; b += 256) acc += partial[b];
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) acc += __shfl_xor(acc, off);
  if (__lane_id() == 0) s_sum[threadIdx.x / 64] = acc;
  __syncthreads();
  if (threadIdx.x == 0) *out = (s_sum[0] + s_sum[1]) + (s_sum[2] + s_sum[3]);
}

__global__ __launch_bounds__(256) void adam_kernel(float* __restrict__ p, const float* __restrict__ g,
                                                   float* __restrict__ m, float* __restrict__ v, int64_t n,
                                                   AdamArgs h) {
  const int64_t k0 = (int64_t(blockIdx.x) * 256 + threadIdx.x) * 4;
  if (k0 + 4 <= n && (reinterpret_cast<uintptr_t>(p + k0) & 15) == 0 && (reinterpret_cast<uintptr_t>(g + k0) & 15) == 0 &&
      (reinterpret_cast<uintptr_t>(m + k0) & 15) == 0 && (reinterpret_cast<uintptr_t>(v + k0) & 15) == 0) {
    float4 pp = *reinterpret_cast<float4*>(p + k0);
    const float4 gg = *reinterpret_cast<const float4*>(g + k0);
    float4 mm = *reinterpret_cast<float4*>(m + k0);
    float4 vv = *reinterpret_cast<float4*>(v + k0);
    float* pa = &pp.x;
    const float* ga = &gg.x;
    float* ma = &mm.x;
    float* va = &vv.x;
#pragma unroll
    for (int u = 0; u < 4; ++u) {
      ma[u] = fmaf(h.b1, ma[u], h.one_minus_b1 * ga[u]);
      va[u] = fmaf(h.b2, va[u], h.one_minus_b2 * (ga[u] * ga[u]));
      pa[u] -= h.lr * (ma[u] * h.inv_c1) / (sqrtf(va[u] * h.inv_c2) + h.eps);
    }
    *reinterpret_cast<float4*>(p + k0) = pp;
    *reinterpret_cast<float4*>(m + k0) = mm;
    *reinterpret_cast<float4*>(v + k0) = vv;
  } else {
    for (int64_t k = k0; k < min(n, k0 + 4); ++k) {
      const float gk = g[k];
      const float mk = fmaf(h.b1, m[k], h.one_minus_b1 * gk);
      const float vk = fmaf(h.b2, v[k], h.one_minus_b2 * (gk * gk));
      m[k] = mk;
      v[k] = vk;
      p[k] -= h.lr * (mk * h.inv_c1) / (sqrtf(vk * h.inv_c2) + h.eps);
    }
  }
}

}  // namespace

int64_t l1_partials(int64_t n) { return ceil_div(n, kL1Items); }

hipError_t launch_l1_grad(const float* image, const float* target, int64_t n, float* dl, double* partial,
                          double* loss, hipStream_t s) {
  if (n <= 0) {
    if (loss) return fill_f32(reinterpret_cast<float*>(loss), 0.0f, 2, s);
    return hipSuccess;
  }
  const int64_t nb = l1_partials(n);
  l1_grad_kernel<<<nb, kL1Block, 0, s>>>(image, target, n, dl, loss ? partial : nullptr);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || !loss) return e;
  sum_partials_kernel<<<1, 256, 0, s>>>(partial, nb, loss);
  return hipGetLastError();
}

hipError_t launch_adam(float* p, const float* g, float* m, float* v, int64_t n, const AdamArgs& h, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  adam_kernel<<<ceil_div(n, 1024), 256, 0, s>>>(p, g, m, v, n, h);
  return hipGetLastError();
}

}  // namespace gart
