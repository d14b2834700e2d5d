// Elementwise kernels of the exponential parametrizations:
//
//   exponential map (Appendix A.3, "Exponential Map with Spectral
//   Normalization"): A = W - W^T; after the spectral-normalization kernels
//   have produced 1/sigma, Ahat = A / sigma and the series accumulator
//   starts as I + Ahat; the powers Ahat^k / k! then run on the fp32 tile
//   GEMM with the series epilogue (P_k = P_{k-1} Ahat / k, What += P_k).
//
//   explicit conv exponential (Appendix B.2, theorem "Explicit conv
//   exponential", Adaptive-SOC): L = scale (K - K*) with
//   K*[o, i, a, b] = K[i, o, k-1-a, k-1-b] (the adjoint conv's kernel), as
//   a compact k x k tap grid; the accumulator (S x S taps, S = p (k-1) + 1)
//   starts as the centred identity plus the centred L; the block-convolution
//   powers L^(⊛j) / j! run on the tile GEMM (every tap of a power sums up to
//   k^2 tap products) with the series epilogue.
//
// Tap (a, b) of an h x w grid is the c x c matrix at element offset
// (a w + b) c^2.  HBM-bound, one pass each.
#include "internal.h"

namespace orth {
namespace {

__global__ __launch_bounds__(256) void exp_skew_kernel(const ExpItem* __restrict__ items, int conv, int in_dtype) {
  const ExpItem it = items[blockIdx.y];
  const int c = it.c, k = it.k;
  const int64_t cc = (int64_t)c * c;
  const int64_t total = conv ? (int64_t)k * k * cc : cc;
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    if (!conv) {
      const int i = (int)(e / c), j = (int)(e % c);
      it.a[e] = load_as_f32(it.in, (int64_t)i * it.ld_in + j, in_dtype) -
                load_as_f32(it.in, (int64_t)j * it.ld_in + i, in_dtype);
    } else {
      // e enumerates (tap (a, b), o, i) of the compact grid
      const int64_t oi = e % cc;
      const int tap = (int)(e / cc);
      const int a = tap / k, b = tap % k;
      const int o = (int)(oi / c), i = (int)(oi % c);
      const int64_t kk = (int64_t)k * k;
      const float v = load_as_f32(it.in, ((int64_t)o * c + i) * kk + a * k + b, in_dtype) -
                      load_as_f32(it.in, ((int64_t)i * c + o) * kk + (k - 1 - a) * k + (k - 1 - b), in_dtype);
      it.a[e] = it.scale * v;
    }
  }
}

__global__ __launch_bounds__(256) void exp_init_kernel(const ExpItem* __restrict__ items, int conv) {
  const ExpItem it = items[blockIdx.y];
  const int c = it.c;
  const int64_t cc = (int64_t)c * c;
  if (!conv) {
    const float inv = *it.inv;
    for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < cc; e += (int64_t)gridDim.x * 256) {
      const float ah = it.a[e] * inv;
      it.p0[e] = ah;
      it.out[e] = (e / c == e % c ? 1.f : 0.f) + ah;
    }
    return;
  }
  const int S = it.size, k = it.k, mid = (S - 1) / 2, off = (S - k) / 2;
  const int64_t total = (int64_t)S * S * cc;
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int64_t oi = e % cc;
    const int tap = (int)(e / cc);
    const int y = tap / S, x = tap % S;
    float v = (y == mid && x == mid && oi / c == oi % c) ? 1.f : 0.f;
    const int ly = y - off, lx = x - off;
    if (ly >= 0 && ly < k && lx >= 0 && lx < k) v += it.a[(int64_t)(ly * k + lx) * cc + oi];
    it.out[e] = v;
  }
}

unsigned grid_x(int64_t max_elems) {
  int64_t b = (max_elems + 255) / 256;
  if (b < 1) b = 1;
  if (b > 2048) b = 2048;
  return (unsigned)b;
}

}  // namespace

hipError_t launch_exp_skew(const ExpItem* items, int n_items, int conv, int in_dtype, int64_t max_elems,
                           hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  timing_begin("exp_skew", s);
  hipLaunchKernelGGL(exp_skew_kernel, dim3(grid_x(max_elems), n_items), dim3(256), 0, s, items, conv, in_dtype);
  hipError_t e = hipGetLastError();
  timing_end("exp_skew", s);
  return e;
}

hipError_t launch_exp_init(const ExpItem* items, int n_items, int conv, int64_t max_elems, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  timing_begin("exp_init", s);
  hipLaunchKernelGGL(exp_init_kernel, dim3(grid_x(max_elems), n_items), dim3(256), 0, s, items, conv);
  hipError_t e = hipGetLastError();
  timing_end("exp_init", s);
  return e;
}

}  // namespace orth
