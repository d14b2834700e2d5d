// Layout and pre-scaling kernels of the Björck vector-Jacobian product.
//
//   load_grad   : dL/d(output) from the caller's layout and dtype into the
//                 tall, zero-padded fp32 gradient iterate (plus its bf16
//                 copy for bf16 products)
//   dot_partial : per 64x64 tile of the caller's layout, sum of
//                 dL/dW_0 * W in fp64 (fixed order inside the tile)
//   dot_finish  : per matrix, <dL/dW_0, W_0> = inv * (fixed-order sum)
//   writeout    : the derivative of W_0 = W / ||W||_F,
//                   dL/dW = inv (Y_0 - <Y_0, W_0> W_0),  W_0 = inv W,
//                 (Y_0 itself without pre-scaling), in the caller's layout;
//                 zero for a zero matrix and NaN for a non-finite one.
//                 Spectral pre-scaling, W_0 = W / sigma, inv = 1 / sigma:
//                   dL/dW = inv (Y_0 - dscale W) + sum_p a_p b_p^T
//                 with dscale and the rank-1 pairs (tall orientation) from
//                 the backward through the power steps (power.hip).
//
// HBM-bound; the transposed (wide) case goes through an LDS tile so that
// both sides are accessed with coalesced rows.
#include "internal.h"

namespace orth {
namespace {

constexpr int TB = 64;

// tile[x][y] = dL/dW_0 at caller element (R + x, C + y), 0 outside the
// padded tall grid
__device__ inline void caller_tile(const TiledMat& d, const float* y, int R, int C, float (*tile)[TB + 1]) {
  for (int e = threadIdx.x; e < TB * TB; e += 256) {
    const int a = e / TB, b = e % TB;
    if (!d.transposed) {
      const int r = R + a, c = C + b;
      tile[a][b] = (r < d.Mp && c < d.Np) ? gld_f32(y, (int64_t)r * d.Np + c) : 0.f;
    } else {
      // caller (R + b, C + a) is tall (C + a, R + b): rows of the tall
      // buffer are read along b
      const int tr = C + a, tc = R + b;
      tile[b][a] = (tr < d.Mp && tc < d.Np) ? gld_f32(y, (int64_t)tr * d.Np + tc) : 0.f;
    }
  }
  __syncthreads();
}

__global__ __launch_bounds__(256) void vjp_load_grad_kernel(const TiledMat* __restrict__ mats,
                                                            const TileItem* __restrict__ items, int gout_dtype) {
  __shared__ float tile[TB][TB + 1];
  const TileItem it = items[blockIdx.x];
  const TiledMat& d = mats[it.mat];
  const int R = it.ti * TB, C = it.tj * TB;  // tile origin in the tall padded layout
  float* y = d.gy[0];
  uint16_t* yc = static_cast<uint16_t*>(d.yc[0]);
  float* yt = d.gyt[0];
  if (!d.transposed && !yt && R + TB <= d.M && C + TB <= d.N && vec8_ok(d.gout, d.ld_gout, gout_dtype) &&
      vec8_ok(y, d.Np, ORTH_F32) && (!yc || vec8_ok(yc, d.Np, ORTH_BF16))) {
    // interior tile of an untransposed matrix: 16-byte vectors, no staging
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = R + (threadIdx.x >> 3) + 32 * h, c = C + 8 * (threadIdx.x & 7);
      float v[8];
      load8_f32(d.gout, (int64_t)r * d.ld_gout + c, gout_dtype, v);
      const int64_t off = (int64_t)r * d.Np + c;
      store8_f32(y, off, ORTH_F32, v);
      if (yc) store8_f32(yc, off, ORTH_BF16, v);
    }
    return;
  }
  for (int e = threadIdx.x; e < TB * TB; e += 256) {
    const int a = e / TB, b = e % TB;
    if (!d.transposed) {
      const int r = R + a, c = C + b;
      tile[a][b] = (r < d.M && c < d.N) ? load_as_f32(d.gout, (int64_t)r * d.ld_gout + c, gout_dtype) : 0.f;
    } else {
      // caller element (C + a, R + b) is tall element (R + b, C + a)
      const int orow = C + a, ocol = R + b;
      tile[b][a] =
          (orow < d.N && ocol < d.M) ? load_as_f32(d.gout, (int64_t)orow * d.ld_gout + ocol, gout_dtype) : 0.f;
    }
  }
  __syncthreads();
  for (int e = threadIdx.x; e < TB * TB; e += 256) {
    const int a = e / TB, b = e % TB;
    const int64_t off = (int64_t)(R + a) * d.Np + C + b;
    gst_f32(y, off, tile[a][b]);
    if (yc) gst_u16(yc, off, f32_to_bf16(tile[a][b]));
    // fp32 products: the transpose too, Np x Mp (consecutive threads along
    // a, so its rows are written coalesced)
    if (yt) gst_f32(yt, (int64_t)(C + a) * d.Mp + R + b, tile[b][a]);
  }
}

__device__ inline double block_sum_256(double v, double* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  const int w = threadIdx.x >> 6;
  if ((threadIdx.x & 63) == 0) red[w] = v;
  __syncthreads();
  double t = 0.0;
  if (threadIdx.x == 0) t = ((red[0] + red[1]) + red[2]) + red[3];
  return t;  // valid in thread 0
}

__global__ __launch_bounds__(256) void vjp_dot_partial_kernel(const TiledMat* __restrict__ mats,
                                                              const TileItem* __restrict__ items, int in_dtype,
                                                              double* __restrict__ partials) {
  __shared__ float tile[TB][TB + 1];
  __shared__ double red[4];
  const TileItem it = items[blockIdx.x];
  const TiledMat& d = mats[it.mat];
  const int R = it.ti * TB, C = it.tj * TB;  // caller layout
  const float* gy = d.gy[d.gy_final];
  double acc = 0.0;
  if (!d.transposed && R + TB <= d.rows && C + TB <= d.cols && vec8_ok(d.in, d.ld_in, in_dtype) &&
      vec8_ok(gy, d.Np, ORTH_F32)) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = R + (threadIdx.x >> 3) + 32 * h, c = C + 8 * (threadIdx.x & 7);
      float g[8], w[8];
      load8_f32(gy, (int64_t)r * d.Np + c, ORTH_F32, g);
      load8_f32(d.in, (int64_t)r * d.ld_in + c, in_dtype, w);
#pragma unroll
      for (int i = 0; i < 8; ++i) acc += (double)g[i] * (double)w[i];
    }
  } else {
    caller_tile(d, gy, R, C, tile);
    for (int e = threadIdx.x; e < TB * TB; e += 256) {
      const int x = e / TB, y = e % TB;
      const int r = R + x, c = C + y;
      if (r < d.rows && c < d.cols)
        acc += (double)tile[x][y] * (double)load_as_f32(d.in, (int64_t)r * d.ld_in + c, in_dtype);
    }
  }
  const double tot = block_sum_256(acc, red);
  if (threadIdx.x == 0) {
    const int tiles_c = (d.cols + TB - 1) / TB;
    partials[d.partial_base + it.ti * tiles_c + it.tj] = tot;
  }
}

__global__ __launch_bounds__(256) void vjp_dot_finish_kernel(const TiledMat* __restrict__ mats,
                                                             const double* __restrict__ partials) {
  __shared__ double red[4];
  const TiledMat& d = mats[blockIdx.x];
  if (d.fused) return;   // handled by the fused small-matrix kernel
  double ss = 0.0;
  for (int i = threadIdx.x; i < d.n_partials; i += 256) ss += partials[d.partial_base + i];
  const double tot = block_sum_256(ss, red);
  if (threadIdx.x == 0) *d.dot = tot * (double)*d.inv_norm;
}

__global__ __launch_bounds__(256) void vjp_writeout_kernel(const TiledMat* __restrict__ mats,
                                                           const TileItem* __restrict__ items, int in_dtype,
                                                           int prescale, const int32_t* __restrict__ status) {
  __shared__ float tile[TB][TB + 1];
  const TileItem it = items[blockIdx.x];
  const TiledMat& d = mats[it.mat];
  const int R = it.ti * TB, C = it.tj * TB;  // caller layout
  const float* gy = d.gy[d.gy_final];
  const int st = status[d.status_index];
  const float inv = *d.inv_norm;
  const bool spec = prescale == ORTH_PRESCALE_SPECTRAL;
  const bool frob = prescale == ORTH_PRESCALE_FROBENIUS || spec;   // a term in W
  const float dscale = st != ORTH_MAT_OK ? 0.f : spec ? (float)d.sb[SB_DSCALE] : (float)(*d.dot) * inv;
  // rank-1 pairs of the power-iteration branch
  const int npair = spec && st == ORTH_MAT_OK && d.sb[SB_BRANCH] != 0.0 ? 2 * d.pq : 0;
  const int64_t pstride = (int64_t)d.M + d.N;
  auto rank1 = [&](int ti, int tj) {   // tall row, tall column
    double a = 0.0;
    for (int p = 0; p < npair; ++p) a += d.pair[p * pstride + ti] * d.pair[p * pstride + d.M + tj];
    return (float)a;
  };
  if (!d.transposed && R + TB <= d.rows && C + TB <= d.cols && vec8_ok(d.in, d.ld_in, in_dtype) &&
      vec8_ok(d.out, d.ld_out, in_dtype) && vec8_ok(gy, d.Np, ORTH_F32)) {
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = R + (threadIdx.x >> 3) + 32 * h, c = C + 8 * (threadIdx.x & 7);
      float v[8];
      if (st == ORTH_MAT_NONFINITE || st == ORTH_MAT_ZERO) {
        const float f = st == ORTH_MAT_ZERO ? 0.f : __builtin_nanf("");
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = f;
      } else {
        load8_f32(gy, (int64_t)r * d.Np + c, ORTH_F32, v);
        if (frob) {
          float w[8];
          load8_f32(d.in, (int64_t)r * d.ld_in + c, in_dtype, w);
#pragma unroll
          for (int i = 0; i < 8; ++i) v[i] = inv * (v[i] - dscale * w[i]);
        }
        if (npair)
          for (int i = 0; i < 8; ++i) v[i] += rank1(r, c + i);
      }
      store8_f32(d.out, (int64_t)r * d.ld_out + c, in_dtype, v);
    }
    return;
  }
  caller_tile(d, gy, R, C, tile);
  for (int e = threadIdx.x; e < TB * TB; e += 256) {
    const int x = e / TB, y = e % TB;
    const int r = R + x, c = C + y;
    if (r >= d.rows || c >= d.cols) continue;
    float v;
    if (st == ORTH_MAT_NONFINITE) {
      v = __builtin_nanf("");
    } else if (st == ORTH_MAT_ZERO) {
      v = 0.f;
    } else if (frob) {
      const float w = load_as_f32(d.in, (int64_t)r * d.ld_in + c, in_dtype);
      v = inv * (tile[x][y] - dscale * w);
      if (npair) v += d.transposed ? rank1(c, r) : rank1(r, c);
    } else {
      v = tile[x][y];
    }
    store_from_f32(d.out, (int64_t)r * d.ld_out + c, in_dtype, v);
  }
}

}  // namespace

hipError_t launch_vjp_load_grad(const TiledMat* mats, const TileItem* items, int n_items, int gout_dtype,
                                hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  timing_begin("vjp_load_grad", s);
  hipLaunchKernelGGL(vjp_load_grad_kernel, dim3(n_items), dim3(256), 0, s, mats, items, gout_dtype);
  hipError_t e = hipGetLastError();
  timing_end("vjp_load_grad", s);
  return e;
}

hipError_t launch_vjp_dot_partial(const TiledMat* mats, const TileItem* items, int n_items, int in_dtype,
                                  double* partials, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  timing_begin("vjp_dot_partial", s);
  hipLaunchKernelGGL(vjp_dot_partial_kernel, dim3(n_items), dim3(256), 0, s, mats, items, in_dtype, partials);
  hipError_t e = hipGetLastError();
  timing_end("vjp_dot_partial", s);
  return e;
}

hipError_t launch_vjp_dot_finish(const TiledMat* mats, int n_mats, const double* partials, hipStream_t s) {
  if (n_mats <= 0) return hipSuccess;
  timing_begin("vjp_dot_finish", s);
  hipLaunchKernelGGL(vjp_dot_finish_kernel, dim3(n_mats), dim3(256), 0, s, mats, partials);
  hipError_t e = hipGetLastError();
  timing_end("vjp_dot_finish", s);
  return e;
}

hipError_t launch_vjp_writeout(const TiledMat* mats, const TileItem* items, int n_items, int in_dtype,
                               int prescale, const int32_t* status, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  timing_begin("vjp_writeout", s);
  hipLaunchKernelGGL(vjp_writeout_kernel, dim3(n_items), dim3(256), 0, s, mats, items, in_dtype, prescale, status);
  hipError_t e = hipGetLastError();
  timing_end("vjp_writeout", s);
  return e;
}

}  // namespace orth
