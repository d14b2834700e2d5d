// Frobenius pre-scaling and layout kernels of the tiled Björck path.
//
//   partial  : squared norm of every 64x64 tile of every input (fp64 sums,
//              NaN when the tile holds a non-finite value)
//   finish   : per matrix, fixed-order sum of its partials -> the scale
//              (1/||W||_F, or 1/sigma from the power iteration of power.hip)
//              and the per-matrix status (deterministic: no atomics)
//   scale    : W_0 = W / ||W||_F in the tall orientation, zero padded to the
//              tile grid, written as the fp32 iterate plus its bf16 copy
//              (bf16 products) or its transpose (fp32 products)
//   writeout : the fp32 iterate back to the caller's orientation and dtype
//
// All four are HBM-bound; tiles go through LDS so that both the row-major
// and the transposed sides are read and written with coalesced accesses.
#include "internal.h"

namespace orth {
namespace {

constexpr int TB = 64;  // tile edge

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

__global__ __launch_bounds__(256) void prescale_partial_kernel(const TiledMat* __restrict__ mats,
                                                               const TileItem* __restrict__ items,
                                                               int in_dtype, double* __restrict__ partials) {
  __shared__ double red[4];
  __shared__ int bad_any;
  const TileItem it = items[blockIdx.x];
  const TiledMat& d = mats[it.mat];
  if (threadIdx.x == 0) bad_any = 0;
  __syncthreads();
  double ss = 0.0;
  int bad = 0;
  const int R = it.ti * TB, C = it.tj * TB;
  if (R + TB <= d.rows && C + TB <= d.cols && vec8_ok(d.in, d.ld_in, in_dtype)) {
    // interior tile: 16-byte vector loads, rows t / 8 and t / 8 + 32,
    // columns 8 (t % 8) .. + 7
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      float v[8];
      load8_f32(d.in, (int64_t)(R + (threadIdx.x >> 3) + 32 * h) * d.ld_in + C + 8 * (threadIdx.x & 7), in_dtype, v);
#pragma unroll
      for (int i = 0; i < 8; ++i) {
        bad |= !isfinite(v[i]);
        ss += (double)v[i] * (double)v[i];
      }
    }
  } else {
    for (int e = threadIdx.x; e < TB * TB; e += 256) {
      const int r = R + e / TB, c = C + (e % TB);
      if (r < d.rows && c < d.cols) {
        const float v = load_as_f32(d.in, (int64_t)r * d.ld_in + c, in_dtype);
        bad |= !isfinite(v);
        ss += (double)v * (double)v;
      }
    }
  }
  if (bad) atomicOr(&bad_any, 1);
  const double tot = block_sum_256(ss, red);
  if (threadIdx.x == 0) {
    const int tiles_c = (d.cols + TB - 1) / TB;
    partials[d.partial_base + it.ti * tiles_c + it.tj] = bad_any ? __builtin_nan("") : tot;
  }
}

__global__ __launch_bounds__(256) void prescale_finish_kernel(const TiledMat* __restrict__ mats,
                                                              const double* __restrict__ partials,
                                                              int prescale, int32_t* __restrict__ status,
                                                              int write_u) {
  __shared__ double red[4];
  const TiledMat& d = mats[blockIdx.x];
  if (d.fused) return;   // pre-scaled inside the fused small-matrix kernel
  double ss = 0.0;
  for (int i = threadIdx.x; i < d.n_partials; i += 256) ss += partials[d.partial_base + i];
  const double tot = block_sum_256(ss, red);
  __shared__ int st_sh;
  if (threadIdx.x == 0) {
    int st = ORTH_MAT_OK;
    float inv = 1.f;
    if (isnan(tot)) {
      st = ORTH_MAT_NONFINITE;
      inv = __builtin_nanf("");
    } else if (prescale != ORTH_PRESCALE_NONE && tot == 0.0) {
      st = ORTH_MAT_ZERO;
      inv = 0.f;
    } else if (prescale == ORTH_PRESCALE_FROBENIUS) {
      inv = (float)(1.0 / sqrt(tot));
    } else if (prescale == ORTH_PRESCALE_SPECTRAL) {
      // both terms are lower bounds of the largest singular value
      const double sigma = fmax(*d.sig, sqrt(tot) / sqrt((double)d.N));
      inv = (float)(1.0 / sigma);
      if (d.sb) {
        d.sb[SB_FRO] = sqrt(tot);
        d.sb[SB_SIGMA] = sigma;
      }
    }
    *d.inv_norm = inv;
    if (status) status[d.status_index] = st;
    st_sh = st;
  }
  __syncthreads();
  // spectral: hand the new estimate back (a degenerate matrix keeps the old one)
  if (prescale == ORTH_PRESCALE_SPECTRAL && st_sh == ORTH_MAT_OK && write_u)
    for (int j = threadIdx.x; j < d.N; j += 256) d.u[j] = (float)d.pv[j];
}

__global__ __launch_bounds__(256) void prescale_scale_kernel(const TiledMat* __restrict__ mats,
                                                             const TileItem* __restrict__ items,
                                                             int in_dtype, int compute) {
  __shared__ float tile[TB][TB + 1];
  const TileItem it = items[blockIdx.x];
  const TiledMat& d = mats[it.mat];
  const int R = it.ti * TB, C = it.tj * TB;  // tile origin in the tall padded layout
  const float inv = *d.inv_norm;
  if (!d.transposed && compute == ORTH_COMPUTE_BF16 && R + TB <= d.M && C + TB <= d.N &&
      vec8_ok(d.in, d.ld_in, in_dtype) && vec8_ok(d.master[0], d.Np, ORTH_F32) &&
      (!d.xc[0] || vec8_ok(d.xc[0], d.Np, ORTH_BF16))) {
    // interior tile of an untransposed matrix: no staging, 16-byte vectors
    // (rows t / 8 and t / 8 + 32, columns 8 (t % 8) .. + 7)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int r = R + (threadIdx.x >> 3) + 32 * h, c = C + 8 * (threadIdx.x & 7);
      float v[8];
      load8_f32(d.in, (int64_t)r * d.ld_in + c, in_dtype, v);
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] *= inv;
      const int64_t off = (int64_t)r * d.Np + c;
      store8_f32(d.master[0], off, ORTH_F32, v);
      if (d.xc[0]) store8_f32(d.xc[0], off, ORTH_BF16, v);
    }
    return;
  }
  for (int e = threadIdx.x; e < TB * TB; e += 256) {
    const int a = e / TB, b = e % TB;
    if (!d.transposed) {
      const int r = R + a, c = C + b;   // tall == original
      float v = 0.f;
      if (r < d.M && c < d.N) v = load_as_f32(d.in, (int64_t)r * d.ld_in + c, in_dtype);
      tile[a][b] = v * inv;
    } else {
      // original element (C + a, R + b) is tall element (R + b, C + a)
      const int orow = C + a, ocol = R + b;
      float v = 0.f;
      if (orow < d.N && ocol < d.M) v = load_as_f32(d.in, (int64_t)orow * d.ld_in + ocol, in_dtype);
      tile[b][a] = v * inv;
    }
  }
  __syncthreads();
  float* master = d.master[0];
  for (int e = threadIdx.x; e < TB * TB; e += 256) {
    const int a = e / TB, b = e % TB;
    const int64_t off = (int64_t)(R + a) * d.Np + C + b;
    const float v = tile[a][b];
    gst_f32(master, off, v);
    // bf16 products: the bf16 copy; fp32 products: the transposed iterate
    // xt[(C + a)][(R + b)] = tile[b][a] (each only where the plan has one)
    if (compute == ORTH_COMPUTE_BF16 && d.xc[0]) gst_u16(d.xc[0], off, f32_to_bf16(v));
    if (compute != ORTH_COMPUTE_BF16 && d.xt)
      gst_f32(d.xt, (int64_t)(C + a) * d.Mp + R + b, tile[b][a]);
  }
}

__global__ __launch_bounds__(256) void writeout_kernel(const TiledMat* __restrict__ mats,
                                                       const TileItem* __restrict__ items,
                                                       int master_index, int out_dtype) {
  __shared__ float tile[TB][TB + 1];
  const TileItem it = items[blockIdx.x];
  const TiledMat& d = mats[it.mat];
  const float* master = d.master[master_index];
  const int R = it.ti * TB, C = it.tj * TB;  // tile origin in the ORIGINAL layout
  if (!d.transposed) {
    if (R + TB <= d.rows && C + TB <= d.cols && vec8_ok(d.out, d.ld_out, out_dtype) &&
        vec8_ok(master, d.Np, ORTH_F32)) {
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int r = R + (threadIdx.x >> 3) + 32 * h, c = C + 8 * (threadIdx.x & 7);
        float v[8];
        load8_f32(master, (int64_t)r * d.Np + c, ORTH_F32, v);
        store8_f32(d.out, (int64_t)r * d.ld_out + c, out_dtype, v);
      }
      return;
    }
    for (int e = threadIdx.x; e < TB * TB; e += 256) {
      const int r = R + e / TB, c = C + e % TB;
      if (r < d.rows && c < d.cols)
        store_from_f32(d.out, (int64_t)r * d.ld_out + c, out_dtype, gld_f32(master, (int64_t)r * d.Np + c));
    }
    return;
  }
  // original (R + x, C + y) is tall (C + y, R + x)
  for (int e = threadIdx.x; e < TB * TB; e += 256) {
    const int a = e / TB, b = e % TB;
    const int tr = C + a, tc = R + b;  // tall row / col
    tile[a][b] = (tr < d.Mp && tc < d.Np) ? gld_f32(master, (int64_t)tr * d.Np + tc) : 0.f;
  }
  __syncthreads();
  for (int e = threadIdx.x; e < TB * TB; e += 256) {
    const int x = e / TB, y = e % TB;
    const int r = R + x, c = C + y;
    if (r < d.rows && c < d.cols) store_from_f32(d.out, (int64_t)r * d.ld_out + c, out_dtype, tile[y][x]);
  }
}

__global__ void fill_f32_kernel(float* p, int64_t n, float v) {
  for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n; i += (int64_t)gridDim.x * blockDim.x)
    p[i] = v;
}

}  // namespace

hipError_t launch_prescale_partial(const TiledMat* mats, const TileItem* items, int n_items, int in_dtype,
                                   double* partials, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  timing_begin("prescale_partial", s);
  hipLaunchKernelGGL(prescale_partial_kernel, dim3(n_items), dim3(256), 0, s, mats, items, in_dtype, partials);
  hipError_t e = hipGetLastError();
  timing_end("prescale_partial", s);
  return e;
}

hipError_t launch_prescale_finish(const TiledMat* mats, int n_mats, const double* partials, int prescale,
                                  int32_t* status, hipStream_t s, int write_u) {
  if (n_mats <= 0) return hipSuccess;
  timing_begin("prescale_finish", s);
  hipLaunchKernelGGL(prescale_finish_kernel, dim3(n_mats), dim3(256), 0, s, mats, partials, prescale, status,
                     write_u);
  hipError_t e = hipGetLastError();
  timing_end("prescale_finish", s);
  return e;
}

hipError_t launch_prescale_scale(const TiledMat* mats, const TileItem* items, int n_items, int in_dtype,
                                 int compute, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  timing_begin("prescale_scale", s);
  hipLaunchKernelGGL(prescale_scale_kernel, dim3(n_items), dim3(256), 0, s, mats, items, in_dtype, compute);
  hipError_t e = hipGetLastError();
  timing_end("prescale_scale", s);
  return e;
}

hipError_t launch_writeout(const TiledMat* mats, const TileItem* items, int n_items, int master_index,
                           int out_dtype, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  timing_begin("writeout", s);
  hipLaunchKernelGGL(writeout_kernel, dim3(n_items), dim3(256), 0, s, mats, items, master_index, out_dtype);
  hipError_t e = hipGetLastError();
  timing_end("writeout", s);
  return e;
}

hipError_t launch_fill_f32(float* p, int64_t n, float v, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  int64_t blocks = (n + 255) / 256;
  if (blocks > 4096) blocks = 4096;
  hipLaunchKernelGGL(fill_f32_kernel, dim3((unsigned)blocks), dim3(256), 0, s, p, n, v);
  return hipGetLastError();
}

}  // namespace orth
