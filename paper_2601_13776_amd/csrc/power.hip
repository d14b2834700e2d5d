// Batched power iteration for spectral pre-scaling (App. A.5, Section 2):
// with X the tall orientation of W and v the cached vector,
//     x = X v,  y = X^T x,  sigma_hat = |y| / |x|,  v = y / |y|,
// for every tiled matrix of a batch at once.  The two matrix-vector
// products run on the caller's W directly (row dot products for W v or W x,
// column dot products for W^T v or W^T x, depending on the orientation);
// vectors and sums are fp64, every reduction has a fixed order.  One pass
// over W per product: HBM-bound.
#include "internal.h"

namespace orth {
namespace {

__device__ inline double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}

// sum over the 256 threads of a block, fixed order; valid in every thread
__device__ inline double block_sum(double v, double* red) {
  v = wave_sum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return ((red[0] + red[1]) + red[2]) + red[3];
}

// v = u / |u| (ones / sqrt(N) for a zero or non-finite u)
__global__ __launch_bounds__(256) void power_init_kernel(const TiledMat* __restrict__ mats) {
  __shared__ double red[4];
  const TiledMat& d = mats[blockIdx.x];
  double ss = 0.0;
  for (int j = threadIdx.x; j < d.N; j += 256) {
    const double u = d.u[j];
    ss += u * u;
  }
  const double nu = sqrt(block_sum(ss, red));
  const bool ok = nu > 0.0 && isfinite(nu);
  for (int j = threadIdx.x; j < d.N; j += 256) d.pv[j] = ok ? d.u[j] / nu : 1.0 / sqrt((double)d.N);
}

__global__ __launch_bounds__(256) void power_dot_kernel(const TiledMat* __restrict__ mats,
                                                        const PowerItem* __restrict__ items, int in_dtype) {
  __shared__ double part[4][64];
  const PowerItem it = items[blockIdx.x];
  const TiledMat& d = mats[it.mat];
  const double* in = it.second ? d.px : d.pv;
  double* out = it.second ? d.py : d.px;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  // rows and columns start 16-byte aligned: runs of 8 elements are loaded
  // with one 16-byte (bf16) or two (fp32) vector loads
  const bool vec = vec8_ok(d.in, d.ld_in, in_dtype);
  if (!it.coldot && vec) {
    // out[r] = sum_c W[r][c] in[c]: a wave per row, lanes along the row in
    // 8-element runs; the vector goes through LDS one chunk of columns at a
    // time, so that the 64 rows of the block share each load of it
    constexpr int CH = 2048;
    __shared__ double vin[CH];
    const int cols8 = d.cols / 8 * 8;
    double acc[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) acc[k] = 0.0;
    for (int cb = 0; cb < cols8; cb += CH) {
      const int cn = cols8 - cb < CH ? cols8 - cb : CH;
      __syncthreads();   // the previous chunk's reads are done
      for (int j = threadIdx.x; j < cn; j += 256) vin[j] = in[cb + j];
      __syncthreads();
#pragma unroll
      for (int k = 0; k < 16; ++k) {
        const int r = it.block * 64 + wave + 4 * k;
        if (r < d.rows) {
          const int64_t row = (int64_t)r * d.ld_in + cb;
          for (int c0 = lane * 8; c0 < cn; c0 += 512) {
            float w[8];
            load8_f32(d.in, row + c0, in_dtype, w);
#pragma unroll
            for (int q = 0; q < 8; ++q) acc[k] += (double)w[q] * vin[c0 + q];
          }
        }
      }
    }
#pragma unroll
    for (int k = 0; k < 16; ++k) {
      const int r = it.block * 64 + wave + 4 * k;
      if (r < d.rows) {
        const int64_t row = (int64_t)r * d.ld_in;
        for (int c = cols8 + lane; c < d.cols; c += 64) acc[k] += (double)load_as_f32(d.in, row + c, in_dtype) * in[c];
        const double t = wave_sum(acc[k]);
        if (lane == 0) out[r] = t;
      }
    }
  } else if (!it.coldot) {
    // out[r] = sum_c W[r][c] in[c]: a wave per row, lanes along the row
    for (int i = wave; i < 64; i += 4) {
      const int r = it.block * 64 + i;
      if (r >= d.rows) break;
      double acc = 0.0;
      const int64_t row = (int64_t)r * d.ld_in;
      for (int c = lane; c < d.cols; c += 64) acc += (double)load_as_f32(d.in, row + c, in_dtype) * in[c];
      acc = wave_sum(acc);
      if (lane == 0) out[r] = acc;
    }
  } else if (vec && (d.cols - it.block * 64 >= 64 || d.cols % 8 == 0)) {
    // out[c] = sum_r W[r][c] in[r] over this item's 64 columns: eight lanes
    // cover them with 8-element runs, a wave reads eight rows at a time
    const int cg = lane & 7, rsub = lane >> 3;
    const int c0 = it.block * 64 + cg * 8;
    double acc[8] = {};
    if (c0 < d.cols)
      for (int r = wave * 8 + rsub; r < d.rows; r += 32) {
        float w[8];
        load8_f32(d.in, (int64_t)r * d.ld_in + c0, in_dtype, w);
        const double x = in[r];
#pragma unroll
        for (int q = 0; q < 8; ++q) acc[q] += (double)w[q] * x;
      }
    // fixed-order reduction: over the eight row groups of a wave (lanes
    // with the same column group), then over the four waves
#pragma unroll
    for (int q = 0; q < 8; ++q) {
#pragma unroll
      for (int off = 8; off < 64; off <<= 1) acc[q] += __shfl_xor(acc[q], off, 64);
    }
    __shared__ double colsum[4][64];
    if (rsub == 0)
#pragma unroll
      for (int q = 0; q < 8; ++q) colsum[wave][cg * 8 + q] = acc[q];
    __syncthreads();
    const int c = it.block * 64 + lane;
    if (wave == 0 && c < d.cols) out[c] = ((colsum[0][lane] + colsum[1][lane]) + colsum[2][lane]) + colsum[3][lane];
  } else {
    // out[c] = sum_r W[r][c] in[r]: lanes along 64 columns, waves interleave rows
    const int c = it.block * 64 + lane;
    double acc = 0.0;
    if (c < d.cols)
      for (int r = wave; r < d.rows; r += 4)
        acc += (double)load_as_f32(d.in, (int64_t)r * d.ld_in + c, in_dtype) * in[r];
    part[wave][lane] = acc;
    __syncthreads();
    if (wave == 0 && c < d.cols) out[c] = ((part[0][lane] + part[1][lane]) + part[2][lane]) + part[3][lane];
  }
}

// sigma_hat = |y| / |x| and v = y / |y| (v and sigma_hat = 0 kept if y = 0)
__global__ __launch_bounds__(256) void power_normalize_kernel(const TiledMat* __restrict__ mats) {
  __shared__ double red[4];
  const TiledMat& d = mats[blockIdx.x];
  double sx = 0.0, sy = 0.0;
  for (int i = threadIdx.x; i < d.M; i += 256) sx += d.px[i] * d.px[i];
  for (int j = threadIdx.x; j < d.N; j += 256) sy += d.py[j] * d.py[j];
  const double nx = sqrt(block_sum(sx, red));
  const double ny = sqrt(block_sum(sy, red));
  if (ny == 0.0) {
    if (threadIdx.x == 0) *d.sig = 0.0;
    return;
  }
  if (threadIdx.x == 0) *d.sig = ny / nx;
  for (int j = threadIdx.x; j < d.N; j += 256) d.pv[j] = d.py[j] / ny;
}

}  // namespace

hipError_t launch_power_init(const TiledMat* mats, int n_mats, hipStream_t s) {
  if (n_mats <= 0) return hipSuccess;
  timing_begin("power_init", s);
  hipLaunchKernelGGL(power_init_kernel, dim3(n_mats), dim3(256), 0, s, mats);
  hipError_t e = hipGetLastError();
  timing_end("power_init", s);
  return e;
}

hipError_t launch_power_dot(const TiledMat* mats, const PowerItem* items, int n_items, int in_dtype,
                            hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  timing_begin("power_dot", s);
  hipLaunchKernelGGL(power_dot_kernel, dim3(n_items), dim3(256), 0, s, mats, items, in_dtype);
  hipError_t e = hipGetLastError();
  timing_end("power_dot", s);
  return e;
}

hipError_t launch_power_normalize(const TiledMat* mats, int n_mats, hipStream_t s) {
  if (n_mats <= 0) return hipSuccess;
  timing_begin("power_normalize", s);
  hipLaunchKernelGGL(power_normalize_kernel, dim3(n_mats), dim3(256), 0, s, mats);
  hipError_t e = hipGetLastError();
  timing_end("power_normalize", s);
  return e;
}

}  // namespace orth
