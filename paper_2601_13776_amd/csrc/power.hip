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
  if (d.fused) return;   // handled by the fused small-matrix kernel
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
      for (int j = threadIdx.x; j < cn; j += 256) vin[j] = gld_f64(in, cb + j);
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
        for (int c = cols8 + lane; c < d.cols; c += 64)
          acc[k] += (double)load_as_f32(d.in, row + c, in_dtype) * gld_f64(in, c);
        const double t = wave_sum(acc[k]);
        if (lane == 0) gst_f64(out, r, t);
      }
    }
  } else if (!it.coldot) {
    // out[r] = sum_c W[r][c] in[c]: a wave per row, lanes along the row
    for (int i = wave; i < 64; i += 4) {
      const int r = it.block * 64 + i;
      if (r >= d.rows) break;
      double acc = 0.0;
      const int64_t row = (int64_t)r * d.ld_in;
      for (int c = lane; c < d.cols; c += 64) acc += (double)load_as_f32(d.in, row + c, in_dtype) * gld_f64(in, c);
      acc = wave_sum(acc);
      if (lane == 0) gst_f64(out, r, acc);
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
        const double x = gld_f64(in, r);
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
    if (wave == 0 && c < d.cols)
      gst_f64(out, c, ((colsum[0][lane] + colsum[1][lane]) + colsum[2][lane]) + colsum[3][lane]);
  } else {
    // out[c] = sum_r W[r][c] in[r]: lanes along 64 columns, waves interleave rows
    const int c = it.block * 64 + lane;
    double acc = 0.0;
    if (c < d.cols)
      for (int r = wave; r < d.rows; r += 4)
        acc += (double)load_as_f32(d.in, (int64_t)r * d.ld_in + c, in_dtype) * gld_f64(in, r);
    part[wave][lane] = acc;
    __syncthreads();
    if (wave == 0 && c < d.cols) gst_f64(out, c, ((part[0][lane] + part[1][lane]) + part[2][lane]) + part[3][lane]);
  }
}

// sigma_hat = |y| / |x| and v = y / |y| (v and sigma_hat = 0 kept if y = 0)
__global__ __launch_bounds__(256) void power_normalize_kernel(const TiledMat* __restrict__ mats) {
  __shared__ double red[4];
  const TiledMat& d = mats[blockIdx.x];
  if (d.fused) return;
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

// ---------------------------------------------------------------------------
// Vector-Jacobian product through spectral pre-scaling.  With X the tall
// orientation of the caller's W, sigma = max(sigma_hat, ||X||_F / sqrt(N)),
// G_0 = dL/dX_0 and c = -<G_0, X> / sigma^2 = -<G_0, X_0> / sigma:
//   dL/dX = G_0 / sigma + c X / (||X||_F sqrt(N))        (the floor is the max)
//   dL/dX = G_0 / sigma + sum of 2q rank-1 terms           (sigma_hat is)
// where the rank-1 terms come from the chain rule through the q power
// steps, the cached vector being constant: with a = |y_q|, b = |x_q|,
//   yh = c y_q / (a b),  gx = -c a x_q / b^3 + X yh:  x_q yh^T + gx v_{q-1}^T,
//   gv = X^T gx, then for k = q-1 .. 1:
//   gy = (gv - <gv, v_k> v_k) / |y_k|:  x_k gy^T + (X gy) v_{k-1}^T,
//   gv = X^T X gy.
// The matrix-vector products run on power_dot_kernel with the backward table
// `bw` (pv, px, py pointing at the backward's vectors); the kernels below are
// the per-matrix glue between them (one block per matrix, fp64).

// v_k of the forward's power steps into the per-step store (k >= 1: also
// that step's x_k = X v_{k-1} and y_k = X^T x_k)
__global__ __launch_bounds__(256) void power_keep_kernel(const TiledMat* __restrict__ mats, int k) {
  const TiledMat& d = mats[blockIdx.x];
  if (d.fused || !d.pst) return;
  const int M = d.M, N = d.N, q = d.pq;
  double* V = d.pst;
  double* Xs = V + (int64_t)(q + 1) * N;
  double* Ys = Xs + (int64_t)q * M;
  for (int j = threadIdx.x; j < N; j += 256) V[(int64_t)k * N + j] = d.pv[j];
  if (k >= 1) {
    for (int i = threadIdx.x; i < M; i += 256) Xs[(int64_t)(k - 1) * M + i] = d.px[i];
    for (int j = threadIdx.x; j < N; j += 256) Ys[(int64_t)(k - 1) * N + j] = d.py[j];
  }
}

// branch, writeout coefficient, and (power-iteration branch) pair 0 =
// (x_q, yh), the start of pair 1 = (-c a x_q / b^3, v_{q-1}); bw.pv = yh
__global__ __launch_bounds__(256) void spec_bwd_start_kernel(const TiledMat* __restrict__ mats,
                                                             const TiledMat* __restrict__ bw,
                                                             const int32_t* __restrict__ status) {
  __shared__ double red[4];
  const TiledMat& d = mats[blockIdx.x];
  if (d.fused || !d.sb) return;
  const TiledMat& b = bw[blockIdx.x];
  const int M = d.M, N = d.N, q = d.pq;
  const int st = status[d.status_index];
  const double F = d.sb[SB_FRO], sigma = d.sb[SB_SIGMA], sh = *d.sig;
  const double dot = *d.dot;
  const double c = -dot / sigma;
  const bool power = st == ORTH_MAT_OK && q > 0 && sh > 0.0 && sh >= F / sqrt((double)N);
  if (threadIdx.x == 0) {
    d.sb[SB_BRANCH] = power ? 1.0 : 0.0;
    d.sb[SB_DSCALE] = st == ORTH_MAT_OK && !power ? dot / (F * sqrt((double)N)) : 0.0;
    d.sb[SB_C] = c;
  }
  if (!power) return;
  const double* V = d.pst;
  const double* x = V + (int64_t)(q + 1) * N + (int64_t)(q - 1) * M;
  const double* y = V + (int64_t)(q + 1) * N + (int64_t)q * M + (int64_t)(q - 1) * N;
  double sx = 0.0, sy = 0.0;
  for (int i = threadIdx.x; i < M; i += 256) sx += x[i] * x[i];
  for (int j = threadIdx.x; j < N; j += 256) sy += y[j] * y[j];
  const double bn = sqrt(block_sum(sx, red));
  const double a = sqrt(block_sum(sy, red));
  double* p0 = d.pair;
  double* p1 = d.pair + (M + N);
  const double xs = -c * a / (bn * bn * bn);
  for (int i = threadIdx.x; i < M; i += 256) {
    p0[i] = x[i];
    p1[i] = xs * x[i];
  }
  const double ys = c / (a * bn);
  for (int j = threadIdx.x; j < N; j += 256) {
    const double yh = ys * y[j];
    p0[M + j] = yh;
    b.pv[j] = yh;
    p1[M + j] = V[(int64_t)(q - 1) * N + j];
  }
}

// gx = pair 1's start + X yh (bw.px): pair 1's a, and bw.px = gx for X^T gx
__global__ __launch_bounds__(256) void spec_bwd_gx_kernel(const TiledMat* __restrict__ mats,
                                                          const TiledMat* __restrict__ bw) {
  const TiledMat& d = mats[blockIdx.x];
  if (d.fused || !d.sb || d.sb[SB_BRANCH] == 0.0) return;
  const TiledMat& b = bw[blockIdx.x];
  double* p1 = d.pair + (d.M + d.N);
  for (int i = threadIdx.x; i < d.M; i += 256) {
    const double g = p1[i] + b.px[i];
    p1[i] = g;
    b.px[i] = g;
  }
}

// earlier step k: gy from gv = bw.py; pair 2 (q - k) = (x_k, gy); bw.pv = gy
__global__ __launch_bounds__(256) void spec_bwd_gy_kernel(const TiledMat* __restrict__ mats,
                                                          const TiledMat* __restrict__ bw, int k) {
  __shared__ double red[4];
  const TiledMat& d = mats[blockIdx.x];
  if (d.fused || !d.sb || d.sb[SB_BRANCH] == 0.0) return;
  const TiledMat& b = bw[blockIdx.x];
  const int M = d.M, N = d.N, q = d.pq;
  const double* vk = d.pst + (int64_t)k * N;
  const double* xk = d.pst + (int64_t)(q + 1) * N + (int64_t)(k - 1) * M;
  const double* yk = d.pst + (int64_t)(q + 1) * N + (int64_t)q * M + (int64_t)(k - 1) * N;
  double sd = 0.0, sy = 0.0;
  for (int j = threadIdx.x; j < N; j += 256) {
    sd += b.py[j] * vk[j];
    sy += yk[j] * yk[j];
  }
  const double dv = block_sum(sd, red);
  const double ny = sqrt(block_sum(sy, red));
  double* p = d.pair + (int64_t)(2 * (q - k)) * (M + N);
  for (int i = threadIdx.x; i < M; i += 256) p[i] = xk[i];
  for (int j = threadIdx.x; j < N; j += 256) {
    const double gy = (b.py[j] - dv * vk[j]) / ny;
    p[M + j] = gy;
    b.pv[j] = gy;
  }
}

// pair 2 (q - k) + 1 = (X gy (bw.px), v_{k-1}); bw.px stays as the input of
// the next X^T product
__global__ __launch_bounds__(256) void spec_bwd_xg_kernel(const TiledMat* __restrict__ mats,
                                                          const TiledMat* __restrict__ bw, int k) {
  const TiledMat& d = mats[blockIdx.x];
  if (d.fused || !d.sb || d.sb[SB_BRANCH] == 0.0) return;
  const TiledMat& b = bw[blockIdx.x];
  const int M = d.M, N = d.N, q = d.pq;
  double* p = d.pair + (int64_t)(2 * (q - k) + 1) * (M + N);
  const double* vk1 = d.pst + (int64_t)(k - 1) * N;
  for (int i = threadIdx.x; i < M; i += 256) p[i] = b.px[i];
  for (int j = threadIdx.x; j < N; j += 256) p[M + j] = vk1[j];
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

namespace orth {

hipError_t launch_power_keep(const TiledMat* mats, int n_mats, int k, hipStream_t s) {
  if (n_mats <= 0) return hipSuccess;
  timing_begin("power_keep", s);
  hipLaunchKernelGGL(power_keep_kernel, dim3(n_mats), dim3(256), 0, s, mats, k);
  hipError_t e = hipGetLastError();
  timing_end("power_keep", s);
  return e;
}

// The whole backward through the power steps; the matrix-vector products
// run for every tiled matrix (those in the floor branch ignore theirs).
hipError_t launch_spec_bwd(const TiledMat* mats, const TiledMat* bw, int n_mats, const PowerItem* items0,
                           int n_items0, const PowerItem* items1, int n_items1, int q, int in_dtype,
                           const int32_t* status, hipStream_t s) {
  if (n_mats <= 0) return hipSuccess;
  auto glue = [&](auto kern, auto... args) {
    timing_begin("spec_bwd", s);
    hipLaunchKernelGGL(kern, dim3(n_mats), dim3(256), 0, s, mats, bw, args...);
    hipError_t e = hipGetLastError();
    timing_end("spec_bwd", s);
    return e;
  };
  hipError_t e = glue(spec_bwd_start_kernel, status);
  if (e == hipSuccess) e = launch_power_dot(bw, items0, n_items0, in_dtype, s);      // X yh
  if (e == hipSuccess) e = glue(spec_bwd_gx_kernel);
  if (e == hipSuccess && q > 1) e = launch_power_dot(bw, items1, n_items1, in_dtype, s);   // X^T gx
  for (int k = q - 1; k >= 1 && e == hipSuccess; --k) {
    e = glue(spec_bwd_gy_kernel, k);
    if (e == hipSuccess) e = launch_power_dot(bw, items0, n_items0, in_dtype, s);    // X gy
    if (e == hipSuccess) e = glue(spec_bwd_xg_kernel, k);
    if (e == hipSuccess && k > 1) e = launch_power_dot(bw, items1, n_items1, in_dtype, s);   // X^T X gy
  }
  return e;
}

}  // namespace orth
