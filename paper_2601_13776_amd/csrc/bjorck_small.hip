// Fused Björck for small matrices: one workgroup owns one matrix and keeps
// it in LDS for the whole run — load (transposing wide inputs to the tall
// orientation), Frobenius or spectral pre-scaling, T steps of
//     E = I - X^T X,   X <- X + beta X E      (Appendix A.5, E-form of
//                                              (1+beta) X - beta X X^T X)
// and the final store.  Products run on fp32 MFMA (v_mfma_f32_32x32x2f32);
// zero padding of X to a 32 x NP grid is exact (padded rows and columns of
// X stay zero and the padded diagonal of E is 1).
#include "internal.h"

namespace orth {

typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace {

__device__ inline double wave_sum(double v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  return v;
}
__device__ inline int wave_or(int v) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v |= __shfl_xor(v, off, 64);
  return v;
}

// 32x32 accumulator layout of the 32x32xK MFMAs: element r of lane l sits at
// row 8 (r / 4) + 4 (l / 32) + (r % 4), column l % 32.
__device__ inline int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// sum over the block, fixed order; valid in every thread
template <int NWAVES>
__device__ inline double block_sum(double v, double* red) {
  v = wave_sum(v);
  __syncthreads();
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  double t = 0.0;
#pragma unroll
  for (int w = 0; w < NWAVES; ++w) t += red[w];
  return t;
}

// The caller's M x N matrix (or its transpose, for a wide one) into the tall
// zero-padded Mp x NP LDS layout (pitch NP + 1), with U independent loads
// of every thread in flight before their LDS stores.  With `stats`, also
// the finiteness flag and the squared norm (fp64) of the loaded values.
template <int NP, int NTHR>
__device__ inline void load_tall(float* dst, const void* src, int64_t ld, int transposed, int M, int N, int Mp,
                                 int dtype, bool stats, double& ss, int& bad) {
  constexpr int U = 8, XP = NP + 1;
  const int total = Mp * NP;
  const int sh = dtype == ORTH_BF16 ? 16 : 0;
  for (int base = 0; base < total; base += NTHR * U) {
    // raw bits, widened after the batch (a conversion inside the guarded
    // load would make each load wait for its data)
    uint32_t w[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int idx = base + u * NTHR + (int)threadIdx.x;
      const int r = idx / NP, c = idx % NP;
      w[u] = 0;
      if (idx < total && r < M && c < N) {
        const int64_t e = transposed ? (int64_t)c * ld + r : (int64_t)r * ld + c;
        w[u] = dtype == ORTH_BF16 ? (uint32_t)gld_u16(src, e) : gld_u32(src, e);
      }
    }
    float v[U];
#pragma unroll
    for (int u = 0; u < U; ++u) {
      asm volatile("" : "+v"(w[u]));
      v[u] = __uint_as_float(w[u] << sh);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
      const int idx = base + u * NTHR + (int)threadIdx.x;
      if (idx < total) {
        const int r = idx / NP, c = idx % NP;
        dst[r * XP + c] = v[u];
        if (stats && r < M && c < N) {
          bad |= !isfinite(v[u]);
          ss += (double)v[u] * (double)v[u];
        }
      }
    }
  }
}

// Spectral pre-scaling on the unscaled tall X in LDS (power iteration on
// X^T X from the caller's cached vector, fp64): returns
// max(|X^T X v| / |X v|, ||X||_F / sqrt(N)) and writes the new vector back.
template <int NP, int NWAVES>
__device__ double spectral_sigma(const float* X, const SmallMat& d, int power_iters, double tot, double* red) {
  constexpr int XP = NP + 1, NTHR = 64 * NWAVES;
  __shared__ double v[NP], y[NP], x[128];
  const int tid = threadIdx.x, M = d.M, N = d.N;
  double ss = 0.0;
  for (int j = tid; j < N; j += NTHR) {
    const double u = d.u[j];
    ss += u * u;
  }
  const double nu = sqrt(block_sum<NWAVES>(ss, red));
  const bool ok = nu > 0.0 && isfinite(nu);
  for (int j = tid; j < N; j += NTHR) v[j] = ok ? d.u[j] / nu : 1.0 / sqrt((double)N);
  __syncthreads();
  double sig = 0.0;
  for (int q = 0; q < power_iters; ++q) {
    for (int i = tid; i < M; i += NTHR) {
      double a = 0.0;
      for (int j = 0; j < N; ++j) a += (double)X[i * XP + j] * v[j];
      x[i] = a;
    }
    __syncthreads();
    for (int j = tid; j < N; j += NTHR) {
      double a = 0.0;
      for (int i = 0; i < M; ++i) a += (double)X[i * XP + j] * x[i];
      y[j] = a;
    }
    __syncthreads();
    double sx = 0.0, sy = 0.0;
    for (int i = tid; i < M; i += NTHR) sx += x[i] * x[i];
    for (int j = tid; j < N; j += NTHR) sy += y[j] * y[j];
    const double nx = sqrt(block_sum<NWAVES>(sx, red));
    const double ny = sqrt(block_sum<NWAVES>(sy, red));
    if (ny == 0.0) {   // uniform: v stays, and so would every later step
      sig = 0.0;
      break;
    }
    sig = ny / nx;
    for (int j = tid; j < N; j += NTHR) v[j] = y[j] / ny;
    __syncthreads();
  }
  for (int j = tid; j < N; j += NTHR) d.u[j] = (float)v[j];
  return fmax(sig, sqrt(tot) / sqrt((double)N));
}

// The power steps of spectral_sigma for a vector-Jacobian product: from the
// cached vector the differentiated forward started from, every step's
// vectors kept in d.pst (v_0 .. v_q, then x_1 .. x_q, then y_1 .. y_q, fp64)
// and the cached vector left untouched.  Returns sigma_hat.
template <int NP, int NWAVES>
__device__ double spectral_keep(const float* X, const SmallVjpMat& d, int q, double* red) {
  constexpr int XP = NP + 1, NTHR = 64 * NWAVES;
  __shared__ double v[NP], y[NP], x[128];
  const int tid = threadIdx.x, M = d.M, N = d.N;
  double* V = d.pst;
  double* Xs = V + (int64_t)(q + 1) * N;
  double* Ys = Xs + (int64_t)q * M;
  double ss = 0.0;
  for (int j = tid; j < N; j += NTHR) {
    const double u = d.u[j];
    ss += u * u;
  }
  const double nu = sqrt(block_sum<NWAVES>(ss, red));
  const bool ok = nu > 0.0 && isfinite(nu);
  for (int j = tid; j < N; j += NTHR) {
    v[j] = ok ? d.u[j] / nu : 1.0 / sqrt((double)N);
    V[j] = v[j];
  }
  __syncthreads();
  double sig = 0.0;
  for (int k = 1; k <= q; ++k) {
    for (int i = tid; i < M; i += NTHR) {
      double a = 0.0;
      for (int j = 0; j < N; ++j) a += (double)X[i * XP + j] * v[j];
      x[i] = a;
      Xs[(int64_t)(k - 1) * M + i] = a;
    }
    __syncthreads();
    for (int j = tid; j < N; j += NTHR) {
      double a = 0.0;
      for (int i = 0; i < M; ++i) a += (double)X[i * XP + j] * x[i];
      y[j] = a;
      Ys[(int64_t)(k - 1) * N + j] = a;
    }
    __syncthreads();
    double sx = 0.0, sy = 0.0;
    for (int i = tid; i < M; i += NTHR) sx += x[i] * x[i];
    for (int j = tid; j < N; j += NTHR) sy += y[j] * y[j];
    const double nx = sqrt(block_sum<NWAVES>(sx, red));
    const double ny = sqrt(block_sum<NWAVES>(sy, red));
    if (ny == 0.0) {   // uniform: the floor of the max is the scale
      sig = 0.0;
      break;
    }
    sig = ny / nx;
    for (int j = tid; j < N; j += NTHR) {
      v[j] = y[j] / ny;
      V[(int64_t)k * N + j] = v[j];
    }
    __syncthreads();
  }
  return sig;
}

// The backward through the power steps (the power-iteration branch of the
// max): the 2q rank-1 pairs (a: M values, b: N values) of dL/dX, written
// after the kept vectors in d.pst.  X holds X_0 = X / sigma; c = -<G_0, X_0>
// / sigma.  With a = |y_q|, b = |x_q|: yh = c y_q / (a b), gx = -c a x_q /
// b^3 + X yh give x_q yh^T + gx v_{q-1}^T; then gv = X^T gx and for
// k = q-1 .. 1: gy = (gv - <gv, v_k> v_k) / |y_k| gives x_k gy^T +
// (X gy) v_{k-1}^T, and gv = X^T X gy.
template <int NP, int NWAVES>
__device__ void spectral_small_bwd(const float* X, const SmallVjpMat& d, int q, double sigma, double c,
                                   double* red) {
  constexpr int XP = NP + 1, NTHR = 64 * NWAVES;
  __shared__ double vn[NP], vm[128];
  const int tid = threadIdx.x, M = d.M, N = d.N;
  const double* V = d.pst;
  const double* Xs = V + (int64_t)(q + 1) * N;
  const double* Ys = Xs + (int64_t)q * M;
  double* pair = d.pst + (int64_t)(q + 1) * N + (int64_t)q * (M + N);
  const int64_t ps = (int64_t)M + N;
  const double* x = Xs + (int64_t)(q - 1) * M;
  const double* y = Ys + (int64_t)(q - 1) * N;
  double sx = 0.0, sy = 0.0;
  for (int i = tid; i < M; i += NTHR) sx += x[i] * x[i];
  for (int j = tid; j < N; j += NTHR) sy += y[j] * y[j];
  const double bn = sqrt(block_sum<NWAVES>(sx, red));
  const double a = sqrt(block_sum<NWAVES>(sy, red));
  for (int j = tid; j < N; j += NTHR) {
    vn[j] = c * y[j] / (a * bn);
    pair[M + j] = vn[j];                          // pair 0: (x_q, yh)
    pair[ps + M + j] = V[(int64_t)(q - 1) * N + j];   // pair 1's b: v_{q-1}
  }
  __syncthreads();
  const double xs = -c * a / (bn * bn * bn);
  for (int i = tid; i < M; i += NTHR) {
    double t = 0.0;
    for (int j = 0; j < N; ++j) t += (double)X[i * XP + j] * vn[j];
    vm[i] = xs * x[i] + sigma * t;                // gx
    pair[i] = x[i];
    pair[ps + i] = vm[i];
  }
  __syncthreads();
  for (int k = q - 1; k >= 1; --k) {
    // gv = X^T (gx or X gy) into vn
    for (int j = tid; j < N; j += NTHR) {
      double t = 0.0;
      for (int i = 0; i < M; ++i) t += (double)X[i * XP + j] * vm[i];
      vn[j] = sigma * t;
    }
    __syncthreads();
    const double* vk = V + (int64_t)k * N;
    const double* yk = Ys + (int64_t)(k - 1) * N;
    double sd = 0.0, sk = 0.0;
    for (int j = tid; j < N; j += NTHR) {
      sd += vn[j] * vk[j];
      sk += yk[j] * yk[j];
    }
    const double dv = block_sum<NWAVES>(sd, red);
    const double nk = sqrt(block_sum<NWAVES>(sk, red));
    double* p = pair + (int64_t)(2 * (q - k)) * ps;
    for (int j = tid; j < N; j += NTHR) {
      vn[j] = (vn[j] - dv * vk[j]) / nk;          // gy
      p[M + j] = vn[j];
      p[ps + M + j] = V[(int64_t)(k - 1) * N + j];
    }
    for (int i = tid; i < M; i += NTHR) p[i] = Xs[(int64_t)(k - 1) * M + i];
    __syncthreads();
    for (int i = tid; i < M; i += NTHR) {
      double t = 0.0;
      for (int j = 0; j < N; ++j) t += (double)X[i * XP + j] * vn[j];
      vm[i] = sigma * t;                          // X gy
      p[ps + i] = vm[i];
    }
    __syncthreads();
  }
}

template <int NP, int NWAVES>
__global__ __launch_bounds__(64 * NWAVES) void bjorck_small_kernel(const SmallMat* __restrict__ mats, int iters,
                                                                  float beta, int prescale, int power_iters,
                                                                  int in_dtype, int out_dtype,
                                                                  int32_t* __restrict__ status) {
  constexpr int NT = NP / 32;
  constexpr int XP = NP + 1;                      // row pitch of X and E in LDS (floats)
  constexpr int MAXT = (4 * NT + NWAVES - 1) / NWAVES;  // update tiles per wave (Mp <= 128)
  constexpr int NTHR = 64 * NWAVES;
  extern __shared__ float smem[];
  __shared__ double red[NWAVES];
  __shared__ int bad_any;
  const SmallMat d = mats[blockIdx.x];
  float* X = smem;
  float* E = smem + d.Mp * XP;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int M = d.M, N = d.N, Mp = d.Mp;

  // -- load, checking finiteness and accumulating the squared norm in fp64
  if (tid == 0) bad_any = 0;
  __syncthreads();
  double ss = 0.0;
  int bad = 0;
  load_tall<NP, NTHR>(X, d.in, d.ld_in, d.transposed, M, N, Mp, in_dtype, true, ss, bad);
  ss = wave_sum(ss);
  if (wave_or(bad) && lane == 0) bad_any = 1;
  if (lane == 0) red[wave] = ss;
  __syncthreads();
  double tot = 0.0;
#pragma unroll
  for (int w = 0; w < NWAVES; ++w) tot += red[w];   // fixed order: deterministic
  int st = ORTH_MAT_OK;
  float scale = 1.f;
  if (bad_any) {
    st = ORTH_MAT_NONFINITE;
    scale = __builtin_nanf("");
  } else if (prescale != ORTH_PRESCALE_NONE && tot == 0.0) {
    st = ORTH_MAT_ZERO;
    scale = 0.f;
  } else if (prescale == ORTH_PRESCALE_FROBENIUS) {
    scale = (float)(1.0 / sqrt(tot));
  } else if (prescale == ORTH_PRESCALE_SPECTRAL) {
    scale = (float)(1.0 / spectral_sigma<NP, NWAVES>(X, d, power_iters, tot, red));
  }
  if (tid == 0 && status) status[d.status_index] = st;
  for (int idx = tid; idx < Mp * NP; idx += NTHR) {
    const int r = idx / NP, c = idx - (idx / NP) * NP;
    X[r * XP + c] *= scale;   // NaN scale turns the whole matrix into NaN
  }
  __syncthreads();

  const int half = lane >> 5, col = lane & 31;
  const int MT = Mp / 32;
  for (int t = 0; t < iters; ++t) {
    // E = I - X^T X: the NT x NT output tiles are shared out over the waves
    for (int tile = wave; tile < NT * NT; tile += NWAVES) {
      const int gi = tile / NT, gj = tile % NT;
      f32x16 acc = {};
      for (int kk = 0; kk < Mp; kk += 2) {
        const float* row = X + (kk + half) * XP;
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(row[gi * 32 + col], row[gj * 32 + col], acc, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = gi * 32 + acc_row(r, lane), j = gj * 32 + col;
        E[i * XP + j] = (i == j ? 1.f : 0.f) - acc[r];
      }
    }
    __syncthreads();
    // X <- X + beta X E: every wave computes its tiles from the old X, then
    // all write after a barrier
    f32x16 acc[MAXT];
#pragma unroll
    for (int q = 0; q < MAXT; ++q) {
      acc[q] = f32x16{};
      const int tile = wave + q * NWAVES;
      if (tile < MT * NT) {
        const int ri = tile / NT, cj = tile % NT;
        const float* xrow = X + (ri * 32 + col) * XP;
        for (int kk = 0; kk < NP; kk += 2)
          acc[q] = __builtin_amdgcn_mfma_f32_32x32x2f32(xrow[kk + half], E[(kk + half) * XP + cj * 32 + col], acc[q],
                                                        0, 0, 0);
      }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < MAXT; ++q) {
      const int tile = wave + q * NWAVES;
      if (tile < MT * NT) {
        const int ri = tile / NT, cj = tile % NT;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = ri * 32 + acc_row(r, lane), j = cj * 32 + col;
          X[i * XP + j] += beta * acc[q][r];
        }
      }
    }
    __syncthreads();
  }

  // -- store in the caller's orientation and dtype
  for (int idx = tid; idx < M * N; idx += NTHR) {
    const int r = idx / N, c = idx - (idx / N) * N;
    const int64_t dst = d.transposed ? (int64_t)c * d.ld_out + r : (int64_t)r * d.ld_out + c;
    store_from_f32(d.out, dst, out_dtype, X[r * XP + c]);
  }
}


// Vector-Jacobian product of the fused small-matrix Björck (Appendix A.5
// iteration, differentiated): with Y the gradient with respect to X_{t+1},
//     S' = -(X_t^T Y + Y^T X_t),   Y <- Y + beta (Y E_t + X_t S'),
// for t = T-1 .. 0, after a forward recomputation that saves X_t and E_t;
// then the pre-scaling derivative dL/dW = inv (Y_0 - <Y_0, X_0> X_0)
// (Frobenius, X_0 = inv W) or Y_0 (none), written in the caller's layout.
// LDS holds X, E, Y and S' (row pitch NP + 1 floats).
template <int NP, int NWAVES>
__global__ __launch_bounds__(64 * NWAVES) void bjorck_small_vjp_kernel(const SmallVjpMat* __restrict__ mats,
                                                                      int iters, float beta, int prescale,
                                                                      int power_iters, int in_dtype,
                                                                      int gout_dtype,
                                                                      int32_t* __restrict__ status) {
  constexpr int NT = NP / 32;
  constexpr int XP = NP + 1;
  constexpr int MAXT = (4 * NT + NWAVES - 1) / NWAVES;  // update tiles per wave (Mp <= 128)
  constexpr int NTHR = 64 * NWAVES;
  extern __shared__ float smem[];
  __shared__ double red[NWAVES];
  __shared__ int bad_any;
  const SmallVjpMat d = mats[blockIdx.x];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int M = d.M, N = d.N, Mp = d.Mp, MT = Mp / 32;
  float* X = smem;
  float* Y = X + Mp * XP;
  float* E = Y + Mp * XP;
  float* S = E + NP * XP;
  const int half = lane >> 5, col = lane & 31;
  const int64_t step_floats = (int64_t)Mp * NP + NP * NP;

  // -- W into X (tall), finiteness and squared norm (fp64, fixed order)
  if (tid == 0) bad_any = 0;
  __syncthreads();
  double ss = 0.0;
  int bad = 0;
  load_tall<NP, NTHR>(X, d.w, d.ld_w, d.transposed, M, N, Mp, in_dtype, true, ss, bad);
  ss = wave_sum(ss);
  if (wave_or(bad) && lane == 0) bad_any = 1;
  if (lane == 0) red[wave] = ss;
  __syncthreads();
  double tot = 0.0;
#pragma unroll
  for (int w = 0; w < NWAVES; ++w) tot += red[w];
  int st = ORTH_MAT_OK;
  float scale = 1.f;
  double sig_hat = 0.0, sigma = 0.0;
  if (bad_any) {
    st = ORTH_MAT_NONFINITE;
    scale = __builtin_nanf("");
  } else if (prescale != ORTH_PRESCALE_NONE && tot == 0.0) {
    st = ORTH_MAT_ZERO;
    scale = 0.f;
  } else if (prescale == ORTH_PRESCALE_FROBENIUS) {
    scale = (float)(1.0 / sqrt(tot));
  } else if (prescale == ORTH_PRESCALE_SPECTRAL) {
    sig_hat = spectral_keep<NP, NWAVES>(X, d, power_iters, red);
    sigma = fmax(sig_hat, sqrt(tot) / sqrt((double)N));
    scale = (float)(1.0 / sigma);
  }
  if (tid == 0 && status) status[d.status_index] = st;
  for (int idx = tid; idx < Mp * NP; idx += NTHR) {
    const int r = idx / NP, c = idx - (idx / NP) * NP;
    X[r * XP + c] *= scale;
  }
  __syncthreads();

  // E = I - X^T X into E
  auto gram = [&]() {
    for (int tile = wave; tile < NT * NT; tile += NWAVES) {
      const int gi = tile / NT, gj = tile % NT;
      f32x16 acc = {};
      for (int kk = 0; kk < Mp; kk += 2) {
        const float* row = X + (kk + half) * XP;
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(row[gi * 32 + col], row[gj * 32 + col], acc, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i = gi * 32 + acc_row(r, lane), j = gj * 32 + col;
        E[i * XP + j] = (i == j ? 1.f : 0.f) - acc[r];
      }
    }
  };
  // P <- P + beta (P Q + P2 Q2) over the Mp x NP update tiles (P2 may be
  // null); every wave computes from the old P, then all write after a barrier
  auto update = [&](float* P, const float* Q, const float* P2, const float* Q2) {
    f32x16 acc[MAXT];
#pragma unroll
    for (int q = 0; q < MAXT; ++q) {
      acc[q] = f32x16{};
      const int tile = wave + q * NWAVES;
      if (tile < MT * NT) {
        const int ri = tile / NT, cj = tile % NT;
        const float* prow = P + (ri * 32 + col) * XP;
        for (int kk = 0; kk < NP; kk += 2)
          acc[q] = __builtin_amdgcn_mfma_f32_32x32x2f32(prow[kk + half], Q[(kk + half) * XP + cj * 32 + col], acc[q],
                                                        0, 0, 0);
        if (P2) {
          const float* p2row = P2 + (ri * 32 + col) * XP;
          for (int kk = 0; kk < NP; kk += 2)
            acc[q] = __builtin_amdgcn_mfma_f32_32x32x2f32(p2row[kk + half], Q2[(kk + half) * XP + cj * 32 + col],
                                                          acc[q], 0, 0, 0);
        }
      }
    }
    __syncthreads();
#pragma unroll
    for (int q = 0; q < MAXT; ++q) {
      const int tile = wave + q * NWAVES;
      if (tile < MT * NT) {
        const int ri = tile / NT, cj = tile % NT;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = ri * 32 + acc_row(r, lane), j = cj * 32 + col;
          P[i * XP + j] += beta * acc[q][r];
        }
      }
    }
    __syncthreads();
  };
  // LDS <-> the saved slot of step t (pitch NP in memory)
  auto save_step = [&](int t) {
    float* xs = d.save + t * step_floats;
    float* es = xs + (int64_t)Mp * NP;
    for (int idx = tid; idx < Mp * NP; idx += NTHR) gst_f32(xs, idx, X[(idx / NP) * XP + idx % NP]);
    for (int idx = tid; idx < NP * NP; idx += NTHR) gst_f32(es, idx, E[(idx / NP) * XP + idx % NP]);
  };
  // (X and E are contiguous in the slot: 16-byte loads, U of them in
  // flight per thread before their LDS stores)
  auto load_step = [&](int t) {
    constexpr int U = 4;
    const float4* src = reinterpret_cast<const float4*>(d.save + t * step_floats);
    const int xq = Mp * NP / 4, total = xq + NP * NP / 4;
    for (int base = 0; base < total; base += NTHR * U) {
      float4 v[U];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int q = base + u * NTHR + tid;
        if (q < total) v[u] = gld_f32x4(src + q);
      }
#pragma unroll
      for (int u = 0; u < U; ++u) {
        const int q = base + u * NTHR + tid;
        if (q < total) {
          const int e = 4 * (q < xq ? q : q - xq);
          float* dst = (q < xq ? X : E) + (e / NP) * XP + e % NP;
          dst[0] = v[u].x;
          dst[1] = v[u].y;
          dst[2] = v[u].z;
          dst[3] = v[u].w;
        }
      }
    }
    __syncthreads();
  };

  // -- forward recomputation: X_t, E_t saved for t < T (X_T is never needed)
  for (int t = 0; t < iters; ++t) {
    gram();
    __syncthreads();
    save_step(t);
    if (t + 1 < iters) update(X, E, nullptr, nullptr);
  }

  // -- dL/dX_T from the caller's layout (tall, zero padded)
  load_tall<NP, NTHR>(Y, d.gout, d.ld_gout, d.transposed, M, N, Mp, gout_dtype, false, ss, bad);
  __syncthreads();

  // -- gradient recurrence, last step first (X_{T-1}, E_{T-1} are in LDS)
  for (int t = iters - 1; t >= 0; --t) {
    if (t + 1 < iters) load_step(t);
    for (int tile = wave; tile < NT * NT; tile += NWAVES) {
      const int gi = tile / NT, gj = tile % NT;
      f32x16 acc = {};
      for (int kk = 0; kk < Mp; kk += 2) {
        const float* xr = X + (kk + half) * XP;
        const float* yr = Y + (kk + half) * XP;
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(xr[gi * 32 + col], yr[gj * 32 + col], acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(yr[gi * 32 + col], xr[gj * 32 + col], acc, 0, 0, 0);
      }
#pragma unroll
      for (int r = 0; r < 16; ++r) S[(gi * 32 + acc_row(r, lane)) * XP + gj * 32 + col] = -acc[r];
    }
    __syncthreads();
    update(Y, E, X, S);
  }

  // -- pre-scaling derivative (X holds X_0 here) in the caller's layout
  float dot = 0.f;
  double dotd = 0.0;
  if (prescale != ORTH_PRESCALE_NONE && st == ORTH_MAT_OK) {
    double a = 0.0;
    for (int idx = tid; idx < M * N; idx += NTHR) {
      const int r = idx / N, c = idx - (idx / N) * N;
      a += (double)Y[r * XP + c] * (double)X[r * XP + c];
    }
    dotd = block_sum<NWAVES>(a, red);
    dot = (float)dotd;
  }
  // spectral pre-scaling: dL/dX = Y_0 / sigma - <Y_0, X_0> X_0 / (||X||_F
  // sqrt(N)) when the floor is the max, else Y_0 / sigma plus the rank-1
  // pairs of the power steps
  int npair = 0;
  float xcoef = 0.f;
  if (prescale == ORTH_PRESCALE_SPECTRAL && st == ORTH_MAT_OK) {
    const double fro = sqrt(tot);
    if (power_iters > 0 && sig_hat > 0.0 && sig_hat >= fro / sqrt((double)N)) {
      spectral_small_bwd<NP, NWAVES>(X, d, power_iters, sigma, -dotd / sigma, red);
      npair = 2 * power_iters;
    } else {
      xcoef = (float)(-dotd / (fro * sqrt((double)N)));
    }
  }
  const double* pairs = npair ? d.pst + (int64_t)(power_iters + 1) * N + (int64_t)power_iters * (M + N) : nullptr;
  for (int idx = tid; idx < M * N; idx += NTHR) {
    const int r = idx / N, c = idx - (idx / N) * N;
    float v;
    if (st == ORTH_MAT_NONFINITE)
      v = __builtin_nanf("");
    else if (st == ORTH_MAT_ZERO)
      v = 0.f;
    else if (prescale == ORTH_PRESCALE_FROBENIUS)
      v = scale * (Y[r * XP + c] - dot * X[r * XP + c]);
    else if (prescale == ORTH_PRESCALE_SPECTRAL) {
      double a = 0.0;
      for (int p = 0; p < npair; ++p) a += pairs[p * (M + N) + r] * pairs[p * (M + N) + M + c];
      v = scale * Y[r * XP + c] + xcoef * X[r * XP + c] + (float)a;
    } else
      v = Y[r * XP + c];
    const int64_t dst = d.transposed ? (int64_t)c * d.ld_gin + r : (int64_t)r * d.ld_gin + c;
    store_from_f32(d.gin, dst, in_dtype, v);
  }
}

}  // namespace

hipError_t launch_bjorck_small(const SmallMat* mats, int n, int np, int max_mp, int iters, float beta,
                               int prescale, int power_iters, int in_dtype, int out_dtype, int32_t* status,
                               hipStream_t s) {
  if (n <= 0) return hipSuccess;
  // dynamic LDS sized for the tallest matrix of this launch (max_mp <= 128)
  const size_t lds = (size_t)(max_mp + np) * (np + 1) * sizeof(float);
  timing_begin("bjorck_small", s);
  // 32-wide matrices: one wavefront each (a single Gram tile); 64-wide: four
  // wavefronts share the 4 Gram tiles and up to 8 update tiles
  if (np == 32)
    hipLaunchKernelGGL((bjorck_small_kernel<32, 1>), dim3(n), dim3(64), lds, s, mats, iters, beta, prescale,
                       power_iters, in_dtype, out_dtype, status);
  else
    hipLaunchKernelGGL((bjorck_small_kernel<64, 4>), dim3(n), dim3(256), lds, s, mats, iters, beta, prescale,
                       power_iters, in_dtype, out_dtype, status);
  hipError_t e = hipGetLastError();
  timing_end("bjorck_small", s);
  return e;
}

hipError_t launch_bjorck_small_vjp(const SmallVjpMat* mats, int n, int np, int max_mp, int iters, float beta,
                                   int prescale, int power_iters, int in_dtype, int gout_dtype, int32_t* status,
                                   hipStream_t s) {
  if (n <= 0) return hipSuccess;
  // X and Y (max_mp rows), E and S' (np rows), pitch np + 1: at most 99.8 KB
  const size_t lds = (size_t)(2 * max_mp + 2 * np) * (np + 1) * sizeof(float);
  timing_begin("bjorck_small_vjp", s);
  hipError_t e;
  if (np == 32) {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&bjorck_small_vjp_kernel<32, 1>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e == hipSuccess)
      hipLaunchKernelGGL((bjorck_small_vjp_kernel<32, 1>), dim3(n), dim3(64), lds, s, mats, iters, beta, prescale,
                         power_iters, in_dtype, gout_dtype, status);
  } else {
    e = hipFuncSetAttribute(reinterpret_cast<const void*>(&bjorck_small_vjp_kernel<64, 4>),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (e == hipSuccess)
      hipLaunchKernelGGL((bjorck_small_vjp_kernel<64, 4>), dim3(n), dim3(256), lds, s, mats, iters, beta, prescale,
                         power_iters, in_dtype, gout_dtype, status);
  }
  if (e == hipSuccess) e = hipGetLastError();
  timing_end("bjorck_small_vjp", s);
  return e;
}

}  // namespace orth
