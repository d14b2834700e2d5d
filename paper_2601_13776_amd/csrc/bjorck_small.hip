// Fused Björck for small matrices: one wavefront owns one matrix and keeps
// it in LDS for the whole run — load (transposing wide inputs to the tall
// orientation), Frobenius pre-scaling, T steps of
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

template <int NP>
__global__ __launch_bounds__(64) void bjorck_small_kernel(const SmallMat* __restrict__ mats, int iters,
                                                          float beta, int prescale, int in_dtype,
                                                          int out_dtype, int32_t* __restrict__ status) {
  constexpr int NT = NP / 32;
  constexpr int XP = NP + 1;  // row pitch of X and E in LDS (floats)
  extern __shared__ float smem[];
  const SmallMat d = mats[blockIdx.x];
  float* X = smem;
  float* E = smem + d.Mp * XP;
  const int lane = threadIdx.x;
  const int M = d.M, N = d.N, Mp = d.Mp;

  // -- load, checking finiteness and accumulating the squared norm in fp64
  double ss = 0.0;
  int bad = 0;
  for (int idx = lane; idx < Mp * NP; idx += 64) {
    const int r = idx / NP, c = idx - (idx / NP) * NP;
    float v = 0.f;
    if (r < M && c < N) {
      const int64_t src = d.transposed ? (int64_t)c * d.ld_in + r : (int64_t)r * d.ld_in + c;
      v = load_as_f32(d.in, src, in_dtype);
      bad |= !isfinite(v);
      ss += (double)v * (double)v;
    }
    X[r * XP + c] = v;
  }
  ss = wave_sum(ss);
  bad = wave_or(bad);
  int st = ORTH_MAT_OK;
  float scale = 1.f;
  if (bad) {
    st = ORTH_MAT_NONFINITE;
    scale = __builtin_nanf("");
  } else if (prescale == ORTH_PRESCALE_FROBENIUS) {
    if (ss == 0.0) {
      st = ORTH_MAT_ZERO;
      scale = 0.f;
    } else {
      scale = (float)(1.0 / sqrt(ss));
    }
  }
  if (lane == 0 && status) status[d.status_index] = st;
  __syncthreads();
  for (int idx = lane; idx < Mp * NP; idx += 64) {
    const int r = idx / NP, c = idx - (idx / NP) * NP;
    X[r * XP + c] *= scale;   // NaN scale turns the whole matrix into NaN
  }
  __syncthreads();

  const int half = lane >> 5, col = lane & 31;
  const int MT = Mp / 32;
  for (int t = 0; t < iters; ++t) {
    // E = I - X^T X   (NT x NT tiles, contraction over the Mp rows)
#pragma unroll
    for (int gi = 0; gi < NT; ++gi) {
#pragma unroll
      for (int gj = 0; gj < NT; ++gj) {
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
    }
    __syncthreads();
    // X <- X + beta X E, one 32-row block at a time (a block only reads its
    // own rows of X, so it can be overwritten right after)
    for (int ri = 0; ri < MT; ++ri) {
      f32x16 acc[NT];
#pragma unroll
      for (int cj = 0; cj < NT; ++cj) acc[cj] = f32x16{};
      const float* xrow = X + (ri * 32 + col) * XP;
      for (int kk = 0; kk < NP; kk += 2) {
        const float a = xrow[kk + half];
        const float* erow = E + (kk + half) * XP;
#pragma unroll
        for (int cj = 0; cj < NT; ++cj)
          acc[cj] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, erow[cj * 32 + col], acc[cj], 0, 0, 0);
      }
      __syncthreads();
#pragma unroll
      for (int cj = 0; cj < NT; ++cj)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i = ri * 32 + acc_row(r, lane), j = cj * 32 + col;
          X[i * XP + j] += beta * acc[cj][r];
        }
      __syncthreads();
    }
  }

  // -- store in the caller's orientation and dtype
  for (int idx = lane; idx < M * N; idx += 64) {
    const int r = idx / N, c = idx - (idx / N) * N;
    const int64_t dst = d.transposed ? (int64_t)c * d.ld_out + r : (int64_t)r * d.ld_out + c;
    store_from_f32(d.out, dst, out_dtype, X[r * XP + c]);
  }
}

}  // namespace

hipError_t launch_bjorck_small(const SmallMat* mats, int n, int np, int max_mp, int iters, float beta,
                               int prescale, int in_dtype, int out_dtype, int32_t* status, hipStream_t s) {
  if (n <= 0) return hipSuccess;
  // dynamic LDS sized for the tallest matrix of this launch (max_mp <= 128)
  const size_t lds = (size_t)(max_mp + np) * (np + 1) * sizeof(float);
  if (np == 32) {
    timing_begin("bjorck_small", s);
    hipLaunchKernelGGL(bjorck_small_kernel<32>, dim3(n), dim3(64), lds, s, mats, iters, beta, prescale,
                       in_dtype, out_dtype, status);
  } else {
    timing_begin("bjorck_small", s);
    hipLaunchKernelGGL(bjorck_small_kernel<64>, dim3(n), dim3(64), lds, s, mats, iters, beta, prescale,
                       in_dtype, out_dtype, status);
  }
  hipError_t e = hipGetLastError();
  timing_end("bjorck_small", s);
  return e;
}

}  // namespace orth
