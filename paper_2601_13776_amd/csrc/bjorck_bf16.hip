// Tiled Björck products for bf16 operands with fp32 accumulation on gfx950
// MFMA (v_mfma_f32_32x32x16_bf16).  Both products are "NT" GEMMs (every
// operand is read along its contiguous K dimension):
//
//   Gram   : E = I - X^T X = I - Xt Xt^T   (Xt = X^T, Np x Mp, K = Mp).
//            Only tiles with ti <= tj are launched; an off-diagonal tile
//            also writes its mirror, so E is stored whole.
//   Update : X <- X + beta X E            (A = bf16 copy of X, Mp x Np;
//            B = E, symmetric, so its rows are its columns; K = Np).
//            The epilogue updates the fp32 iterate in place (each tile
//            reads and writes only its own elements) and emits the next
//            bf16 copy (ping-pong: other tiles still read this one) and
//            the transposed bf16 copy for the next Gram.
//
// One workgroup of 4 waves (2 x 2) computes a BM x BN tile; each wave holds
// a (BM/2) x (BN/2) block of 32x32 accumulators.  K advances in steps of
// 64 through a 2-stage LDS ring (rows padded by 16 bytes, which spreads the
// 16-byte fragment reads of 16 consecutive rows over all banks); the next
// step's global loads are in flight while the MFMAs of the current step run.
// Work items (matrix, tile row, tile column) come from a table that the
// host orders so that consecutive tiles of one matrix land on one XCD.
#include "internal.h"

namespace orth {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace {

__device__ inline int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

__device__ inline uint2 pack4_bf16(float a, float b, float c, float d) {
  uint2 p;
  p.x = (uint32_t)f32_to_bf16(a) | ((uint32_t)f32_to_bf16(b) << 16);
  p.y = (uint32_t)f32_to_bf16(c) | ((uint32_t)f32_to_bf16(d) << 16);
  return p;
}

template <int BM, int BN, int MODE>
__global__ __launch_bounds__(256, 1) void bjorck_bf16_kernel(const TiledMat* __restrict__ mats,
                                                             const TileItem* __restrict__ items, int parity,
                                                             float beta) {
  constexpr int BK = 64;
  constexpr int PITCH = BK + 8;  // bf16 elements per LDS row (144 bytes)
  constexpr int WTM = BM / 2, WTN = BN / 2;
  constexpr int MI = WTM / 32, NI = WTN / 32;
  constexpr int ACH = BM * BK / 8 / 256;  // 16-byte chunks per thread
  constexpr int BCH = BN * BK / 8 / 256;
  __shared__ __attribute__((aligned(16))) uint16_t As[2][BM * PITCH];
  __shared__ __attribute__((aligned(16))) uint16_t Bs[2][BN * PITCH];

  const TileItem it = items[blockIdx.x];
  const TiledMat* d = mats + it.mat;
  const int Mp = d->Mp, Np = d->Np;
  const uint16_t* A;
  const uint16_t* B;
  int64_t lda, ldb;
  int K;
  if (MODE == 0) {
    const uint16_t* xt = static_cast<const uint16_t*>(d->xt);
    A = xt + (int64_t)it.ti * BM * Mp;
    B = xt + (int64_t)it.tj * BN * Mp;
    lda = ldb = Mp;
    K = Mp;
  } else {
    A = static_cast<const uint16_t*>(d->xc[parity]) + (int64_t)it.ti * BM * Np;
    B = static_cast<const uint16_t*>(d->e) + (int64_t)it.tj * BN * Np;
    lda = ldb = Np;
    K = Np;
  }

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  uint4 ra[ACH], rb[BCH];
  auto gload = [&](int k0) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + 256 * i;
      ra[i] = *reinterpret_cast<const uint4*>(A + (int64_t)(c >> 3) * lda + k0 + (c & 7) * 8);
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int c = tid + 256 * i;
      rb[i] = *reinterpret_cast<const uint4*>(B + (int64_t)(c >> 3) * ldb + k0 + (c & 7) * 8);
    }
  };
  auto sstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      const int c = tid + 256 * i;
      *reinterpret_cast<uint4*>(&As[buf][(c >> 3) * PITCH + (c & 7) * 8]) = ra[i];
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      const int c = tid + 256 * i;
      *reinterpret_cast<uint4*>(&Bs[buf][(c >> 3) * PITCH + (c & 7) * 8]) = rb[i];
    }
  };

  f32x16 acc[MI][NI];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = f32x16{};

  const int nk = K / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  const int arow = (wm * WTM + (lane & 31)) * PITCH + (lane >> 5) * 8;
  const int brow = (wn * WTN + (lane & 31)) * PITCH + (lane >> 5) * 8;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      bf16x8 a[MI], b[NI];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
        a[mi] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(&As[buf][arow + mi * 32 * PITCH + kk * 16]));
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
        b[ni] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(&Bs[buf][brow + ni * 32 * PITCH + kk * 16]));
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mi], b[ni], acc[mi][ni], 0, 0, 0);
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // ------------------------------------------------------------ epilogue --
  const int col = lane & 31;
  if (MODE == 0) {
    uint16_t* E = static_cast<uint16_t*>(d->e);
    const bool mirror = it.ti != it.tj;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) {
        const int j = it.tj * BN + wn * WTN + ni * 32 + col;
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int i0 = it.ti * BM + wm * WTM + mi * 32 + acc_row(rg * 4, lane);
          float v[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            v[q] = (i0 + q == j ? 1.f : 0.f) - acc[mi][ni][rg * 4 + q];
            E[(int64_t)(i0 + q) * Np + j] = f32_to_bf16(v[q]);
          }
          if (mirror) *reinterpret_cast<uint2*>(E + (int64_t)j * Np + i0) = pack4_bf16(v[0], v[1], v[2], v[3]);
        }
      }
  } else {
    float* Xm = d->master[0];
    uint16_t* Xo = static_cast<uint16_t*>(d->xc[parity ^ 1]);
    uint16_t* Xt = static_cast<uint16_t*>(d->xt);
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) {
        const int j = it.tj * BN + wn * WTN + ni * 32 + col;
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int i0 = it.ti * BM + wm * WTM + mi * 32 + acc_row(rg * 4, lane);
          float v[4];
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            const int64_t off = (int64_t)(i0 + q) * Np + j;
            v[q] = Xm[off] + beta * acc[mi][ni][rg * 4 + q];
            Xm[off] = v[q];
            Xo[off] = f32_to_bf16(v[q]);
          }
          *reinterpret_cast<uint2*>(Xt + (int64_t)j * Mp + i0) = pack4_bf16(v[0], v[1], v[2], v[3]);
        }
      }
  }
}

}  // namespace

hipError_t launch_bf16_gram(int big, const TiledMat* mats, const TileItem* items, int n_items, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  const char* name = big ? "bjorck_gram_bf16_256" : "bjorck_gram_bf16_128";
  timing_begin(name, s);
  if (big)
    hipLaunchKernelGGL((bjorck_bf16_kernel<256, 256, 0>), dim3(n_items), dim3(256), 0, s, mats, items, 0, 0.f);
  else
    hipLaunchKernelGGL((bjorck_bf16_kernel<128, 128, 0>), dim3(n_items), dim3(256), 0, s, mats, items, 0, 0.f);
  hipError_t e = hipGetLastError();
  timing_end(name, s);
  return e;
}

hipError_t launch_bf16_update(int big, const TiledMat* mats, const TileItem* items, int n_items, int parity,
                              float beta, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  const char* name = big ? "bjorck_update_bf16_256" : "bjorck_update_bf16_128";
  timing_begin(name, s);
  if (big)
    hipLaunchKernelGGL((bjorck_bf16_kernel<256, 256, 1>), dim3(n_items), dim3(256), 0, s, mats, items, parity,
                       beta);
  else
    hipLaunchKernelGGL((bjorck_bf16_kernel<128, 128, 1>), dim3(n_items), dim3(256), 0, s, mats, items, parity,
                       beta);
  hipError_t e = hipGetLastError();
  timing_end(name, s);
  return e;
}

}  // namespace orth
