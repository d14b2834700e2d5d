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

// 16-byte chunk swizzle of a 128-byte LDS row: chunk c of row r lives at
// position c ^ swz(r).  Eight consecutive rows get eight distinct positions,
// and so do the even (odd) rows among sixteen consecutive ones, so the
// fragment reads below (one row per lane, same chunk) are bank-conflict
// free whether the LDS serves 8 or 16 lanes of a 16-byte read per cycle.
__device__ __forceinline__ int swz(int r) { return (r ^ (r >> 3)) & 7; }

// 16-byte direct global -> LDS load of every lane (gfx950
// global_load_lds_dwordx4): lane l's bytes land at lds + 16 l.  Kept in a
// plain device function: used directly in a kernel template, the builtin
// stops the host pass from emitting the kernel's launch stub.
__device__ __forceinline__ void dma16(const void* g, void* lds) { __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0); }

template <int BM, int BN, int WM, int WN, int MODE>
__global__ __launch_bounds__(64 * WM * WN, 1) void bjorck_bf16_kernel(const TiledMat* __restrict__ mats,
                                                                      const TileItem* __restrict__ items,
                                                                      int parity, float beta) {
  constexpr int BK = 64;                  // bf16 elements per LDS row (128 bytes)
  constexpr int NW = WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int MI = TM / 32, NI = TN / 32;
  constexpr int ABLK = BM / (8 * NW);     // 1 KB direct-to-LDS blocks per wave and k-step
  constexpr int BBLK = BN / (8 * NW);
  // Two LDS stages held in distinct arrays and selected at compile time, so
  // that the compiler can tell the reads of one stage from the asynchronous
  // direct-to-LDS writes into the other.
  __shared__ __attribute__((aligned(1024))) uint16_t sA0[BM * BK];
  __shared__ __attribute__((aligned(1024))) uint16_t sB0[BN * BK];
  __shared__ __attribute__((aligned(1024))) uint16_t sA1[BM * BK];
  __shared__ __attribute__((aligned(1024))) uint16_t sB1[BN * BK];

  const TileItem it = items[blockIdx.x];
  const TiledMat* d = mats + it.mat;
  const int Mp = d->Mp, Np = d->Np;
  const uint16_t* A;
  const uint16_t* B;
  int lda;
  int K;
  if (MODE == 0) {
    const uint16_t* xt = static_cast<const uint16_t*>(d->xt);
    A = xt + (int64_t)it.ti * BM * Mp;
    B = xt + (int64_t)it.tj * BN * Mp;
    lda = Mp;
    K = Mp;
  } else {
    A = static_cast<const uint16_t*>(d->xc[parity]) + (int64_t)it.ti * BM * Np;
    B = static_cast<const uint16_t*>(d->e) + (int64_t)it.tj * BN * Np;
    lda = Np;
    K = Np;
  }

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WN, wn = wave % WN;

  // Direct-to-LDS operand loads: one instruction moves 64 lanes x 16 bytes
  // = 8 rows of a tile into a contiguous 1 KB LDS block; lane l fills row
  // l / 8 of the block at chunk position l % 8, so it fetches the global
  // chunk that the swizzle maps there.  Byte offsets stay below 2^29.
  uint32_t aoff[ABLK], boff[BBLK];
#pragma unroll
  for (int i = 0; i < ABLK; ++i) {
    const int r = (i * NW + wave) * 8 + (lane >> 3);
    aoff[i] = ((uint32_t)r * lda + ((lane & 7) ^ swz(r)) * 8) * 2;
  }
#pragma unroll
  for (int i = 0; i < BBLK; ++i) {
    const int r = (i * NW + wave) * 8 + (lane >> 3);
    boff[i] = ((uint32_t)r * lda + ((lane & 7) ^ swz(r)) * 8) * 2;
  }
  auto issue = [&](uint16_t* la, uint16_t* lb, int k0) {
    const char* ab = reinterpret_cast<const char*>(A) + (int64_t)k0 * 2;
    const char* bb = reinterpret_cast<const char*>(B) + (int64_t)k0 * 2;
#pragma unroll
    for (int i = 0; i < ABLK; ++i)
      dma16(ab + aoff[i], la + (i * NW + wave) * 512);
#pragma unroll
    for (int i = 0; i < BBLK; ++i)
      dma16(bb + boff[i], lb + (i * NW + wave) * 512);
  };

  // fragment addressing: row R of the wave tile, chunk (2 kk + lane / 32)
  int arow[MI], axor[MI], brow[NI], bxor[NI];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
    const int R = wm * TM + mi * 32 + (lane & 31);
    arow[mi] = R * BK;
    axor[mi] = swz(R) ^ (lane >> 5);
  }
#pragma unroll
  for (int ni = 0; ni < NI; ++ni) {
    const int R = wn * TN + ni * 32 + (lane & 31);
    brow[ni] = R * BK;
    bxor[ni] = swz(R) ^ (lane >> 5);
  }

  f32x16 acc[MI][NI];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = f32x16{};

  // MFMAs over one LDS stage.  Each 16-deep sub-step is fenced into its own
  // scheduling region holding the LDS reads of the next sub-step's
  // fragments and the current sub-step's independent MFMAs, so the reads
  // are always in flight behind a full set of MFMAs.
  auto compute = [&](const uint16_t* pa, const uint16_t* pb) {
    bf16x8 a[2][MI], b[2][NI];
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
      a[0][mi] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(pa + arow[mi] + (axor[mi] << 3)));
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
      b[0][ni] = __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(pb + brow[ni] + (bxor[ni] << 3)));
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kk = 0; kk < BK / 16; ++kk) {
      const int cur = kk & 1;
      if (kk + 1 < BK / 16) {
#pragma unroll
        for (int mi = 0; mi < MI; ++mi)
          a[cur ^ 1][mi] = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const uint4*>(pa + arow[mi] + (((2 * (kk + 1)) ^ axor[mi]) << 3)));
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
          b[cur ^ 1][ni] = __builtin_bit_cast(
              bf16x8, *reinterpret_cast<const uint4*>(pb + brow[ni] + (((2 * (kk + 1)) ^ bxor[ni]) << 3)));
      }
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[cur][mi], b[cur][ni], acc[mi][ni], 0, 0, 0);
      if (kk + 1 < BK / 16) __builtin_amdgcn_sched_group_barrier(0x100, MI + NI, 0);  // LDS reads first
      __builtin_amdgcn_sched_group_barrier(0x008, MI * NI, 0);                       // then the MFMAs
      __builtin_amdgcn_sched_barrier(0);
    }
  };

  const int nk = K / BK;  // even: K is a multiple of 128
  issue(sA0, sB0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  for (int kt = 0; kt < nk; kt += 2) {
    issue(sA1, sB1, (kt + 1) * BK);
    compute(sA0, sB0);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    __syncthreads();
    if (kt + 2 < nk) issue(sA0, sB0, (kt + 2) * BK);
    compute(sA1, sB1);
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
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
        const int j = it.tj * BN + wn * TN + ni * 32 + col;
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int i0 = it.ti * BM + wm * TM + mi * 32 + acc_row(rg * 4, lane);
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
        const int j = it.tj * BN + wn * TN + ni * 32 + col;
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
          const int i0 = it.ti * BM + wm * TM + mi * 32 + acc_row(rg * 4, lane);
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
    hipLaunchKernelGGL((bjorck_bf16_kernel<256, 256, 2, 2, 0>), dim3(n_items), dim3(256), 0, s, mats, items, 0, 0.f);
  else
    hipLaunchKernelGGL((bjorck_bf16_kernel<128, 128, 2, 2, 0>), dim3(n_items), dim3(256), 0, s, mats, items, 0, 0.f);
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
    hipLaunchKernelGGL((bjorck_bf16_kernel<256, 256, 2, 2, 1>), dim3(n_items), dim3(256), 0, s, mats, items, parity,
                       beta);
  else
    hipLaunchKernelGGL((bjorck_bf16_kernel<128, 128, 2, 2, 1>), dim3(n_items), dim3(256), 0, s, mats, items, parity,
                       beta);
  hipError_t e = hipGetLastError();
  timing_end(name, s);
  return e;
}

}  // namespace orth
