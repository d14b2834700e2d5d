// Tiled Björck products for bf16 operands with fp32 accumulation on gfx950
// MFMA (v_mfma_f32_32x32x16_bf16).  Both products are "NT" GEMMs (every
// operand is read along its contiguous K dimension):
//
// A launch may mix Gram tiles of some matrices with update tiles of others
// (the host pipelines two groups of matrices this way); every work item
// names its matrix, tile and mode.
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
// a (BM/2) x (BN/2) block of 32x32 accumulators.  K advances in steps of 64
// through a 2-stage LDS ring filled by direct global->LDS loads; 16-byte
// chunks are XOR-swizzled so fragment reads are bank-conflict free.  The
// scheduling fences below keep LDS reads and loads interleaved with MFMAs.
// Work items come from a table that the host orders so that consecutive
// tiles of one matrix land on one XCD.
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

// Scheduling fence for one sub-step: NDMA direct-to-LDS loads first (their
// M0 writes would otherwise force waits on the LDS reads in flight), then
// NMFMA MFMAs with one LDS fragment read after each of the first NREADS.
template <int NMFMA, int NREADS, int NDMA>
__device__ __forceinline__ void fence_substep() {
  if constexpr (NDMA > 0) __builtin_amdgcn_sched_group_barrier(0x010, NDMA, 0);
#pragma unroll
  for (int q = 0; q < NMFMA; ++q) {
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if (q < NREADS) __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
  }
  __builtin_amdgcn_sched_barrier(0);
}
__device__ __forceinline__ void lds_settle() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

template <int BM, int BN, int WM, int WN>
__global__ __launch_bounds__(64 * WM * WN, 1) void bjorck_bf16_kernel(const TiledMat* __restrict__ mats,
                                                                      const TileItem* __restrict__ items,
                                                                      float beta) {
  constexpr int BK = 64;                  // bf16 elements per LDS row (128 bytes)
  constexpr int NW = WM * WN;
  constexpr int TM = BM / WM, TN = BN / WN;
  constexpr int MI = TM / 32, NI = TN / 32;
  constexpr int ABLK = BM / (8 * NW);     // 1 KB direct-to-LDS blocks per wave and k-step
  constexpr int BBLK = BN / (8 * NW);
  static_assert(MI * NI >= MI + NI, "a sub-step needs at least as many MFMAs as fragment reads");
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
  const int MODE = it.flags & TILE_UPDATE ? 1 : 0;   // uniform per workgroup
  const int parity = it.flags & TILE_PARITY ? 1 : 0;
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
  // half h of the loads of k-step k0 (0: the A rows, 1: the B rows)
  auto issue_half = [&](uint16_t* la, uint16_t* lb, int k0, int h) {
    if (h == 0) {
      const char* ab = reinterpret_cast<const char*>(A) + (int64_t)k0 * 2;
#pragma unroll
      for (int i = 0; i < ABLK; ++i) dma16(ab + aoff[i], la + (i * NW + wave) * 512);
    } else {
      const char* bb = reinterpret_cast<const char*>(B) + (int64_t)k0 * 2;
#pragma unroll
      for (int i = 0; i < BBLK; ++i) dma16(bb + boff[i], lb + (i * NW + wave) * 512);
    }
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

  // two register sets of fragments: sub-step kk uses set kk & 1
  bf16x8 fa[2][MI], fb[2][NI];
  auto rd = [&](int set, const uint16_t* pa, const uint16_t* pb, int kk) {
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
      fa[set][mi] = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const uint4*>(pa + arow[mi] + (((2 * kk) ^ axor[mi]) << 3)));
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
      fb[set][ni] = __builtin_bit_cast(
          bf16x8, *reinterpret_cast<const uint4*>(pb + brow[ni] + (((2 * kk) ^ bxor[ni]) << 3)));
  };
  auto mma = [&](int set) {
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
        acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[set][mi], fb[set][ni], acc[mi][ni], 0, 0, 0);
  };

  // One k-step over stage (ca, cb) while stage (na, nb) is filled with the
  // next k-step.  Sub-steps 0-2 each run their MFMAs with the next
  // sub-step's fragment reads interleaved (the first two also issue half of
  // the next stage's loads); then every wave waits for its loads and meets
  // the others at the barrier, after which sub-step 3 (fragments already in
  // registers) keeps the MFMA pipe busy while the first fragments of the
  // next stage are read.  The last k-step re-loads a valid k-step into the
  // idle stage instead of branching, which keeps the loop body one block.
  constexpr int NR = MI + NI, NM = MI * NI;
  const int nk = K / BK;  // even: K is a multiple of 128
  auto kstep = [&](uint16_t* ca, uint16_t* cb, uint16_t* na, uint16_t* nb, int kt) {
    const int kn = (kt + 1 < nk ? kt + 1 : nk - 1) * BK;
    lds_settle();
    rd(1, ca, cb, 1);
    issue_half(na, nb, kn, 0);
    mma(0);
    fence_substep<NM, NR, ABLK>();
    lds_settle();
    rd(0, ca, cb, 2);
    issue_half(na, nb, kn, 1);
    mma(1);
    fence_substep<NM, NR, BBLK>();
    lds_settle();
    rd(1, ca, cb, 3);
    mma(0);
    fence_substep<NM, NR, 0>();
    asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
    __syncthreads();
    __builtin_amdgcn_sched_barrier(0);
    rd(0, na, nb, 0);
    mma(1);
    fence_substep<NM, NR, 0>();
  };
  issue_half(sA0, sB0, 0, 0);
  issue_half(sA0, sB0, 0, 1);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  rd(0, sA0, sB0, 0);
  __builtin_amdgcn_sched_barrier(0);
  for (int kt = 0; kt < nk; kt += 2) {
    kstep(sA0, sB0, sA1, sB1, kt);
    kstep(sA1, sB1, sA0, sB0, kt + 1);
  }

  // ------------------------------------------------------------ epilogue --
  // Each wave stages its accumulators 32 rows at a time through a private
  // fp32 LDS buffer (32 x TN, 16-byte chunks XOR-swizzled so that the two
  // half-waves, which hold rows 4 apart, hit disjoint banks).  From there
  // the row-major outputs are handled as 16-byte vectors along rows and the
  // transposed output as 8-element runs down columns, so every global
  // access is a coalesced 8- or 16-byte vector access.
  float* buf;
  if (BM == 256)
    buf = reinterpret_cast<float*>((wave < 2 ? sA0 : sB0) + (wave & 1) * (32 * TN * 2));
  else
    buf = reinterpret_cast<float*>(wave == 0 ? sA0 : wave == 1 ? sB0 : wave == 2 ? sA1 : sB1);
  auto bidx = [&](int r, int c) {  // float index of element (r, c) of the staging buffer
    return r * TN + ((((c >> 2) ^ (((r >> 2) & 1) << 3))) << 2) + (c & 3);
  };
  const int col = lane & 31, half = lane >> 5;
  const int gi0 = it.ti * BM + wm * TM;  // first global row of this wave
  const int gj0 = it.tj * BN + wn * TN;  // first global column
  const bool mirror = MODE == 0 && it.ti != it.tj;
  uint16_t* E = static_cast<uint16_t*>(d->e);
  float* Xm = d->master[0];
  uint16_t* Xo = static_cast<uint16_t*>(d->xc[parity ^ 1]);
  uint16_t* Xt = static_cast<uint16_t*>(d->xt);
  __syncthreads();
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
    // (1) accumulators -> LDS, row-major
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) buf[bidx(acc_row(r, lane), ni * 32 + col)] = acc[mi][ni][r];
    // (2) row-major pass: 4 consecutive columns per lane
    const int gi = gi0 + mi * 32;
#pragma unroll 4
    for (int q = 0; q < 32 * TN / 256; ++q) {
      const int e4 = q * 64 + lane;            // index of a 4-column group
      const int r = e4 / (TN / 4), c = (e4 % (TN / 4)) * 4;
      float4 v = *reinterpret_cast<const float4*>(&buf[bidx(r, c)]);
      const int64_t off = (int64_t)(gi + r) * Np + gj0 + c;
      if (MODE == 0) {
        const int dg = (gi + r) - (gj0 + c);   // diagonal hits column c + dg
        v.x = (dg == 0 ? 1.f : 0.f) - v.x;
        v.y = (dg == 1 ? 1.f : 0.f) - v.y;
        v.z = (dg == 2 ? 1.f : 0.f) - v.z;
        v.w = (dg == 3 ? 1.f : 0.f) - v.w;
        *reinterpret_cast<uint2*>(E + off) = pack4_bf16(v.x, v.y, v.z, v.w);
      } else {
        const float4 m = *reinterpret_cast<const float4*>(Xm + off);
        v.x = m.x + beta * v.x;
        v.y = m.y + beta * v.y;
        v.z = m.z + beta * v.z;
        v.w = m.w + beta * v.w;
        *reinterpret_cast<float4*>(Xm + off) = v;
        *reinterpret_cast<uint2*>(Xo + off) = pack4_bf16(v.x, v.y, v.z, v.w);
      }
      if (MODE == 1 || mirror) *reinterpret_cast<float4*>(&buf[bidx(r, c)]) = v;
    }
    // (3) transposed pass: 8 consecutive rows of one column per lane
    if (MODE == 1 || mirror) {
      uint16_t* T = MODE == 0 ? E : Xt;
      const int64_t ldt = MODE == 0 ? Np : Mp;
#pragma unroll 2
      for (int q = 0; q < TN * 4 / 64; ++q) {
        const int c = (q * 64 + lane) % TN;  // lanes 0..15 share a row group
        const int g = (q * 64 + lane) / TN;  // 8-row group 0..3
        float v[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) v[j] = buf[bidx(g * 8 + j, c)];
        uint4 p;
        const uint2 lo = pack4_bf16(v[0], v[1], v[2], v[3]);
        const uint2 hi = pack4_bf16(v[4], v[5], v[6], v[7]);
        p.x = lo.x; p.y = lo.y; p.z = hi.x; p.w = hi.y;
        *reinterpret_cast<uint4*>(T + (int64_t)(gj0 + c) * ldt + gi + g * 8) = p;
      }
    }
  }
  (void)half;
}

}  // namespace

// One launch over a table of Gram and/or update tiles (each item carries its
// own mode and ping-pong parity).
hipError_t launch_bf16_tiles(int big, const TiledMat* mats, const TileItem* items, int n_items, float beta,
                             hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  const char* name = big ? "bjorck_bf16_256" : "bjorck_bf16_128";
  timing_begin(name, s);
  if (big)
    hipLaunchKernelGGL((bjorck_bf16_kernel<256, 256, 2, 2>), dim3(n_items), dim3(256), 0, s, mats, items, beta);
  else
    hipLaunchKernelGGL((bjorck_bf16_kernel<128, 128, 2, 2>), dim3(n_items), dim3(256), 0, s, mats, items, beta);
  hipError_t e = hipGetLastError();
  timing_end(name, s);
  return e;
}

}  // namespace orth
