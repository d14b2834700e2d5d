// Table-driven fp32 "NT" GEMM on gfx950 fp32 MFMA (v_mfma_f32_32x32x2f32):
// every work item is one product C = A B^T (+ A2 B2^T and any further pairs
// from a table, accumulated into the same tile) with its own operands,
// shapes and epilogue, and every block one 64 x 64 tile of such an item
// (from a tile list), so a single launch covers a whole ragged batch
// (all matrices of a Björck step, all tap products of a composition step,
// all Gram checks).  Operands may be fp32 or bf16 and stored either
// K-contiguous ([M][K]) or transposed ([K][M]); loads are bounds-checked
// with zero fill, with a vectorized fast path for aligned in-bounds fp32
// K-contiguous tiles.  A launch's step argument moves each operand by its
// item's per-step offset, so one table serves every step of a recurrence
// whose buffers are laid out step after step.
//
// Four waves (2 x 2) each own one 32x32 accumulator.  The K loop steps by
// 32 through a 2-stage LDS ring; the next step's loads are in flight while
// the current step's MFMAs run.  The fp32 MFMA consumes one k per lane half
// per instruction; a 16-byte LDS read gives each lane four consecutive k, so
// instruction s of a group uses k = g*8 + 4*(lane/32) + s for both operands.
#include "internal.h"

namespace orth {

typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace {

__device__ inline int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

// KM: every tile of the launch is of a single-pair product whose operands
// are both stored k-major ([K][M] and [K][N]); each thread then loads eight
// consecutive rows of one k (16-byte vectors along the stored rows) and
// writes them to the [row][k] LDS tile one element at a time.  A separate
// instantiation, so that the general loads keep their registers.
template <bool KM>
__global__ __launch_bounds__(256) void gemm_f32_kernel(const GemmItem* __restrict__ items,
                                                       const GemmTile* __restrict__ tiles, int step,
                                                       const GemmPair* __restrict__ extra) {
  constexpr int BM = 64, BN = 64, BK = 32, PITCH = BK + 4;
  __shared__ __attribute__((aligned(16))) float As[2][BM * PITCH];
  __shared__ __attribute__((aligned(16))) float Bs[2][BN * PITCH];
  const GemmTile tl = tiles[blockIdx.x];
  const GemmItem* g = items + tl.item;
  const int M = g->M, N = g->N;
  const int row0 = tl.ti * BM, col0 = tl.tj * BN;
  const bool mirror = g->mirror != 0 && tl.ti != tl.tj;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int64_t st = step;

  f32x16 acc = {};
  const int aoff = (wm * 32 + (lane & 31)) * PITCH + (lane >> 5) * 4;
  const int boff = (wn * 32 + (lane & 31)) * PITCH + (lane >> 5) * 4;
  const int npairs = 2 + g->pair_count;
  for (int pair = 0; pair < npairs; ++pair) {
    // pairs 0 and 1 live in the item (with per-step offsets), the others in
    // the launch's pair table; all are stored like the first
    const GemmPair* xp = pair >= 2 ? extra + g->pair_base + (pair - 2) : nullptr;
    const int K = xp ? xp->K : (pair ? g->K2 : g->K);
    if (K <= 0) continue;
    const int adt = g->a_dtype, bdt = g->b_dtype;
    const int atr = xp ? xp->a_trans : (pair ? g->a2_trans : g->a_trans);
    const int btr = xp ? xp->b_trans : (pair ? g->b2_trans : g->b_trans);
    const int64_t lda = xp ? xp->lda : (pair ? g->lda2 : g->lda), ldb = xp ? xp->ldb : (pair ? g->ldb2 : g->ldb);
    const int esz_a = adt == ORTH_BF16 ? 2 : 4, esz_b = bdt == ORTH_BF16 ? 2 : 4;
    const void* A = xp ? xp->A
                       : static_cast<const char*>(pair ? g->A2 : g->A) + (pair ? g->a2_step : g->a_step) * st * esz_a;
    const void* B = xp ? xp->B
                       : static_cast<const char*>(pair ? g->B2 : g->B) + (pair ? g->b2_step : g->b_step) * st * esz_b;

    // thread -> (row, first k of 8) for each operand; KM: (first row of 8, k)
    const int ar = KM ? (tid & 7) * 8 : atr ? (tid & 63) : (tid >> 2);
    const int ak = KM ? (tid >> 3) : atr ? (tid >> 6) * 8 : (tid & 3) * 8;
    const int br = KM ? (tid & 7) * 8 : btr ? (tid & 63) : (tid >> 2);
    const int bk = KM ? (tid >> 3) : btr ? (tid >> 6) * 8 : (tid & 3) * 8;

    // Raw operand words: fp32 bits, bf16 bits in the low half (widened at
    // the LDS store), or (packed) eight bf16 values in words 0-3 from one
    // 16-byte load.  Widening only at the store keeps each guarded load
    // from waiting for its data.
    uint32_t ra[8], rb[8];
    bool apk = false, bpk = false;
    auto load_op = [&](const void* P, int64_t ld, int dt, int tr, int r, int kq, int rows_lim, int rbase, int k0,
                       uint32_t* dst, bool& packed) {
      const int gr = rbase + r;
      const int gk = k0 + kq;
      packed = false;
      if (!tr && gr < rows_lim && gk + 8 <= K) {
        if (dt == ORTH_F32) {
          const float* p = static_cast<const float*>(P) + (int64_t)gr * ld + gk;
          if ((reinterpret_cast<uintptr_t>(p) & 15) == 0) {
            const uint4 x = gld_u32x4(p);
            const uint4 y = gld_u32x4(p + 4);
            dst[0] = x.x; dst[1] = x.y; dst[2] = x.z; dst[3] = x.w;
            dst[4] = y.x; dst[5] = y.y; dst[6] = y.z; dst[7] = y.w;
            return;
          }
        } else {
          const uint16_t* p = static_cast<const uint16_t*>(P) + (int64_t)gr * ld + gk;
          if ((reinterpret_cast<uintptr_t>(p) & 15) == 0) {
            const uint4 x = gld_u32x4(p);
            dst[0] = x.x; dst[1] = x.y; dst[2] = x.z; dst[3] = x.w;
            packed = true;
            return;
          }
        }
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        uint32_t v = 0;
        if (gr < rows_lim && gk + q < K) {
          const int64_t idx = tr ? (int64_t)(gk + q) * ld + gr : (int64_t)gr * ld + gk + q;
          v = dt == ORTH_BF16 ? (uint32_t)gld_u16(P, idx) : gld_u32(P, idx);
        }
        dst[q] = v;
      }
    };
    // KM: rows r .. r + 7 of stored row k (eight consecutive elements)
    auto load_km = [&](const void* P, int64_t ld, int dt, int r, int kq, int rows_lim, int rbase, int k0,
                       uint32_t* dst, bool& packed) {
      const int gr = rbase + r;
      const int gk = k0 + kq;
      packed = false;
      if (gk < K && gr + 8 <= rows_lim) {
        if (dt == ORTH_F32) {
          const float* p = static_cast<const float*>(P) + (int64_t)gk * ld + gr;
          if ((reinterpret_cast<uintptr_t>(p) & 15) == 0) {
            const uint4 x = gld_u32x4(p);
            const uint4 y = gld_u32x4(p + 4);
            dst[0] = x.x; dst[1] = x.y; dst[2] = x.z; dst[3] = x.w;
            dst[4] = y.x; dst[5] = y.y; dst[6] = y.z; dst[7] = y.w;
            return;
          }
        } else {
          const uint16_t* p = static_cast<const uint16_t*>(P) + (int64_t)gk * ld + gr;
          if ((reinterpret_cast<uintptr_t>(p) & 15) == 0) {
            const uint4 x = gld_u32x4(p);
            dst[0] = x.x; dst[1] = x.y; dst[2] = x.z; dst[3] = x.w;
            packed = true;
            return;
          }
        }
      }
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        uint32_t v = 0;
        if (gk < K && gr + q < rows_lim) {
          const int64_t idx = (int64_t)gk * ld + gr + q;
          v = dt == ORTH_BF16 ? (uint32_t)gld_u16(P, idx) : gld_u32(P, idx);
        }
        dst[q] = v;
      }
    };
    auto gload = [&](int k0) {
      if constexpr (KM) {
        load_km(A, lda, adt, ar, ak, M, row0, k0, ra, apk);
        load_km(B, ldb, bdt, br, bk, N, col0, k0, rb, bpk);
      } else {
        load_op(A, lda, adt, atr, ar, ak, M, row0, k0, ra, apk);
        load_op(B, ldb, bdt, btr, br, bk, N, col0, k0, rb, bpk);
      }
    };
    auto widen = [&](const uint32_t* w, bool packed, int dt, float* f) {
      if (packed) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          f[2 * q] = __uint_as_float(w[q] << 16);
          f[2 * q + 1] = __uint_as_float(w[q] & 0xffff0000u);
        }
      } else {
        const int sh = dt == ORTH_BF16 ? 16 : 0;
#pragma unroll
        for (int q = 0; q < 8; ++q) f[q] = __uint_as_float(w[q] << sh);
      }
    };
    auto sstore = [&](int buf) {
#pragma unroll
      for (int q = 0; q < 8; ++q) {
        asm volatile("" : "+v"(ra[q]));
        asm volatile("" : "+v"(rb[q]));
      }
      float fa[8], fb[8];
      widen(ra, apk, adt, fa);
      widen(rb, bpk, bdt, fb);
      if constexpr (KM) {
#pragma unroll
        for (int q = 0; q < 8; ++q) {
          As[buf][(ar + q) * PITCH + ak] = fa[q];
          Bs[buf][(br + q) * PITCH + bk] = fb[q];
        }
        return;
      }
      float4* pa = reinterpret_cast<float4*>(&As[buf][ar * PITCH + ak]);
      pa[0] = make_float4(fa[0], fa[1], fa[2], fa[3]);
      pa[1] = make_float4(fa[4], fa[5], fa[6], fa[7]);
      float4* pb = reinterpret_cast<float4*>(&Bs[buf][br * PITCH + bk]);
      pb[0] = make_float4(fb[0], fb[1], fb[2], fb[3]);
      pb[1] = make_float4(fb[4], fb[5], fb[6], fb[7]);
    };

    // stage 0 is free here: every wave passed the last barrier of the
    // previous pair after its final reads
    const int nk = (K + BK - 1) / BK;
    gload(0);
    sstore(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
      const int buf = kt & 1;
      if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
      for (int gq = 0; gq < BK / 8; ++gq) {
        const float4 a4 = *reinterpret_cast<const float4*>(&As[buf][aoff + gq * 8]);
        const float4 b4 = *reinterpret_cast<const float4*>(&Bs[buf][boff + gq * 8]);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.x, b4.x, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.y, b4.y, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.z, b4.z, acc, 0, 0, 0);
        acc = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.w, b4.w, acc, 0, 0, 0);
      }
      if (kt + 1 < nk) sstore(buf ^ 1);
      __syncthreads();
    }
  }

  // ------------------------------------------------------------ epilogue --
  const int epi = g->epi;
  const int j = col0 + wn * 32 + (lane & 31);
  const int ibase = row0 + wm * 32;
  if (epi == EPI_MAXDEV) {
    float m = 0.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = ibase + acc_row(r, lane);
      if (i < M && j < N) {
        const float v = fabsf((i == j ? 1.f : 0.f) - acc[r]);
        m = (v > m || isnan(v)) ? v : m;
      }
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const float o = __shfl_xor(m, off, 64);
      m = (o > m || isnan(o)) ? o : m;
    }
    if (lane == 0) atomicMax(reinterpret_cast<unsigned int*>(g->red), __float_as_uint(m));
    return;
  }
  // update tiles stage their transposed copy through LDS with every lane
  if (j >= N && epi != EPI_UPDATE) return;
  float* C = static_cast<float*>(g->C) + g->c_step * st;
  const int64_t ldc = g->ldc;
  if (epi == EPI_STORE) {
    const int cdt = g->c_dtype;
    void* Cv = static_cast<char*>(g->C) + g->c_step * st * (cdt == ORTH_BF16 ? 2 : 4);
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = ibase + acc_row(r, lane);
      if (i < M) store_from_f32(Cv, (int64_t)i * ldc + j, cdt, acc[r]);
    }
  } else if (epi == EPI_GRAM_E) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = ibase + acc_row(r, lane);
      if (i < M) {
        const float v = (i == j ? 1.f : 0.f) - acc[r];
        gst_f32(C, (int64_t)i * ldc + j, v);
        if (mirror) gst_f32(C, (int64_t)j * ldc + i, v);
      }
    }
  } else if (epi == EPI_SERIES) {
    float* dst2 = g->dst2;
    const int64_t ld2 = g->ld2;
    const float beta = g->beta;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = ibase + acc_row(r, lane);
      if (i < M) {
        const float v = beta * acc[r];
        gst_f32(C, (int64_t)i * ldc + j, v);
        // each element belongs to one item of the launch
        gst_f32(dst2, (int64_t)i * ld2 + j, gld_f32(dst2, (int64_t)i * ld2 + j) + v);
      }
    }
  } else if (epi == EPI_NEG) {
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = ibase + acc_row(r, lane);
      if (i < M) {
        gst_f32(C, (int64_t)i * ldc + j, -acc[r]);
        if (mirror) gst_f32(C, (int64_t)j * ldc + i, -acc[r]);
      }
    }
  } else {  // EPI_UPDATE
    const float* src = g->src + g->src_step * st;
    float* dst2 = g->dst2 ? g->dst2 + g->d2_step * st : nullptr;
    const int64_t lds_ = g->ld_src, ld2 = g->ld2;
    const float beta = g->beta;
    float v[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int i = ibase + acc_row(r, lane);
      v[r] = 0.f;
      if (i < M && j < N) {
        v[r] = gld_f32(src, (int64_t)i * lds_ + j) + beta * acc[r];
        gst_f32(C, (int64_t)i * ldc + j, v[r]);
      }
    }
    if (dst2) {
      // the wave's 32 x 32 block transposed through LDS (its own 32 x 33
      // region of As, free after the last k-step's barrier), so that every
      // row of the copy is written as 16-byte pieces
      float* Tt = &As[0][0] + wave * (32 * 33);
#pragma unroll
      for (int r = 0; r < 16; ++r) Tt[(lane & 31) * 33 + acc_row(r, lane)] = v[r];
      __syncthreads();
      const int jbase = col0 + wn * 32;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int e = q * 64 + lane;
        const int jj = e >> 3, c4 = (e & 7) * 4;
        const int gj = jbase + jj, gi = ibase + c4;
        if (gj >= N) continue;
        const float* t = Tt + jj * 33 + c4;
        float* d = dst2 + (int64_t)gj * ld2 + gi;
        if (gi + 4 <= M && (reinterpret_cast<uintptr_t>(d) & 15) == 0) {
          gst_f32x4(d, make_float4(t[0], t[1], t[2], t[3]));
        } else {
#pragma unroll
          for (int k = 0; k < 4; ++k)
            if (gi + k < M) gst_f32(d, k, t[k]);
        }
      }
    }
  }
}

}  // namespace

hipError_t launch_gemm_f32(const GemmItem* items, const GemmTile* tiles, int n_tiles, const char* name,
                           hipStream_t s, int step, const GemmPair* pairs, int n_km) {
  if (n_tiles <= 0) return hipSuccess;
  if (n_km < 0 || n_km > n_tiles) return hipErrorInvalidValue;
  timing_begin(name, s);
  hipError_t e = hipSuccess;
  if (n_tiles > n_km) {
    hipLaunchKernelGGL(gemm_f32_kernel<false>, dim3(n_tiles - n_km), dim3(256), 0, s, items, tiles, step, pairs);
    e = hipGetLastError();
  }
  if (e == hipSuccess && n_km > 0) {
    hipLaunchKernelGGL(gemm_f32_kernel<true>, dim3(n_km), dim3(256), 0, s, items, tiles + (n_tiles - n_km), step,
                       pairs);
    e = hipGetLastError();
  }
  timing_end(name, s);
  return e;
}

}  // namespace orth
