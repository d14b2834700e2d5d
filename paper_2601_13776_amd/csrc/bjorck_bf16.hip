// Tiled Björck products for bf16 operands with fp32 accumulation on gfx950
// MFMA (v_mfma_f32_32x32x16_bf16).  With X the current iterate (tall,
// Mp x Np, a bf16 copy of the fp32 iterate) and E = I - X^T X:
//
//   Gram   : E tile (I, J) = I - X[:, I]^T X[:, J], for I <= J only (E is
//            symmetric and only its upper tiles are ever read).  Both
//            operands are column panels of row-major X: they are staged in
//            LDS as [k][column] and read with transposing LDS reads.
//   Update : X <- X + beta X E.  A is a row panel of X ([row][k] in LDS,
//            plain 16-byte reads).  B = E[:, J]: for k in or above tile J
//            the stored rows E[J, k] are read directly, below it the stored
//            upper tile E[k-block, J] is read transposed.  The epilogue
//            updates the fp32 iterate in place (each tile reads and writes
//            only its own elements) and emits the next bf16 copy (ping-pong:
//            other tiles still read the current one); the last two k-steps
//            already load the first two 32-row chunks of the iterate in
//            place of the loads that would only re-read a k-step.
//
// Every work item names its matrix, tile, mode (Gram or update) and
// ping-pong parity, so one launch can cover any mix of tiles.
//
// Vector-Jacobian product (second instantiation): with X_t and E_t the saved
// bf16 iterate and E of step t and Y the gradient with respect to X_{t+1},
// the derivative of the update gives
//   dL/dX_t = Y + beta (Y E_t + X_t S'),   S' = -(X_t^T Y + Y^T X_t),
// computed as S' tiles (two transposed-panel products, upper tiles only, no
// identity) and then update-like tiles with two panel-times-symmetric
// products, the fp32 gradient iterate updated in place.
//
// One workgroup of 4 waves (2 x 2) computes a BM x BN tile; each wave holds
// a (BM/2) x (BN/2) block of 32x32 accumulators.  K advances in steps of 64
// through five LDS buffers (160 KB for 256-tiles) filled by direct
// global->LDS loads up to two k-steps ahead; 16-byte chunks are
// XOR-swizzled so fragment reads are bank-conflict free.  The scheduling
// fences keep LDS reads and loads interleaved with MFMAs.  Work items come
// from a table whose order the host chooses so that concurrently running
// tiles share operand panels through the caches.
#include <type_traits>

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

// Swizzle of a [row][k] tile (128-byte rows of 8 16-byte chunks): chunk c
// of row r lives at position c ^ swz(r).  Eight consecutive rows get eight
// distinct positions, and so do the even (odd) rows among sixteen
// consecutive ones, so the 16-byte fragment reads (one row per lane, same
// chunk) are conflict free whether the LDS serves 8 or 16 lanes per cycle.
__device__ __forceinline__ int swz(int r) { return (r ^ (r >> 3)) & 7; }

// Swizzle of a [k][column] tile (rows of 16 or 32 chunks): chunk c of row k
// lives at c ^ swt(k).  A transposing read touches 4 consecutive rows and 2
// (16 lanes) or 4 (32 lanes) consecutive chunks; the values {0, 6, 10, 12}
// differ in bits 1-2 and in bits 2-3, which keeps both cases conflict free.
__device__ __forceinline__ int swt(int k) { return (0xCA60 >> ((k & 3) * 4)) & 15; }

// Global-memory accesses of the epilogues.  The kernel takes its data
// pointers from the descriptor table, and the compiler cannot prove that
// a pointer loaded from memory points to global memory, so plain accesses
// through it become FLAT instructions, which count against the LDS counter
// as well: every wait for an LDS result (the staging buffer's reads) would
// then also wait for the epilogue's stores in flight.
// (The address-space attribute takes effect on vector-extension types,
// not on HIP's float4 / uint2 classes.)
typedef float f32x4v __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));
typedef __attribute__((address_space(1))) f32x4v g_f32x4;
typedef __attribute__((address_space(1))) u32x2v g_u32x2;
__device__ __forceinline__ float4 gload4(const float* p) {
  const f32x4v v = *(const g_f32x4*)(p);
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void gstore4(float* p, float4 v) { *(g_f32x4*)(p) = f32x4v{v.x, v.y, v.z, v.w}; }
__device__ __forceinline__ void gstore2(uint16_t* p, uint2 v) { *(g_u32x2*)(p) = u32x2v{v.x, v.y}; }

// 16-byte direct global -> LDS load of every lane (gfx950
// global_load_lds_dwordx4): lane l's bytes land at lds + 16 l.  Kept in a
// plain device function: used directly in a kernel template, the builtin
// stops the host pass from emitting the kernel's launch stub.
__device__ __forceinline__ void dma16(const void* g, void* lds) { __builtin_amdgcn_global_load_lds(g, lds, 16, 0, 0); }

// Transposing 8-byte LDS read (gfx950 ds_read_b64_tr_b16).  Within each
// group of 16 lanes, if lane j addresses row k0 + j / 4, columns
// c0 + 4 (j % 4) .. + 3 of a [k][column] bf16 tile, lane l receives
// columns c0 + l, rows k0 .. k0 + 3: half of an MFMA A/B fragment.
// The address is cast pointer to pointer (not through an integer) so that
// alias analysis still sees which LDS array it reads: a read of one stage
// then needs no wait for the asynchronous loads into the other.
typedef short s16x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ uint2 lds_read_tr(const uint16_t* p) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(const_cast<uint16_t*>(p)));
  return __builtin_bit_cast(uint2, v);
}

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

// Scheduling plan of one sub-step of NMFMA MFMAs: its NDMA loads go out
// DPS per MFMA over the first slots (each load sets M0, and an M0 write
// waits for every LDS read in flight, so no read is issued before them),
// then its NREADS fragment reads are spread over the following slots, and
// the last TAIL MFMAs issue no read, so that the reads have returned when
// the next sub-step waits for them.
template <int Q, int NMFMA, int NREADS, int NDMA, int DPS, int TAIL>
__device__ __forceinline__ void plan_slots() {
  if constexpr (Q < NMFMA) {
    constexpr int DSLOTS = (NDMA + DPS - 1) / DPS;
    constexpr int RSLOTS = NMFMA - TAIL - DSLOTS;
    static_assert(RSLOTS > 0 || NREADS == 0, "no MFMA slot left for the fragment reads");
    __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
    if constexpr (Q < DSLOTS) {
      constexpr int n = (Q + 1) * DPS <= NDMA ? DPS : NDMA - Q * DPS;
      __builtin_amdgcn_sched_group_barrier(0x010, n, 0);
    } else if constexpr (Q < DSLOTS + RSLOTS) {
      constexpr int slot = Q - DSLOTS;
      constexpr int lo = slot * NREADS / RSLOTS, hi = (slot + 1) * NREADS / RSLOTS;
      if constexpr (hi > lo) __builtin_amdgcn_sched_group_barrier(0x100, hi - lo, 0);
    }
    plan_slots<Q + 1, NMFMA, NREADS, NDMA, DPS, TAIL>();
  }
}
template <int NMFMA, int NREADS, int NDMA, int DPS, int TAIL>
__device__ __forceinline__ void fence_plan() {
  plan_slots<0, NMFMA, NREADS, NDMA, DPS, TAIL>();
  __builtin_amdgcn_sched_barrier(0);
}

// One operand of the tile product, staged in LDS either as [row][k]
// (TRANS = false: the operand's rows are contiguous along k in memory) or
// as [k][row] (TRANS = true: memory holds it k-major, each k a contiguous
// run of ROWS elements).  Each wave moves its share of the 64-deep k-step
// with 1 KB direct-to-LDS loads and reads its fragments.
template <int ROWS, int NW, int NF, bool TRANS>
struct Operand {
  static constexpr int BK = 64;
  static constexpr int NBLK = ROWS * BK * 2 / 1024 / NW;  // 1 KB loads per wave and k-step
  static constexpr int CPR = TRANS ? ROWS / 8 : BK / 8;   // 16-byte chunks per LDS row
  static constexpr int RPB = 64 / CPR;                    // LDS rows per 1 KB block
  const char* base;   // operand origin in global memory (row 0 / k 0)
  int64_t ld;         // elements between consecutive memory rows
  uint32_t off[NBLK]; // per-load byte offsets without the k-step term
  int fr[NF];         // per-fragment element offsets in the tile (k term excluded)

  __device__ __forceinline__ void init(const uint16_t* p, int64_t ld_, int wave, int lane, int wrow0) {
    base = reinterpret_cast<const char*>(p);
    ld = ld_;
#pragma unroll
    for (int i = 0; i < NBLK; ++i) {
      const int row = (i * NW + wave) * RPB + lane / CPR;  // LDS row of this lane's chunk
      const int pos = lane % CPR;
      const int c = TRANS ? pos ^ swt(row) : pos ^ swz(row);
      off[i] = ((uint32_t)row * (uint32_t)ld + c * 8) * 2;
    }
#pragma unroll
    for (int f = 0; f < NF; ++f) {
      if (!TRANS) {
        const int R = wrow0 + f * 32 + (lane & 31);
        fr[f] = R * BK + ((swz(R) ^ (lane >> 5)) << 3);
      } else {
        const int g = lane >> 4, j = lane & 15;
        const int col = wrow0 + f * 32 + (g & 1) * 16 + 4 * (j & 3);
        const int krow = (g >> 1) * 8 + (j >> 2);   // k within a 16-deep sub-step, excluding 4 h
        fr[f] = krow * ROWS + ((((col >> 3) ^ swt(krow)) << 3) | (col & 7));
      }
    }
  }
  // the loads of the k-step starting at k0 into LDS stage `lds`
  __device__ __forceinline__ void issue(uint16_t* lds, int k0, int wave) const {
    const char* b = base + (TRANS ? (int64_t)k0 * ld * 2 : (int64_t)k0 * 2);
#pragma unroll
    for (int i = 0; i < NBLK; ++i) dma16(b + off[i], lds + (i * NW + wave) * 512);
  }
  // the same loads, or (pf: a k-step past the end, whose loads only keep
  // the wait counts) 1 KB pieces q0 + i of an epilogue prefetch: a piece is
  // RPP rows of TN fp32 values starting at row RPP q of chunk base pfb (row
  // stride pfr bytes), 4 values per lane
  template <int TN>
  __device__ __forceinline__ void issue_pf(uint16_t* lds, int k0, int wave, int lane, bool pf, const char* pfb,
                                           int64_t pfr, int q0) const {
    constexpr int RPP = 256 / TN;
    const char* b = base + (TRANS ? (int64_t)k0 * ld * 2 : (int64_t)k0 * 2);
    // both addresses are formed and one is kept by a mask (a uniform
    // condition would otherwise become a branch inside the scheduled k-step)
    const uint64_t keep = pf ? ~0ull : 0ull;
#pragma unroll
    for (int i = 0; i < NBLK; ++i) {
      const uint64_t a = reinterpret_cast<uint64_t>(b + off[i]);
      const uint64_t p = reinterpret_cast<uint64_t>(pfb) +
                         (uint64_t)(((q0 + i) * RPP + lane / (TN / 4)) * pfr + (lane % (TN / 4)) * 16);
      dma16(reinterpret_cast<const char*>((a & ~keep) | (p & keep)), lds + (i * NW + wave) * 512);
    }
  }
  // fragment f of sub-step kk (16 k) from LDS stage `lds`
  __device__ __forceinline__ bf16x8 frag(const uint16_t* lds, int f, int kk) const {
    if (!TRANS) {
      // chunk (2 kk + lane / 32) of the row: the swizzle term was folded in fr
      return __builtin_bit_cast(bf16x8, *reinterpret_cast<const uint4*>(lds + (fr[f] ^ ((2 * kk) << 3))));
    } else {
      const uint2 lo = lds_read_tr(lds + fr[f] + (kk * 16) * ROWS);
      const uint2 hi = lds_read_tr(lds + fr[f] + (kk * 16 + 4) * ROWS);
      return __builtin_bit_cast(bf16x8, make_uint4(lo.x, lo.y, hi.x, hi.y));
    }
  }
};

// Measured on the 256-tiles: one load per MFMA slot and four read-free MFMAs
// at the end of each sub-step (two loads per slot or no tail were slower).
constexpr int DMA_PER_SLOT = 1;
constexpr int READ_TAIL = 4;

template <int BM, int BN, int WM, int WN>
struct Tile {
  static constexpr int BK = 64, NW = WM * WN, TM = BM / WM, TN = BN / WN, MI = TM / 32, NI = TN / 32;
};

// K loop over [kb, ke) (multiples of 64) of one tile, through five LDS
// buffers: the A operand cycles through three, B through two.  In k-step t,
// sub-step 0 sends the A loads of k-step t + 2 into the free A buffer;
// sub-steps 0-2 run their MFMAs with the next sub-step's fragment reads
// interleaved; then every wave waits for the loads of k-step t + 1 (the
// newest A loads may stay in flight) and meets the others at the barrier,
// after which sub-step 3 (fragments already in registers) keeps the MFMA
// pipe busy while the first fragments of k-step t + 1 are read and the B
// loads of k-step t + 2 go into the B buffer just read.  A loads get seven
// sub-steps to land, B loads four (two stages: three and two; measured 4%
// faster).  Past the end, loads re-read a valid k-step instead of
// branching: the barrier's partial wait relies on this k-step's A loads
// being the newest in flight (skipped, they would let the next k-step's B
// loads pass the barrier unfinished).
// Epilogue prefetch of an update tile: in the last two k-steps of its final
// K loop the loads would re-read a valid k-step (see kloop); instead they
// fetch the first two 32-row chunks of this wave's part of the fp32
// iterate, A loads the first pieces and B loads the rest of a chunk.  The
// chunk of k-step kt (kt + 2 - nk = 0 or 1) lands in that k-step's free A
// buffer and its B buffer (blocks (i * 4 + wave), as the operand loads).
struct Prefetch {
  const char* base = nullptr;   // the wave's part of the iterate (wave-uniform)
  int64_t row = 0;              // bytes between iterate rows
};

template <int BM, int BN, int WM, int WN, bool AT, bool BT, bool PF = false>
__device__ __forceinline__ void kloop(f32x16 (&acc)[BM / WM / 32][BN / WN / 32], const uint16_t* A, int64_t lda,
                                      const uint16_t* B, int64_t ldb, int kb, int ke, uint16_t* sA0, uint16_t* sB0,
                                      uint16_t* sA1, uint16_t* sB1, uint16_t* sX, int wave, int lane, int wm,
                                      int wn, Prefetch pf = Prefetch()) {
  using T = Tile<BM, BN, WM, WN>;
  constexpr int MI = T::MI, NI = T::NI, BK = T::BK;
  const int nk = (ke - kb) / BK;
  if (nk <= 0) return;
  Operand<BM, T::NW, MI, AT> oa;
  Operand<BN, T::NW, NI, BT> ob;
  oa.init(A, lda, wave, lane, wm * T::TM);
  ob.init(B, ldb, wave, lane, wn * T::TN);
  bf16x8 fa[2][MI], fb[2][NI];
  auto rd = [&](int set, const uint16_t* pa, const uint16_t* pb, int kk) {
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) fa[set][mi] = oa.frag(pa, mi, kk);
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) fb[set][ni] = ob.frag(pb, ni, kk);
  };
  auto mma = [&](int set) {
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
        acc[mi][ni] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fa[set][mi], fb[set][ni], acc[mi][ni], 0, 0, 0);
  };
  constexpr int NR = (AT ? 2 : 1) * MI + (BT ? 2 : 1) * NI, NM = MI * NI;
  constexpr int NRF = NR < NM ? NR : NM;
  // The loads of a sub-step go out before its fragment reads: every load sets
  // M0, and an M0 write waits for all LDS reads in flight, so reads issued
  // ahead of the loads would stall the wave (with the MFMA pipe draining)
  // until they return.  On 256-tiles the loads ride along the first MFMAs of
  // the sub-step (fence_plan); on 128-tiles, with four MFMAs per sub-step,
  // they go out first behind a scheduling barrier.
  constexpr int NA = decltype(oa)::NBLK, NBL = decltype(ob)::NBLK;
  static_assert(NA == 8 || NA == 4, "wait counts are spelled out for 4 or 8 loads");
  // ca/cb: this k-step's stage; na/nb: the next one's; sa: free buffer that
  // receives A of k-step kt + 2 in sub-step 0; B of kt + 2 goes into cb
  // after the barrier
  auto kstep = [&](uint16_t* ca, uint16_t* cb, uint16_t* na, uint16_t* nb, uint16_t* sa, int kt) {
    const int kn2 = kb + (kt + 2 < nk ? kt + 2 : nk - 1) * BK;
    constexpr bool BIG = NM >= 16;   // 256-tiles: loads and reads spread over the sub-step
    const bool pfk = PF && kt + 2 >= nk;
    const char* pfb = PF ? pf.base + (pfk ? (int64_t)(kt + 2 - nk) * 32 * pf.row : 0) : nullptr;
    lds_settle();
    if constexpr (PF)
      oa.template issue_pf<BN / WN>(sa, kn2, wave, lane, pfk, pfb, pf.row, 0);
    else
      oa.issue(sa, kn2, wave);
    if constexpr (!BIG) __builtin_amdgcn_sched_barrier(0);
    rd(1, ca, cb, 1);
    mma(0);
    if constexpr (BIG)
      fence_plan<NM, NR, NA, DMA_PER_SLOT, READ_TAIL>();
    else
      fence_substep<NM, NRF, 0>();
    lds_settle();
    rd(0, ca, cb, 2);
    mma(1);
    if constexpr (BIG)
      fence_plan<NM, NR, 0, 1, READ_TAIL>();
    else
      fence_substep<NM, NRF, 0>();
    lds_settle();
    rd(1, ca, cb, 3);
    mma(0);
    if constexpr (BIG)
      fence_plan<NM, NR, 0, 1, READ_TAIL>();
    else
      fence_substep<NM, NRF, 0>();
    // every load but this k-step's A loads for k-step kt + 2 has landed and
    // every LDS read is done; a plain s_barrier (a workgroup fence would
    // wait for all loads)
    // (s_waitcnt vmcnt(NA) expcnt(7) lgkmcnt(0) as a builtin, so that the
    // compiler's own wait analysis sees it)
    __builtin_amdgcn_s_waitcnt((NA & 15) | (7 << 4) | ((NA >> 4) << 14));
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    if constexpr (PF)
      ob.template issue_pf<BN / WN>(cb, kn2, wave, lane, pfk, pfb, pf.row, NA);
    else
      ob.issue(cb, kn2, wave);
    if constexpr (!BIG) __builtin_amdgcn_sched_barrier(0);
    rd(0, na, nb, 0);
    mma(1);
    if constexpr (BIG)
      fence_plan<NM, NR, NBL, DMA_PER_SLOT, READ_TAIL>();
    else
      fence_substep<NM, NRF, 0>();
  };
  // A cycles through three buffers (sA0, sA1, sX), B through two (sB0,
  // sB1): the pattern repeats every six k-steps
  oa.issue(sA0, kb, wave);
  ob.issue(sB0, kb, wave);
  oa.issue(sA1, kb + (nk > 1 ? BK : 0), wave);
  ob.issue(sB1, kb + (nk > 1 ? BK : 0), wave);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  rd(0, sA0, sB0, 0);
  __builtin_amdgcn_sched_barrier(0);
  // whole periods in the loop; the remainder in straight-line code, so that
  // the loop head only ever follows the last k-step of a period (the
  // compiler's wait analysis then sees which buffers have loads in flight)
  int kt = 0;
  for (; kt + 6 <= nk; kt += 6) {
    kstep(sA0, sB0, sA1, sB1, sX, kt);
    kstep(sA1, sB1, sX, sB0, sA0, kt + 1);
    kstep(sX, sB0, sA0, sB1, sA1, kt + 2);
    kstep(sA0, sB1, sA1, sB0, sX, kt + 3);
    kstep(sA1, sB0, sX, sB1, sA0, kt + 4);
    kstep(sX, sB1, sA0, sB0, sA1, kt + 5);
  }
  if (kt < nk) {
    kstep(sA0, sB0, sA1, sB1, sX, kt);
    if (kt + 1 < nk) {
      kstep(sA1, sB1, sX, sB0, sA0, kt + 1);
      if (kt + 2 < nk) {
        kstep(sX, sB0, sA0, sB1, sA1, kt + 2);
        if (kt + 3 < nk) {
          kstep(sA0, sB1, sA1, sB0, sX, kt + 3);
          if (kt + 4 < nk) kstep(sA1, sB0, sX, sB1, sA0, kt + 4);
        }
      }
    }
  }
  // every wave is done with both stages before anyone refills them
  asm volatile("s_waitcnt vmcnt(0) lgkmcnt(0)" ::: "memory");
  __syncthreads();
}

template <int BM, int BN, int WM, int WN, bool VJP>
__global__ __launch_bounds__(64 * WM * WN, 1) void bjorck_bf16_kernel(const TiledMat* __restrict__ mats,
                                                                      const TileItem* __restrict__ items,
                                                                      float beta, int step) {
  using T = Tile<BM, BN, WM, WN>;
  constexpr int BK = T::BK, TM = T::TM, TN = T::TN, MI = T::MI, NI = T::NI;
  static_assert(MI * NI >= MI + NI, "a sub-step needs at least as many MFMAs as fragment reads");
  // Five LDS buffers held in distinct arrays and selected at compile time,
  // so that the compiler can tell the reads of one buffer from the
  // asynchronous direct-to-LDS writes into the others.
  __shared__ __attribute__((aligned(1024))) uint16_t sA0[BM * BK];
  __shared__ __attribute__((aligned(1024))) uint16_t sB0[BN * BK];
  __shared__ __attribute__((aligned(1024))) uint16_t sA1[BM * BK];
  __shared__ __attribute__((aligned(1024))) uint16_t sB1[BN * BK];
  __shared__ __attribute__((aligned(1024))) uint16_t sX[BM * BK];

  const TileItem it = items[blockIdx.x];
  const TiledMat* d = mats + it.mat;
  const int Mp = d->Mp, Np = d->Np;
  const int MODE = it.flags & TILE_UPDATE ? 1 : 0;   // uniform per workgroup
  const int parity = it.flags & TILE_PARITY ? 1 : 0;
  // saved-iterate mode: step t reads the t-th saved iterate and E
  const int64_t xoff = (int64_t)step * d->xstep, eoff = (int64_t)step * d->estep;
  const uint16_t* X = static_cast<const uint16_t*>(d->xc[VJP ? 0 : parity]) + xoff;
  const uint16_t* Ep = static_cast<const uint16_t*>(d->e) + eoff;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wm = wave / WN, wn = wave % WN;

  f32x16 acc[MI][NI];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = f32x16{};

  // row panel I of P times the symmetric matrix Q (upper tiles stored) at
  // column panel J: below tile J the stored tiles Q[k-block, J] are read
  // transposed, from tile J on the stored rows Q[J, k] directly
  // (PF: the final K loop prefetches the iterate for the epilogue)
  auto panel_times_sym = [&](const uint16_t* P, const uint16_t* Q, auto pf_tag, Prefetch pf) {
    constexpr bool PF = decltype(pf_tag)::value;
    const int ksplit = it.tj * BN;
    kloop<BM, BN, WM, WN, false, true>(acc, P + (int64_t)it.ti * BM * Np, Np, Q + (int64_t)it.tj * BN, Np, 0,
                                       ksplit, sA0, sB0, sA1, sB1, sX, wave, lane, wm, wn);
    kloop<BM, BN, WM, WN, false, false, PF>(acc, P + (int64_t)it.ti * BM * Np, Np, Q + (int64_t)it.tj * BN * Np,
                                            Np, ksplit, Np, sA0, sB0, sA1, sB1, sX, wave, lane, wm, wn, pf);
  };
  // column panels I of P and J of Q, k over all Mp rows: P[:, I]^T Q[:, J]
  auto cols_t_cols = [&](const uint16_t* P, const uint16_t* Q) {
    kloop<BM, BN, WM, WN, true, true>(acc, P + (int64_t)it.ti * BM, Np, Q + (int64_t)it.tj * BN, Np, 0, Mp, sA0,
                                      sB0, sA1, sB1, sX, wave, lane, wm, wn);
  };

  // forward update tiles: this wave's part of the fp32 iterate, prefetched
  // by the final K loop (a k-step's A loads carry half a chunk, its B loads
  // the other half; the loop has at least two k-steps: BN / BK >= 2)
  static_assert(32 * TN / 256 / 2 == BM * BK * 2 / 1024 / T::NW && BM == BN && BN / BK >= 2,
                "an update tile's k-step loads must cover one 32-row chunk of its iterate");
  Prefetch pf;
  if (!VJP && MODE == 1) {
    pf.base = reinterpret_cast<const char*>(d->master[0] + (int64_t)(it.ti * BM + wm * TM) * Np + it.tj * BN +
                                            wn * TN);
    pf.row = (int64_t)Np * 4;
  }

  const uint16_t* Y = nullptr;
  if constexpr (!VJP) {
    if (MODE == 0)
      cols_t_cols(X, X);            // Gram tile of I - X^T X
    else
      panel_times_sym(X, Ep, std::true_type(), pf);   // update tile of X E
  } else {
    Y = static_cast<const uint16_t*>(d->yc[parity]);
    const uint16_t* S = static_cast<const uint16_t*>(d->s);
    if (MODE == 0) {
      cols_t_cols(X, Y);            // S tile: X^T Y + Y^T X
      cols_t_cols(Y, X);
    } else {
      panel_times_sym(Y, Ep, std::false_type(), pf);   // Y E + X S' with S' = -(X^T Y + Y^T X)
      panel_times_sym(X, S, std::false_type(), pf);
    }
  }

  // ------------------------------------------------------------ epilogue --
  float* Xm = VJP ? d->gy[0] : d->master[0];   // the fp32 iterate an update tile advances
  const int gi0 = it.ti * BM + wm * TM;  // first global row of this wave
  const int gj0 = it.tj * BN + wn * TN;  // first global column
  uint16_t* Xo = static_cast<uint16_t*>(VJP ? d->yc[parity ^ 1] : d->xc[parity ^ 1]) + (VJP ? 0 : xoff);
  if (!VJP && MODE == 1) {
    // Update tiles advance the fp32 iterate in place and emit its next bf16
    // copy.  Chunks 0 and 1 (32 rows each) of this wave's part of the
    // iterate were loaded by the final K loop's last two k-steps, into
    // those k-steps' free A buffers (A rotates through sX, sA0, sA1) and
    // their B buffers (sB0, sB1 alternately): piece q (1 KB: 256 / TN rows,
    // 4 values per lane) of chunk c sits in block q * 4 + wave of the A
    // buffer (q < NQ / 2) or of the B buffer (the rest).  On 256-tiles
    // chunk 2 is loaded into registers as the epilogue starts and chunk 3
    // as chunk 2 starts (both at once would spill), in the same 4-column
    // pieces per lane as the stores; loads into LDS would make the compiler
    // wait for them before every access of the staging buffer, as it
    // cannot tell the run-time-chosen buffers apart.  The accumulators are
    // staged 16 rows at a time in the last k-step's A buffer, the one
    // buffer left free.
    const int nkf = (Np - it.tj * BN) / BK;
    auto abuf = [&](int t) { const int r = t % 3; return r == 0 ? sX : r == 1 ? sA0 : sA1; };
    auto cbuf = [&](int t) { const int r = t % 3; return r == 0 ? sA0 : r == 1 ? sA1 : sX; };
    constexpr int NQ = 32 * TN / 256;   // pieces per chunk
    uint16_t* pa[2] = {abuf(nkf - 2), abuf(nkf - 1)};
    uint16_t* pb[2] = {(nkf - 2) & 1 ? sB1 : sB0, (nkf - 1) & 1 ? sB1 : sB0};
    float* sbuf = reinterpret_cast<float*>(cbuf(nkf - 1) + wave * (16 * TN * 2));
    auto piece = [&](int mi, int q) {
      return q < NQ / 2 ? pa[mi & 1] + (q * 4 + wave) * 512 : pb[mi & 1] + ((q - NQ / 2) * 4 + wave) * 512;
    };
    auto bidx = [&](int r, int c) {     // float index of element (r, c) of sbuf (16-byte chunks swizzled)
      return r * TN + ((((c >> 2) ^ (((r >> 2) & 1) << 3))) << 2) + (c & 3);
    };
    const int col = lane & 31;
    static_assert(MI <= 4, "chunks past the fourth have no registers");
    constexpr int MR = MI > 2 ? MI - 2 : 1;   // chunks read into registers
    float4 mreg[MR][NQ];
    auto load_reg = [&](int j) {
#pragma unroll
      for (int q = 0; q < NQ; ++q) {
        const int e4 = q * 64 + lane;
        const int r = e4 / (TN / 4), c = (e4 % (TN / 4)) * 4;
        mreg[j][q] = gload4(Xm + (int64_t)(gi0 + (j + 2) * 32 + r) * Np + gj0 + c);
      }
    };
    if (MI > 2) load_reg(0);
#pragma unroll
    for (int mi = 0; mi < MI; ++mi) {
      const int gi = gi0 + mi * 32;
      if (mi == 2 && MI > 3) load_reg(1);
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        // this half's iterate values
        float4 mpre[NQ / 2];
#pragma unroll
        for (int q = 0; q < NQ / 2; ++q)
          mpre[q] = mi < 2 ? *reinterpret_cast<const float4*>(piece(mi, h * NQ / 2 + q) + lane * 8)
                           : mreg[mi < 2 ? 0 : mi - 2][h * NQ / 2 + q];
        // accumulator rows 16 h .. 16 h + 15 of the chunk -> sbuf
#pragma unroll
        for (int ni = 0; ni < NI; ++ni)
#pragma unroll
          for (int r = 8 * h; r < 8 * h + 8; ++r)
            sbuf[bidx(acc_row(r, lane) - 16 * h, ni * 32 + col)] = acc[mi][ni][r];
        // row-major pass: 4 consecutive columns per lane
#pragma unroll
        for (int q = h * NQ / 2; q < (h + 1) * NQ / 2; ++q) {
          const int e4 = q * 64 + lane;
          const int r = e4 / (TN / 4), c = (e4 % (TN / 4)) * 4;
          float4 v = *reinterpret_cast<const float4*>(&sbuf[bidx(r - 16 * h, c)]);
          const int64_t off = (int64_t)(gi + r) * Np + gj0 + c;
          const float4 m = mpre[q - h * NQ / 2];
          v.x = m.x + beta * v.x;
          v.y = m.y + beta * v.y;
          v.z = m.z + beta * v.z;
          v.w = m.w + beta * v.w;
          gstore4(Xm + off, v);
          gstore2(Xo + off, pack4_bf16(v.x, v.y, v.z, v.w));
        }
      }
    }
    return;
  }
  // Other tiles: each wave stages its accumulators through a private fp32
  // LDS buffer (rows of TN floats, 16-byte chunks XOR-swizzled so that the
  // two half-waves, which hold rows 4 apart, hit disjoint banks) and writes
  // its outputs as coalesced 8- or 16-byte vectors along rows.
  auto bidx = [&](int r, int c) {  // float index of element (r, c) of a staging buffer
    return r * TN + ((((c >> 2) ^ (((r >> 2) & 1) << 3))) << 2) + (c & 3);
  };
  const int col = lane & 31;
  constexpr int NQ = 32 * TN / 256;        // 1 KB pieces (4 columns per lane) of a 32-row chunk
  // Gram-like tiles write E (or S' in VJP mode) with the identity (or
  // none) subtracted from; gradient-update tiles advance the fp32 gradient
  // iterate in place and emit its next bf16 copy, each wave's iterate chunk
  // (32 x TN) loaded by direct-to-LDS loads into a second private buffer,
  // chunk mi + 1 in flight while chunk mi is written.  The accumulators are
  // staged 32 rows at a time (every buffer is free after the loop).
  float* buf;
  uint16_t* mbuf;
  if (BM == 256) {
    buf = reinterpret_cast<float*>((wave < 2 ? sA0 : sB0) + (wave & 1) * (32 * TN * 2));
    mbuf = (wave < 2 ? sA1 : sB1) + (wave & 1) * (32 * TN * 2);
  } else {
    buf = reinterpret_cast<float*>(wave == 0 ? sA0 : wave == 1 ? sB0 : wave == 2 ? sA1 : sB1);
    mbuf = (wave == 0 ? sA0 : wave == 1 ? sB0 : wave == 2 ? sA1 : sB1) + 32 * TN * 2;
  }
  uint16_t* E = static_cast<uint16_t*>(VJP ? d->s : d->e) + (VJP ? 0 : eoff);
  constexpr float DELTA = VJP ? 0.f : 1.f;
  const bool upd = VJP && MODE == 1;
  // chunk mi of the iterate into mbuf, row-major (TN floats per row): load q
  // of a lane covers the same (row, 4 columns) that its row-major pass reads
  auto load_chunk = [&](int mi) {
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int e4 = q * 64 + lane;
      const int r = e4 / (TN / 4), c = (e4 % (TN / 4)) * 4;
      dma16(Xm + (int64_t)(gi0 + mi * 32 + r) * Np + gj0 + c, mbuf + q * 512);
    }
  };
  if (upd) load_chunk(0);
#pragma unroll
  for (int mi = 0; mi < MI; ++mi) {
    const int gi = gi0 + mi * 32;
    float4 mpre[NQ];
    if (upd) {
      // this chunk's iterate from LDS, then the next chunk's loads
      asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
#pragma unroll
      for (int q = 0; q < NQ; ++q)
        mpre[q] = *reinterpret_cast<const float4*>(mbuf + q * 512 + lane * 8);
      if (mi + 1 < MI) {
        lds_settle();
        load_chunk(mi + 1);
      }
    }
    // accumulators -> LDS, row-major
#pragma unroll
    for (int ni = 0; ni < NI; ++ni)
#pragma unroll
      for (int r = 0; r < 16; ++r) buf[bidx(acc_row(r, lane), ni * 32 + col)] = acc[mi][ni][r];
    // row-major pass: 4 consecutive columns per lane
#pragma unroll
    for (int q = 0; q < NQ; ++q) {
      const int e4 = q * 64 + lane;
      const int r = e4 / (TN / 4), c = (e4 % (TN / 4)) * 4;
      float4 v = *reinterpret_cast<const float4*>(&buf[bidx(r, c)]);
      const int64_t off = (int64_t)(gi + r) * Np + gj0 + c;
      if (!upd) {
        const int dg = (gi + r) - (gj0 + c);   // the diagonal hits column c + dg
        v.x = (dg == 0 ? DELTA : 0.f) - v.x;
        v.y = (dg == 1 ? DELTA : 0.f) - v.y;
        v.z = (dg == 2 ? DELTA : 0.f) - v.z;
        v.w = (dg == 3 ? DELTA : 0.f) - v.w;
        gstore2(E + off, pack4_bf16(v.x, v.y, v.z, v.w));
      } else {
        const float4 m = mpre[q];
        v.x = m.x + beta * v.x;
        v.y = m.y + beta * v.y;
        v.z = m.z + beta * v.z;
        v.w = m.w + beta * v.w;
        gstore4(Xm + off, v);
        gstore2(Xo + off, pack4_bf16(v.x, v.y, v.z, v.w));
      }
    }
  }
}

}  // namespace

// One launch over a table of Gram and/or update tiles (each item carries its
// own mode and ping-pong parity); vjp selects the gradient modes, step the
// saved iterate.
hipError_t launch_bf16_tiles(int big, const TiledMat* mats, const TileItem* items, int n_items, float beta,
                             hipStream_t s, int vjp, int step) {
  if (n_items <= 0) return hipSuccess;
  const char* name = vjp ? (big ? "bjorck_vjp_bf16_256" : "bjorck_vjp_bf16_128")
                         : (big ? "bjorck_bf16_256" : "bjorck_bf16_128");
  timing_begin(name, s);
  if (big && !vjp)
    hipLaunchKernelGGL((bjorck_bf16_kernel<256, 256, 2, 2, false>), dim3(n_items), dim3(256), 0, s, mats, items,
                       beta, step);
  else if (!vjp)
    hipLaunchKernelGGL((bjorck_bf16_kernel<128, 128, 2, 2, false>), dim3(n_items), dim3(256), 0, s, mats, items,
                       beta, step);
  else if (big)
    hipLaunchKernelGGL((bjorck_bf16_kernel<256, 256, 2, 2, true>), dim3(n_items), dim3(256), 0, s, mats, items,
                       beta, step);
  else
    hipLaunchKernelGGL((bjorck_bf16_kernel<128, 128, 2, 2, true>), dim3(n_items), dim3(256), 0, s, mats, items,
                       beta, step);
  hipError_t e = hipGetLastError();
  timing_end(name, s);
  return e;
}

}  // namespace orth
