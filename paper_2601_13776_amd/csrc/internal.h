// Internal declarations shared by the HIP kernels and the host side of
// liborth.  Not part of the public ABI (include/orth.h is).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <utility>

#include "../../include/orth.h"

namespace orth {

// ---------------------------------------------------------------------------
// bfloat16 <-> fp32.  Round to nearest, ties to even; NaN stays a quiet NaN.
// ---------------------------------------------------------------------------
__host__ __device__ inline float bf16_to_f32(uint16_t b) {
  return __uint_as_float(static_cast<uint32_t>(b) << 16);
}
__device__ inline uint16_t f32_to_bf16(float f) {
  uint32_t u = __float_as_uint(f);
  if ((u & 0x7fffffffu) > 0x7f800000u) return 0x7fc0;
  u += 0x7fffu + ((u >> 16) & 1u);
  return static_cast<uint16_t>(u >> 16);
}
// ---------------------------------------------------------------------------
// Global-memory accesses.  Kernels take their data pointers from descriptor
// tables, and the compiler cannot prove that a pointer loaded from memory
// addresses global memory: plain accesses through it become FLAT
// instructions, which count against the LDS counter as well, so every wait
// for an LDS result also waits for the global loads and stores in flight.
// These helpers access through global-address-space pointers (the attribute
// takes effect on scalar and vector-extension types, not on HIP's vector
// classes).  Every pointer passed to them must address global memory.
// ---------------------------------------------------------------------------
#define ORTH_GLOBAL __attribute__((address_space(1)))
typedef uint32_t orth_u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t orth_u32x2 __attribute__((ext_vector_type(2)));
typedef float orth_f32x4 __attribute__((ext_vector_type(4)));
__device__ __forceinline__ float gld_f32(const void* p, int64_t i) { return ((const ORTH_GLOBAL float*)p)[i]; }
__device__ __forceinline__ uint32_t gld_u32(const void* p, int64_t i) { return ((const ORTH_GLOBAL uint32_t*)p)[i]; }
__device__ __forceinline__ uint16_t gld_u16(const void* p, int64_t i) { return ((const ORTH_GLOBAL uint16_t*)p)[i]; }
__device__ __forceinline__ double gld_f64(const void* p, int64_t i) { return ((const ORTH_GLOBAL double*)p)[i]; }
__device__ __forceinline__ uint4 gld_u32x4(const void* p) {
  const orth_u32x4 v = *(const ORTH_GLOBAL orth_u32x4*)p;
  return make_uint4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ float4 gld_f32x4(const void* p) {
  const orth_f32x4 v = *(const ORTH_GLOBAL orth_f32x4*)p;
  return make_float4(v.x, v.y, v.z, v.w);
}
__device__ __forceinline__ void gst_f32(void* p, int64_t i, float v) { ((ORTH_GLOBAL float*)p)[i] = v; }
__device__ __forceinline__ void gst_u16(void* p, int64_t i, uint16_t v) { ((ORTH_GLOBAL uint16_t*)p)[i] = v; }
__device__ __forceinline__ void gst_f64(void* p, int64_t i, double v) { ((ORTH_GLOBAL double*)p)[i] = v; }
__device__ __forceinline__ void gst_f32x4(void* p, float4 v) {
  *(ORTH_GLOBAL orth_f32x4*)p = orth_f32x4{v.x, v.y, v.z, v.w};
}
__device__ __forceinline__ void gst_u32x4(void* p, uint4 v) { *(ORTH_GLOBAL orth_u32x4*)p = orth_u32x4{v.x, v.y, v.z, v.w}; }
__device__ __forceinline__ void gst_u32x2(void* p, uint2 v) { *(ORTH_GLOBAL orth_u32x2*)p = orth_u32x2{v.x, v.y}; }

__device__ inline float load_as_f32(const void* p, int64_t idx, int dtype) {
  return dtype == ORTH_BF16 ? bf16_to_f32(gld_u16(p, idx)) : gld_f32(p, idx);
}
__device__ inline void store_from_f32(void* p, int64_t idx, int dtype, float v) {
  if (dtype == ORTH_BF16)
    gst_u16(p, idx, f32_to_bf16(v));
  else
    gst_f32(p, idx, v);
}

// Runs of 8 consecutive elements moved as 16-byte vectors (one for bf16,
// two for fp32).  vec8_ok tells whether every run starting at a multiple
// of 8 of every row of a (pointer, leading dim) pair is 16-byte aligned.
__device__ inline bool vec8_ok(const void* p, int64_t ld, int dtype) {
  const int64_t es = dtype == ORTH_BF16 ? 2 : 4;
  return ((reinterpret_cast<uintptr_t>(p) | (uintptr_t)(ld * es)) & 15) == 0;
}
__device__ inline void load8_f32(const void* p, int64_t idx, int dtype, float (&v)[8]) {
  if (dtype == ORTH_BF16) {
    const uint4 q = gld_u32x4(static_cast<const uint16_t*>(p) + idx);
    const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = __uint_as_float(w[i] << 16);
      v[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
    }
  } else {
    const float4 a = gld_f32x4(static_cast<const float*>(p) + idx);
    const float4 b = gld_f32x4(static_cast<const float*>(p) + idx + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}
__device__ inline uint4 pack8_bf16(const float (&v)[8]) {
  uint32_t w[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) w[i] = (uint32_t)f32_to_bf16(v[2 * i]) | ((uint32_t)f32_to_bf16(v[2 * i + 1]) << 16);
  return make_uint4(w[0], w[1], w[2], w[3]);
}
__device__ inline void store8_f32(void* p, int64_t idx, int dtype, const float (&v)[8]) {
  if (dtype == ORTH_BF16) {
    gst_u32x4(static_cast<uint16_t*>(p) + idx, pack8_bf16(v));
  } else {
    gst_f32x4(static_cast<float*>(p) + idx, make_float4(v[0], v[1], v[2], v[3]));
    gst_f32x4(static_cast<float*>(p) + idx + 4, make_float4(v[4], v[5], v[6], v[7]));
  }
}

// ---------------------------------------------------------------------------
// Björck batch descriptors (device-resident tables built by the host).
// Every matrix is processed in its tall orientation M x N (M >= N); a wide
// input (rows < cols) is transposed on the way in and out.
// ---------------------------------------------------------------------------
struct TiledMat {
  const void* in;
  void* out;
  int64_t ld_in, ld_out;
  int32_t rows, cols;        // as given by the caller
  int32_t M, N;              // tall orientation
  int32_t Mp, Np;            // padded to the tile grid (zero padding is exact)
  int32_t transposed;        // rows < cols
  int32_t status_index;      // index in the batch (status array slot)
  int32_t partial_base;      // first slot of this matrix's partial sums
  int32_t n_partials;
  float* master[2];          // fp32 iterate, Mp x Np (bf16 mode uses [0] only)
  void* xc[2];               // bf16 mode: bf16 copies of the iterate, Mp x Np
  void* xt;                  // fp32 products only: transposed iterate, Np x Mp
  void* e;                   // I - X^T X in compute dtype, Np x Np (bf16: upper tiles only)
  float* inv_norm;           // this matrix's pre-scale factor
  // Saved-iterate mode (vector-Jacobian product): step t of a launch reads
  // xc[p] + t xstep and e + t estep (both 0 outside that mode).
  int64_t xstep, estep;
  // Vector-Jacobian product only.
  const void* gout;          // dL/d(output) in the caller's layout
  int64_t ld_gout;
  float* gy[2];              // fp32 gradient iterate, Mp x Np (bf16 mode: [0], in place)
  float* gyt[2];             // fp32 products: its transposes, Np x Mp (the X^T Y operands)
  void* yc[2];               // bf16 copies of the gradient iterate (bf16 mode)
  void* s;                   // -(X^T Y + Y^T X), Np x Np (bf16: upper tiles only)
  double* dot;               // <Y_0, W_0>, one per matrix
  int32_t gy_final;          // gy[] index holding dL/dW_0 after the last step
  int32_t fused;             // 1: handled whole by the small-matrix kernel (per-matrix
                             // finish kernels skip it)
  // Spectral pre-scaling only.
  float* u;                  // the caller's cached vector (N values)
  double* pv;                // power-iteration vector v (N)
  double* px;                // X v (M)
  double* py;                // X^T X v (N)
  double* sig;               // sigma_hat
  // Spectral pre-scaling in a vector-Jacobian product: the vectors of every
  // power step (v_0 .. v_q at pst, then x_1 .. x_q, then y_1 .. y_q), the
  // backward scalars (SB_* slots) and the 2q rank-1 pairs (a: M values, then
  // b: N values, each pair M + N apart) that the power steps add to dL/dX.
  double* pst;
  double* sb;
  double* pair;
  int32_t pq;                // power steps q
};

// Slots of TiledMat::sb.
enum { SB_FRO = 0, SB_SIGMA = 1, SB_BRANCH = 2, SB_DSCALE = 3, SB_C = 4, SB_SLOTS = 8 };

struct TileItem {
  int32_t mat;
  int32_t ti, tj;
  int32_t flags;             // TILE_* bits
};
enum : int32_t {
  TILE_UPDATE = 1,           // bf16 Björck: update tile (else Gram tile)
  TILE_PARITY = 2,           // bf16 Björck: the update reads xc[1] and writes xc[0]
  TILE_VJP = 4               // with TILE_UPDATE: Y <- Y + beta (Y E + X S), else S tile
};

struct SmallMat {
  const void* in;
  void* out;
  int64_t ld_in, ld_out;
  int32_t rows, cols;
  int32_t M, N;              // tall orientation
  int32_t Mp;                // M rounded up to 32
  int32_t transposed;
  int32_t status_index;
  int32_t pad;
  float* u;                  // spectral pre-scaling: the caller's cached vector
};

// A small matrix (N <= 64, M <= 128) of the vector-Jacobian product: the
// whole computation (forward recomputation, gradient recurrence, pre-scaling
// derivative) runs in one workgroup; X_t and E_t of the recomputation go to
// `save` (T (Mp NP + NP NP) floats, pitch NP) for the way back.
struct SmallVjpMat {
  const void* w;             // the forward's input, caller layout
  const void* gout;          // dL/d(output), caller layout
  void* gin;                 // dL/dW, caller layout (dtype of w)
  int64_t ld_w, ld_gout, ld_gin;
  int32_t rows, cols;
  int32_t M, N;              // tall orientation
  int32_t Mp;                // M rounded up to 32
  int32_t transposed;
  int32_t status_index;
  int32_t np;                // LDS columns: 32 or 64
  float* save;
  // spectral pre-scaling: the cached vector the differentiated forward
  // started from (read only) and fp64 storage for the power steps' vectors
  // and the rank-1 pairs of the backward
  const float* u;
  double* pst;
};

// One batched power-iteration work item: 64 outputs of a matrix-vector
// product with a matrix in the caller's layout.
struct PowerItem {
  int32_t mat;
  int32_t block;             // outputs [64 block, 64 block + 64)
  int32_t coldot;            // 0: out[r] = sum_c W[r][c] in[c]; 1: out[c] = sum_r W[r][c] in[r]
  int32_t second;            // 0: v -> x, 1: x -> y
};

// Generic bounds-checked fp32 GEMM work item: C = A * B^T (+ A2 * B2^T)
// over one 64 x 64 output tile, A logically M x K, B logically N x K, A2
// M x K2, B2 N x K2 (K2 = 0: no second pair).
enum GemmEpi : int32_t {
  EPI_STORE = 0,     // C[i][j] = acc
  EPI_GRAM_E = 1,    // C[i][j] = delta_ij - acc  (and C[j][i] if mirror)
  EPI_UPDATE = 2,    // v = src[i][j] + beta acc; C[i][j] = v; dst2[j][i] = v if dst2
  EPI_MAXDEV = 3,    // red[0] = max(red[0], |delta_ij - acc|)
  EPI_NEG = 4,       // C[i][j] = -acc  (and C[j][i] if mirror)
  EPI_SERIES = 5     // v = beta acc; C[i][j] = v (fp32); dst2[i][j] += v (ld2)
};

// A further operand pair of a GEMM item (same storage dtypes as the item's
// first pair): C += A B^T with A logically M x K, B logically N x K.
struct GemmPair {
  const void* A;
  const void* B;
  int64_t lda, ldb;
  int32_t K;
  int32_t a_trans, b_trans;
  int32_t pad;
};

struct GemmItem {
  const void* A;
  const void* B;
  const void* A2;
  const void* B2;
  void* C;
  const float* src;
  float* dst2;
  float* red;
  int64_t lda, ldb, lda2, ldb2, ldc, ld_src, ld2;
  // element offsets added per unit of the launch's step argument
  int64_t a_step, b_step, a2_step, b2_step, c_step, src_step, d2_step;
  int32_t M, N, K, K2;
  int32_t ti, tj;
  int32_t a_dtype, b_dtype;  // storage of A and A2, of B and B2
  int32_t a_trans, b_trans;  // 0: row-major [M][K]; 1: stored [K][M]
  int32_t a2_trans, b2_trans;
  int32_t epi;
  int32_t mirror;
  float beta;
  int32_t c_dtype;           // EPI_STORE: storage of C
  int32_t pair_base;         // further operand pairs: the launch's pair table
  int32_t pair_count;        //   [pair_base, pair_base + pair_count)
};

// One 64 x 64 output tile of a GemmItem's product (the item's own ti, tj are
// not read on the device).  With a product's `mirror` set, its off-diagonal
// tiles also write the transposed tile.
struct GemmTile {
  int32_t item;
  int32_t ti, tj;
  int32_t pad;
};

// Compose (AOC) descriptors: one entry per (layer, group).
struct ComposeGroup {
  const void* rko;           // this group's RKO matrix, cout_g x (c s^2)
  const void* proj;          // this group's projector factors, nproj x c x h
  void* kernel;              // whole layer kernel (OIHW); group offset applied in-kernel
  float* taps[2];            // ping-pong tap buffers, k*k taps of cout_g x c
  float* y;                  // tap products, k*k taps of cout_g x c
  float* p;                  // projectors, nproj x c x c
  int32_t cout_g, c, h;      // h = floor(c / 2)
  int32_t k, s, group, nproj;
  int32_t cur;               // which taps[] holds the current kernel
  int32_t pad;
};

// One tap-combination work item of a block step.
struct CombineItem {
  int32_t grp;               // ComposeGroup index
  int32_t vertical;          // 0: horizontal block, 1: vertical block
  int32_t in_h, in_w;        // tap grid before the step
  int32_t src;               // taps[src] is read, taps[src ^ 1] written
  int32_t pad;
};

// One elementwise work item of the composition's vector-Jacobian product.
// Tap grids are compact: tap (a, b) of an h x w grid is the og x c matrix at
// element offset (a w + b) og c.
struct TapItem {
  const void* a;             // first source (see the kernel using the item)
  const void* b;             // second source
  void* out;
  void* out2;
  int32_t og, c;             // tap matrix shape
  int32_t h, w;              // grid of the tap buffer the item is defined on
  int32_t vertical;          // block direction of a combine step
  int32_t pad;
};

// ---------------------------------------------------------------------------
// Launch helpers (host).
// ---------------------------------------------------------------------------
struct LaunchCtx {
  hipStream_t stream;
};

// Hooks around every launch: per-kernel event timing when enabled, the
// launch trace of ORTH_LOG=2 and the per-launch synchronization of
// ORTH_DEBUG_SYNC=1.
void timing_begin(const char* name, hipStream_t s);
void timing_end(const char* name, hipStream_t s);
// Sets the calling thread's last-error message and returns `code`.
int report_error(int code, const char* msg);
// ORTH_LOG level (0 when unset) and one stderr line prefixed "[orth] ".
int log_level();
void log_line(const char* fmt, ...) __attribute__((format(printf, 1, 2)));

// Copies a call's descriptor tables into its workspace `dst` on stream s:
// n_spans spans (workspace offset, bytes) whose bytes lie back to back in
// `data`.  Returns an orth_status.
typedef int (*TableUploader)(const unsigned char* data, const std::pair<size_t, size_t>* spans, size_t n_spans,
                             void* dst, hipStream_t s);
// The orthogonalization of one batch (validation, planning, table upload
// and every launch) on stream s into `workspace`; side_streams lets the
// small-matrix kernels run on the calling thread's side streams; upload
// nullptr copies the tables from the library's pinned staging pool.
int ortho_enqueue(const orth_mat* mats, int32_t n, const orth_bjorck_opts* opts, void* workspace,
                  size_t workspace_bytes, int32_t* status_dev, hipStream_t s, bool side_streams,
                  TableUploader upload, const char* entry);

// Kernel launchers (defined next to their kernels).
hipError_t launch_bjorck_small(const SmallMat* mats, int n, int np, int max_mp, int iters, float beta,
                               int prescale, int power_iters, int in_dtype, int out_dtype, int32_t* status,
                               hipStream_t s);
hipError_t launch_bjorck_small_vjp(const SmallVjpMat* mats, int n, int np, int max_mp, int iters, float beta,
                                   int prescale, int power_iters, int in_dtype, int gout_dtype, int32_t* status,
                                   hipStream_t s);
hipError_t launch_power_init(const TiledMat* mats, int n_mats, hipStream_t s);
// vector-Jacobian product through spectral pre-scaling: the forward's power
// vectors kept per step, then the backward through the steps (bw: the same
// matrices with pv / px / py pointing at the backward's vectors)
hipError_t launch_power_keep(const TiledMat* mats, int n_mats, int k, hipStream_t s);
hipError_t launch_spec_bwd(const TiledMat* mats, const TiledMat* bw, int n_mats, const PowerItem* items0,
                           int n_items0, const PowerItem* items1, int n_items1, int q, int in_dtype,
                           const int32_t* status, hipStream_t s);
hipError_t launch_power_dot(const TiledMat* mats, const PowerItem* items, int n_items, int in_dtype,
                            hipStream_t s);
hipError_t launch_power_normalize(const TiledMat* mats, int n_mats, hipStream_t s);
hipError_t launch_prescale_partial(const TiledMat* mats, const TileItem* items, int n_items,
                                   int in_dtype, double* partials, hipStream_t s);
// write_u = 0: the spectral estimate is not handed back (a vector-Jacobian
// product's recomputation); matrices with sb record ||W||_F and the scale
hipError_t launch_prescale_finish(const TiledMat* mats, int n_mats, const double* partials,
                                  int prescale, int32_t* status, hipStream_t s, int write_u = 1);
hipError_t launch_prescale_scale(const TiledMat* mats, const TileItem* items, int n_items,
                                 int in_dtype, int compute, hipStream_t s);
hipError_t launch_writeout(const TiledMat* mats, const TileItem* items, int n_items,
                           int master_index, int out_dtype, hipStream_t s);
hipError_t launch_bf16_tiles(int big, const TiledMat* mats, const TileItem* items, int n_items, float beta,
                             hipStream_t s, int vjp = 0, int step = 0);
// The last n_km tiles must be of single-pair products with both operands
// stored k-major; they run on the k-major instantiation.
hipError_t launch_gemm_f32(const GemmItem* items, const GemmTile* tiles, int n_tiles, const char* name,
                           hipStream_t s, int step = 0, const GemmPair* pairs = nullptr, int n_km = 0);
hipError_t launch_vjp_load_grad(const TiledMat* mats, const TileItem* items, int n_items, int gout_dtype,
                                hipStream_t s);
hipError_t launch_vjp_dot_partial(const TiledMat* mats, const TileItem* items, int n_items, int in_dtype,
                                  double* partials, hipStream_t s);
hipError_t launch_vjp_dot_finish(const TiledMat* mats, int n_mats, const double* partials, hipStream_t s);
hipError_t launch_vjp_writeout(const TiledMat* mats, const TileItem* items, int n_items, int in_dtype,
                               int prescale, const int32_t* status, hipStream_t s);
hipError_t launch_compose_init(const ComposeGroup* groups, int n_groups, int dtype, int64_t max_elems,
                               hipStream_t s);
hipError_t launch_compose_combine(const ComposeGroup* groups, const CombineItem* items, int n_items,
                                  int64_t max_elems, hipStream_t s);
hipError_t launch_fill_f32(float* p, int64_t n, float v, hipStream_t s);
// kind: 0 taps from the RKO matrix, 1 taps from an OIHW kernel gradient,
// 2 RKO gradient (or any OIHW tensor: the composed kernel) from taps,
// 3 forward combine, 4 adjoint combine; name: the timing name (default:
// the kind's role in the composition VJP)
hipError_t launch_tap_items(int kind, const TapItem* items, int n_items, int dtype, int64_t max_elems,
                            hipStream_t s, const char* name = nullptr);

// Exponentials (expo.hip).  One item per matrix or conv layer.
struct ExpItem {
  const void* in;            // W (C x C, caller layout) or the kernel K (c x c x k x k, OIHW)
  float* a;                  // exp map: A = W - W^T (C x C); conv: L taps (k x k grid)
  float* out;                // the fp32 series accumulator (C x C, or S x S taps)
  float* p0;                 // exp map: first power Ahat; unused for conv
  const float* inv;          // exp map: 1 / sigma of A (from the spectral pre-scaling kernels)
  int64_t ld_in;
  int32_t c;                 // C, or channels c
  int32_t k;                 // conv: kernel size (1 for the exp map)
  int32_t size;              // conv: S = terms (k - 1) + 1 (1 for the exp map)
  float scale;               // conv: L = scale (K - K*)
};
hipError_t launch_exp_skew(const ExpItem* items, int n_items, int conv, int in_dtype, int64_t max_elems,
                           hipStream_t s);
hipError_t launch_exp_init(const ExpItem* items, int n_items, int conv, int64_t max_elems, hipStream_t s);
hipError_t launch_conv_apply(const orth_conv_apply_args* a, hipStream_t s);
hipError_t launch_conv_check(const orth_check_args* a, const void* kernel, const float* x,
                             double* partial, float* out, int adjoint, hipStream_t s);

}  // namespace orth
