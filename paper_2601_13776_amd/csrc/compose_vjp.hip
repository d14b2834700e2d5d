// Elementwise kernels of the composition's vector-Jacobian product
// (Appendix B.1 construction, differentiated).  Tap grids are compact:
// tap (a, b) of an h x w grid is the og x c matrix at offset (a w + b) og c.
//
// With a block of taps P and I - P along direction (da, db) = (0, 1)
// (horizontal) or (1, 0) (vertical), one forward step is
//     T'[a][b] = Y[a][b] + T[a-da][b-db] - Y[a-da][b-db],   Y = T P,
// (terms outside T's grid are zero), and its adjoint, for the gradient G of
// T' and Z = G P, is
//     dT[a][b] = Z[a][b] + G[a+da][b+db] - Z[a+da][b+db],
//     dP      = sum over T's taps of T[a][b]^T D[a][b],
//               D[a][b] = G[a][b] - G[a+da][b+db].
// The tap products (Y, Z, dP) run on the fp32 tile GEMM; these kernels do the
// gathers, scatters and combines, all HBM-bound.
#include "internal.h"

namespace orth {
namespace {

// Layout changes between a tap grid and the per-(o, i) layout, both seen as
// matrices with M = og c and T = n^2 (n x n grid of taps):
// kind 0: out = taps (s x s grid) of the RKO matrix a (og x c s^2, dtype):
//         out[(x s + y)][o][i] = a[o][i s^2 + x s + y]
// kind 1: out = taps (k x k grid) of an OIHW kernel slice a (og x c x k x k):
//         out[(x k + y)][o][i] = a[o][i][x][y]
// kind 2: out (RKO matrix, dtype) from taps a (s x s grid), inverse of 0
// Kinds 0 and 1 transpose a [M][T] matrix into [T][M], kind 2 the reverse.
// Each tile of 64 (o, i) rows and up to 64 taps goes through LDS so that
// both the reads and the writes are contiguous runs (a tile of all T taps
// covers one contiguous span of the [M][T] side).
template <int KIND>
__global__ __launch_bounds__(256) void tap_layout_kernel(const TapItem* __restrict__ items, int dtype) {
  constexpr int TM = 64, TTMAX = 64;
  __shared__ float tile[TTMAX][TM + 1];
  const TapItem it = items[blockIdx.y];
  const int n = it.h;
  const int T = n * n;
  const int64_t M = (int64_t)it.og * it.c;
  if (T == 0 || M == 0) return;
  const int TT = T < TTMAX ? T : TTMAX;
  const int64_t mt = (M + TM - 1) / TM;
  const int64_t ntiles = mt * ((T + TT - 1) / TT);
  for (int64_t q = blockIdx.x; q < ntiles; q += gridDim.x) {
    const int64_t m0 = (q % mt) * TM;
    const int t0 = (int)(q / mt) * TT;
    const int tn = T - t0 < TT ? T - t0 : TT;
    const int mn = M - m0 < TM ? (int)(M - m0) : TM;
    __syncthreads();  // the previous tile's reads of `tile` are done
    if (KIND == 0 || KIND == 1) {
      // read [M][T] side: row m holds tn contiguous taps
      for (int j = threadIdx.x; j < mn * tn; j += 256) {
        const int m = j / tn, t = j - m * tn;
        tile[t][m] = load_as_f32(it.a, (m0 + m) * T + t0 + t, dtype);
      }
      __syncthreads();
      for (int j = threadIdx.x; j < tn * TM; j += 256) {
        const int t = j >> 6, m = j & 63;
        if (m < mn) gst_f32(it.out, (int64_t)(t0 + t) * M + m0 + m, tile[t][m]);
      }
    } else {
      for (int j = threadIdx.x; j < tn * TM; j += 256) {
        const int t = j >> 6, m = j & 63;
        if (m < mn) tile[t][m] = gld_f32(it.a, (int64_t)(t0 + t) * M + m0 + m);
      }
      __syncthreads();
      for (int j = threadIdx.x; j < mn * tn; j += 256) {
        const int m = j / tn, t = j - m * tn;
        store_from_f32(it.out, (m0 + m) * T + t0 + t, dtype, tile[t][m]);
      }
    }
  }
}

// forward combine: a = T (h x w grid), b = Y (same grid), out = T' grid
__global__ __launch_bounds__(256) void combine_fwd_kernel(const TapItem* __restrict__ items) {
  const TapItem it = items[blockIdx.y];
  const int v = it.vertical, h = it.h, w = it.w;
  const int oh = h + v, ow = w + 1 - v;
  const int64_t tap = (int64_t)it.og * it.c;
  const int64_t total = (int64_t)oh * ow * tap;
  const float* T = static_cast<const float*>(it.a);
  const float* Y = static_cast<const float*>(it.b);
  float* O = static_cast<float*>(it.out);
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int64_t m = e % tap;
    const int t = (int)(e / tap);
    const int a = t / ow, b = t % ow;
    const int pa = a - v, pb = b - (1 - v);
    float val = 0.f;
    if (a < h && b < w) val += Y[(int64_t)(a * w + b) * tap + m];
    if (pa >= 0 && pb >= 0) {
      const int64_t po = (int64_t)(pa * w + pb) * tap + m;
      val += T[po] - Y[po];
    }
    O[e] = val;
  }
}

// adjoint combine: a = G, b = Z (both on the grid (h + v) x (w + 1 - v)),
// out = dT and out2 = D (both on the h x w grid)
__global__ __launch_bounds__(256) void combine_bwd_kernel(const TapItem* __restrict__ items) {
  const TapItem it = items[blockIdx.y];
  const int v = it.vertical, h = it.h, w = it.w;
  const int gw = w + 1 - v;
  const int64_t tap = (int64_t)it.og * it.c;
  const int64_t total = (int64_t)h * w * tap;
  const float* G = static_cast<const float*>(it.a);
  const float* Z = static_cast<const float*>(it.b);
  float* dT = static_cast<float*>(it.out);
  float* D = static_cast<float*>(it.out2);
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int64_t m = e % tap;
    const int t = (int)(e / tap);
    const int a = t / w, b = t % w;
    const int64_t here = (int64_t)(a * gw + b) * tap + m;
    const int64_t next = (int64_t)((a + v) * gw + b + 1 - v) * tap + m;
    const float g0 = G[here], g1 = G[next];
    dT[e] = Z[here] + g1 - Z[next];
    D[e] = g0 - g1;
  }
}

unsigned grid_x(int64_t max_elems) {
  int64_t b = (max_elems + 255) / 256;
  if (b < 1) b = 1;
  if (b > 1024) b = 1024;
  return (unsigned)b;
}

}  // namespace

hipError_t launch_tap_items(int kind, const TapItem* items, int n_items, int dtype, int64_t max_elems,
                            hipStream_t s, const char* name) {
  if (n_items <= 0) return hipSuccess;
  static const char* names[5] = {"conv_vjp_rko_taps", "conv_vjp_grad_taps", "conv_vjp_rko_grad",
                                 "conv_vjp_combine_fwd", "conv_vjp_combine_bwd"};
  if (kind < 0 || kind > 4) return hipErrorInvalidValue;
  if (!name) name = names[kind];
  timing_begin(name, s);
  // the layout kernels take a 64 x 64 tile per grid-stride step
  const dim3 grid(kind <= 2 ? grid_x((max_elems + 15) / 16) : grid_x(max_elems), n_items);
  switch (kind) {
    case 0: hipLaunchKernelGGL(tap_layout_kernel<0>, grid, dim3(256), 0, s, items, dtype); break;
    case 1: hipLaunchKernelGGL(tap_layout_kernel<1>, grid, dim3(256), 0, s, items, dtype); break;
    case 2: hipLaunchKernelGGL(tap_layout_kernel<2>, grid, dim3(256), 0, s, items, dtype); break;
    case 3: hipLaunchKernelGGL(combine_fwd_kernel, grid, dim3(256), 0, s, items); break;
    default: hipLaunchKernelGGL(combine_bwd_kernel, grid, dim3(256), 0, s, items); break;
  }
  hipError_t e = hipGetLastError();
  timing_end(name, s);
  return e;
}

}  // namespace orth
