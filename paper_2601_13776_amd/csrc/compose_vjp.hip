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

// kind 0: out = taps (s x s grid) of the RKO matrix a (og x c s^2, dtype):
//         out[(x s + y)][o][i] = a[o][i s^2 + x s + y]
// kind 1: out = taps (k x k grid) of an OIHW kernel slice a (og x c x k x k):
//         out[(x k + y)][o][i] = a[o][i][x][y]
// kind 2: out (RKO matrix, dtype) from taps a (s x s grid), inverse of 0
template <int KIND>
__global__ __launch_bounds__(256) void tap_layout_kernel(const TapItem* __restrict__ items, int dtype) {
  const TapItem it = items[blockIdx.y];
  const int og = it.og, c = it.c, n = it.h;   // square grid of n x n taps
  const int64_t total = (int64_t)n * n * og * c;
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    // e enumerates (o, i, x, y) with y fastest: the OIHW / RKO side is contiguous
    const int y = (int)(e % n);
    const int x = (int)((e / n) % n);
    const int64_t oi = e / ((int64_t)n * n);
    const int64_t t = ((int64_t)(x * n + y) * og) * c + oi;
    if (KIND == 0 || KIND == 1)
      static_cast<float*>(it.out)[t] = load_as_f32(it.a, e, dtype);
    else
      store_from_f32(it.out, e, dtype, static_cast<const float*>(it.a)[t]);
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
                            hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  static const char* names[5] = {"conv_vjp_rko_taps", "conv_vjp_grad_taps", "conv_vjp_rko_grad",
                                 "conv_vjp_combine_fwd", "conv_vjp_combine_bwd"};
  if (kind < 0 || kind > 4) return hipErrorInvalidValue;
  timing_begin(names[kind], s);
  const dim3 grid(grid_x(max_elems), n_items);
  switch (kind) {
    case 0: hipLaunchKernelGGL(tap_layout_kernel<0>, grid, dim3(256), 0, s, items, dtype); break;
    case 1: hipLaunchKernelGGL(tap_layout_kernel<1>, grid, dim3(256), 0, s, items, dtype); break;
    case 2: hipLaunchKernelGGL(tap_layout_kernel<2>, grid, dim3(256), 0, s, items, dtype); break;
    case 3: hipLaunchKernelGGL(combine_fwd_kernel, grid, dim3(256), 0, s, items); break;
    default: hipLaunchKernelGGL(combine_bwd_kernel, grid, dim3(256), 0, s, items); break;
  }
  hipError_t e = hipGetLastError();
  timing_end(names[kind], s);
  return e;
}

}  // namespace orth
