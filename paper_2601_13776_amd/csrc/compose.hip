// AOC kernel composition (Appendix B.1: AOC = RKO ⊛ K_BCOP).
//
// The kernel of one group is kept as a grid of "taps": tap (a, b) is the
// cout_g x c matrix K[:, :, a, b] (tap-major, fixed k x k slots).  Composing
// the current kernel T with a horizontal block (taps P and I - P) gives one
// more column of taps:
//     T'[a][b] = T[a][b] P + T[a][b-1] (I - P) = Y[a][b] + T[a][b-1] - Y[a][b-1]
// with Y[a][b] = T[a][b] P; a vertical block does the same along a.  The
// products Y run as a batched GEMM (gemm_f32.hip); the kernels here build
// the initial s x s taps from the RKO matrix, combine taps after each block
// step and scatter the final taps into the OIHW kernel of the layer.
// All three are elementwise and HBM-bound.
#include "internal.h"

namespace orth {
namespace {

// taps[a][b] = M[:, i s^2 + a s + b]  (M is cout_g x c s^2, row-major)
__global__ __launch_bounds__(256) void compose_init_kernel(const ComposeGroup* __restrict__ groups, int dtype) {
  const ComposeGroup& g = groups[blockIdx.y];
  const int s = g.s, c = g.c, og = g.cout_g;
  const int64_t tap = (int64_t)og * c;
  const int64_t total = (int64_t)s * s * tap;
  float* T = g.taps[0];
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    // e enumerates (o, i, a, b) with b fastest so reads of M are contiguous
    const int b = (int)(e % s);
    const int a = (int)((e / s) % s);
    const int64_t oi = e / ((int64_t)s * s);
    const int i = (int)(oi % c);
    const int o = (int)(oi / c);
    const float v = load_as_f32(g.rko, (int64_t)o * c * s * s + (int64_t)i * s * s + a * s + b, dtype);
    T[(int64_t)(a * g.k + b) * tap + (int64_t)o * c + i] = v;
  }
}

__global__ __launch_bounds__(256) void compose_combine_kernel(const ComposeGroup* __restrict__ groups,
                                                              const CombineItem* __restrict__ items) {
  const CombineItem it = items[blockIdx.y];
  const ComposeGroup& g = groups[it.grp];
  const int k = g.k;
  const int64_t tap = (int64_t)g.cout_g * g.c;
  const int out_h = it.in_h + (it.vertical ? 1 : 0);
  const int out_w = it.in_w + (it.vertical ? 0 : 1);
  const int64_t total = (int64_t)out_h * out_w * tap;
  const float* T = g.taps[it.src];
  float* TN = g.taps[it.src ^ 1];
  const float* Y = g.y;
  for (int64_t e = blockIdx.x * 256 + threadIdx.x; e < total; e += (int64_t)gridDim.x * 256) {
    const int64_t w = e % tap;
    const int t = (int)(e / tap);
    const int a = t / out_w, b = t % out_w;
    // this tap of the block (a, b) and the tap it shifts in (pa, pb)
    const int pa = it.vertical ? a - 1 : a;
    const int pb = it.vertical ? b : b - 1;
    float v = 0.f;
    if (a < it.in_h && b < it.in_w) v += Y[(int64_t)(a * k + b) * tap + w];
    if (pa >= 0 && pb >= 0) {
      const int64_t po = (int64_t)(pa * k + pb) * tap + w;
      v += T[po] - Y[po];
    }
    TN[(int64_t)(a * k + b) * tap + w] = v;
  }
}

unsigned grid_x(int64_t max_elems) {
  int64_t b = (max_elems + 255) / 256;
  if (b < 1) b = 1;
  if (b > 1024) b = 1024;
  return (unsigned)b;
}

}  // namespace

hipError_t launch_compose_init(const ComposeGroup* groups, int n_groups, int dtype, int64_t max_elems,
                               hipStream_t s) {
  if (n_groups <= 0) return hipSuccess;
  timing_begin("compose_init", s);
  hipLaunchKernelGGL(compose_init_kernel, dim3(grid_x(max_elems), n_groups), dim3(256), 0, s, groups, dtype);
  hipError_t e = hipGetLastError();
  timing_end("compose_init", s);
  return e;
}

hipError_t launch_compose_combine(const ComposeGroup* groups, const CombineItem* items, int n_items,
                                  int64_t max_elems, hipStream_t s) {
  if (n_items <= 0) return hipSuccess;
  timing_begin("compose_combine", s);
  hipLaunchKernelGGL(compose_combine_kernel, dim3(grid_x(max_elems), n_items), dim3(256), 0, s, groups, items);
  hipError_t e = hipGetLastError();
  timing_end("compose_combine", s);
  return e;
}


}  // namespace orth
