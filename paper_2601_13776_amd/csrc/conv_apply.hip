// Application of an explicit convolution kernel with circular padding, and
// of its transpose (Section 3: AOC layers run as one convolution, natively
// strided, dilated, grouped, and transposed for learnable upsampling).
//
// Forward (cross-correlation, NCHW, kernel cout x c x k x k, c = cin / g):
//   y[b, o, u, v] = sum_{i,a,e} K[o, i, a, e] x[b, g(o) c + i, (s u + d a - pl) mod H, (s v + d e - pl) mod W]
// Transposed (the adjoint, from the cout x H/s x W/s grid to cin x H x W):
//   z[b, g c + i, p, q] = sum_{o,a,e} K[g og + o, i, a, e] y[b, g og + o, u, v]
//   with u = ((p + pl - d a) mod H) / s when that is a multiple of s (else
//   the term is absent), v likewise; pl = floor((d (k - 1) + 1 - s) / 2).
//
// Both run as an implicit GEMM on fp32 MFMA (v_mfma_f32_32x32x2f32): rows
// are output channels (the kernel is the first operand), columns are output
// pixels (the second operand is gathered from the input on the fly), the
// reduction runs over (input channel, tap).  Every output element is written
// once by one lane: deterministic, no atomics.  64 x 64 tiles, four waves of
// 32 x 32, K steps of 32 through two LDS stages.
#include "internal.h"

namespace orth {

typedef float f32x16 __attribute__((ext_vector_type(16)));

namespace {

struct ApplyGeom {
  int cin, cout, k, s, d, g, c, og;
  int H, W, Ho, Wo;      // the forward conv's input and output grids
  int pl;
  int batch;
  int rows, red;         // per group: output channels, reduction length
  int64_t pix;           // output pixels (batch x output grid)
  int kdtype;
};

__device__ inline int pmod(int a, int m) {
  int r = a % m;
  return r < 0 ? r + m : r;
}
__device__ inline int acc_row(int r, int lane) { return 8 * (r >> 2) + 4 * (lane >> 5) + (r & 3); }

template <bool TR>
__global__ __launch_bounds__(256) void conv_apply_kernel(ApplyGeom G, const void* __restrict__ kern,
                                                         const float* __restrict__ x, float* __restrict__ y) {
  constexpr int BM = 64, BN = 64, BK = 32, PITCH = BK + 4;
  __shared__ __attribute__((aligned(16))) float As[2][BM * PITCH];
  __shared__ __attribute__((aligned(16))) float Bs[2][BN * PITCH];
  const int grp = blockIdx.z;
  const int row0 = blockIdx.y * BM;
  const int64_t pix0 = (int64_t)blockIdx.x * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int kk2 = G.k * G.k;

  // first operand: the kernel, thread -> (row, 8 consecutive k)
  const int ar = tid >> 2, ak = (tid & 3) * 8;
  // second operand: gathered pixels, thread -> (pixel, 8 consecutive k)
  const int bp = tid & 63, bk = (tid >> 6) * 8;
  const int64_t pix = pix0 + bp;
  const bool pix_ok = pix < G.pix;
  // decompose this thread's pixel once
  int pb = 0, pu = 0, pv = 0;   // batch, row, column of the output pixel
  if (pix_ok) {
    const int ow = TR ? G.W : G.Wo, oh = TR ? G.H : G.Ho;
    pv = (int)(pix % ow);
    pu = (int)((pix / ow) % oh);
    pb = (int)(pix / ((int64_t)ow * oh));
  }
  const int64_t xplane = TR ? (int64_t)G.Ho * G.Wo : (int64_t)G.H * G.W;
  const int xch = TR ? G.cout : G.cin;
  const float* xb = x + (int64_t)pb * xch * xplane;

  float ra[8], rb[8];
  auto gload = [&](int k0) {
    // kernel values
    {
      const int row = row0 + ar;
      int kk = k0 + ak;
      int ch = kk / kk2, tap = kk - ch * kk2;   // (input channel, tap) or (output channel, tap)
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float v = 0.f;
        if (row < G.rows && kk < G.red) {
          const int64_t idx = TR ? ((int64_t)(grp * G.og + ch) * G.c + row) * kk2 + tap
                                 : (int64_t)(grp * G.og + row) * G.red + kk;
          v = load_as_f32(kern, idx, G.kdtype);
        }
        ra[j] = v;
        ++kk;
        if (++tap == kk2) {
          tap = 0;
          ++ch;
        }
      }
    }
    // gathered input values
    {
      int kk = k0 + bk;
      int ch = kk / kk2, tap = kk - ch * kk2;
      int a = tap / G.k, e = tap - a * G.k;
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        float v = 0.f;
        if (pix_ok && kk < G.red) {
          if (!TR) {
            const int r = pmod(G.s * pu + G.d * a - G.pl, G.H);
            const int q = pmod(G.s * pv + G.d * e - G.pl, G.W);
            v = xb[(int64_t)(grp * G.c + ch) * xplane + (int64_t)r * G.W + q];
          } else {
            const int r = pmod(pu + G.pl - G.d * a, G.H);
            const int q = pmod(pv + G.pl - G.d * e, G.W);
            if (r % G.s == 0 && q % G.s == 0)
              v = xb[(int64_t)(grp * G.og + ch) * xplane + (int64_t)(r / G.s) * G.Wo + q / G.s];
          }
        }
        rb[j] = v;
        ++kk;
        if (++e == G.k) {
          e = 0;
          if (++a == G.k) {
            a = 0;
            ++ch;
          }
        }
      }
    }
  };
  auto sstore = [&](int buf) {
    float4* pa = reinterpret_cast<float4*>(&As[buf][ar * PITCH + ak]);
    pa[0] = make_float4(ra[0], ra[1], ra[2], ra[3]);
    pa[1] = make_float4(ra[4], ra[5], ra[6], ra[7]);
    float4* pbv = reinterpret_cast<float4*>(&Bs[buf][bp * PITCH + bk]);
    pbv[0] = make_float4(rb[0], rb[1], rb[2], rb[3]);
    pbv[1] = make_float4(rb[4], rb[5], rb[6], rb[7]);
  };

  f32x16 acc = {};
  const int nk = (G.red + BK - 1) / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  const int aoff = (wm * 32 + (lane & 31)) * PITCH + (lane >> 5) * 4;
  const int boff = (wn * 32 + (lane & 31)) * PITCH + (lane >> 5) * 4;
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

  // columns are pixels: consecutive lanes store consecutive pixels
  const int64_t p = pix0 + wn * 32 + (lane & 31);
  if (p >= G.pix) return;
  const int ow = TR ? G.W : G.Wo, oh = TR ? G.H : G.Ho;
  const int ov = (int)(p % ow);
  const int ou = (int)((p / ow) % oh);
  const int ob = (int)(p / ((int64_t)ow * oh));
  const int ych = TR ? G.cin : G.cout;
  const int chbase = grp * (TR ? G.c : G.og);
  const int64_t plane = (int64_t)oh * ow;
#pragma unroll
  for (int r = 0; r < 16; ++r) {
    const int ch = row0 + wm * 32 + acc_row(r, lane);
    if (ch < G.rows) y[((int64_t)ob * ych + chbase + ch) * plane + (int64_t)ou * ow + ov] = acc[r];
  }
}

}  // namespace

hipError_t launch_conv_apply(const orth_conv_apply_args* a, hipStream_t s) {
  const orth_conv_geom& g = a->geom;
  ApplyGeom G{};
  G.cin = g.cin;
  G.cout = g.cout;
  G.k = g.k;
  G.s = g.stride;
  G.d = g.dilation;
  G.g = g.groups;
  G.c = g.cin / g.groups;
  G.og = g.cout / g.groups;
  G.H = a->height;
  G.W = a->width;
  G.Ho = a->height / g.stride;
  G.Wo = a->width / g.stride;
  G.pl = (g.dilation * (g.k - 1) + 1 - g.stride) / 2;
  G.batch = a->batch;
  G.rows = a->transposed ? G.c : G.og;
  G.red = (a->transposed ? G.og : G.c) * g.k * g.k;
  G.pix = (int64_t)a->batch * (a->transposed ? (int64_t)G.H * G.W : (int64_t)G.Ho * G.Wo);
  G.kdtype = a->kernel_dtype;
  const dim3 grid((unsigned)((G.pix + 63) / 64), (unsigned)((G.rows + 63) / 64), (unsigned)g.groups);
  const char* name = a->transposed ? "conv_apply_transposed" : "conv_apply";
  timing_begin(name, s);
  if (a->transposed)
    hipLaunchKernelGGL(conv_apply_kernel<true>, grid, dim3(256), 0, s, G, a->kernel, a->x, a->y);
  else
    hipLaunchKernelGGL(conv_apply_kernel<false>, grid, dim3(256), 0, s, G, a->kernel, a->x, a->y);
  hipError_t e = hipGetLastError();
  timing_end(name, s);
  return e;
}

}  // namespace orth
