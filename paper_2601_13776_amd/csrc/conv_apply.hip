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
// once by one lane: deterministic, no atomics.  64 x 64 tiles (the kernel
// also builds 128-wide ones), four waves, K steps of 32 through two LDS
// stages.
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
// a mod m for a in [-m, 2m)
__device__ inline int wrap1(int a, int m) { return a < 0 ? a + m : (a >= m ? a - m : a); }

// WRAP1: every circular index lies within one period of the grid (the host
// checks d (k - 1) and the padding against H and W), so a conditional add
// or subtract replaces the integer modulo in the gather.
// BM x BN tiles (64 or 128 each): four waves of (BM / 2) x (BN / 2), that
// is (BM / 64) x (BN / 64) accumulators of 32 x 32 each.
template <bool TR, bool WRAP1, int BM, int BN>
__global__ __launch_bounds__(256) void conv_apply_kernel(ApplyGeom G, const void* __restrict__ kern,
                                                         const float* __restrict__ x, float* __restrict__ y) {
  constexpr int BK = 32, PITCH = BK + 4;
  static_assert((BM == 64 || BM == 128) && (BN == 64 || BN == 128), "tiles of 64 or 128");
  constexpr int EA = BM * BK / 256, EB = BN * BK / 256;   // elements per thread and k-step
  constexpr int MI = BM / 64, NI = BN / 64;
  __shared__ __attribute__((aligned(16))) float As[2][BM * PITCH];
  __shared__ __attribute__((aligned(16))) float Bs[2][BN * PITCH];
  const int grp = blockIdx.z;
  const int row0 = blockIdx.y * BM;
  const int64_t pix0 = (int64_t)blockIdx.x * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int kk2 = G.k * G.k;

  // first operand: the kernel, thread -> (row, EA consecutive k)
  const int ar = tid / (BK / EA), ak = (tid % (BK / EA)) * EA;
  // second operand: gathered pixels, thread -> (pixel, EB consecutive k)
  const int bp = tid % BN, bk = (tid / BN) * EB;
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

  float ra[EA], rb[EB];
  auto gload = [&](int k0) {
    // kernel values
    {
      const int row = row0 + ar;
      int kk = k0 + ak;
      int ch = kk / kk2, tap = kk - ch * kk2;   // (input channel, tap) or (output channel, tap)
#pragma unroll
      for (int j = 0; j < EA; ++j) {
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
      // window origin of this pixel; the tap moves it by +-(d a, d e)
      const int r0 = TR ? pu + G.pl : G.s * pu - G.pl, q0 = TR ? pv + G.pl : G.s * pv - G.pl;
      int da = G.d * a, de = G.d * e;
      const float* xg = xb + (int64_t)(grp * (TR ? G.og : G.c) + ch) * xplane;
#pragma unroll
      for (int j = 0; j < EB; ++j) {
        float v = 0.f;
        if (pix_ok && kk < G.red) {
          const int rr = TR ? r0 - da : r0 + da, qq = TR ? q0 - de : q0 + de;
          const int r = WRAP1 ? wrap1(rr, G.H) : pmod(rr, G.H);
          const int q = WRAP1 ? wrap1(qq, G.W) : pmod(qq, G.W);
          if (!TR) {
            v = xg[(int64_t)r * G.W + q];
          } else if (G.s == 1) {
            v = xg[(int64_t)r * G.Wo + q];
          } else if (r % G.s == 0 && q % G.s == 0) {
            v = xg[(int64_t)(r / G.s) * G.Wo + q / G.s];
          }
        }
        rb[j] = v;
        ++kk;
        de += G.d;
        if (++e == G.k) {
          e = 0;
          de = 0;
          da += G.d;
          if (++a == G.k) {
            a = 0;
            da = 0;
            ++ch;
            xg += xplane;
          }
        }
      }
    }
  };
  auto sstore = [&](int buf) {
    float4* pa = reinterpret_cast<float4*>(&As[buf][ar * PITCH + ak]);
#pragma unroll
    for (int q = 0; q < EA / 4; ++q) pa[q] = make_float4(ra[4 * q], ra[4 * q + 1], ra[4 * q + 2], ra[4 * q + 3]);
    float4* pbv = reinterpret_cast<float4*>(&Bs[buf][bp * PITCH + bk]);
#pragma unroll
    for (int q = 0; q < EB / 4; ++q) pbv[q] = make_float4(rb[4 * q], rb[4 * q + 1], rb[4 * q + 2], rb[4 * q + 3]);
  };

  f32x16 acc[MI][NI];
#pragma unroll
  for (int mi = 0; mi < MI; ++mi)
#pragma unroll
    for (int ni = 0; ni < NI; ++ni) acc[mi][ni] = f32x16{};
  const int nk = (G.red + BK - 1) / BK;
  gload(0);
  sstore(0);
  __syncthreads();
  const int aoff = (wm * (BM / 2) + (lane & 31)) * PITCH + (lane >> 5) * 4;
  const int boff = (wn * (BN / 2) + (lane & 31)) * PITCH + (lane >> 5) * 4;
  for (int kt = 0; kt < nk; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
    for (int gq = 0; gq < BK / 8; ++gq) {
      float4 a4[MI], b4[NI];
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
        a4[mi] = *reinterpret_cast<const float4*>(&As[buf][aoff + mi * 32 * PITCH + gq * 8]);
#pragma unroll
      for (int ni = 0; ni < NI; ++ni)
        b4[ni] = *reinterpret_cast<const float4*>(&Bs[buf][boff + ni * 32 * PITCH + gq * 8]);
#pragma unroll
      for (int mi = 0; mi < MI; ++mi)
#pragma unroll
        for (int ni = 0; ni < NI; ++ni) {
          f32x16& c = acc[mi][ni];
          c = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[mi].x, b4[ni].x, c, 0, 0, 0);
          c = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[mi].y, b4[ni].y, c, 0, 0, 0);
          c = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[mi].z, b4[ni].z, c, 0, 0, 0);
          c = __builtin_amdgcn_mfma_f32_32x32x2f32(a4[mi].w, b4[ni].w, c, 0, 0, 0);
        }
    }
    if (kt + 1 < nk) sstore(buf ^ 1);
    __syncthreads();
  }

  // columns are pixels: consecutive lanes store consecutive pixels
  const int ow = TR ? G.W : G.Wo, oh = TR ? G.H : G.Ho;
  const int ych = TR ? G.cin : G.cout;
  const int chbase = grp * (TR ? G.c : G.og);
  const int64_t plane = (int64_t)oh * ow;
#pragma unroll
  for (int ni = 0; ni < NI; ++ni) {
    const int64_t p = pix0 + wn * (BN / 2) + ni * 32 + (lane & 31);
    if (p >= G.pix) continue;
    const int ov = (int)(p % ow);
    const int ou = (int)((p / ow) % oh);
    const int ob = (int)(p / ((int64_t)ow * oh));
    float* yp = y + ((int64_t)ob * ych + chbase) * plane + (int64_t)ou * ow + ov;
#pragma unroll
    for (int mi = 0; mi < MI; ++mi)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int ch = row0 + wm * (BM / 2) + mi * 32 + acc_row(r, lane);
        if (ch < G.rows) yp[(int64_t)ch * plane] = acc[mi][ni][r];
      }
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
  // 64 x 64 tiles: measured on the CIFAR- and ImageNet-like stacks, 128 x
  // 128 tiles (four times the MFMA work per gathered element) were no
  // faster on wide layers and up to 2x slower where the small late grids
  // leave few tiles, and 16-deep k-steps won on neither
  constexpr int TB = 64;
  const dim3 grid((unsigned)((G.pix + TB - 1) / TB), (unsigned)((G.rows + TB - 1) / TB), (unsigned)g.groups);
  const char* name = a->transposed ? "conv_apply_transposed" : "conv_apply";
  // circular indices within one period: forward s u + d a - pl over
  // [-pl, H - s + d (k - 1) - pl], transposed p + pl - d a over
  // [pl - d (k - 1), H - 1 + pl] (likewise for W)
  const int span = G.d * (G.k - 1);
  const int lo = a->transposed ? G.pl - span : -G.pl;
  const int hi_h = a->transposed ? G.H - 1 + G.pl : G.H - G.s + span - G.pl;
  const int hi_w = a->transposed ? G.W - 1 + G.pl : G.W - G.s + span - G.pl;
  const bool w1 = lo >= -std::min(G.H, G.W) && hi_h < 2 * G.H && hi_w < 2 * G.W;
  timing_begin(name, s);
#define ORTH_APPLY(TR_, W1_, T_)                                                                              \
  hipLaunchKernelGGL((conv_apply_kernel<TR_, W1_, T_, T_>), grid, dim3(256), 0, s, G, a->kernel, a->x, a->y)
  if (a->transposed && w1) ORTH_APPLY(true, true, TB);
  else if (a->transposed) ORTH_APPLY(true, false, TB);
  else if (w1) ORTH_APPLY(false, true, TB);
  else ORTH_APPLY(false, false, TB);
#undef ORTH_APPLY
  hipError_t e = hipGetLastError();
  timing_end(name, s);
  return e;
}

}  // namespace orth
