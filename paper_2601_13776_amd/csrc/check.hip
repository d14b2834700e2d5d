// Norm-preservation check of an explicit convolution kernel (Section 4 /
// Appendix C: an orthogonal convolution preserves the norm of every input).
// Direct circular-padded cross-correlation (or its transpose), one output
// element per thread; squared norms are reduced per block in fp64 and then
// summed per sample in a fixed order, so the result is deterministic.
#include "internal.h"

namespace orth {
namespace {

struct ConvGeomDev {
  int cin, cout, k, s, d, g, c, og;
  int hin, win, hout, wout;  // input and output grids of the forward conv
  int pl;                    // left/top padding
  int kdtype;
};

__device__ inline int pmod(int a, int m) {
  int r = a % m;
  return r < 0 ? r + m : r;
}

__device__ inline double block_sum(double v, double* red) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
  if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
  __syncthreads();
  return threadIdx.x == 0 ? ((red[0] + red[1]) + red[2]) + red[3] : 0.0;
}

// mode 0: ||conv(K, x_n)||^2 partials; 1: ||conv^T(K, x_n)||^2; 2: ||x_n||^2.
__global__ __launch_bounds__(256) void conv_sq_kernel(ConvGeomDev G, const void* __restrict__ kern,
                                                      const float* __restrict__ x, int mode, int64_t per_sample,
                                                      int64_t in_per_sample, double* __restrict__ partial,
                                                      int blocks_per_sample) {
  __shared__ double red[4];
  const int n = blockIdx.y;
  const int64_t e = (int64_t)blockIdx.x * 256 + threadIdx.x;
  double v2 = 0.0;
  if (e < per_sample) {
    const float* xn = x + (int64_t)n * in_per_sample;
    float v = 0.f;
    if (mode == 2) {
      v = xn[e];
    } else if (mode == 0) {
      // output element (o, u, w) of the forward conv
      const int w = (int)(e % G.wout);
      const int u = (int)((e / G.wout) % G.hout);
      const int o = (int)(e / ((int64_t)G.wout * G.hout));
      const int grp = o / G.og;
      for (int i = 0; i < G.c; ++i) {
        const float* xc = xn + (int64_t)(grp * G.c + i) * G.hin * G.win;
        for (int a = 0; a < G.k; ++a) {
          const int r = pmod(G.s * u + G.d * a - G.pl, G.hin);
          for (int b = 0; b < G.k; ++b) {
            const int q = pmod(G.s * w + G.d * b - G.pl, G.win);
            const float kv = load_as_f32(kern, (((int64_t)o * G.c + i) * G.k + a) * G.k + b, G.kdtype);
            v += kv * xc[(int64_t)r * G.win + q];
          }
        }
      }
    } else {
      // input-grid element (ci, p, q) of the transposed conv; x holds y
      const int q = (int)(e % G.win);
      const int p = (int)((e / G.win) % G.hin);
      const int ci = (int)(e / ((int64_t)G.win * G.hin));
      const int grp = ci / G.c, i = ci % G.c;
      for (int oo = 0; oo < G.og; ++oo) {
        const int o = grp * G.og + oo;
        const float* yo = xn + (int64_t)o * G.hout * G.wout;
        for (int a = 0; a < G.k; ++a) {
          const int tr = pmod(p - G.d * a + G.pl, G.hin);
          if (tr % G.s) continue;
          const int u = tr / G.s;
          for (int b = 0; b < G.k; ++b) {
            const int tc = pmod(q - G.d * b + G.pl, G.win);
            if (tc % G.s) continue;
            const int w = tc / G.s;
            const float kv = load_as_f32(kern, (((int64_t)o * G.c + i) * G.k + a) * G.k + b, G.kdtype);
            v += kv * yo[(int64_t)u * G.wout + w];
          }
        }
      }
    }
    v2 = (double)v * (double)v;
  }
  const double t = block_sum(v2, red);
  if (threadIdx.x == 0) partial[(int64_t)n * blocks_per_sample + blockIdx.x] = t;
}

__global__ __launch_bounds__(256) void conv_ratio_kernel(const double* __restrict__ num, int nb_num,
                                                         const double* __restrict__ den, int nb_den,
                                                         float* __restrict__ out) {
  __shared__ double red[4];
  const int n = blockIdx.x;
  double a = 0.0, b = 0.0;
  for (int i = threadIdx.x; i < nb_num; i += 256) a += num[(int64_t)n * nb_num + i];
  const double sa = block_sum(a, red);
  __syncthreads();
  for (int i = threadIdx.x; i < nb_den; i += 256) b += den[(int64_t)n * nb_den + i];
  const double sb = block_sum(b, red);
  if (threadIdx.x == 0) out[n] = (float)sqrt(sa / sb);
}

}  // namespace

// partial must hold batch * (blocks for the numerator + blocks for x) doubles.
hipError_t launch_conv_check(const orth_check_args* a, const void* kernel, const float* x, double* partial,
                             float* out, int adjoint, hipStream_t s) {
  ConvGeomDev G;
  G.cin = a->geom.cin;
  G.cout = a->geom.cout;
  G.k = a->geom.k;
  G.s = a->geom.stride;
  G.d = a->geom.dilation;
  G.g = a->geom.groups;
  G.c = G.cin / G.g;
  G.og = G.cout / G.g;
  G.pl = (G.d * (G.k - 1) + 1 - G.s) / 2;
  G.kdtype = a->kernel_dtype;
  if (!adjoint) {
    G.hin = a->height;
    G.win = a->width;
    G.hout = a->height / G.s;
    G.wout = a->width / G.s;
  } else {
    G.hout = a->height;
    G.wout = a->width;
    G.hin = a->height * G.s;
    G.win = a->width * G.s;
  }
  const int64_t in_ps = adjoint ? (int64_t)G.cout * G.hout * G.wout : (int64_t)G.cin * G.hin * G.win;
  const int64_t out_ps = adjoint ? (int64_t)G.cin * G.hin * G.win : (int64_t)G.cout * G.hout * G.wout;
  const int nb_out = (int)((out_ps + 255) / 256);
  const int nb_in = (int)((in_ps + 255) / 256);
  double* p_out = partial;
  double* p_in = partial + (int64_t)a->batch * nb_out;
  timing_begin("conv_check", s);
  hipLaunchKernelGGL(conv_sq_kernel, dim3(nb_out, a->batch), dim3(256), 0, s, G, kernel, x, adjoint ? 1 : 0,
                     out_ps, in_ps, p_out, nb_out);
  hipLaunchKernelGGL(conv_sq_kernel, dim3(nb_in, a->batch), dim3(256), 0, s, G, kernel, x, 2, in_ps, in_ps, p_in,
                     nb_in);
  hipLaunchKernelGGL(conv_ratio_kernel, dim3(a->batch), dim3(256), 0, s, p_out, nb_out, p_in, nb_in, out);
  hipError_t e = hipGetLastError();
  timing_end("conv_check", s);
  return e;
}

}  // namespace orth
