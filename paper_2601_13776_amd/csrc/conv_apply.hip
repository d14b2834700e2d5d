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

  uint32_t ra[EA];
  float rb[EB];
  auto gload = [&](int k0) {
    // kernel values
    {
      const int row = row0 + ar;
      int kk = k0 + ak;
      int ch = kk / kk2, tap = kk - ch * kk2;   // (input channel, tap) or (output channel, tap)
      // raw bits, widened at the LDS store (a conversion inside the guarded
      // load would make every load wait for its data)
#pragma unroll
      for (int j = 0; j < EA; ++j) {
        uint32_t v = 0;
        if (row < G.rows && kk < G.red) {
          const int64_t idx = TR ? ((int64_t)(grp * G.og + ch) * G.c + row) * kk2 + tap
                                 : (int64_t)(grp * G.og + row) * G.red + kk;
          v = G.kdtype == ORTH_BF16 ? (uint32_t) static_cast<const uint16_t*>(kern)[idx]
                                    : static_cast<const uint32_t*>(kern)[idx];
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
    // the raw values materialize here, after the MFMAs that the loads
    // overlap (otherwise the widening shift is moved into each guarded
    // load's block, where it waits for the data)
#pragma unroll
    for (int j = 0; j < EA; ++j) asm volatile("" : "+v"(ra[j]));
    float4* pa = reinterpret_cast<float4*>(&As[buf][ar * PITCH + ak]);
    const int sh = G.kdtype == ORTH_BF16 ? 16 : 0;
#pragma unroll
    for (int q = 0; q < EA / 4; ++q)
      pa[q] = make_float4(__uint_as_float(ra[4 * q] << sh), __uint_as_float(ra[4 * q + 1] << sh),
                          __uint_as_float(ra[4 * q + 2] << sh), __uint_as_float(ra[4 * q + 3] << sh));
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


// ---------------------------------------------------------------------------
// Halo-staged variant for k <= 3: per chunk of CB = 8 reduction channels,
// every input row that a 64-pixel tile needs (per output row it touches and
// per tap row) is staged once in LDS, circularly extended by the taps'
// reach, and all k^2 taps read from there.  The per-element global gather
// (index arithmetic, wraps and one load per tap) becomes one load per
// staged element (each read by up to k^2 taps x pixels) plus one LDS read
// per MFMA operand value; the offsets of every staged element are computed
// once per block.
//
// Staged layout per chunk: [ch][j][a][col], j the tile's output row slot
// (J of them), a the tap row, col in [0, WX):
//   forward    input row (s u + d a - pl) mod H of output row u, input
//              column (col - pl) mod W; pixel v at tap e reads col s v + d e
//   transposed row (u + pl - d a) mod H and column (col - span + pl) mod W of
//              the stride-upsampled input (zero off the stride lattice);
//              pixel v at tap e reads col v + span - d e
struct HaloGeom {
  int J;            // output rows a 64-pixel tile touches, at most
  int RC;           // staged rows per channel: J k
  int WX;           // staged columns
  int tpr_log2;     // threads per staged row: 1 << tpr_log2 >= WX
  int b_floats;     // CB RC WX rounded up to 4
  int nch;          // reduction channels per group (c forward, og transposed)
  int Hout, Wout;   // the output grid
  int nchunks;      // ceil(nch / CB)
};

// 64 x 64 pixels per workgroup (128 pixels, for twice the reuse of the
// staged kernel tile, measured 25-50% slower: more staged rows per chunk)
constexpr int HALO_CB = 8, HALO_BNP = 64, HALO_MAXE = 24;

// 64 output rows x BN pixels per workgroup; each wave 32 rows x BN / 2
// pixels (NI accumulators)
// VECA (fp32 kernel, rows of a multiple of four elements): each chunk's
// kernel tile is loaded as 16-byte vectors, with the offsets computed once
// per workgroup.  Forward: along the kernel rows.  Transposed: the chunk's
// channels o each hold the tile's 64 rows x k^2 taps contiguously
// (K[o][i][tap]), read as one run per o and scattered to the LDS rows.
template <bool TR, int KS, int BN, bool KBF16, bool VECA>
__global__ __launch_bounds__(256) void conv_apply_halo_kernel(ApplyGeom G, HaloGeom Hg,
                                                              const void* __restrict__ kern,
                                                              const float* __restrict__ x, float* __restrict__ y) {
  constexpr int CB = HALO_CB, KK = KS * KS, KCH = CB * KK, AP = KCH + 4, NI = BN / 64;
  constexpr int MAXA = (64 * KCH + 255) / 256;
  static_assert(KCH % 8 == 0, "a chunk is a whole number of 8-deep groups");
  extern __shared__ float smem[];
  float* const As = smem;
  float* const Bs = smem + 64 * AP;
  int* koff = reinterpret_cast<int*>(Bs + Hg.b_floats);

  const int grp = blockIdx.z;
  const int row0 = blockIdx.y * 64;
  const int64_t p0 = (int64_t)blockIdx.x * BN;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int span = G.d * (KS - 1);
  const int WX = Hg.WX, RC = Hg.RC;

  // LDS offset of tap (ch, a, e) relative to a pixel's base
  for (int kk = tid; kk < KCH; kk += 256) {
    const int ch = kk / KK, tap = kk % KK, a = tap / KS, e = tap % KS;
    koff[kk] = ch * RC * WX + a * WX + (TR ? -G.d * e : G.d * e);
  }
  // this lane's B-operand pixel: its base offset in a channel's block
  const int64_t first_row = p0 / Hg.Wout;
  int poff[NI];
#pragma unroll
  for (int ni = 0; ni < NI; ++ni) {
    const int64_t pn = p0 + wn * (BN / 2) + ni * 32 + (lane & 31);
    poff[ni] = 0;
    if (pn < G.pix) {
      const int64_t orow = pn / Hg.Wout;
      const int v = (int)(pn - orow * Hg.Wout);
      poff[ni] = (int)(orow - first_row) * KS * WX + (TR ? v + span : G.s * v);
    }
  }

  // staged elements of this thread: rows r = (tid >> tpr_log2) + i RPP,
  // column tid & (TPR - 1); offsets relative to the chunk's first channel
  const int rpp = 256 >> Hg.tpr_log2;
  const int scol = tid & ((1 << Hg.tpr_log2) - 1);
  const int srow0 = tid >> Hg.tpr_log2;
  const int64_t cplane = TR ? (int64_t)G.Ho * G.Wo : (int64_t)G.H * G.W;   // one channel of the source
  const int src_ch = TR ? G.cout : G.cin;
  const int ch_base = grp * Hg.nch;
  int boff[HALO_MAXE];
#pragma unroll
  for (int i = 0; i < HALO_MAXE; ++i) {
    boff[i] = -1;
    const int r = srow0 + i * rpp;
    if (r >= CB * RC || scol >= WX) continue;
    const int ch = r / RC, rr = r - ch * RC, j = rr / KS, a = rr - j * KS;
    const int64_t orow = first_row + j;
    const int64_t b = orow / Hg.Hout;
    const int u = (int)(orow - b * Hg.Hout);
    if (b >= G.batch) continue;
    int off;
    if (!TR) {
      const int sr = pmod(G.s * u + G.d * a - G.pl, G.H), sc = pmod(scol - G.pl, G.W);
      off = (int)(((b * src_ch + ch_base + ch) * cplane) + (int64_t)sr * G.W + sc);
    } else {
      const int R = pmod(u + G.pl - G.d * a, G.H), C = pmod(scol - span + G.pl, G.W);
      if (R % G.s || C % G.s) continue;
      off = (int)(((b * src_ch + ch_base + ch) * cplane) + (int64_t)(R / G.s) * G.Wo + C / G.s);
    }
    boff[i] = off;
  }
  // VECA: float4 f = tid + j 256 of the 64 x KCH tile: global offset (-1:
  // row past the end), column within the chunk, LDS offset
  // (transposed: f over CB runs of 64 KK floats; vcol = element within the
  // run, vlo = the run's channel o; elim = valid elements of a run)
  constexpr int Q4 = KCH / 4, NV = (64 * Q4 + 255) / 256, QR = 64 * KK / 4;
  int vgo[VECA ? NV : 1], vcol[VECA ? NV : 1], vlo[VECA ? NV : 1];
  const int elim = TR ? (G.rows - row0 < 64 ? G.rows - row0 : 64) * KK : 0;
  if constexpr (VECA && !TR) {
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int f = tid + j * 256, row = f / Q4, c4 = f - row * Q4;
      vgo[j] = f < 64 * Q4 && row0 + row < G.rows ? (grp * G.og + row0 + row) * G.red + c4 * 4 : -1;
      vcol[j] = c4 * 4;
      vlo[j] = f < 64 * Q4 ? row * AP + c4 * 4 : -1;
    }
  } else if constexpr (VECA && TR) {
#pragma unroll
    for (int j = 0; j < NV; ++j) {
      const int f = tid + j * 256, o = f / QR, w4 = f - o * QR;
      vgo[j] = f < 64 * Q4 ? ((grp * G.og + o) * G.c + row0) * KK + w4 * 4 : -1;
      vcol[j] = w4 * 4;
      vlo[j] = o;
    }
  }
  // kernel elements of this thread: e = tid + i 256 over 64 rows x KCH
  int aoff[VECA ? 1 : MAXA];
#pragma unroll
  for (int i = 0; i < (VECA ? 0 : MAXA); ++i) {
    aoff[i] = -1;
    const int e = tid + i * 256;
    if (e >= 64 * KCH) continue;
    const int row = e / KCH, col = e - (e / KCH) * KCH;
    if (row0 + row >= G.rows) continue;
    if (!TR)
      aoff[i] = (grp * G.og + row0 + row) * G.red + col;            // + ch0 KK per chunk
    else
      aoff[i] = ((grp * G.og + col / KK) * G.c + row0 + row) * KK + col % KK;   // + ch0 c KK
  }

  // one LDS stage: every chunk is staged (all loads in flight, then the
  // stores), computed between two barriers; the two or three other
  // workgroups on the compute unit overlap their staging with this one's
  // MFMAs
  // loads address a uniform base (this chunk's first channel) plus a
  // 32-bit byte offset (the host keeps both tensors below 2^30 elements),
  // one VGPR per address
  auto stage = [&](int ch0) {
    const int nvalid = Hg.nch - ch0;   // channels of this chunk that exist
    constexpr int kes = KBF16 ? 2 : 4;   // kernel element bytes
    const char* kq = static_cast<const char*>(kern) + (TR ? (int64_t)ch0 * G.c * KK : (int64_t)ch0 * KK) * kes;
    const char* xq = reinterpret_cast<const char*>(x + (int64_t)ch0 * cplane);
    // raw bits first, widened at the LDS store: a conversion inside the
    // guarded load would make every load wait for its data
    uint32_t ra[VECA ? 1 : MAXA];
    float4 va[VECA ? NV : 1];
    float rb[HALO_MAXE];
    if constexpr (VECA) {
      // valid elements of this thread's runs: forward, the chunk's valid
      // columns; transposed, the rows that exist (channels checked apart)
      const int lim = TR ? elim : (nvalid >= CB ? KCH : nvalid * KK);
      const float* kf = reinterpret_cast<const float*>(kq);
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        float4 v = make_float4(0.f, 0.f, 0.f, 0.f);
        const int col = vcol[j];
        if (vgo[j] >= 0 && (!TR || vlo[j] < nvalid)) {
          const float* p = kf + (uint32_t)vgo[j];
          if (col + 4 <= lim) {
            v = *reinterpret_cast<const float4*>(p);
          } else {
            if (col < lim) v.x = p[0];
            if (col + 1 < lim) v.y = p[1];
            if (col + 2 < lim) v.z = p[2];
          }
        }
        va[j] = v;
      }
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        asm volatile("" : "+v"(va[j].x));
        asm volatile("" : "+v"(va[j].y));
        asm volatile("" : "+v"(va[j].z));
        asm volatile("" : "+v"(va[j].w));
      }
    } else {
#pragma unroll
      for (int i = 0; i < MAXA; ++i) {
        const int e = tid + i * 256, col = e - (e / KCH) * KCH;
        uint32_t v = 0;
        if (aoff[i] >= 0 && col / KK < nvalid) {
          const uint32_t bo = (uint32_t)aoff[i] * (uint32_t)kes;
          if constexpr (KBF16)
            v = *reinterpret_cast<const uint16_t*>(kq + bo);
          else
            v = *reinterpret_cast<const uint32_t*>(kq + bo);
        }
        ra[i] = v;
      }
      // materialize the raw values after the guarded loads (otherwise the
      // widening shift is moved into each guarded block, where it waits)
#pragma unroll
      for (int i = 0; i < MAXA; ++i) asm volatile("" : "+v"(ra[i]));
    }
#pragma unroll
    for (int i = 0; i < HALO_MAXE; ++i) {
      const int r = srow0 + i * rpp;
      float v = 0.f;
      if (boff[i] >= 0 && r < nvalid * RC) v = *reinterpret_cast<const float*>(xq + (uint32_t)boff[i] * 4u);
      rb[i] = v;
    }
    if constexpr (VECA && !TR) {
#pragma unroll
      for (int j = 0; j < NV; ++j)
        if (vlo[j] >= 0) *reinterpret_cast<float4*>(&As[vlo[j]]) = va[j];
    } else if constexpr (VECA && TR) {
      // element e of channel o's run is row e / KK, tap e % KK
#pragma unroll
      for (int j = 0; j < NV; ++j) {
        if (vgo[j] < 0) continue;
        const float w[4] = {va[j].x, va[j].y, va[j].z, va[j].w};
#pragma unroll
        for (int q = 0; q < 4; ++q) {
          const int e = vcol[j] + q, row = e / KK;
          As[row * AP + vlo[j] * KK + (e - row * KK)] = w[q];
        }
      }
    } else {
#pragma unroll
      for (int i = 0; i < MAXA; ++i) {
        const int e = tid + i * 256;
        if (e < 64 * KCH) As[(e / KCH) * AP + e % KCH] = __uint_as_float(KBF16 ? ra[i] << 16 : ra[i]);
      }
    }
#pragma unroll
    for (int i = 0; i < HALO_MAXE; ++i) {
      const int r = srow0 + i * rpp;
      if (r < CB * RC && scol < WX) Bs[r * WX + scol] = rb[i];
    }
  };

  f32x16 acc[NI];
#pragma unroll
  for (int ni = 0; ni < NI; ++ni) acc[ni] = f32x16{};
  const int aread = (wm * 32 + (lane & 31)) * AP + (lane >> 5) * 4;
  for (int q = 0; q < Hg.nchunks; ++q) {
    stage(q * CB);
    __syncthreads();
#pragma unroll
    for (int g8 = 0; g8 < KCH / 8; ++g8) {
      // k = 8 g8 + 4 (lane / 32) + t for instruction t, on both operands
      const float4 a4 = *reinterpret_cast<const float4*>(&As[aread + g8 * 8]);
      const int4 k4 = *reinterpret_cast<const int4*>(&koff[g8 * 8 + (lane >> 5) * 4]);
#pragma unroll
      for (int ni = 0; ni < NI; ++ni) {
        const float* bs = Bs + poff[ni];
        acc[ni] = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.x, bs[k4.x], acc[ni], 0, 0, 0);
        acc[ni] = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.y, bs[k4.y], acc[ni], 0, 0, 0);
        acc[ni] = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.z, bs[k4.z], acc[ni], 0, 0, 0);
        acc[ni] = __builtin_amdgcn_mfma_f32_32x32x2f32(a4.w, bs[k4.w], acc[ni], 0, 0, 0);
      }
    }
    __syncthreads();
  }

  const int ow = Hg.Wout, oh = Hg.Hout;
  const int ych = TR ? G.cin : G.cout;
  const int chb = grp * (TR ? G.c : G.og);
  const int64_t plane = (int64_t)oh * ow;
#pragma unroll
  for (int ni = 0; ni < NI; ++ni) {
    const int64_t pn = p0 + wn * (BN / 2) + ni * 32 + (lane & 31);
    if (pn >= G.pix) continue;
    const int ov = (int)(pn % ow);
    const int ou = (int)((pn / ow) % oh);
    const int ob = (int)(pn / ((int64_t)ow * oh));
#pragma unroll
    for (int r = 0; r < 16; ++r) {
      const int ch = row0 + wm * 32 + acc_row(r, lane);
      if (ch < G.rows) y[((int64_t)ob * ych + chb + ch) * plane + (int64_t)ou * ow + ov] = acc[ni][r];
    }
  }
}

template <bool TR, int KS, bool KBF16, bool VECA>
hipError_t launch_halo_k(const ApplyGeom& G, const HaloGeom& Hg, dim3 grid, size_t lds, const orth_conv_apply_args* a,
                         hipStream_t s) {
  hipError_t e = hipFuncSetAttribute(
      reinterpret_cast<const void*>(&conv_apply_halo_kernel<TR, KS, HALO_BNP, KBF16, VECA>),
      hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  if (e != hipSuccess) return e;
  hipLaunchKernelGGL((conv_apply_halo_kernel<TR, KS, HALO_BNP, KBF16, VECA>), grid, dim3(256), lds, s, G, Hg,
                     a->kernel, a->x, a->y);
  return hipGetLastError();
}
template <bool TR, int KS>
hipError_t launch_halo(const ApplyGeom& G, const HaloGeom& Hg, dim3 grid, size_t lds, const orth_conv_apply_args* a,
                       hipStream_t s) {
  if (G.kdtype == ORTH_BF16) return launch_halo_k<TR, KS, true, false>(G, Hg, grid, lds, a, s);
  // 16-byte kernel loads: runs of a multiple of four floats, a 16-byte
  // aligned kernel
  const int64_t run = TR ? (int64_t)G.c * G.k * G.k : G.red;   // elements between consecutive runs
  if (run % 4 == 0 && (reinterpret_cast<uintptr_t>(a->kernel) & 15) == 0)
    return launch_halo_k<TR, KS, false, true>(G, Hg, grid, lds, a, s);
  return launch_halo_k<TR, KS, false, false>(G, Hg, grid, lds, a, s);
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
  // halo-staged kernel where it applies (k <= 3, staged rows within the
  // per-thread budget, three workgroups' LDS per compute unit)
  if (g.k <= 3) {
    const bool TRn = a->transposed != 0;
    HaloGeom Hg{};
    Hg.Hout = TRn ? G.H : G.Ho;
    Hg.Wout = TRn ? G.W : G.Wo;
    Hg.nch = TRn ? G.og : G.c;
    const int span = G.d * (G.k - 1);
    Hg.J = (Hg.Wout - 1 + HALO_BNP - 1) / Hg.Wout + 1;
    Hg.RC = Hg.J * G.k;
    Hg.WX = TRn ? G.W + span : G.s * (G.Wo - 1) + span + 1;
    int t = 0;
    while ((1 << t) < Hg.WX) ++t;
    Hg.tpr_log2 = t;
    Hg.b_floats = (HALO_CB * Hg.RC * Hg.WX + 3) / 4 * 4;
    Hg.nchunks = (Hg.nch + HALO_CB - 1) / HALO_CB;
    const int kch = HALO_CB * G.k * G.k;
    const size_t lds = (size_t)(64 * (kch + 4) + Hg.b_floats + kch) * sizeof(float);
    const int64_t src_elems = (int64_t)G.batch * (TRn ? (int64_t)G.cout * G.Ho * G.Wo : (int64_t)G.cin * G.H * G.W);
    const bool fits = t <= 8 && (HALO_CB * Hg.RC + (256 >> t) - 1) / (256 >> t) <= HALO_MAXE && lds <= 52 * 1024 &&
                      src_elems < ((int64_t)1 << 30) && (int64_t)G.cout * G.c * G.k * G.k < ((int64_t)1 << 30) &&
                      Hg.nch > 0;
    if (fits) {
      const dim3 grid((unsigned)((G.pix + HALO_BNP - 1) / HALO_BNP), (unsigned)((G.rows + 63) / 64),
                      (unsigned)g.groups);
      const char* name = TRn ? "conv_apply_transposed" : "conv_apply";
      timing_begin(name, s);
      hipError_t e;
      if (TRn)
        e = G.k == 1 ? launch_halo<true, 1>(G, Hg, grid, lds, a, s)
                     : G.k == 2 ? launch_halo<true, 2>(G, Hg, grid, lds, a, s) : launch_halo<true, 3>(G, Hg, grid, lds, a, s);
      else
        e = G.k == 1 ? launch_halo<false, 1>(G, Hg, grid, lds, a, s)
                     : G.k == 2 ? launch_halo<false, 2>(G, Hg, grid, lds, a, s)
                                : launch_halo<false, 3>(G, Hg, grid, lds, a, s);
      timing_end(name, s);
      return e;
    }
  }
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
