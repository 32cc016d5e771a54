// Quantized convolution / FC (the C-Block contraction, Sec. "Integer-Only
// Inference"): implicit GEMM over NHWC int8 codes and KRSC int8 weights with
// int32 accumulation on the gfx950 int8 matrix cores (v_mfma_i32_32x32x32_i8).
//
//   rows    m = (n, oh, ow)          M = N * Ho * Wo
//   columns j = output channel       N = K
//   depth   k = (r, s, c), c fastest K = R * S * C
//
// A block computes a BM x BN tile with 4 waves of 64 x 64 (2 x 2 MFMA tiles),
// stepping through depth in 64-byte slabs staged in LDS (double buffered, the
// next slab's global loads in flight during the current slab's MFMAs).  No
// im2col buffer: each thread gathers its rows' 16-byte chunks straight from
// the NHWC tensor, with zero padding (code 0, or -128 for codes stored as
// u - 128, both meaning the value 0).
//
// Epilogue: for inputs stored as u - 128 the exact accumulator is restored by
// adding 128 * (sum of the filter's codes).  The int32 accumulators are
// stored; optionally the exact min / max of the C-Block values (bias, Scale,
// ReLU applied in fp64, exact below 2^53) are reduced for the FxP-QLayer.
#include <limits.h>
#include <math.h>

#include "values.hpp"

namespace fxpq {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BK = 64;
constexpr int LDS_STRIDE = 80;  // bytes per staged row: 64 + 16 to spread LDS banks

enum Loader { LD_FAST64 = 0, LD_GEN16 = 1, LD_RGB4 = 2 };

struct ConvArgs {
  const int8_t* x;
  const int8_t* w;
  const int32_t* colsum;
  int32_t* acc;
  int N, H, W, C, K, R, S, stride, pad, Ho, Wo;
  int M;        // rows
  int kdepth;   // R * S * C
  int wrow;     // bytes per weight row (kdepth, or padded to 64 for RGB4)
  int x_type;
  int want_mm;  // reduce min / max of the epilogue values
  SrcDev ep;    // kind == FXPQ_SRC_ACC when an epilogue is given
  int has_ep;
  double* mm_part;
};

template <int BM, int BN, int LOADER>
__global__ __launch_bounds__(256) void k_qconv(ConvArgs a) {
  constexpr int WN = BN / 64;   // waves along N
  constexpr int ACH = BM / 64;  // A chunks (16 B) per thread per slab
  constexpr int BCH = BN / 64;
  __shared__ __attribute__((aligned(16))) int8_t As[2][BM * LDS_STRIDE];
  __shared__ __attribute__((aligned(16))) int8_t Bs[2][BN * LDS_STRIDE];
  __shared__ int rs_tab[128];
  __shared__ double shd[8];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave / WN, wn = wave % WN;
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
  const int kc = tid & 3;

  int a_off = 0;
  if (a.x_type == FXPQ_U8OFF) a_off = 1;
  else if (a.x_type == FXPQ_C8) a_off = (a.has_ep && a.ep.fin->sign == 0) ? 1 : 0;
  const int padw = a_off ? (int)0x80808080 : 0;
  const v4i padv = {padw, padw, padw, padw};

  if (LOADER == LD_RGB4) {
    for (int i = tid; i < 128; i += 256) rs_tab[i] = (i < a.R * a.S) ? ((i / a.S) << 16) | (i % a.S) : -1;
    __syncthreads();
  }

  // Rows owned by this thread for A loads.
  const int8_t* abase[ACH];
  int ih0[ACH], iw0[ACH];
  bool aval[ACH];
  const int hw_out = a.Ho * a.Wo;
#pragma unroll
  for (int i = 0; i < ACH; ++i) {
    int row = m0 + (tid >> 2) + 64 * i;
    aval[i] = row < a.M;
    int rr = aval[i] ? row : a.M - 1;
    int n = rr / hw_out, rem = rr - n * hw_out;
    int oh = rem / a.Wo, ow = rem - oh * a.Wo;
    ih0[i] = oh * a.stride - a.pad;
    iw0[i] = ow * a.stride - a.pad;
    abase[i] = a.x + (int64_t)n * a.H * a.W * a.C;
  }
  const int8_t* bptr[BCH];
#pragma unroll
  for (int i = 0; i < BCH; ++i) {
    int col = n0 + (tid >> 2) + 64 * i;
    int cc = col < a.K ? col : a.K - 1;
    bptr[i] = a.w + (int64_t)cc * a.wrow;
  }

  v4i regA[ACH], regB[BCH];
  auto gload = [&](int kt) {
    const int k0 = kt * BK;
    if constexpr (LOADER == LD_FAST64) {
      int rs = k0 / a.C, c0 = k0 - rs * a.C;
      int r = rs / a.S, s = rs - r * a.S;
#pragma unroll
      for (int i = 0; i < ACH; ++i) {
        int ih = ih0[i] + r, iw = iw0[i] + s;
        bool ok = aval[i] && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
        const int8_t* p = abase[i] + ((int64_t)ih * a.W + iw) * a.C + c0 + kc * 16;
        regA[i] = ok ? *reinterpret_cast<const v4i*>(p) : padv;
      }
    } else if constexpr (LOADER == LD_GEN16) {
      int k = k0 + kc * 16;
      int rs = k / a.C, c0 = k - rs * a.C;
      int r = rs / a.S, s = rs - r * a.S;
      bool kin = k < a.kdepth;
#pragma unroll
      for (int i = 0; i < ACH; ++i) {
        int ih = ih0[i] + r, iw = iw0[i] + s;
        bool ok = kin && aval[i] && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
        const int8_t* p = abase[i] + ((int64_t)ih * a.W + iw) * a.C + c0;
        regA[i] = ok ? *reinterpret_cast<const v4i*>(p) : padv;
      }
    } else {  // LD_RGB4: four 4-byte pixels per 16-byte chunk
#pragma unroll
      for (int i = 0; i < ACH; ++i) {
        v4i v;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          int rs = (k0 + kc * 16 + 4 * j) >> 2;
          int t = (rs < 128) ? rs_tab[rs] : -1;
          int word = padw;
          if (t >= 0 && aval[i]) {
            int ih = ih0[i] + (t >> 16), iw = iw0[i] + (t & 0xFFFF);
            if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W)
              word = *reinterpret_cast<const int*>(abase[i] + ((int64_t)ih * a.W + iw) * 4);
          }
          v[j] = word;
        }
        regA[i] = v;
      }
    }
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      int k = k0 + kc * 16;
      if (LOADER == LD_GEN16 && k >= a.kdepth)
        regB[i] = v4i{0, 0, 0, 0};
      else
        regB[i] = *reinterpret_cast<const v4i*>(bptr[i] + k);
    }
  };
  auto lstore = [&](int buf) {
#pragma unroll
    for (int i = 0; i < ACH; ++i)
      *reinterpret_cast<v4i*>(&As[buf][((tid >> 2) + 64 * i) * LDS_STRIDE + kc * 16]) = regA[i];
#pragma unroll
    for (int i = 0; i < BCH; ++i)
      *reinterpret_cast<v4i*>(&Bs[buf][((tid >> 2) + 64 * i) * LDS_STRIDE + kc * 16]) = regB[i];
  };

  v16i acc[2][2];
#pragma unroll
  for (int mi = 0; mi < 2; ++mi)
#pragma unroll
    for (int ni = 0; ni < 2; ++ni)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[mi][ni][e] = 0;

  const int ktiles = (a.kdepth + BK - 1) / BK;
  gload(0);
  lstore(0);
  __syncthreads();
  for (int kt = 0; kt < ktiles; ++kt) {
    const int buf = kt & 1;
    if (kt + 1 < ktiles) gload(kt + 1);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      v4i af[2], bf[2];
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
        af[mi] = *reinterpret_cast<const v4i*>(
            &As[buf][(wm * 64 + mi * 32 + (lane & 31)) * LDS_STRIDE + kk * 32 + (lane >> 5) * 16]);
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        bf[ni] = *reinterpret_cast<const v4i*>(
            &Bs[buf][(wn * 64 + ni * 32 + (lane & 31)) * LDS_STRIDE + kk * 32 + (lane >> 5) * 16]);
#pragma unroll
      for (int mi = 0; mi < 2; ++mi)
#pragma unroll
        for (int ni = 0; ni < 2; ++ni)
          acc[mi][ni] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[mi], bf[ni], acc[mi][ni], 0, 0, 0);
    }
    if (kt + 1 < ktiles) lstore(buf ^ 1);
    __syncthreads();
  }

  // ---- epilogue ----
  double mn = INFINITY, mx = -INFINITY;
  EpiU eu;
  if (a.want_mm) eu = epi_uniform(a.ep);
#pragma unroll
  for (int ni = 0; ni < 2; ++ni) {
    const int col = n0 + wn * 64 + ni * 32 + (lane & 31);
    const int cc = col < a.K ? col : a.K - 1;
    const int corr = a_off ? 128 * a.colsum[cc] : 0;
    double Mc = 1.0, Ac = 0.0;
    if (a.want_mm) epi_channel(a.ep, eu, cc, Mc, Ac);
#pragma unroll
    for (int mi = 0; mi < 2; ++mi) {
#pragma unroll
      for (int e = 0; e < 16; ++e) {
        const int row = m0 + wm * 64 + mi * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
        const int v = acc[mi][ni][e] + corr;
        if (row < a.M && col < a.K) {
          a.acc[(int64_t)row * a.K + col] = v;
          if (a.want_mm) {
            double val = fma((double)v, Mc, Ac);
            if (a.ep.ep_relu) val = fmax(val, 0.0);
            mn = fmin(mn, val);
            mx = fmax(mx, val);
          }
        }
      }
    }
  }
  if (!a.want_mm) return;
  mn = block_reduce(mn, OpMin(), shd);
  mx = block_reduce(mx, OpMax(), shd);
  const int bid = blockIdx.y * gridDim.x + blockIdx.x;
  if (tid == 0) {
    a.mm_part[2 * bid] = mn;
    a.mm_part[2 * bid + 1] = mx;
  }
}

template <int BM, int BN>
static void conv_dispatch_loader(int loader, dim3 grid, hipStream_t st, const ConvArgs& a) {
  if (loader == LD_FAST64)
    k_qconv<BM, BN, LD_FAST64><<<grid, 256, 0, st>>>(a);
  else if (loader == LD_GEN16)
    k_qconv<BM, BN, LD_GEN16><<<grid, 256, 0, st>>>(a);
  else
    k_qconv<BM, BN, LD_RGB4><<<grid, 256, 0, st>>>(a);
}

hipError_t launch_conv(const Ctx& c, const fxpq_conv_desc& d, const void* x, int x_type,
                       const int8_t* w, const int32_t* colsum, const SrcDev* ep, int32_t* acc,
                       double* d_minmax) {
  ConvArgs a;
  a.x = static_cast<const int8_t*>(x);
  a.w = w;
  a.colsum = colsum;
  a.acc = acc;
  a.N = d.n; a.H = d.h; a.W = d.w; a.C = d.c; a.K = d.k; a.R = d.r; a.S = d.s;
  a.stride = d.stride; a.pad = d.pad;
  a.Ho = (d.h + 2 * d.pad - d.r) / d.stride + 1;
  a.Wo = (d.w + 2 * d.pad - d.s) / d.stride + 1;
  a.M = d.n * a.Ho * a.Wo;
  a.kdepth = d.r * d.s * d.c;
  int loader = (d.c % 64 == 0) ? LD_FAST64 : (d.c == 4 ? LD_RGB4 : LD_GEN16);
  a.wrow = (loader == LD_RGB4) ? (a.kdepth + 63) / 64 * 64 : a.kdepth;
  if (loader == LD_RGB4) a.kdepth = a.wrow;
  a.x_type = x_type;
  a.has_ep = ep != nullptr;
  if (ep) a.ep = *ep;
  a.want_mm = (ep != nullptr && d_minmax != nullptr);
  a.mm_part = c.sc.minmax_part;
  bool timed = timer_begin(c, FXPQ_TIMER_QCONV);
  dim3 grid;
  if (d.k <= 64) {
    grid = dim3((a.M + 255) / 256, (d.k + 63) / 64);
    conv_dispatch_loader<256, 64>(loader, grid, c.stream, a);
  } else {
    grid = dim3((a.M + 127) / 128, (d.k + 127) / 128);
    conv_dispatch_loader<128, 128>(loader, grid, c.stream, a);
  }
  timer_end(c, timed, 2.0 * (double)a.M * (double)d.k * (double)(d.r * d.s * d.c));
  if (a.want_mm) return launch_minmax_fin(c, a.mm_part, (int)(grid.x * grid.y), d_minmax);
  return hipGetLastError();
}

}  // namespace fxpq
