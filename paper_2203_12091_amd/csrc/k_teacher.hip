// FP32 teacher: the full-precision network whose activations are the
// reference of the layer error in the per-layer sensitivity sweep (Sec.
// "Data-Structures Sensitivity to Quantization"; the full-precision model as
// teacher, Sec. "Quantization Parameters Optimization").  Its arithmetic is
// fixed so that any implementation gets the same bits:
//   conv / FC   fp64 sum of the fp32 x fp32 products (exact in fp64) in the
//               order r, s, c with padded taps skipped, rounded once to fp32;
//   BN-as-Scale one fp32 fma per value; bias one fp32 add;
//   ReLU        every value <= 0 becomes +0;
//   residual    one fp32 add, then ReLU;
//   max-pool    the largest in-range tap;
//   avg-pool    (float)(fp64 sum in pixel order / pixels).
// Reference data only: computed once per sweep, outside its timing.
#include <math.h>

#include "common.hpp"

namespace fxpq {

// x NHWC fp32, w RSCK fp32 (output channels contiguous), y NHWK fp32; one
// thread per output, output channels fastest so a wave reads one input
// pixel and 64 consecutive filters.
__global__ __launch_bounds__(256) void k_teacher_conv(const float* x, const float* w, float* y,
                                                      int N, int H, int W, int C, int K, int R,
                                                      int S, int stride, int pad, int Ho, int Wo) {
  const int64_t total = (int64_t)N * Ho * Wo * K;
  for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total;
       o += (int64_t)gridDim.x * blockDim.x) {
    const int k = (int)(o % K);
    int64_t pix = o / K;
    const int ow = (int)(pix % Wo);
    pix /= Wo;
    const int oh = (int)(pix % Ho);
    const int n = (int)(pix / Ho);
    double acc = 0.0;
    for (int r = 0; r < R; ++r) {
      const int ih = oh * stride - pad + r;
      if (ih < 0 || ih >= H) continue;
      for (int s = 0; s < S; ++s) {
        const int iw = ow * stride - pad + s;
        if (iw < 0 || iw >= W) continue;
        const float* xp = x + (((int64_t)n * H + ih) * W + iw) * C;
        const float* wp = w + ((int64_t)(r * S + s) * C) * K + k;
        for (int c = 0; c < C; ++c) acc = fma((double)xp[c], (double)wp[(int64_t)c * K], acc);
      }
    }
    y[o] = (float)acc;
  }
}

// Per channel (innermost, `channels` of them): fmaf(t, a1, a2) or t + bias,
// then ReLU.  In place allowed.
__global__ __launch_bounds__(256) void k_teacher_affine(const float* t, int64_t n, int channels,
                                                        const float* a1, const float* a2,
                                                        const float* bias, int relu, float* y) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(i % channels);
    float v = t[i];
    if (a1) v = fmaf(v, a1[c], a2[c]);
    else if (bias) v = v + bias[c];
    if (relu) v = v > 0.0f ? v : 0.0f;
    y[i] = v;
  }
}

__global__ __launch_bounds__(256) void k_teacher_add(const float* a, const float* b, int64_t n,
                                                     int relu, float* y) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    float v = a[i] + b[i];
    if (relu) v = v > 0.0f ? v : 0.0f;
    y[i] = v;
  }
}

// NHWC max-pool; out-of-range taps are skipped.
__global__ __launch_bounds__(256) void k_teacher_maxpool(const float* x, float* y, int N, int H,
                                                         int W, int C, int ks, int stride, int pad,
                                                         int Ho, int Wo) {
  const int64_t total = (int64_t)N * Ho * Wo * C;
  for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total;
       o += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(o % C);
    int64_t pix = o / C;
    const int ow = (int)(pix % Wo);
    pix /= Wo;
    const int oh = (int)(pix % Ho);
    const int n = (int)(pix / Ho);
    float m = -INFINITY;
    for (int r = 0; r < ks; ++r) {
      const int ih = oh * stride - pad + r;
      if (ih < 0 || ih >= H) continue;
      for (int s = 0; s < ks; ++s) {
        const int iw = ow * stride - pad + s;
        if (iw < 0 || iw >= W) continue;
        m = fmaxf(m, x[(((int64_t)n * H + ih) * W + iw) * C + c]);
      }
    }
    y[o] = m;
  }
}

// x [n][hw][c] -> y [n][c].
__global__ __launch_bounds__(256) void k_teacher_avgpool(const float* x, float* y, int N, int hw,
                                                         int C) {
  const int64_t total = (int64_t)N * C;
  for (int64_t o = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; o < total;
       o += (int64_t)gridDim.x * blockDim.x) {
    const int c = (int)(o % C);
    const int n = (int)(o / C);
    double acc = 0.0;
    for (int p = 0; p < hw; ++p) acc = acc + (double)x[((int64_t)n * hw + p) * C + c];
    y[o] = (float)(acc / (double)hw);
  }
}

static int elem_grid(int64_t n) {
  int64_t b = (n + 255) / 256;
  return (int)(b < 65536 ? (b < 1 ? 1 : b) : 65536);
}

hipError_t launch_teacher_conv(const Ctx& c, const fxpq_conv_desc& d, const float* x,
                               const float* w, float* y) {
  const int Ho = (d.h + 2 * d.pad - d.r) / d.stride + 1;
  const int Wo = (d.w + 2 * d.pad - d.s) / d.stride + 1;
  const int64_t total = (int64_t)d.n * Ho * Wo * d.k;
  k_teacher_conv<<<elem_grid(total), 256, 0, c.stream>>>(x, w, y, d.n, d.h, d.w, d.c, d.k, d.r,
                                                         d.s, d.stride, d.pad, Ho, Wo);
  return hipGetLastError();
}

hipError_t launch_teacher_affine(const Ctx& c, const float* t, int64_t n, int channels,
                                 const float* a1, const float* a2, const float* bias, int relu,
                                 float* y) {
  k_teacher_affine<<<elem_grid(n), 256, 0, c.stream>>>(t, n, channels, a1, a2, bias, relu, y);
  return hipGetLastError();
}

hipError_t launch_teacher_add(const Ctx& c, const float* a, const float* b, int64_t n, int relu,
                              float* y) {
  k_teacher_add<<<elem_grid(n), 256, 0, c.stream>>>(a, b, n, relu, y);
  return hipGetLastError();
}

hipError_t launch_teacher_maxpool(const Ctx& c, const float* x, int n, int h, int w, int ch,
                                  int ks, int stride, int pad, float* y) {
  const int Ho = (h + 2 * pad - ks) / stride + 1, Wo = (w + 2 * pad - ks) / stride + 1;
  k_teacher_maxpool<<<elem_grid((int64_t)n * Ho * Wo * ch), 256, 0, c.stream>>>(
      x, y, n, h, w, ch, ks, stride, pad, Ho, Wo);
  return hipGetLastError();
}

hipError_t launch_teacher_avgpool(const Ctx& c, const float* x, int n, int hw, int ch, float* y) {
  k_teacher_avgpool<<<elem_grid((int64_t)n * ch), 256, 0, c.stream>>>(x, y, n, hw, ch);
  return hipGetLastError();
}

}  // namespace fxpq
