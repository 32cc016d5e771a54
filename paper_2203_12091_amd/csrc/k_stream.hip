// Streaming kernels of the hot path: min/max of FxP-QLayer inputs, the DFX
// quantizer / FxP-QLayer requantization (Eq. 10-12), the layer error
// (Eq. 14, 16, 18), pooling on codes and small helpers.  All HBM-bound: each
// thread moves 16-byte groups, grid-strided with a stride that keeps its
// channels fixed (see values.hpp).
#include <math.h>

#include <mutex>
#include <unordered_map>

#include "fls.hpp"

namespace fxpq {

// ----------------------------------------------------------------------------
// Grid sizing shared by the streaming launchers.
// ----------------------------------------------------------------------------
static int64_t gcd64(int64_t a, int64_t b) {
  while (b) {
    int64_t t = a % b;
    a = b;
    b = t;
  }
  return a;
}

int resident_blocks(const Ctx& c, const void* kernel) {
  static std::mutex mu;
  static std::unordered_map<const void*, int> per_cu;
  int b = 0;
  {
    std::lock_guard<std::mutex> lock(mu);
    auto it = per_cu.find(kernel);
    if (it != per_cu.end()) {
      b = it->second;
    } else {
      if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&b, kernel, kThreads, 0) != hipSuccess) b = 0;
      per_cu[kernel] = b;
    }
  }
  return b > 0 ? b * c.cus : 0;
}

// One block per kThreads groups of `vec` values, capped at one full round of
// resident blocks (the grid-stride loop covers the rest: a partial second
// round would leave most of the chip idle at its end).  When a bound on the
// values per thread asks for more blocks, whole rounds.  Then rounded so the
// grid stride is a multiple of `channels`.
int stream_grid(int64_t n, int channels, int64_t max_per_thread, int vec, int resident) {
  const int64_t cap = resident > 0 ? resident : kMaxStreamBlocks;
  int64_t groups = (n + vec - 1) / vec;
  int64_t blocks = (groups + kThreads - 1) / kThreads;
  if (blocks > cap) blocks = cap;
  if (max_per_thread > 0) {
    int64_t need = (n + (int64_t)kThreads * max_per_thread - 1) / ((int64_t)kThreads * max_per_thread);
    if (need > blocks) blocks = (need + cap - 1) / cap * cap;
  }
  if (blocks < 1) blocks = 1;
  if (channels > 0) {
    int64_t g = channels / gcd64(channels, (int64_t)vec * kThreads);
    blocks = (blocks + g - 1) / g * g;
  }
  return (int)blocks;
}

// ----------------------------------------------------------------------------
// min / max
// ----------------------------------------------------------------------------
template <int KIND, int DT>
__global__ __launch_bounds__(kThreads) void k_minmax(SrcDev s, int64_t n, double* part,
                                                     unsigned* flags) {
  __shared__ double sh[8];
  using PK = Pack<KIND, DT>;
  const int64_t gtid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  ThreadVals<PK::V> t;
  thread_vals_init<KIND, DT>(s, (int64_t)blockIdx.x * kThreads * PK::V, t);
  double mn = INFINITY, mx = -INFINITY;
  bool bad = false;
  const int64_t nfull = n - n % PK::EP;
  bool done = false;
  if constexpr (KIND == FXPQ_SRC_ADD) {
    if (t.sa <= kAddMaxShift && t.sb <= kAddMaxShift) {
      // eltwise sums in integers: value = relu(x + k) is non-decreasing in
      // x = (a << sa) + (b << sb) (|x| < 2^30), so the extremes of the values
      // are those of x, finished once
      int lo = INT_MAX, hi = INT_MIN;
      stream_packets<KIND, DT, false, 2, false, true>(
          s, n, t, [&](const Raw<KIND, DT>& r, int64_t, int) {
            const int wa[4] = {r.a.x, r.a.y, r.a.z, r.a.w};
            const int wb[4] = {r.b.x, r.b.y, r.b.z, r.b.w};
#pragma unroll
            for (int j = 0; j < PK::EP; ++j) {
              const int ca = (wa[j / 4] << (24 - 8 * (j % 4))) >> 24;
              const int cb = (wb[j / 4] << (24 - 8 * (j % 4))) >> 24;
              const int x = (ca << t.sa) + (cb << t.sb);
              lo = min(lo, x);
              hi = max(hi, x);
            }
          });
      if (lo <= hi) {
        mn = fmax((double)lo + t.k, t.relo);
        mx = fmax((double)hi + t.k, t.relo);
      }
      done = true;
    }
  }
  if (!done)
    stream_values<KIND, DT>(s, n, t, [&](double v, int64_t) {
      mn = fmin(mn, v);
      mx = fmax(mx, v);
      if (KIND == FXPQ_SRC_F32) bad |= !isfinite(v);
    });
  if (gtid == 0) {
    for (int64_t i = nfull; i < n; ++i) {
      double v = load1<KIND, DT>(s, i);
      mn = fmin(mn, v);
      mx = fmax(mx, v);
      if (KIND == FXPQ_SRC_F32) bad |= !isfinite(v);
    }
  }
  int any_bad = __syncthreads_or(bad);
  mn = block_reduce(mn, OpMin(), sh);
  mx = block_reduce(mx, OpMax(), sh);
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = any_bad ? NAN : mn;
    part[2 * blockIdx.x + 1] = mx;
    if (any_bad) raise_flag(flags, FXPQ_FLAG_NONFINITE);
  }
}

// One block: reduces nb (min, max) partials; a NaN partial marks non-finite input.
constexpr int kMmFinThreads = 1024;

__global__ __launch_bounds__(kMmFinThreads) void k_minmax_fin(const double* part, int nb, double* out) {
  __shared__ double sh[kMmFinThreads / 64];
  double a = INFINITY, b = -INFINITY;
  bool nan_seen = false;
#pragma unroll 4
  for (int i = threadIdx.x; i < nb; i += kMmFinThreads) {
    double p0 = part[2 * i], p1 = part[2 * i + 1];
    nan_seen |= isnan(p0);
    a = fmin(a, p0);
    b = fmax(b, p1);
  }
  int nan_any = __syncthreads_or(nan_seen);
  a = block_reduce(a, OpMin(), sh);
  b = block_reduce(b, OpMax(), sh);
  if (threadIdx.x == 0) {
    out[0] = nan_any ? NAN : a;
    out[1] = b;
  }
}

hipError_t launch_minmax_fin(const Ctx& c, const double* part, int nb, double* out) {
  k_minmax_fin<<<1, kMmFinThreads, 0, c.stream>>>(part, nb, out);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Quantize / requantize.
// ----------------------------------------------------------------------------
// dst[i] = src[i] for i < n over the grid (both 16-byte aligned).
__device__ inline void copy_bytes(const int8_t* src, int8_t* dst, int64_t n) {
  const int64_t n16 = n / 16;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n16; i += stride)
    reinterpret_cast<int4*>(dst)[i] = reinterpret_cast<const int4*>(src)[i];
  if (blockIdx.x == 0 && threadIdx.x < n % 16) dst[16 * n16 + threadIdx.x] = src[16 * n16 + threadIdx.x];
}

template <int OUT, int V>
__device__ inline void storev(void* codes, int64_t i, const int c[V]) {
  if constexpr (OUT == FXPQ_I8 || OUT == FXPQ_U8OFF || OUT == FXPQ_C8) {
    if constexpr (V == 2) {
      *reinterpret_cast<uint16_t*>(static_cast<int8_t*>(codes) + i) =
          (uint16_t)((c[0] & 0xFF) | ((c[1] & 0xFF) << 8));
    } else {
      uint32_t w[V / 4];
#pragma unroll
      for (int q = 0; q < V / 4; ++q)
        w[q] = (uint32_t)(c[4 * q] & 0xFF) | ((uint32_t)(c[4 * q + 1] & 0xFF) << 8) |
               ((uint32_t)(c[4 * q + 2] & 0xFF) << 16) | ((uint32_t)(c[4 * q + 3] & 0xFF) << 24);
      uint32_t* dst = reinterpret_cast<uint32_t*>(static_cast<int8_t*>(codes) + i);
      if constexpr (V == 16) {
        *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
      } else {
        dst[0] = w[0];
      }
    }
  } else if constexpr (OUT == FXPQ_I16) {
    uint32_t* dst = reinterpret_cast<uint32_t*>(static_cast<int16_t*>(codes) + i);
#pragma unroll
    for (int q = 0; q < V / 2; ++q)
      dst[q] = (uint32_t)(c[2 * q] & 0xFFFF) | ((uint32_t)(c[2 * q + 1] & 0xFFFF) << 16);
  } else {
    int32_t* dst = static_cast<int32_t*>(codes) + i;
    if constexpr (V % 4 == 0) {
#pragma unroll
      for (int q = 0; q < V / 4; ++q)
        reinterpret_cast<int4*>(dst)[q] = make_int4(c[4 * q], c[4 * q + 1], c[4 * q + 2], c[4 * q + 3]);
    } else {
#pragma unroll
      for (int q = 0; q < V / 2; ++q) reinterpret_cast<int2*>(dst)[q] = make_int2(c[2 * q], c[2 * q + 1]);
    }
  }
}

template <int OUT>
__device__ inline void store1(void* codes, int64_t i, int c) {
  if constexpr (OUT == FXPQ_I8 || OUT == FXPQ_U8OFF || OUT == FXPQ_C8)
    static_cast<int8_t*>(codes)[i] = (int8_t)c;
  else if constexpr (OUT == FXPQ_I16)
    static_cast<int16_t*>(codes)[i] = (int16_t)c;
  else
    static_cast<int32_t*>(codes)[i] = c;
}

template <int KIND, int DT, int OUT>
__global__ __launch_bounds__(kThreads) void k_requant(SrcDev s, int64_t n, const fxpq_fmt* fmt,
                                                      void* codes, unsigned* flags,
                                                      const FlsPlan* gate, const int8_t* alt) {
  if (gate && gate->spec && fmt->status == 0) {
    // fused FxP-QLayer: the search already wrote the codes of its window
    const int fl = fmt->fl;
    if (fl == gate->spec_fl[0]) return;
    if (fl == gate->spec_fl[1]) {
      copy_bytes(alt, static_cast<int8_t*>(codes), n);
      return;
    }
  }
  const int sv = src_scale(s);
  const QFmt q = qfmt_setup<OUT>(fmt, sv, flags);
  if (!q.ok) return;
  if constexpr (KIND == FXPQ_SRC_INT && DT == FXPQ_I64) {
    // int64 values (wide C-Blocks, pooled sums): the exact integer quantizer
    const int sh = fmt->fl - sv;
    const int64_t* x = static_cast<const int64_t*>(s.x);
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * kThreads)
      store1<OUT>(codes, i, quant_one_i64(x[i], sh, q));
    return;
  }
  using PK = Pack<KIND, DT>;
  const int64_t gtid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  ThreadVals<PK::V> t;
  thread_vals_init<KIND, DT>(s, (int64_t)blockIdx.x * kThreads * PK::V, t);
  const int64_t nfull = n - n % PK::EP;
  // fp32 sources (quantize, Eq. 10): NaN / Inf has no code; it raises the
  // sticky non-finite flag (its code is unspecified)
  bool bad = false;
  stream_packets<KIND, DT>(s, n, t, [&](const double* v, int64_t i0, int) {
    int c[PK::EP];
#pragma unroll
    for (int j = 0; j < PK::EP; ++j) {
      if constexpr (KIND == FXPQ_SRC_F32) bad |= !isfinite(v[j]);
      c[j] = quant_one<OUT>(v[j], q);
    }
    storev<OUT, PK::EP>(codes, i0, c);
  });
  if (gtid == 0) {
    for (int64_t i = nfull; i < n; ++i) {
      const double v = load1<KIND, DT>(s, i);
      if constexpr (KIND == FXPQ_SRC_F32) bad |= !isfinite(v);
      store1<OUT>(codes, i, quant_one<OUT>(v, q));
    }
  }
  if constexpr (KIND == FXPQ_SRC_F32) {
    if (bad) raise_flag(flags, FXPQ_FLAG_NONFINITE);
  }
}

// ----------------------------------------------------------------------------
// Layer error.
// ----------------------------------------------------------------------------
template <int CT>
__device__ inline double code_at(const void* codes, int64_t i) {
  if constexpr (CT == FXPQ_I16) return static_cast<const int16_t*>(codes)[i];
  else if constexpr (CT == FXPQ_I32) return static_cast<const int32_t*>(codes)[i];
  else if constexpr (CT == FXPQ_U32) return static_cast<const uint32_t*>(codes)[i];
  else if constexpr (CT == FXPQ_F32) return static_cast<const float*>(codes)[i];
  else return static_cast<const int8_t*>(codes)[i];
}

template <int CT>
__global__ __launch_bounds__(kThreads) void k_layer_error(const float* ref, const void* codes,
                                                          const fxpq_fmt* fmt, int64_t n,
                                                          double* part) {
  __shared__ double sh[8];
  // fp32 values (CT == FXPQ_F32) are compared as they are
  const double step = (CT == FXPQ_F32) ? 1.0 : ldexp(1.0, -fmt->fl);
  const double off = (CT == FXPQ_U8OFF || (CT == FXPQ_C8 && fmt->sign == 0)) ? 128.0 : 0.0;
  const int64_t gtid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  const int64_t stride = (int64_t)gridDim.x * kThreads;
  double sse = 0.0, mn = INFINITY, mx = -INFINITY, s1 = 0.0, s2 = 0.0;
  auto add = [&](double r, double c) {
    const double d = r - (c + off) * step;
    sse = fma(d, d, sse);
    mn = fmin(mn, r);
    mx = fmax(mx, r);
    s1 += r;
    s2 = fma(r, r, s2);
  };
  // four grid strides per iteration: their loads are issued together
  int64_t i = gtid;
  for (; i + 3 * stride < n; i += 4 * stride) {
    double r[4], c[4];
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      r[k] = ref[i + k * stride];
      c[k] = code_at<CT>(codes, i + k * stride);
    }
#pragma unroll
    for (int k = 0; k < 4; ++k) add(r[k], c[k]);
  }
  for (; i < n; i += stride) add(ref[i], code_at<CT>(codes, i));
  sse = block_reduce(sse, OpAddD(), sh);
  mn = block_reduce(mn, OpMin(), sh);
  mx = block_reduce(mx, OpMax(), sh);
  s1 = block_reduce(s1, OpAddD(), sh);
  s2 = block_reduce(s2, OpAddD(), sh);
  if (threadIdx.x == 0) {
    double* p = part + 5 * blockIdx.x;
    p[0] = sse; p[1] = mn; p[2] = mx; p[3] = s1; p[4] = s2;
  }
}

__global__ __launch_bounds__(kThreads) void k_layer_error_fin(const double* part, int nb, int64_t n,
                                                              double* out) {
  __shared__ double sh[8];
  double a = 0.0, b = INFINITY, c = -INFINITY, d = 0.0, e = 0.0;
  for (int i = threadIdx.x; i < nb; i += kThreads) {
    const double* p = part + 5 * i;
    a += p[0];
    b = fmin(b, p[1]);
    c = fmax(c, p[2]);
    d += p[3];
    e += p[4];
  }
  a = block_reduce(a, OpAddD(), sh);
  b = block_reduce(b, OpMin(), sh);
  c = block_reduce(c, OpMax(), sh);
  d = block_reduce(d, OpAddD(), sh);
  e = block_reduce(e, OpAddD(), sh);
  if (threadIdx.x == 0) {
    double mean = d / (double)n;
    double var = e / (double)n - mean * mean;
    out[0] = a;
    out[1] = b;
    out[2] = c;
    out[3] = sqrt(var > 0.0 ? var : 0.0);
  }
}

// ----------------------------------------------------------------------------
// Pooling and helpers.
// ----------------------------------------------------------------------------
template <int VEC>
__global__ __launch_bounds__(kThreads) void k_maxpool(const int8_t* x, int n, int h, int w, int ch,
                                                      int ks, int stride, int pad, int ho, int wo,
                                                      int8_t* y) {
  const int cg = ch / VEC;
  const int64_t total = (int64_t)n * ho * wo * cg;
  for (int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * kThreads) {
    int g = (int)(idx % cg);
    int64_t pix = idx / cg;
    int ow = (int)(pix % wo);
    int oh = (int)((pix / wo) % ho);
    int b = (int)(pix / ((int64_t)wo * ho));
    union {
      int4 v16;
      char4 v4;
      int8_t b[16];
    } best;
#pragma unroll
    for (int j = 0; j < 16; ++j) best.b[j] = -128;
    if (VEC == 16 && ks == 3) {
      // 3x3 windows: the nine loads issued together (a tap outside the image
      // reads the window's clamped pixel and is then left out), so that the
      // thread waits for one round trip instead of nine
      int4 v[9];
      unsigned okm = 0;
#pragma unroll
      for (int r = 0; r < 3; ++r) {
#pragma unroll
        for (int q = 0; q < 3; ++q) {
          const int ih = oh * stride - pad + r, iw = ow * stride - pad + q;
          const bool ok = ih >= 0 && ih < h && iw >= 0 && iw < w;
          const int ihc = min(max(ih, 0), h - 1), iwc = min(max(iw, 0), w - 1);
          v[3 * r + q] = *reinterpret_cast<const int4*>(
              x + (((int64_t)b * h + ihc) * w + iwc) * ch + (int64_t)g * VEC);
          okm |= ok ? 1u << (3 * r + q) : 0u;
        }
      }
#pragma unroll
      for (int k = 0; k < 9; ++k) {
        if (!((okm >> k) & 1u)) continue;
        const int8_t* pv = reinterpret_cast<const int8_t*>(&v[k]);
#pragma unroll
        for (int j = 0; j < 16; ++j) best.b[j] = pv[j] > best.b[j] ? pv[j] : best.b[j];
      }
    } else
    for (int r = 0; r < ks; ++r) {
      int ih = oh * stride - pad + r;
      if (ih < 0 || ih >= h) continue;
      for (int q = 0; q < ks; ++q) {
        int iw = ow * stride - pad + q;
        if (iw < 0 || iw >= w) continue;
        const int8_t* src = x + (((int64_t)b * h + ih) * w + iw) * ch + (int64_t)g * VEC;
        if constexpr (VEC == 16) {
          int4 v = *reinterpret_cast<const int4*>(src);
          const int8_t* pv = reinterpret_cast<const int8_t*>(&v);
#pragma unroll
          for (int j = 0; j < 16; ++j) best.b[j] = pv[j] > best.b[j] ? pv[j] : best.b[j];
        } else {
          char4 v = *reinterpret_cast<const char4*>(src);
          best.b[0] = v.x > best.b[0] ? v.x : best.b[0];
          best.b[1] = v.y > best.b[1] ? v.y : best.b[1];
          best.b[2] = v.z > best.b[2] ? v.z : best.b[2];
          best.b[3] = v.w > best.b[3] ? v.w : best.b[3];
        }
      }
    }
    int8_t* dst = y + pix * ch + (int64_t)g * VEC;
    if constexpr (VEC == 16) {
      *reinterpret_cast<int4*>(dst) = best.v16;
    } else {
      *reinterpret_cast<char4*>(dst) = best.v4;
    }
  }
}

template <int CT>
__global__ __launch_bounds__(kThreads) void k_avgpool(const int8_t* x, const fxpq_fmt* fmt, int n,
                                                      int hw, int ch, int64_t recip, int64_t* y) {
  const int64_t off = code_is_off(CT, fmt) ? 128 : 0;
  const int64_t total = (int64_t)n * ch;
  for (int64_t idx = (int64_t)blockIdx.x * kThreads + threadIdx.x; idx < total;
       idx += (int64_t)gridDim.x * kThreads) {
    int c = (int)(idx % ch);
    int64_t b = idx / ch;
    int64_t s = 0;
    const int8_t* p = x + b * hw * ch + c;
    // seven pixels per step, their loads issued together (an exact integer
    // sum: the order does not matter)
    int q = 0;
    for (; q + 7 <= hw; q += 7) {
      int v[7];
#pragma unroll
      for (int k = 0; k < 7; ++k) v[k] = p[(int64_t)(q + k) * ch];
#pragma unroll
      for (int k = 0; k < 7; ++k) s += (int64_t)v[k] + off;
    }
    for (; q < hw; ++q) s += (int64_t)p[(int64_t)q * ch] + off;
    y[idx] = s * recip;
  }
}

__global__ __launch_bounds__(kThreads) void k_colsum(const int8_t* w, int64_t len, int32_t* out) {
  __shared__ long long sh[8];
  const int8_t* row = w + (int64_t)blockIdx.x * len;
  long long s = 0;
  for (int64_t j = threadIdx.x; j < len; j += kThreads) s += row[j];
  s = block_reduce(s, OpAddL(), sh);
  if (threadIdx.x == 0) out[blockIdx.x] = (int32_t)s;
}

__global__ void k_epi_scale(SrcDev s, int32_t* out) {
  if (threadIdx.x == 0 && blockIdx.x == 0) out[0] = src_scale(s);
}

// ----------------------------------------------------------------------------
// Launchers.
// ----------------------------------------------------------------------------
#define FXPQ_DISPATCH_SRC(KIND_VAR, DT_VAR, CALL)                                   \
  switch (KIND_VAR) {                                                               \
    case FXPQ_SRC_F32: { constexpr int K_ = FXPQ_SRC_F32, D_ = FXPQ_F32; CALL; } break; \
    case FXPQ_SRC_INT:                                                              \
      if (DT_VAR == FXPQ_I64) { constexpr int K_ = FXPQ_SRC_INT, D_ = FXPQ_I64; CALL; } \
      else { constexpr int K_ = FXPQ_SRC_INT, D_ = FXPQ_I32; CALL; }                \
      break;                                                                        \
    case FXPQ_SRC_ACC: { constexpr int K_ = FXPQ_SRC_ACC, D_ = FXPQ_I32; CALL; } break; \
    default: { constexpr int K_ = FXPQ_SRC_ADD, D_ = FXPQ_I8; CALL; } break;        \
  }

static int src_channels(const SrcDev& s) { return s.kind == FXPQ_SRC_ACC ? s.channels : 0; }

static int src_vec(const SrcDev& s) {
  return s.kind == FXPQ_SRC_ADD ? 16 : 4;
}  // values per thread per block iteration (Pack<>::V)

// Blocks (one min / max partial each) of launch_minmax's first kernel.
int minmax_blocks(const Ctx& c, const SrcDev& s, int64_t n) {
  int blocks = 1;
  FXPQ_DISPATCH_SRC(s.kind, s.dtype,
                    (blocks = stream_grid(n, src_channels(s), 0, src_vec(s),
                                          resident_blocks(c, (const void*)&k_minmax<K_, D_>))));
  return blocks;
}

hipError_t launch_minmax(const Ctx& c, const SrcDev& s, int64_t n, double* out) {
  int blocks = 1;
  FXPQ_DISPATCH_SRC(s.kind, s.dtype,
                    (blocks = stream_grid(n, src_channels(s), 0, src_vec(s),
                                          resident_blocks(c, (const void*)&k_minmax<K_, D_>)),
                     k_minmax<K_, D_><<<blocks, kThreads, 0, c.stream>>>(s, n, c.sc.minmax_part,
                                                                        c.sc.flags)));
  k_minmax_fin<<<1, kMmFinThreads, 0, c.stream>>>(c.sc.minmax_part, blocks, out);
  return hipGetLastError();
}

// Requantization of C-Block values, plus the min / max of the residual sum
// that consumes the codes written: relu?(code * 2^(F - fl_out) + b * 2^(F -
// fl_b)) in units of 2^-F, F = max(fl_out, fl_b), the same exact values an
// eltwise source over (codes, b) yields.  Block partials to `part`.
template <int OUT>
__global__ __launch_bounds__(kThreads) void k_requant_addmm(SrcDev s, int64_t n,
                                                            const fxpq_fmt* fmt, void* codes,
                                                            const int8_t* b, int b_type,
                                                            const fxpq_fmt* fmt_b, int relu,
                                                            double* part, unsigned* flags) {
  constexpr int KIND = FXPQ_SRC_ACC, DT = FXPQ_I32;
  using PK = Pack<KIND, DT>;
  __shared__ double sh[8];
  const int sv = src_scale(s);
  const QFmt q = qfmt_setup<OUT>(fmt, sv, flags);
  double mn = INFINITY, mx = -INFINITY;
  if (q.ok) {
    const int F = imax(fmt->fl, fmt_b->fl);
    const double ca = ldexp(1.0, F - fmt->fl), cb = ldexp(1.0, F - fmt_b->fl);
    const double offa = (double)q.off;
    const double offb = code_is_off(b_type, fmt_b) ? 128.0 : 0.0;
    const double relo = relu ? 0.0 : -INFINITY;
    auto add_value = [&](int stored_a, int stored_b) {
      const double va = ((double)stored_a + offa) * ca;
      return fmax(fma((double)stored_b + offb, cb, va), relo);
    };
    const int64_t gtid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    ThreadVals<PK::V> t;
    thread_vals_init<KIND, DT>(s, (int64_t)blockIdx.x * kThreads * PK::V, t);
    const int64_t nfull = n - n % PK::EP;
    stream_packets<KIND, DT, true>(s, n, t, [&](const double* v, int64_t i0, int bw) {
      int c[PK::EP];
#pragma unroll
      for (int j = 0; j < PK::EP; ++j) c[j] = quant_one(v[j], q);
      storev<OUT, PK::EP>(codes, i0, c);
#pragma unroll
      for (int j = 0; j < PK::EP; ++j) {
        const double x = add_value(c[j], (bw << (24 - 8 * j)) >> 24);
        mn = fmin(mn, x);
        mx = fmax(mx, x);
      }
    }, b);
    if (gtid == 0) {
      for (int64_t i = nfull; i < n; ++i) {
        const int ci = quant_one(load1<KIND, DT>(s, i), q);
        store1<OUT>(codes, i, ci);
        const double x = add_value(ci, b[i]);
        mn = fmin(mn, x);
        mx = fmax(mx, x);
      }
    }
  }
  mn = block_reduce(mn, OpMin(), sh);
  mx = block_reduce(mx, OpMax(), sh);
  if (threadIdx.x == 0) {
    part[2 * blockIdx.x] = mn;
    part[2 * blockIdx.x + 1] = mx;
  }
}

// The gated launch after a fused FxP-QLayer usually finds its codes written
// and does nothing: a grid of at most kGatedBlocks keeps that launch short
// (a real requantization then loops more per thread).
constexpr int kGatedBlocks = 256;

template <int OUT>
static void requant_out(const Ctx& c, const SrcDev& s, int64_t n, const fxpq_fmt* fmt,
                        void* codes, const FlsPlan* gate = nullptr, const int8_t* alt = nullptr) {
  int blocks = 1;
  const int cap = gate ? kGatedBlocks : 0;
  FXPQ_DISPATCH_SRC(s.kind, s.dtype,
                    (blocks = stream_grid(n, src_channels(s), 0, src_vec(s),
                                          cap ? cap : resident_blocks(c, (const void*)&k_requant<K_, D_, OUT>)),
                     k_requant<K_, D_, OUT><<<blocks, kThreads, 0, c.stream>>>(s, n, fmt, codes,
                                                                             c.sc.flags, gate, alt)));
}

hipError_t launch_requant_gated(const Ctx& c, const SrcDev& s, int64_t n, const fxpq_fmt* fmt,
                                int8_t* codes, const FlsPlan* plan, const int8_t* alt) {
  requant_out<FXPQ_C8>(c, s, n, fmt, codes, plan, alt);
  return hipGetLastError();
}

hipError_t launch_requant(const Ctx& c, const SrcDev& s, int64_t n, const fxpq_fmt* fmt,
                          void* codes, int code_type) {
  const double in_b = (s.kind == FXPQ_SRC_ADD) ? 2.0 : (s.kind == FXPQ_SRC_INT && s.dtype == FXPQ_I64) ? 8.0 : 4.0;
  const double out_b = (code_type == FXPQ_I32 || code_type == FXPQ_U32) ? 4.0 : (code_type == FXPQ_I16 ? 2.0 : 1.0);
  bool timed = timer_begin(c, FXPQ_TIMER_REQUANT);
  switch (code_type) {
    case FXPQ_I8: requant_out<FXPQ_I8>(c, s, n, fmt, codes); break;
    case FXPQ_U8OFF: requant_out<FXPQ_U8OFF>(c, s, n, fmt, codes); break;
    case FXPQ_C8: requant_out<FXPQ_C8>(c, s, n, fmt, codes); break;
    case FXPQ_I16: requant_out<FXPQ_I16>(c, s, n, fmt, codes); break;
    case FXPQ_U32: requant_out<FXPQ_U32>(c, s, n, fmt, codes); break;
    default: requant_out<FXPQ_I32>(c, s, n, fmt, codes); break;
  }
  timer_end(c, timed, (in_b + out_b) * (double)n);
  return hipGetLastError();
}

hipError_t launch_requant_addmm(const Ctx& c, const SrcDev& s, int64_t n, const fxpq_fmt* fmt,
                                void* codes, int code_type, const int8_t* b, int b_type,
                                const fxpq_fmt* fmt_b, int relu, double* d_add_minmax) {
  bool timed = timer_begin(c, FXPQ_TIMER_REQUANT);
  double* part = c.sc.minmax_part;
  auto run = [&](auto kernel) {
    const int blocks = stream_grid(n, src_channels(s), 0, src_vec(s),
                                   resident_blocks(c, (const void*)kernel));
    kernel<<<blocks, kThreads, 0, c.stream>>>(s, n, fmt, codes, b, b_type, fmt_b, relu, part,
                                              c.sc.flags);
    return blocks;
  };
  int blocks;
  switch (code_type) {
    case FXPQ_I8: blocks = run(&k_requant_addmm<FXPQ_I8>); break;
    case FXPQ_U8OFF: blocks = run(&k_requant_addmm<FXPQ_U8OFF>); break;
    default: blocks = run(&k_requant_addmm<FXPQ_C8>); break;
  }
  timer_end(c, timed, 6.0 * (double)n);
  return launch_minmax_fin(c, part, blocks, d_add_minmax);
}

hipError_t launch_layer_error(const Ctx& c, const float* ref, const void* codes, int code_type,
                              const fxpq_fmt* fmt, int64_t n, double* out) {
  double* part = c.sc.minmax_part;  // 5 doubles per block fits (kMaxConvBlocks * 2)
  auto run = [&](auto kernel) {
    const int blocks = stream_grid(n, 0, 0, 4, resident_blocks(c, (const void*)kernel));
    kernel<<<blocks, kThreads, 0, c.stream>>>(ref, codes, fmt, n, part);
    return blocks;
  };
  int blocks;
  switch (code_type) {
    case FXPQ_I16: blocks = run(&k_layer_error<FXPQ_I16>); break;
    case FXPQ_I32: blocks = run(&k_layer_error<FXPQ_I32>); break;
    case FXPQ_U32: blocks = run(&k_layer_error<FXPQ_U32>); break;
    case FXPQ_U8OFF: blocks = run(&k_layer_error<FXPQ_U8OFF>); break;
    case FXPQ_C8: blocks = run(&k_layer_error<FXPQ_C8>); break;
    case FXPQ_F32: blocks = run(&k_layer_error<FXPQ_F32>); break;
    default: blocks = run(&k_layer_error<FXPQ_I8>); break;
  }
  k_layer_error_fin<<<1, kThreads, 0, c.stream>>>(part, blocks, n, out);
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Dequantization (Eq. 1): out[i] = code_i * 2^-fl (+128 for codes stored as
// u - 128), exact in fp32 for codes below 2^24 in magnitude.
// ----------------------------------------------------------------------------
template <int CT>
__global__ __launch_bounds__(kThreads) void k_dequant(const void* codes, const fxpq_fmt* fmt,
                                                      int64_t n, float* out) {
  const double step = ldexp(1.0, -fmt->fl);
  const double off = (CT == FXPQ_U8OFF || (CT == FXPQ_C8 && fmt->sign == 0)) ? 128.0 : 0.0;
  for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kThreads)
    out[i] = (float)((code_at<CT>(codes, i) + off) * step);
}

hipError_t launch_dequant(const Ctx& c, const void* codes, int code_type, const fxpq_fmt* fmt,
                          int64_t n, float* out) {
  auto run = [&](auto kernel) {
    const int blocks = stream_grid(n, 0, 0, 1, resident_blocks(c, (const void*)kernel));
    kernel<<<blocks, kThreads, 0, c.stream>>>(codes, fmt, n, out);
  };
  switch (code_type) {
    case FXPQ_I16: run(&k_dequant<FXPQ_I16>); break;
    case FXPQ_I32: run(&k_dequant<FXPQ_I32>); break;
    case FXPQ_U32: run(&k_dequant<FXPQ_U32>); break;
    case FXPQ_U8OFF: run(&k_dequant<FXPQ_U8OFF>); break;
    case FXPQ_C8: run(&k_dequant<FXPQ_C8>); break;
    default: run(&k_dequant<FXPQ_I8>); break;
  }
  return hipGetLastError();
}

// ----------------------------------------------------------------------------
// Prediction ties of a classifier (Eq. 19-20): per row of `rows` x `cols`
// scores, the number c of classes sharing the highest score (exact
// comparison); out[0] = number of rows with c > 1, out[1] = sum of (c - 1).
// One block; a wave per row.
// ----------------------------------------------------------------------------
template <typename T>
__global__ __launch_bounds__(kThreads) void k_logit_ties(const T* s, int rows, int cols,
                                                         long long* out) {
  __shared__ long long sh[2][kThreads / 64];
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  long long un = 0, extra = 0;
  for (int r = w; r < rows; r += kThreads / 64) {
    const T* row = s + (int64_t)r * cols;
    T mx = row[lane < cols ? lane : 0];
    for (int j = lane; j < cols; j += 64) mx = row[j] > mx ? row[j] : mx;
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) {
      const T o = __shfl_xor(mx, off, 64);
      mx = o > mx ? o : mx;
    }
    int cnt = 0;
    for (int j = lane; j < cols; j += 64) cnt += (row[j] == mx) ? 1 : 0;
    cnt = wave_reduce(cnt, [](int a, int b) { return a + b; });
    un += (cnt > 1) ? 1 : 0;
    extra += cnt - 1;
  }
  if (lane == 0) {
    sh[0][w] = un;
    sh[1][w] = extra;
  }
  __syncthreads();
  if (threadIdx.x == 0) {
    long long a = 0, b = 0;
    for (int i = 0; i < kThreads / 64; ++i) {
      a += sh[0][i];
      b += sh[1][i];
    }
    out[0] = a;
    out[1] = b;
  }
}

hipError_t launch_logit_ties(const Ctx& c, const void* scores, int dtype, int rows, int cols,
                             long long* out) {
  if (dtype == FXPQ_F32)
    k_logit_ties<float><<<1, kThreads, 0, c.stream>>>(static_cast<const float*>(scores), rows, cols, out);
  else
    k_logit_ties<int32_t><<<1, kThreads, 0, c.stream>>>(static_cast<const int32_t*>(scores), rows, cols, out);
  return hipGetLastError();
}

hipError_t launch_maxpool(const Ctx& c, const int8_t* x, int n, int h, int w, int ch, int ks,
                          int stride, int pad, int8_t* y) {
  int ho = (h + 2 * pad - ks) / stride + 1, wo = (w + 2 * pad - ks) / stride + 1;
  int vec = (ch % 16 == 0) ? 16 : 4;
  int64_t total = (int64_t)n * ho * wo * (ch / vec);
  int64_t blocks = (total + kThreads - 1) / kThreads;
  if (blocks > 65536) blocks = 65536;
  if (blocks < 1) blocks = 1;
  if (vec == 16)
    k_maxpool<16><<<(int)blocks, kThreads, 0, c.stream>>>(x, n, h, w, ch, ks, stride, pad, ho, wo, y);
  else
    k_maxpool<4><<<(int)blocks, kThreads, 0, c.stream>>>(x, n, h, w, ch, ks, stride, pad, ho, wo, y);
  return hipGetLastError();
}

hipError_t launch_avgpool(const Ctx& c, const int8_t* x, int dtype, const fxpq_fmt* fmt, int n,
                          int hw, int ch, int64_t recip, int64_t* y) {
  int64_t total = (int64_t)n * ch;
  int64_t blocks = (total + kThreads - 1) / kThreads;
  if (blocks > 65536) blocks = 65536;
  if (dtype == FXPQ_U8OFF)
    k_avgpool<FXPQ_U8OFF><<<(int)blocks, kThreads, 0, c.stream>>>(x, fmt, n, hw, ch, recip, y);
  else if (dtype == FXPQ_C8)
    k_avgpool<FXPQ_C8><<<(int)blocks, kThreads, 0, c.stream>>>(x, fmt, n, hw, ch, recip, y);
  else
    k_avgpool<FXPQ_I8><<<(int)blocks, kThreads, 0, c.stream>>>(x, fmt, n, hw, ch, recip, y);
  return hipGetLastError();
}

hipError_t launch_colsum(const Ctx& c, const int8_t* w, int64_t k, int64_t len, int32_t* out) {
  k_colsum<<<(int)k, kThreads, 0, c.stream>>>(w, len, out);
  return hipGetLastError();
}

hipError_t launch_epi_scale(const Ctx& c, const SrcDev& s, int32_t* out) {
  k_epi_scale<<<1, 64, 0, c.stream>>>(s, out);
  return hipGetLastError();
}

}  // namespace fxpq

namespace fxpq {

// ----------------------------------------------------------------------------
// Preprocessor initial format (Sec. "Initial Design Generation", Eq. 6-9).
// With psi = r / D for an extreme r of the data (exact double, r > 0) and an
// integer D, beta_hat = -log2(psi):
//   floor(beta_hat) = largest b with r 2^b <= D,
//   ceil(beta_hat)  = smallest b with r 2^b >= D,
//   nearest         = largest b with (r 2^b)^2 <= 2 D^2 (beta_hat is never a
//                     half-integer: psi is rational).
// Every comparison is exact: r 2^b is exact in fp64, and the squared one falls
// back to 128-bit integers when fp64 cannot tell.
// ----------------------------------------------------------------------------
__device__ inline bool sq_le_2d2(double y, double d) {
  const double l = y * y, r = 2.0 * d * d;
  if (l < r * (1.0 - 0x1p-48)) return true;
  if (l > r * (1.0 + 0x1p-48)) return false;
  // near the boundary: y = M 2^E (M < 2^53), both sides below 2^110
  int e;
  const double m = frexp(y, &e);  // y = m 2^e, 0.5 <= m < 1
  const unsigned long long M = (unsigned long long)ldexp(m, 53);
  const int E = e - 53;
  const unsigned __int128 L0 = (unsigned __int128)M * M;
  const unsigned long long D = (unsigned long long)d;
  const unsigned __int128 R0 = (unsigned __int128)(2ull * D) * D;
  if (E >= 0) return (L0 << (2 * E)) <= R0;
  return L0 <= (R0 << (-2 * E));
}

// Ratio side: value magnitude r (in real units, exact) over the integer D.
struct PsiSide {
  double r, d;
  bool ok;
};

__device__ inline bool side_le(const PsiSide& p, int b, bool squared) {
  const double y = ldexp(p.r, b);
  return squared ? sq_le_2d2(y, p.d) : y <= p.d;
}
__device__ inline bool side_ge(const PsiSide& p, int b) { return ldexp(p.r, b) >= p.d; }

__global__ void k_preprocess(SrcDev s, const double* mm, int wl, int strategy, int rule, int fl_lo,
                             int fl_hi, fxpq_fmt* out, unsigned* flags) {
  if (blockIdx.x != 0 || threadIdx.x != 0) return;
  const int sv = src_scale(s);
  const double mn = ldexp(mm[0], -sv), mx = ldexp(mm[1], -sv);  // real units, exact
  if (!isfinite(mn) || !isfinite(mx)) {
    *out = fxpq_fmt{wl, 0, 0, 1};
    raise_flag(flags, FXPQ_FLAG_RANGE);
    return;
  }
  const int sign = mn < 0.0 ? 1 : 0;
  PsiSide a{0.0, 1.0, false}, c{0.0, 1.0, false};  // psi = min / max of a and c
  if (sign == 0) {
    a = PsiSide{mx, ldexp(1.0, wl) - 1.0, mx > 0.0};
  } else {
    a = PsiSide{-mn, ldexp(1.0, wl - 1), true};
    c = PsiSide{mx, ldexp(1.0, wl - 1) - 1.0, mx > 0.0};
  }
  int fl = fl_hi;
  if (a.ok) {
    const bool use_min = (rule == FXPQ_PSI_PRINTED);
    // psi 2^b <= bound: min rule -> either side, max rule -> both (sides
    // that are not ok are left out)
    auto le = [&](int b, bool sq) {
      const bool x = side_le(a, b, sq);
      if (!c.ok) return x;
      const bool y = side_le(c, b, sq);
      return use_min ? (x || y) : (x && y);
    };
    auto ge = [&](int b) {
      const bool x = side_ge(a, b);
      if (!c.ok) return x;
      const bool y = side_ge(c, b);
      return use_min ? (x && y) : (x || y);
    };
    if (strategy == FXPQ_ROUND_AGGRESSIVE) {
      fl = fl_hi;
      for (int b = fl_lo; b <= fl_hi; ++b)
        if (ge(b)) {
          fl = b;
          break;
        }
    } else {
      const bool sq = (strategy == FXPQ_ROUND_NEUTRAL);
      fl = fl_lo;
      for (int b = fl_hi; b >= fl_lo; --b)
        if (le(b, sq)) {
          fl = b;
          break;
        }
    }
  }
  *out = fxpq_fmt{wl, fl, sign, 0};
}

hipError_t launch_preprocess(const Ctx& c, const SrcDev& s, const double* d_minmax, int wl,
                             int strategy, int rule, int fl_lo, int fl_hi, fxpq_fmt* out) {
  k_preprocess<<<1, 64, 0, c.stream>>>(s, d_minmax, wl, strategy, rule, fl_lo, fl_hi, out,
                                       c.sc.flags);
  return hipGetLastError();
}

}  // namespace fxpq
