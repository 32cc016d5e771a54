// C-Blocks over codes wider than 8 bits (Sec. "Integer-Only Inference": the
// first and last layers start at 32-bit activations and weights, Sec.
// "Initial Design Generation"), on the int8 matrix cores.
//
// A code of up to 32 bits is written in base 256.  Input codes x split into
// np_x byte planes: planes below the top hold the unsigned bytes (stored as
// byte - 128, the U8OFF storage the int8 contraction already corrects with the
// weight column sums), the top plane holds the rest (signed storage for
// signed formats).  Weight codes split into balanced digits in [-128, 127]
// (int8 as they are).  Then
//     sum_k x_k w_k = sum_{p,q} 256^(p+q) sum_k xp_k wq_k,
// each inner sum an ordinary int8 contraction with exact int32 accumulation;
// the combine kernel adds them with exact shifts in 128-bit integers and
// applies the C-Block epilogue in integers, writing int64 values at the
// epilogue's scale (an FXPQ_SRC_INT source for the FxP-QLayer that follows).
#include "common.hpp"

namespace fxpq {

namespace {

__device__ inline void flag(unsigned* flags, unsigned bit) { atomicOr(flags, bit); }

__global__ __launch_bounds__(kThreads) void k_split_x(const int32_t* __restrict__ x, int64_t n,
                                                      int np, int sign, int64_t ps,
                                                      int8_t* __restrict__ planes,
                                                      unsigned* flags) {
  bool bad = false;
  for (int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kThreads) {
    const int32_t v = x[i];
    for (int p = 0; p < np - 1; ++p) planes[p * ps + i] = (int8_t)(((v >> (8 * p)) & 255) - 128);
    if (sign) {
      const int32_t top = v >> (8 * (np - 1));
      bad |= top < -128 || top > 127;
      planes[(np - 1) * ps + i] = (int8_t)top;
    } else {
      // unsigned codes are read as uint32 (the storage of 32-bit ones)
      const uint32_t top = (uint32_t)v >> (8 * (np - 1));
      bad |= top > 255;
      planes[(np - 1) * ps + i] = (int8_t)((int)top - 128);
    }
  }
  if (bad) flag(flags, FXPQ_FLAG_CODE);
}

__global__ __launch_bounds__(kThreads) void k_split_w(const int32_t* __restrict__ w, int64_t n,
                                                      int np, int sign, int64_t ps,
                                                      int8_t* __restrict__ planes,
                                                      unsigned* flags) {
  bool bad = false;
  for (int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kThreads) {
    // unsigned codes are read as uint32 (the storage of 32-bit ones)
    int64_t r = sign ? (int64_t)w[i] : (int64_t)(uint32_t)w[i];
    for (int p = 0; p < np; ++p) {
      const int d = (int)((r + 128) & 255) - 128;
      planes[p * ps + i] = (int8_t)d;
      r = (r - d) >> 8;
    }
    bad |= r != 0;
  }
  if (bad) flag(flags, FXPQ_FLAG_CODE);
}

// Bits of |v| (0 for v == 0).
__device__ inline int bits128(__int128 v) {
  unsigned __int128 m = v < 0 ? (unsigned __int128)(-v) : (unsigned __int128)v;
  unsigned long long hi = (unsigned long long)(m >> 64), lo = (unsigned long long)m;
  return hi ? 128 - __builtin_clzll(hi) : (lo ? 64 - __builtin_clzll(lo) : 0);
}

// v * 2^sh, with `bad` set where the result would not stay below 2^120.
__device__ inline __int128 shl_checked(__int128 v, int sh, bool& bad) {
  if (v == 0) return 0;
  if (sh > 119 || bits128(v) + sh > 120) {
    bad = true;
    return 0;
  }
  return v * ((__int128)1 << sh);
}

// Bits of |v| (0 for v == 0).
__device__ inline int bits64(int64_t v) {
  const unsigned long long m = v < 0 ? 0ull - (unsigned long long)v : (unsigned long long)v;
  return m ? 64 - __builtin_clzll(m) : 0;
}

// v * 2^sh, with `bad` set where the result would not stay below 2^62.
__device__ inline int64_t shl62(int64_t v, int sh, bool& bad) {
  if (v == 0) return 0;
  if (sh > 61 || bits64(v) + sh > 62) {
    bad = true;
    return 0;
  }
  return v * ((int64_t)1 << sh);
}

// WIDE: the plane sums may exceed 2^62 (combined in 128 bits); otherwise the
// host has shown |sum| < 2^62 and the whole value stays in int64, every step
// checked against 2^62.
template <bool WIDE>
__global__ __launch_bounds__(kThreads) void k_wide_combine(const int32_t* __restrict__ acc,
                                                           int64_t mk, int np_x, int np_w,
                                                           SrcDev ep, int64_t* __restrict__ v,
                                                           int32_t* d_scale, unsigned* flags) {
  const EpiU u = epi_uniform(ep);
  if (blockIdx.x == 0 && threadIdx.x == 0) *d_scale = u.s_out;
  const int K = ep.channels;
  const int64_t step = (int64_t)gridDim.x * kThreads;
  const int cstep = (int)(step % K);
  int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x;
  int c = (int)(i % K);
  bool bad = false;
  for (; i < mk; i += step) {
    const EpiRaw r = epi_channel_load(ep, c);
    bool b = false;
    int64_t out;
    if constexpr (WIDE) {
      __int128 a = 0;
      for (int p = 0; p < np_x; ++p)
        for (int q = 0; q < np_w; ++q)
          a += (__int128)acc[(int64_t)(p * np_w + q) * mk + i] * ((__int128)1 << (8 * (p + q)));
      __int128 t = shl_checked(a, u.sh_acc, b);
      if (ep.bias) t += shl_checked((__int128)r.b, u.sh_bias, b);
      if (ep.scale) {
        if (bits128(t) > 90) b = true;
        else t *= (__int128)r.sc;
      }
      t = shl_checked(t, u.sh_mid, b);
      if (ep.shift) t += shl_checked((__int128)r.sh, u.sh_shift, b);
      if (ep.ep_relu && t < 0) t = 0;
      b |= bits128(t) > 62;
      out = (int64_t)t;
    } else {
      int64_t a = 0;
      for (int p = 0; p < np_x; ++p)
        for (int q = 0; q < np_w; ++q)
          a += (int64_t)acc[(int64_t)(p * np_w + q) * mk + i] * ((int64_t)1 << (8 * (p + q)));
      int64_t t = shl62(a, u.sh_acc, b);
      if (ep.bias) t += shl62((int64_t)r.b, u.sh_bias, b);
      if (ep.scale) {
        if (bits64(t) + 32 > 62) {
          int64_t m;
          b |= __builtin_mul_overflow(t, (int64_t)r.sc, &m);
          t = m;
        } else {
          t *= (int64_t)r.sc;
        }
      }
      t = shl62(t, u.sh_mid, b);
      if (ep.shift) t += shl62((int64_t)r.sh, u.sh_shift, b);
      if (ep.ep_relu && t < 0) t = 0;
      b |= bits64(t) > 62;
      out = t;
    }
    if (b) {
      bad = true;
      out = 0;
    }
    v[i] = out;
    c += cstep;
    if (c >= K) c -= K;
  }
  if (bad) flag(flags, FXPQ_FLAG_RANGE);
}

// Accumulators outside [-2^(bits-1), 2^(bits-1) - 1]: one atomic add per block.
__global__ __launch_bounds__(kThreads) void k_acc_overflow(const int32_t* __restrict__ acc,
                                                           int64_t n, int bits,
                                                           unsigned long long* count) {
  __shared__ unsigned long long part[kThreads / 64];
  const int64_t lo = -((int64_t)1 << (bits - 1)), hi = ((int64_t)1 << (bits - 1)) - 1;
  unsigned long long c = 0;
  for (int64_t i = blockIdx.x * (int64_t)kThreads + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * kThreads) {
    const int64_t a = acc[i];
    c += (a < lo || a > hi) ? 1 : 0;
  }
  for (int off = 32; off > 0; off >>= 1) c += __shfl_down(c, off, 64);
  if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = c;
  __syncthreads();
  if (threadIdx.x == 0) {
    unsigned long long t = 0;
    for (int w = 0; w < kThreads / 64; ++w) t += part[w];
    if (t) atomicAdd(count, t);
  }
}

int stream_blocks(int64_t n) {
  int64_t b = (n + kThreads - 1) / kThreads;
  return (int)(b < 4096 ? (b < 1 ? 1 : b) : 4096);
}

}  // namespace

hipError_t launch_wide_split_x(const Ctx& c, const int32_t* x, int64_t n, int np, int sign,
                               int64_t plane_stride, int8_t* planes) {
  k_split_x<<<stream_blocks(n), kThreads, 0, c.stream>>>(x, n, np, sign, plane_stride, planes,
                                                         c.sc.flags);
  return hipGetLastError();
}

hipError_t launch_wide_split_w(const Ctx& c, const int32_t* w, int64_t n, int np, int sign,
                               int64_t plane_stride, int8_t* planes) {
  k_split_w<<<stream_blocks(n), kThreads, 0, c.stream>>>(w, n, np, sign, plane_stride, planes,
                                                         c.sc.flags);
  return hipGetLastError();
}

hipError_t launch_acc_overflow(const Ctx& c, const int32_t* acc, int64_t n, int bits,
                               int64_t* count) {
  k_acc_overflow<<<stream_blocks(n), kThreads, 0, c.stream>>>(
      acc, n, bits, reinterpret_cast<unsigned long long*>(count));
  return hipGetLastError();
}

hipError_t launch_wide_combine(const Ctx& c, const int32_t* acc, int64_t mk, int np_x, int np_w,
                               const SrcDev& ep, int64_t* v, int32_t* d_scale) {
  // |sum_{p,q} acc_pq 256^(p+q)| < pairs * 2^31 * 256^(np_x + np_w - 2): int64 when below 2^62
  const int pairs = np_x * np_w;
  const int lg = pairs <= 1 ? 0 : 32 - __builtin_clz((unsigned)(pairs - 1));  // ceil(log2 pairs)
  const bool wide = 31 + 8 * (np_x + np_w - 2) + lg >= 62;
  if (wide)
    k_wide_combine<true><<<stream_blocks(mk), kThreads, 0, c.stream>>>(acc, mk, np_x, np_w, ep, v,
                                                                       d_scale, c.sc.flags);
  else
    k_wide_combine<false><<<stream_blocks(mk), kThreads, 0, c.stream>>>(acc, mk, np_x, np_w, ep,
                                                                        v, d_scale, c.sc.flags);
  return hipGetLastError();
}

}  // namespace fxpq
