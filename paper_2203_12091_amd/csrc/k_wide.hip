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
#include <type_traits>

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

// The C-Block epilogue on an exact contraction value a (bias, Scale
// multiply and offset, ReLU; every step exact): 128-bit arithmetic, or int64
// where the host has shown the contraction stays below 2^62 (every step then
// checked against 2^62).  bad: the value leaves [-2^62, 2^62] (written as 0).
__device__ inline int64_t wide_epi(__int128 a, const EpiRaw& r, const EpiU& u, const SrcDev& ep,
                                   bool& bad) {
  bool b = false;
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
  bad |= b;
  return b ? 0 : (int64_t)t;
}

__device__ inline int64_t wide_epi(int64_t a, const EpiRaw& r, const EpiU& u, const SrcDev& ep,
                                   bool& bad) {
  bool b = false;
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
  bad |= b;
  return b ? 0 : t;
}

// WIDE: the plane sums may exceed 2^62 (combined in 128 bits); otherwise the
// host has shown |sum| < 2^62 and the whole value stays in int64.
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
    using Acc = typename std::conditional<WIDE, __int128, int64_t>::type;
    Acc a = 0;
    for (int p = 0; p < np_x; ++p)
      for (int q = 0; q < np_w; ++q)
        a += (Acc)acc[(int64_t)(p * np_w + q) * mk + i] * ((Acc)1 << (8 * (p + q)));
    v[i] = wide_epi(a, r, u, ep, bad);
    c += cstep;
    if (c >= K) c -= K;
  }
  if (bad) flag(flags, FXPQ_FLAG_RANGE);
}

// ---------------------------------------------------------------------------
// One contraction for the whole wide C-Block.  The plane pairs (p, q) are
// walked by shift g = p + q; the pairs of one shift accumulate in the same
// int32 matrix-core accumulators (a pair's sum is at most depth * 2^14 in
// magnitude, the host bounds the group), which then fold into an exact wide
// register accumulator W += (acc + corr_g) * 256^g, corr_g adding back
// 128 * (the weight plane's column sum) for every input plane stored as
// byte - 128.  The epilogue runs on W in the same kernel: no per-pair
// tensors and no combine pass.  Tiles of 128 rows x 64 channels, four waves
// of 32 rows; slabs of 64 bytes of depth staged in LDS (two stages,
// register-staged loads one slab ahead).
// ---------------------------------------------------------------------------
typedef int v4i_w __attribute__((ext_vector_type(4)));
typedef int v16i_w __attribute__((ext_vector_type(16)));

__device__ inline int wlds_off(int row, int chunk) {
  return row * 64 + ((chunk ^ ((row >> 2) & 3)) & 3) * 16;
}

template <bool WIDE>
__global__ __launch_bounds__(kThreads, 2) void k_wide_fused(WideFusedArgs a) {
  constexpr int BM = 128, BN = 64;
  using Acc = typename std::conditional<WIDE, __int128, int64_t>::type;
  __shared__ __attribute__((aligned(16))) int8_t As[2][BM * 64];
  __shared__ __attribute__((aligned(16))) int8_t Bs[2][BN * 64];
  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int m0 = blockIdx.x * BM, n0 = blockIdx.y * BN;
  const int kc = tid & 3;
  const int hw_out = a.Ho * a.Wo;
  const int taps = a.R * a.S;
  const int ktiles = (a.wrow + 63) / 64;
  const int npairs_total = a.np_x * a.np_w;
  // rows this thread loads (two) and their image geometry
  int ih0[2], iw0[2];
  int64_t nbase[2];
#pragma unroll
  for (int i = 0; i < 2; ++i) {
    const int row = m0 + (tid >> 2) + 64 * i;
    const int rr = row < a.M ? row : a.M - 1;
    const int n = rr / hw_out, rem = rr - n * hw_out;
    const int oh = rem / a.Wo, ow = rem - oh * a.Wo;
    ih0[i] = oh * a.stride - a.pad;
    iw0[i] = ow * a.stride - a.pad;
    nbase[i] = (int64_t)n * a.H * a.W * a.C;
  }
  const int bcol = n0 + (tid >> 2);
  const int64_t brow = (int64_t)(bcol < a.K ? bcol : a.K - 1) * a.wrow;
  // pair number j (in shift order) -> (p, q)
  auto pair_of = [&](int j, int& p, int& q) {
    for (int g = 0;; ++g) {
      const int plo = g - a.np_w + 1 > 0 ? g - a.np_w + 1 : 0;
      const int phi = g < a.np_x - 1 ? g : a.np_x - 1;
      const int cnt = phi - plo + 1;
      if (j < cnt) {
        p = plo + j;
        q = g - p;
        return;
      }
      j -= cnt;
    }
  };
  v4i_w ra[2], rb;
  auto gload = [&](int sidx) {
    const int j = sidx / ktiles, kt = sidx - j * ktiles;
    int p, q;
    pair_of(j, p, q);
    const int8_t* xp = a.px + (int64_t)p * a.xs;
    const int padw = (p < a.np_x - 1 || !a.sign_x) ? (int)0x80808080 : 0;  // the value 0
    const int k = kt * 64 + kc * 16;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      v4i_w t = {padw, padw, padw, padw};
      const bool rowok = m0 + (tid >> 2) + 64 * i < a.M;
      if (a.C == 4) {
        // padded RGB: a 16-byte chunk holds four taps of 4 bytes
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int rs = (k >> 2) + e;
          if (rowok && rs < taps) {
            const int r = rs / a.S, sx = rs - r * a.S;
            const int ih = ih0[i] + r, iw = iw0[i] + sx;
            if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W)
              t[e] = *reinterpret_cast<const int*>(xp + nbase[i] + ((int64_t)ih * a.W + iw) * 4);
          }
        }
      } else if (rowok && k < a.kdepth) {
        const int rs = k / a.C, c0 = k - rs * a.C;
        const int r = rs / a.S, sx = rs - r * a.S;
        const int ih = ih0[i] + r, iw = iw0[i] + sx;
        if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W)
          t = *reinterpret_cast<const v4i_w*>(xp + nbase[i] + ((int64_t)ih * a.W + iw) * a.C + c0);
      }
      ra[i] = t;
    }
    const v4i_w z = {0, 0, 0, 0};
    rb = (k < a.wrow) ? *reinterpret_cast<const v4i_w*>(a.pw + (int64_t)q * a.ws + brow + k) : z;
  };
  auto lstore = [&](int st) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
      *reinterpret_cast<v4i_w*>(&As[st][wlds_off((tid >> 2) + 64 * i, kc)]) = ra[i];
    *reinterpret_cast<v4i_w*>(&Bs[st][wlds_off(tid >> 2, kc)]) = rb;
  };
  v16i_w acc[2];
  Acc W[2][16];
#pragma unroll
  for (int ni = 0; ni < 2; ++ni)
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      acc[ni][e] = 0;
      W[ni][e] = 0;
    }
  const int nslabs = npairs_total * ktiles;
  gload(0);
  lstore(0);
  __syncthreads();
  int j = 0;           // pair of the slab being computed
  int gcur = -1;       // shift of that pair
  int corr[2] = {0, 0};
  for (int sidx = 0; sidx < nslabs; ++sidx) {
    const int st = sidx & 1;
    if (sidx + 1 < nslabs) gload(sidx + 1);
    j = sidx / ktiles;
    int p, q;
    pair_of(j, p, q);
    if (p + q != gcur) gcur = p + q;
    if (sidx - j * ktiles == 0 && (p < a.np_x - 1 || !a.sign_x)) {
      // byte - 128 storage: 128 * colsum of this weight plane per column
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
        const int col = n0 + ni * 32 + (lane & 31);
        corr[ni] += 128 * a.cs[(int64_t)q * a.K + (col < a.K ? col : a.K - 1)];
      }
    }
    v4i_w af[2], bf[2][2];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
      af[kk] = *reinterpret_cast<const v4i_w*>(&As[st][wlds_off(wave * 32 + (lane & 31), kk * 2 + (lane >> 5))]);
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        bf[kk][ni] = *reinterpret_cast<const v4i_w*>(&Bs[st][wlds_off(ni * 32 + (lane & 31), kk * 2 + (lane >> 5))]);
    }
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int ni = 0; ni < 2; ++ni)
        acc[ni] = __builtin_amdgcn_mfma_i32_32x32x32_i8(af[kk], bf[kk][ni], acc[ni], 0, 0, 0);
    // end of a shift group: fold into the wide accumulator
    bool last = sidx + 1 == nslabs;
    if (!last) {
      int p2, q2;
      pair_of((sidx + 1) / ktiles, p2, q2);
      last = p2 + q2 != gcur;
    }
    if (last) {
#pragma unroll
      for (int ni = 0; ni < 2; ++ni) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          W[ni][e] += ((Acc)acc[ni][e] + (Acc)corr[ni]) * ((Acc)1 << (8 * gcur));
          acc[ni][e] = 0;
        }
        corr[ni] = 0;
      }
    }
    if (sidx + 1 < nslabs) lstore(st ^ 1);
    __syncthreads();
  }
  // epilogue
  const EpiU u = epi_uniform(a.ep);
  if (blockIdx.x == 0 && blockIdx.y == 0 && tid == 0) *a.d_scale = u.s_out;
  bool bad = false;
#pragma unroll
  for (int ni = 0; ni < 2; ++ni) {
    const int col = n0 + ni * 32 + (lane & 31);
    if (col >= a.K) continue;
    const EpiRaw r = epi_channel_load(a.ep, col);
#pragma unroll
    for (int e = 0; e < 16; ++e) {
      const int row = m0 + wave * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
      if (row < a.M) a.v[(int64_t)row * a.K + col] = wide_epi(W[ni][e], r, u, a.ep, bad);
    }
  }
  if (bad) flag(a.flags, FXPQ_FLAG_RANGE);
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

hipError_t launch_wide_fused(const Ctx& c, const WideFusedArgs& a, bool wide) {
  const dim3 grid((unsigned)((a.M + 127) / 128), (unsigned)((a.K + 63) / 64));
  if (wide) k_wide_fused<true><<<grid, kThreads, 0, c.stream>>>(a);
  else k_wide_fused<false><<<grid, kThreads, 0, c.stream>>>(a);
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
