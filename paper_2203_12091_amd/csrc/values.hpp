// Per-thread loading of FxP-QLayer input values (exact doubles) for every
// source kind.  Streaming kernels walk the tensor in 4-element groups with a
// grid stride that is a multiple of the channel count, so the channels of a
// thread's group never change and their epilogue constants live in registers.
#pragma once

#include "common.hpp"

namespace fxpq {

constexpr double kTwo52 = 4503599627370496.0;  // 2^52
constexpr double kTwo53 = 9007199254740992.0;  // 2^53

// fp64 max / min of values that are never NaN (exact integers and their
// scaled codes), as single v_max_f64 / v_min_f64: written as the instruction
// itself so that the compiler adds no NaN-quieting of the operands (which
// IEEE-mode maxnum semantics would make it add before every use).  Same
// results as fmax / fmin on non-NaN operands (+0 above -0).
__device__ inline double max64(double a, double b) {
  double r;
  asm("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}
__device__ inline double min64(double a, double b) {
  double r;
  asm("v_min_f64 %0, %1, %2" : "=v"(r) : "v"(a), "v"(b));
  return r;
}

// max(a, b) for a wave-uniform b held in scalar registers.
__device__ inline double max64s(double a, double b) {
  double r;
  asm("v_max_f64 %0, %1, %2" : "=v"(r) : "v"(a), "s"(b));
  return r;
}

// max(a, 0) and min(a, 0) with the zero as an inline constant.
__device__ inline double max64z(double a) {
  double r;
  asm("v_max_f64 %0, %1, 0" : "=v"(r) : "v"(a));
  return r;
}
__device__ inline double min64z(double a) {
  double r;
  asm("v_min_f64 %0, %1, 0" : "=v"(r) : "v"(a));
  return r;
}

// Median of three (x clamped to [lo, hi] when lo <= hi) as one v_med3_i32.
__device__ inline int med3i(int x, int lo, int hi) {
  int r;
  asm("v_med3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "v"(lo), "v"(hi));
  return r;
}

// Rounding to nearest even by one addition: for |t| < 2^(51 - k),
// t + 1.5 * 2^(52 - k) is rne(t 2^k) 2^-k + 1.5 * 2^(52 - k) exactly (the
// sum's unit in the last place is 2^-k), and the low 32 bits of that double
// are rne(t 2^k) as a two's-complement int when |rne(t 2^k)| < 2^31.
__device__ inline int rne_lo(double t_plus_magic) {
  return (int)(unsigned)__builtin_bit_cast(unsigned long long, t_plus_magic);
}
constexpr double kRne1 = 0x1.8p51;  // k = 1: rne(2 t)

// Sticky device flags (vector atomic OR at device scope).
__device__ inline void raise_flag(unsigned* flags, unsigned f) {
  __hip_atomic_fetch_or(flags, f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Streaming layout.  A thread handles P packets of 16 bytes per block
// iteration; packet p of thread t covers elements base + (p*kThreads + t)*EP
// ... + EP-1, so every packet load of a wave is one contiguous 1 KiB span.
// EP = values per packet (4 for 4-byte data, 2 for int64, 16 for the two int8
// code tensors of an eltwise source).
template <int KIND, int DT>
struct Pack {
  static constexpr int EP = (KIND == FXPQ_SRC_ADD) ? 16 : (KIND == FXPQ_SRC_INT && DT == FXPQ_I64) ? 2 : 4;
  static constexpr int P = (KIND == FXPQ_SRC_INT && DT == FXPQ_I64) ? 2 : 1;
  static constexpr int V = EP * P;  // values per thread per block iteration
};

template <int V>
struct ThreadVals {
  double M[V], A[V];  // ACC: per-channel multiplier / addend, indexed p * EP + j
  int sa, sb;         // ADD: value = (a << sa) + (b << sb) + k, one shift is 0
  double k;           // ADD: the +128 of offset-stored unsigned codes, aligned
  double relo;        // ReLU as max(v, relo): 0, or -inf without ReLU
};

// Element index of packet p, value 0, for this thread at block base `base`.
template <int EP>
__device__ inline int64_t pk_index(int64_t base, int p) {
  return base + ((int64_t)p * kThreads + threadIdx.x) * EP;
}

template <int KIND, int DT>
__device__ inline void thread_vals_init(const SrcDev& s, int64_t base0,
                                        ThreadVals<Pack<KIND, DT>::V>& t) {
  using PK = Pack<KIND, DT>;
  if constexpr (KIND == FXPQ_SRC_ACC) {
    EpiU u = epi_uniform(s);
#pragma unroll
    for (int p = 0; p < PK::P; ++p) {
      int c0 = (int)(pk_index<PK::EP>(base0, p) % s.channels);
#pragma unroll
      for (int j = 0; j < PK::EP; ++j)
        epi_channel(s, u, (c0 + j) % s.channels, t.M[p * PK::EP + j], t.A[p * PK::EP + j]);
    }
    t.relo = s.ep_relu ? 0.0 : -INFINITY;
  } else if constexpr (KIND == FXPQ_SRC_ADD) {
    int F = imax(s.fa->fl, s.fb->fl);
    t.sa = F - s.fa->fl;
    t.sb = F - s.fb->fl;
    t.k = (code_is_off(s.dtype, s.fa) ? ldexp(128.0, t.sa) : 0.0) +
          (code_is_off(s.dtype2, s.fb) ? ldexp(128.0, t.sb) : 0.0);
    t.relo = s.relu ? 0.0 : -INFINITY;
  }
}

// Exactness of the integer combination of an eltwise source: |code| <= 255,
// so (a << sa) + (b << sb) stays inside int32 for shifts up to 22; larger
// alignments fall back to fp64 arithmetic.
constexpr int kAddMaxShift = 22;

// Raw 16-byte packet(s) of one group of EP values, as loaded.
template <int KIND, int DT>
struct Raw {
  int4 a;
  int4 b;  // second operand of an eltwise source
};

template <int KIND, int DT>
__device__ inline Raw<KIND, DT> load_raw(const SrcDev& s, int64_t i) {
  Raw<KIND, DT> r;
  if constexpr (KIND == FXPQ_SRC_ADD) {
    r.a = *reinterpret_cast<const int4*>(static_cast<const int8_t*>(s.x) + i);
    r.b = *reinterpret_cast<const int4*>(static_cast<const int8_t*>(s.x2) + i);
  } else if constexpr (KIND == FXPQ_SRC_INT && DT == FXPQ_I64) {
    r.a = *reinterpret_cast<const int4*>(static_cast<const int64_t*>(s.x) + i);
  } else if constexpr (KIND == FXPQ_SRC_ACC) {
    // conv accumulators are read once (by the FL search): non-temporal
    typedef int v4 __attribute__((ext_vector_type(4)));
    const v4 t = __builtin_nontemporal_load(
        reinterpret_cast<const v4*>(static_cast<const int32_t*>(s.x) + i));
    r.a = make_int4(t.x, t.y, t.z, t.w);
  } else {
    r.a = *reinterpret_cast<const int4*>(static_cast<const int32_t*>(s.x) + i);
  }
  return r;
}

// Exact doubles of packet p from its raw bytes.
template <int KIND, int DT>
__device__ inline void unpack(const Raw<KIND, DT>& r, const ThreadVals<Pack<KIND, DT>::V>& t,
                              int p, double* v) {
  constexpr int EP = Pack<KIND, DT>::EP;
  if constexpr (KIND == FXPQ_SRC_F32) {
    v[0] = __int_as_float(r.a.x); v[1] = __int_as_float(r.a.y);
    v[2] = __int_as_float(r.a.z); v[3] = __int_as_float(r.a.w);
  } else if constexpr (KIND == FXPQ_SRC_INT && DT == FXPQ_I32) {
    v[0] = r.a.x; v[1] = r.a.y; v[2] = r.a.z; v[3] = r.a.w;
  } else if constexpr (KIND == FXPQ_SRC_INT && DT == FXPQ_I64) {
    v[0] = (double)(((long long)(unsigned)r.a.y << 32) | (unsigned)r.a.x);
    v[1] = (double)(((long long)(unsigned)r.a.w << 32) | (unsigned)r.a.z);
  } else if constexpr (KIND == FXPQ_SRC_ACC) {
    const int raw[4] = {r.a.x, r.a.y, r.a.z, r.a.w};
#pragma unroll
    for (int j = 0; j < EP; ++j) v[j] = fmax(fma((double)raw[j], t.M[p * EP + j], t.A[p * EP + j]), t.relo);
  } else if constexpr (KIND == FXPQ_SRC_ADD) {
    const int wa[4] = {r.a.x, r.a.y, r.a.z, r.a.w};
    const int wb[4] = {r.b.x, r.b.y, r.b.z, r.b.w};
#pragma unroll
    for (int j = 0; j < EP; ++j) {
      const int ca = (wa[j / 4] << (24 - 8 * (j % 4))) >> 24;  // sign-extended byte
      const int cb = (wb[j / 4] << (24 - 8 * (j % 4))) >> 24;
      double x;
      if (t.sa <= kAddMaxShift && t.sb <= kAddMaxShift)
        x = (double)((ca << t.sa) + (cb << t.sb));
      else
        x = fma((double)ca, ldexp(1.0, t.sa), (double)cb * ldexp(1.0, t.sb));
      v[j] = fmax(x + t.k, t.relo);
    }
  }
}

// Drives a streaming kernel over this thread's packets of the grid-stride
// loop: fp(values, index of the first) for every whole packet.  Two register
// sets alternate so that the loads of the next iteration are in flight while
// this one's values are consumed; every load is issued unconditionally (an
// index past the end reads the last whole packet again, which is not
// consumed), so the number of loads in flight is fixed and the wait before
// each use only covers the older one.  Values past the last whole packet are
// left to the caller.
// REV: the thread visits its packets from the last to the first (the same
// packets and channels), so that a pass right after the kernel that wrote the
// tensor starts with its most recently written lines, still in the
// memory-side cache.
// RAWCB: fp receives the packet's raw bytes (Raw<KIND, DT>) instead of its
// values.
template <int KIND, int DT, bool AUX = false, int NSET = 2, bool REV = false, bool RAWCB = false,
          typename F>
__device__ inline void stream_packets(const SrcDev& s, int64_t n, const ThreadVals<Pack<KIND, DT>::V>& t,
                                      F&& fp, const int8_t* aux = nullptr) {
  // AUX: one byte per value of `aux`, loaded with each packet and handed to
  // fp as the packet's EP bytes (4-value packets only).  NSET register sets
  // rotate: NSET - 1 packets stay in flight while one is consumed.
  static_assert(!AUX || Pack<KIND, DT>::EP == 4, "aux bytes need 4-value packets");
  using PK = Pack<KIND, DT>;
  const int64_t chunk = (int64_t)kThreads * PK::V;
  const int64_t stride = (int64_t)gridDim.x * chunk;
  const int64_t nfull = n - n % PK::EP;
  if (nfull == 0) return;
  const int64_t last = nfull - PK::EP;
  auto load_set = [&](int64_t base, Raw<KIND, DT>* r, int* x) {
#pragma unroll
    for (int p = 0; p < PK::P; ++p) {
      int64_t i = pk_index<PK::EP>(base, p);
      i = i < nfull ? i : last;
      r[p] = load_raw<KIND, DT>(s, i);
      if constexpr (AUX) x[p] = *reinterpret_cast<const int*>(aux + i);
    }
  };
  auto use_set = [&](int64_t base, const Raw<KIND, DT>* r, const int* x) {
#pragma unroll
    for (int p = 0; p < PK::P; ++p) {
      const int64_t i = pk_index<PK::EP>(base, p);
      if (i < nfull) {
        if constexpr (RAWCB) {
          fp(r[p], i, x[p]);
        } else {
          double v[PK::EP];
          unpack<KIND, DT>(r[p], t, p, v);
          fp(v, i, x[p]);
        }
      }
    }
  };
  int64_t base = (int64_t)blockIdx.x * chunk;
  Raw<KIND, DT> rs[NSET][PK::P];
  int xs[NSET][PK::P] = {};
  if constexpr (REV) {
    // packets j = 0 .. J-1 at base + j * stride, visited from J-1 down; a
    // load for j < 0 reads packet 0 again and is not consumed
    if (base >= nfull) return;
    const int64_t top = (nfull - 1 - base) / stride;
    auto at = [&](int64_t j) { return base + (j < 0 ? 0 : j) * stride; };
#pragma unroll
    for (int k = 0; k < NSET; ++k) load_set(at(top - k), rs[k], xs[k]);
    for (int64_t j = top; j >= 0; j -= NSET) {
#pragma unroll
      for (int k = 0; k < NSET; ++k) {
        if (j - k >= 0) use_set(at(j - k), rs[k], xs[k]);
        load_set(at(j - NSET - k), rs[k], xs[k]);
      }
    }
    return;
  }
#pragma unroll
  for (int k = 0; k < NSET; ++k) load_set(base + k * stride, rs[k], xs[k]);
  for (; base < nfull; base += NSET * stride) {
#pragma unroll
    for (int k = 0; k < NSET; ++k) {
      use_set(base + k * stride, rs[k], xs[k]);
      load_set(base + (NSET + k) * stride, rs[k], xs[k]);
    }
  }
}

// Per-value form of stream_packets: f(value, index).
template <int KIND, int DT, typename F>
__device__ inline void stream_values(const SrcDev& s, int64_t n, const ThreadVals<Pack<KIND, DT>::V>& t,
                                     F&& f) {
  using PK = Pack<KIND, DT>;
  stream_packets<KIND, DT>(s, n, t, [&](const double* v, int64_t i0, int) {
#pragma unroll
    for (int j = 0; j < PK::EP; ++j) f(v[j], i0 + j);
  });
}

// Loads the single value i (tail elements); computes its own channel constants.
template <int KIND, int DT>
__device__ inline double load1(const SrcDev& s, int64_t i) {
  if constexpr (KIND == FXPQ_SRC_F32) {
    return static_cast<const float*>(s.x)[i];
  } else if constexpr (KIND == FXPQ_SRC_INT && DT == FXPQ_I32) {
    return static_cast<const int32_t*>(s.x)[i];
  } else if constexpr (KIND == FXPQ_SRC_INT && DT == FXPQ_I64) {
    return (double)static_cast<const int64_t*>(s.x)[i];
  } else if constexpr (KIND == FXPQ_SRC_ACC) {
    EpiU u = epi_uniform(s);
    double M, A;
    epi_channel(s, u, (int)(i % s.channels), M, A);
    double r = fma((double)static_cast<const int32_t*>(s.x)[i], M, A);
    return s.ep_relu ? fmax(r, 0.0) : r;  // tail values only
  } else {
    int F = imax(s.fa->fl, s.fb->fl);
    double a = (double)static_cast<const int8_t*>(s.x)[i] + (code_is_off(s.dtype, s.fa) ? 128.0 : 0.0);
    double b = (double)static_cast<const int8_t*>(s.x2)[i] + (code_is_off(s.dtype2, s.fb) ? 128.0 : 0.0);
    double r = fma(a, ldexp(1.0, F - s.fa->fl), b * ldexp(1.0, F - s.fb->fl));
    return s.relu ? fmax(r, 0.0) : r;
  }
}

// ---- quantization to a DFX format (Eq. 1 with round half to even, Eq. 2) ----
struct QFmt {
  double qmin, qmax, mult;
  int off;         // 128 when stored as u - 128
  double lo, hi;   // storage range
  bool binary;     // signed 1-bit format (Eq. 13): stored decoded, -1 or +1
  bool ok;
};

template <int OUT>
__device__ inline QFmt qfmt_setup(const fxpq_fmt* fmt, int sv, unsigned* flags) {
  QFmt q;
  int k = fmt->wl, fl = fmt->fl, sg = fmt->sign;
  q.ok = (fmt->status == 0 && k >= 1 && k <= 32 && (sg == 0 || sg == 1));
  q.binary = (k == 1 && sg == 1);
  if (!q.ok) {
    if (blockIdx.x == 0 && threadIdx.x == 0) raise_flag(flags, FXPQ_FLAG_RANGE);
    return q;
  }
  q.qmax = ldexp(1.0, k - sg) - 1.0;
  q.qmin = sg ? -ldexp(1.0, k - 1) : 0.0;
  q.mult = ldexp(1.0, fl - sv);
  q.off = (OUT == FXPQ_U8OFF || (OUT == FXPQ_C8 && sg == 0)) ? 128 : 0;
  if (OUT == FXPQ_I8 || OUT == FXPQ_U8OFF || OUT == FXPQ_C8) {
    q.lo = -128;
    q.hi = 127;
  } else if (OUT == FXPQ_I16) {
    q.lo = -32768;
    q.hi = 32767;
  } else if (OUT == FXPQ_U32) {
    q.lo = 0;
    q.hi = 4294967295.0;
  } else {
    q.lo = INT32_MIN;
    q.hi = INT32_MAX;
  }
  if (q.qmin - q.off < q.lo || q.qmax - q.off > q.hi) {
    if (blockIdx.x == 0 && threadIdx.x == 0) raise_flag(flags, FXPQ_FLAG_CODE);
  }
  return q;
}

// Exact Eq. 10-13 for an int64 value v at fractional length sv, sh = fl - sv:
// the code of v * 2^sh in integer arithmetic (fp64 holds int64 values exactly
// only below 2^53).  Products beyond the code range saturate (|qmin|, qmax <
// 2^33); right shifts round half to even.
__device__ inline int quant_one_i64(long long v, int sh, const QFmt& q) {
  if (q.binary) return v < 0 ? -1 : 1;
  const long long qmin = (long long)q.qmin, qmax = (long long)q.qmax;
  long long r;
  if (sh >= 0) {
    const unsigned long long m = v < 0 ? 0ull - (unsigned long long)v : (unsigned long long)v;
    if (v == 0) r = 0;
    else if (sh >= 33 || (m >> (33 - sh)) != 0ull) r = v < 0 ? qmin : qmax;
    else r = v * (1ll << sh);
  } else {
    const int d = -sh;
    if (d >= 64) {
      r = 0;  // |v| < 2^63 <= 2^(d - 1): below one half
    } else {
      const __int128 f = (__int128)v >> d;
      const __int128 rem = (__int128)v - f * ((__int128)1 << d);
      const __int128 half = (__int128)1 << (d - 1);
      r = (long long)(f + ((rem > half || (rem == half && (f & 1) != 0)) ? 1 : 0));
    }
  }
  r = r < qmin ? qmin : (r > qmax ? qmax : r);
  long long c = r - q.off;
  const long long lo = (long long)q.lo, hi = (long long)q.hi;
  c = c < lo ? lo : (c > hi ? hi : c);
  return (int)(unsigned)c;  // the storage's 32 bits (uint32 codes keep their bits)
}

template <int OUT = FXPQ_I32>
__device__ inline int quant_one(double v, const QFmt& q) {
  // Eq. 13: negative values take code -1, the rest code 0, which decodes to
  // +1; the decoded value is what is stored, so a C-Block uses it as it is
  if (q.binary) return v < 0.0 ? -1 : 1;
  double r = rint(v * q.mult);  // round half to even
  r = fmin(fmax(r, q.qmin), q.qmax);
  double c = r - (double)q.off;
  c = fmin(fmax(c, q.lo), q.hi);
  if constexpr (OUT == FXPQ_U32) return (int)(unsigned)c;  // uint32 storage bits
  else return (int)c;
}

// ---- wave / block reductions (wave64) ---------------------------------------
template <typename T, typename Op>
__device__ inline T wave_reduce(T v, Op op) {
#pragma unroll
  for (int off = 32; off > 0; off >>= 1) v = op(v, __shfl_xor(v, off, 64));
  return v;
}

// Block-wide reduction; every thread gets the result.  `sh` holds >= 4 T.
template <typename T, typename Op>
__device__ inline T block_reduce(T v, Op op, T* sh) {
  v = wave_reduce(v, op);
  int lane = threadIdx.x & 63, wid = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sh[wid] = v;
  __syncthreads();
  T r = sh[0];
  for (int w = 1; w < (int)(blockDim.x >> 6); ++w) r = op(r, sh[w]);
  return r;
}

struct OpMin {
  __device__ double operator()(double a, double b) const { return fmin(a, b); }
};
struct OpMax {
  __device__ double operator()(double a, double b) const { return fmax(a, b); }
};
struct OpAddD {
  __device__ double operator()(double a, double b) const { return a + b; }
};
struct OpAddL {
  __device__ long long operator()(long long a, long long b) const { return a + b; }
};
struct OpMaxU {
  __device__ unsigned long long operator()(unsigned long long a, unsigned long long b) const {
    return a > b ? a : b;
  }
};



}  // namespace fxpq
