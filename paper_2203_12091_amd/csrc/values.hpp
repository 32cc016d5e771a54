// Per-thread loading of FxP-QLayer input values (exact doubles) for every
// source kind.  Streaming kernels walk the tensor in 4-element groups with a
// grid stride that is a multiple of the channel count, so the channels of a
// thread's group never change and their epilogue constants live in registers.
#pragma once

#include "common.hpp"

namespace fxpq {

constexpr double kTwo52 = 4503599627370496.0;  // 2^52
constexpr double kTwo53 = 9007199254740992.0;  // 2^53

struct ThreadVals {
  double M[4], A[4];  // ACC: per-channel multiplier / addend
  double ca, cb;      // ADD: alignment factors
  double oa, ob;      // ADD: +128 for offset-stored unsigned codes
  int relu;
};

template <int KIND>
__device__ inline void thread_vals_init(const SrcDev& s, int64_t first_elem, ThreadVals& t) {
  if constexpr (KIND == FXPQ_SRC_ACC) {
    EpiU u = epi_uniform(s);
    int c0 = (int)(first_elem % s.channels);
#pragma unroll
    for (int j = 0; j < 4; ++j) epi_channel(s, u, (c0 + j) % s.channels, t.M[j], t.A[j]);
    t.relu = s.ep_relu;
  } else if constexpr (KIND == FXPQ_SRC_ADD) {
    int F = imax(s.fa->fl, s.fb->fl);
    t.ca = ldexp(1.0, F - s.fa->fl);
    t.cb = ldexp(1.0, F - s.fb->fl);
    t.oa = code_is_off(s.dtype, s.fa) ? 128.0 : 0.0;
    t.ob = code_is_off(s.dtype2, s.fb) ? 128.0 : 0.0;
    t.relu = s.relu;
  }
}

// Loads values i..i+3 (i % 4 == 0, all in range).
template <int KIND, int DT>
__device__ inline void load4(const SrcDev& s, const ThreadVals& t, int64_t i, double v[4]) {
  if constexpr (KIND == FXPQ_SRC_F32) {
    float4 f = *reinterpret_cast<const float4*>(static_cast<const float*>(s.x) + i);
    v[0] = f.x; v[1] = f.y; v[2] = f.z; v[3] = f.w;
  } else if constexpr (KIND == FXPQ_SRC_INT && DT == FXPQ_I32) {
    int4 a = *reinterpret_cast<const int4*>(static_cast<const int32_t*>(s.x) + i);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
  } else if constexpr (KIND == FXPQ_SRC_INT && DT == FXPQ_I64) {
    const longlong2* p = reinterpret_cast<const longlong2*>(static_cast<const int64_t*>(s.x) + i);
    longlong2 a = p[0], b = p[1];
    v[0] = (double)a.x; v[1] = (double)a.y; v[2] = (double)b.x; v[3] = (double)b.y;
  } else if constexpr (KIND == FXPQ_SRC_ACC) {
    int4 a = *reinterpret_cast<const int4*>(static_cast<const int32_t*>(s.x) + i);
    double r0 = fma((double)a.x, t.M[0], t.A[0]);
    double r1 = fma((double)a.y, t.M[1], t.A[1]);
    double r2 = fma((double)a.z, t.M[2], t.A[2]);
    double r3 = fma((double)a.w, t.M[3], t.A[3]);
    if (t.relu) {
      r0 = fmax(r0, 0.0); r1 = fmax(r1, 0.0); r2 = fmax(r2, 0.0); r3 = fmax(r3, 0.0);
    }
    v[0] = r0; v[1] = r1; v[2] = r2; v[3] = r3;
  } else if constexpr (KIND == FXPQ_SRC_ADD) {
    char4 a = *reinterpret_cast<const char4*>(static_cast<const int8_t*>(s.x) + i);
    char4 b = *reinterpret_cast<const char4*>(static_cast<const int8_t*>(s.x2) + i);
    double r0 = fma((double)a.x + t.oa, t.ca, ((double)b.x + t.ob) * t.cb);
    double r1 = fma((double)a.y + t.oa, t.ca, ((double)b.y + t.ob) * t.cb);
    double r2 = fma((double)a.z + t.oa, t.ca, ((double)b.z + t.ob) * t.cb);
    double r3 = fma((double)a.w + t.oa, t.ca, ((double)b.w + t.ob) * t.cb);
    if (t.relu) {
      r0 = fmax(r0, 0.0); r1 = fmax(r1, 0.0); r2 = fmax(r2, 0.0); r3 = fmax(r3, 0.0);
    }
    v[0] = r0; v[1] = r1; v[2] = r2; v[3] = r3;
  }
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
    return s.ep_relu ? fmax(r, 0.0) : r;
  } else {
    ThreadVals t;
    thread_vals_init<FXPQ_SRC_ADD>(s, 0, t);
    double a = (double)static_cast<const int8_t*>(s.x)[i] + t.oa;
    double b = (double)static_cast<const int8_t*>(s.x2)[i] + t.ob;
    double r = fma(a, t.ca, b * t.cb);
    return t.relu ? fmax(r, 0.0) : r;
  }
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

__device__ inline void raise_flag(unsigned* flags, unsigned f) {
  __hip_atomic_fetch_or(flags, f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}


}  // namespace fxpq
