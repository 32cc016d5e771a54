// Shared pieces of the exact fractional-length search (used by the search
// kernels and by the fused conv epilogues).
#pragma once

#include <limits.h>
#include <math.h>

#include "values.hpp"

namespace fxpq {

struct FlsPlan {
  int need_general;
  int gen_lo, gen_hi;
  int gen_extra;  // INT_MIN when none
  int sign;
  int status;
  // Codes written by the window pass of a fused FxP-QLayer: when spec != 0,
  // the output codes hold the codes at fl = spec_fl[0] and the alternate
  // buffer those at fl = spec_fl[1].
  int spec;
  int spec_fl[2];
};

enum FlsMode { MODE_SEARCH = 0, MODE_REPORT = 1 };


// ---------------------------------------------------------------------------
// Small signed 512-bit integer (two's complement), used by one thread.
// ---------------------------------------------------------------------------
struct Big {
  unsigned long long w[8];
};

__device__ inline Big big_from_i128(__int128 v) {
  Big b;
  b.w[0] = (unsigned long long)v;
  b.w[1] = (unsigned long long)(v >> 64);
  unsigned long long ext = (v < 0) ? ~0ull : 0ull;
  for (int i = 2; i < 8; ++i) b.w[i] = ext;
  return b;
}

// a * 2^s for 0 <= s < 512 (static indexing only: whole words first, then bits).
__device__ inline Big big_shl(const Big& a, int s) {
  Big r = a;
  const int ws = s >> 6, bs = s & 63;
#pragma unroll
  for (int step = 0; step < 8; ++step) {
    if (step < ws) {
#pragma unroll
      for (int i = 7; i > 0; --i) r.w[i] = r.w[i - 1];
      r.w[0] = 0ull;
    }
  }
  if (bs) {
#pragma unroll
    for (int i = 7; i > 0; --i) r.w[i] = (r.w[i] << bs) | (r.w[i - 1] >> (64 - bs));
    r.w[0] <<= bs;
  }
  return r;
}

__device__ inline Big big_sub(const Big& a, const Big& b) {
  Big r;
  unsigned long long borrow = 0;
  for (int i = 0; i < 8; ++i) {
    unsigned long long x = a.w[i], y = b.w[i];
    unsigned long long d = x - y - borrow;
    borrow = (x < y) || (x - y < borrow) ? 1ull : 0ull;
    r.w[i] = d;
  }
  return r;
}

__device__ inline int big_cmp(const Big& a, const Big& b) {
  bool na = (long long)a.w[7] < 0, nb = (long long)b.w[7] < 0;
  if (na != nb) return na ? -1 : 1;
  for (int i = 7; i >= 0; --i)
    if (a.w[i] != b.w[i]) return a.w[i] < b.w[i] ? -1 : 1;
  return 0;
}

__device__ inline double big_to_double(const Big& a) {
  bool neg = (long long)a.w[7] < 0;
  Big m = a;
  if (neg) {
    Big z;
    for (int i = 0; i < 8; ++i) z.w[i] = 0;
    m = big_sub(z, a);
  }
  double r = 0.0;
  for (int i = 7; i >= 0; --i) r = r * 18446744073709551616.0 + (double)m.w[i];
  return neg ? -r : r;
}

// ---------------------------------------------------------------------------
// Uniform set-up shared by both passes.
// ---------------------------------------------------------------------------
struct FlsU {
  int sv;        // fractional length of the loaded values v
  int sign;
  double qmin, qmax;
  int sigma;     // W = v * 2^(sigma - sv) is an integer where it matters
  double wscale; // 2^(sigma - sv)
  double absmax; // max |v|
  int beta_nosat;
  int ok;        // 0: non-finite input
};

template <int KIND>
__device__ inline FlsU fls_uniform(const SrcDev& s, const double* mm, int wl, int sign_req,
                                   int fl_lo, int fl_hi) {
  FlsU u;
  u.sv = (KIND == FXPQ_SRC_F32) ? 0 : src_scale(s);
  double mn = mm[0], mx = mm[1];
  u.ok = isfinite(mn) && isfinite(mx);
  u.sign = (sign_req == FXPQ_SIGN_AUTO) ? (mn < 0.0 ? 1 : 0) : sign_req;
  u.qmax = ldexp(1.0, wl - u.sign) - 1.0;
  u.qmin = u.sign ? -ldexp(1.0, wl - 1) : 0.0;
  u.absmax = fmax(fabs(mn), fabs(mx));
  u.sigma = (KIND == FXPQ_SRC_F32) ? fl_hi + 24 : u.sv;
  u.wscale = ldexp(1.0, u.sigma - u.sv);
  // largest fl with every value inside [qmin - 1/2, qmax + 1/2] after scaling
  u.beta_nosat = fl_lo - 1;
  if (u.ok) {
    for (int b = fl_hi; b >= fl_lo; --b) {
      double tmax = ldexp(mx, b - u.sv), tmin = ldexp(mn, b - u.sv);
      if (tmax <= u.qmax + 0.5 && tmin >= u.qmin - 0.5) {
        u.beta_nosat = b;
        break;
      }
    }
  }
  return u;
}

// ---------------------------------------------------------------------------
// Pass 1: window search.
// ---------------------------------------------------------------------------
struct WinSetup {
  FlsU u;
  int verdict;  // 0: run window; 1: done (fl_hi); 2: general for all; 3: failure
  int b0, b1, nc, bce;
};

// Decisions every block of a window pass (and its finalize) takes from the
// min / max alone.  One thread adds at most `per_thread` values.  For integer
// sources its sums of W * q stay exact integers below 2^53 when max|W| *
// max|q| * per_thread < 2^53, and a tensor beyond that bound goes to the exact
// general pass.  fp32 values (W up to 2^52) always use the split form
// W = Wh * 2^26 + Wl, exact while 2^26 * max|q| * per_thread < 2^53, which
// the launcher's bound on per_thread guarantees.
template <int KIND>
__device__ inline WinSetup win_setup(const SrcDev& s, const double* mm, int wl, int sign_req,
                                     int fl_lo, int fl_hi, int mode, int64_t per_thread) {
  WinSetup w;
  w.u = fls_uniform<KIND>(s, mm, wl, sign_req, fl_lo, fl_hi);
  const double wmax = w.u.absmax * w.u.wscale;
  const double qabs = fmax(w.u.qmax, -w.u.qmin);
  w.verdict = 0;
  if (!w.u.ok) w.verdict = 3;
  else if (mode == MODE_REPORT || wl > 16 || wl == 1 || wmax >= kTwo52) w.verdict = 2;
  else if (w.u.beta_nosat >= fl_hi) w.verdict = 1;
  else if (KIND != FXPQ_SRC_F32 && wmax * qabs * (double)per_thread >= kTwo53) w.verdict = 2;
  w.b0 = imax(fl_lo, w.u.beta_nosat);
  w.b1 = (w.b0 + kWindow - 1 < fl_hi) ? w.b0 + kWindow - 1 : fl_hi;
  w.nc = w.b1 - w.b0 + 1;
  w.bce = (w.b1 < fl_hi) ? w.b1 + 1 : w.b1;
  return w;
}


// Per-thread accumulators of the window pass: per candidate the exact
// integers sum q^2 and sum W q (as sum Wh q and sum Wl q in the split form;
// all below 2^53, see win_setup), plus the fp64 bound sums: sum W^2 and the
// clipping errors at fl = b1 + 1, b1 + 2, ...
struct WinAcc {
  double A[kWindow], PH[kWindow], PL[kWindow];
  double V2, CE[kCeBounds];
};

constexpr double kTwoM26 = 1.0 / 67108864.0;  // 2^-26
constexpr double kTwo26 = 67108864.0;

// Exact int64 of an integer-valued double below 2^53 in magnitude.
__device__ inline long long exact_i64(double x) {
  const double hi = floor(x * 0x1p-32);
  const double lo = fma(hi, -0x1p32, x);  // in [0, 2^32)
  return (long long)(((unsigned long long)(unsigned)(int)hi << 32) | (unsigned)lo);
}

// Uniform constants of the window pass: candidate and clipping-bound scales.
struct WinCtx {
  double cj[kWindow];
  double cce;
  double qmin, qmax;
};

__device__ inline WinCtx win_ctx(const FlsU& u, const WinSetup& ws) {
  WinCtx c;
#pragma unroll
  for (int j = 0; j < kWindow; ++j) c.cj[j] = ldexp(1.0, (j < ws.nc ? ws.b0 + j : ws.b1) - u.sigma);
  c.cce = ldexp(1.0, ws.bce - u.sigma);
  c.qmin = u.qmin;
  c.qmax = u.qmax;
  return c;
}

__device__ inline void win_acc_zero(WinAcc& acc) {
#pragma unroll
  for (int j = 0; j < kWindow; ++j) acc.A[j] = acc.PH[j] = acc.PL[j] = 0.0;
  acc.V2 = 0.0;
#pragma unroll
  for (int k = 0; k < kCeBounds; ++k) acc.CE[k] = 0.0;
}

// Adds one integer value W = v * 2^sigma.  Specialized on
//   SPLIT    W * q summed as Wh * q and Wl * q (fp32 sources);
// and on what the min/max already tell:
//   NONNEG   every value is >= 0: no lower clamp, no lower clipping term;
//   CLAMP0   the first candidate can saturate (it is not beta_nosat).
template <bool SPLIT, bool NONNEG, bool CLAMP0, int NB = 1>
__device__ inline void win_consume(const WinCtx& c, WinAcc& acc, double W, double (&qo)[kWindow]) {
  double Wh = 0.0, Wl = W;
  if (SPLIT) {
    Wh = floor(W * kTwoM26);
    Wl = fma(-Wh, kTwo26, W);
  }
  acc.V2 = fma(W, W, acc.V2);
#pragma unroll
  for (int j = 0; j < kWindow; ++j) {
    double q = rint(W * c.cj[j]);
    if (j > 0 || CLAMP0) {
      q = min64(q, c.qmax);
      if (!NONNEG) q = max64(q, c.qmin);
    }
    acc.A[j] = fma(q, q, acc.A[j]);
    if (SPLIT) acc.PH[j] = fma(Wh, q, acc.PH[j]);
    acc.PL[j] = fma(Wl, q, acc.PL[j]);
    qo[j] = q;
  }
  // clipping error at the first NB fl above the window: W * 2^(fl - sigma)
  // doubles (exactly) from one to the next
  double t = W * c.cce;
#pragma unroll
  for (int k = 0; k < NB; ++k) {
    if (k) t += t;
    const double d1 = max64z(t - c.qmax);
    acc.CE[k] = fma(d1, d1, acc.CE[k]);
    if (!NONNEG) {
      const double d2 = min64z(t - c.qmin);
      acc.CE[k] = fma(d2, d2, acc.CE[k]);
    }
  }
}

template <bool SPLIT, bool NONNEG, bool CLAMP0, int NB = 1>
__device__ inline void win_consume(const WinCtx& c, WinAcc& acc, double W) {
  double q[kWindow];
  win_consume<SPLIT, NONNEG, CLAMP0, NB>(c, acc, W, q);
}

// Window candidate whose codes a predicted FxP-QLayer writes: the second
// when the format the previous call chose (still in the output format) is
// its fractional length, else the first.
__device__ inline int pred_pick(const WinSetup& ws, const fxpq_fmt& prev) {
  return (ws.nc == 2 && prev.fl == ws.b0 + 1) ? 1 : 0;
}

// Variant index (NONNEG << 1 | CLAMP0).
__device__ inline int win_variant(const FlsU& u, const WinSetup& ws, const double* mm) {
  const bool nonneg = mm[0] >= 0.0;
  const bool clamp0 = ws.b0 != u.beta_nosat;
  return (nonneg ? 2 : 0) | (clamp0 ? 1 : 0);
}

// Records a decision taken before the data is read (verdict != 0): done at
// fl_hi, the general pass over every candidate, or a failure.
__device__ inline void win_verdict_write(const WinSetup& ws, int wl, int fl_lo, int fl_hi,
                                         FlsPlan* plan, fxpq_fmt* out, unsigned* flags) {
  plan->sign = ws.u.sign;
  plan->status = 0;
  plan->need_general = 0;
  plan->gen_extra = INT_MIN;
  plan->spec = 0;
  if (ws.verdict == 1) {
    *out = fxpq_fmt{wl, fl_hi, ws.u.sign, 0};
  } else if (ws.verdict == 2) {
    plan->need_general = 1;
    plan->gen_lo = fl_lo;
    plan->gen_hi = fl_hi;
  } else {
    plan->status = 1;
    *out = fxpq_fmt{wl, 0, ws.u.sign, 1};
    raise_flag(flags, FXPQ_FLAG_RANGE);
  }
}

// LDS table of the block reduction (one row per wave of a 256-thread block).
struct WinShared {
  long long i[4][kWinSums];
  double f[4][kWinPartF];
};

__device__ inline void slot_add(long long* p, long long v) {
  __hip_atomic_fetch_add(reinterpret_cast<unsigned long long*>(p), (unsigned long long)v,
                         __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}
__device__ inline void slot_add(double* p, double v) {
  __hip_atomic_fetch_add(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
}

// Min / max of a predicted call, combined across blocks without a finish
// pass: each fp64 value maps to an unsigned key that orders like the value
// (mm_key), and the slot keeps the 64-bit atomic maximum of the key of the
// max (at kWinSums + 1) and of the complemented key of the min (at
// kWinSums).  Every key of a non-NaN value is above 0, so a cleared slot
// means "no value".
__device__ inline unsigned long long mm_key(double v) {
  const long long b = __double_as_longlong(v);
  return (unsigned long long)(b >= 0 ? b : b ^ 0x7FFFFFFFFFFFFFFFll) ^ 0x8000000000000000ull;
}
__device__ inline double mm_unkey(unsigned long long k) {
  const long long b = (long long)(k ^ 0x8000000000000000ull);
  return __longlong_as_double(b >= 0 ? b : b ^ 0x7FFFFFFFFFFFFFFFll);
}
__device__ inline void slot_max(long long* p, unsigned long long v) {
  __hip_atomic_fetch_max(reinterpret_cast<unsigned long long*>(p), v, __ATOMIC_RELAXED,
                         __HIP_MEMORY_SCOPE_AGENT);
}
// Every lane of the wave passes its min / max (mn > mx: none); lane 0 adds
// the wave's into slot bid % kWinSlots.
__device__ inline void mm_slot_add(double mn, double mx, int64_t bid, long long* part_i) {
  mn = wave_reduce(mn, OpMin());
  mx = wave_reduce(mx, OpMax());
  if ((threadIdx.x & 63) == 0 && mn <= mx) {
    long long* p = part_i + (int)(bid % kWinSlots) * kWinPart + kWinSums;
    slot_max(p, ~mm_key(mn));
    slot_max(p + 1, mm_key(mx));
  }
}

// Block results of the window pass (256 threads).  Each exact per-thread sum
// (below 2^62) is split into its high and low 32-bit halves, summed
// separately over the block and added (int64 atomics: exact, order-free) into
// slot bid % kWinSlots of part_i (kWinPart int64 per slot: per candidate A
// hi/lo, PH hi/lo, PL hi/lo, then two min / max keys, see mm_slot_add); the
// fp64 bound sums (sum W^2, then nb clipping
// bounds) go to part_f (kWinPartF per slot).  The search's decision reads the
// slots; the next search's decision clears them.
__device__ inline void win_write_partials_i64(const long long* A, const long long* PH,
                                              const long long* PL, double V2, const double* CE,
                                              int nb, int64_t bid, long long* part_i,
                                              double* part_f, WinShared& sh) {
  // Each wave reduces every quantity; lane 0 of wave w writes row w of the
  // table; after one barrier thread t adds the four rows of quantity t and
  // adds the result into the slot.
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  long long q[kWinSums];
#pragma unroll
  for (int j = 0; j < kWindow; ++j) {
    const long long q3[3] = {A[j], PH[j], PL[j]};
#pragma unroll
    for (int k = 0; k < 3; ++k) {
      q[6 * j + 2 * k] = q3[k] >> 32;
      q[6 * j + 2 * k + 1] = q3[k] & 0xFFFFFFFFll;
    }
  }
  double f[kWinPartF];
  f[0] = V2;
#pragma unroll
  for (int k = 0; k < kCeBounds; ++k) f[1 + k] = (k < nb) ? CE[k] : 0.0;
#pragma unroll
  for (int i = 0; i < kWinSums; ++i) q[i] = wave_reduce(q[i], OpAddL());
#pragma unroll
  for (int i = 0; i < kWinPartF; ++i) f[i] = wave_reduce(f[i], OpAddD());
  if (lane == 0) {
#pragma unroll
    for (int i = 0; i < kWinSums; ++i) sh.i[w][i] = q[i];
#pragma unroll
    for (int i = 0; i < kWinPartF; ++i) sh.f[w][i] = f[i];
  }
  __syncthreads();
  const int t = threadIdx.x;
  const int slot = (int)(bid % kWinSlots);
  if (t < kWinSums) {
    slot_add(part_i + slot * kWinPart + t, sh.i[0][t] + sh.i[1][t] + sh.i[2][t] + sh.i[3][t]);
  } else if (t < kWinSums + 1 + nb) {
    const int i = t - kWinSums;
    slot_add(part_f + kWinPartF * slot + i, ((sh.f[0][i] + sh.f[1][i]) + sh.f[2][i]) + sh.f[3][i]);
  }
}
__device__ inline void win_write_partials(const WinAcc& acc, int nb, int64_t bid,
                                          long long* part_i, double* part_f, WinShared& sh) {
  long long A[kWindow], PH[kWindow], PL[kWindow];
#pragma unroll
  for (int j = 0; j < kWindow; ++j) {
    A[j] = exact_i64(acc.A[j]);
    PH[j] = exact_i64(acc.PH[j]);
    PL[j] = exact_i64(acc.PL[j]);
  }
  win_write_partials_i64(A, PH, PL, acc.V2, acc.CE, nb, bid, part_i, part_f, sh);
}

// Block results of a window pass over integer values (no W split: PH is
// zero).  Fewer reductions than win_write_partials: sum q^2 per candidate is
// reduced in fp64, where it is exact (below 2^53 for word lengths up to 16
// and at most 2^17 values per block); sum W q as the 32-bit halves of the
// thread's exact int64 sum wq (below 2^62); the bound sums in fp64.  Same
// slot contents.
__device__ inline void win_write_partials_wq(const WinAcc& acc, const long long* wq, int nb,
                                             int64_t bid, long long* part_i, double* part_f,
                                             WinShared& sh) {
  const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
  double a[kWindow];
  long long ph[kWindow], pl[kWindow];
#pragma unroll
  for (int j = 0; j < kWindow; ++j) {
    a[j] = wave_reduce(acc.A[j], OpAddD());
    ph[j] = wave_reduce(wq[j] >> 32, OpAddL());
    pl[j] = wave_reduce(wq[j] & 0xFFFFFFFFll, OpAddL());
  }
  double f[kWinPartF];
  f[0] = wave_reduce(acc.V2, OpAddD());
#pragma unroll
  for (int k = 0; k < kCeBounds; ++k) f[1 + k] = (k < nb) ? wave_reduce(acc.CE[k], OpAddD()) : 0.0;
  if (lane == 0) {
#pragma unroll
    for (int j = 0; j < kWindow; ++j) {
      const long long aj = exact_i64(a[j]);
      sh.i[w][6 * j + 0] = aj >> 32;
      sh.i[w][6 * j + 1] = aj & 0xFFFFFFFFll;
      sh.i[w][6 * j + 2] = 0;  // W q summed unsplit: the high part is zero
      sh.i[w][6 * j + 3] = 0;
      sh.i[w][6 * j + 4] = ph[j];
      sh.i[w][6 * j + 5] = pl[j];
    }
#pragma unroll
    for (int i = 0; i < kWinPartF; ++i) sh.f[w][i] = f[i];
  }
  __syncthreads();
  const int t = threadIdx.x;
  const int slot = (int)(bid % kWinSlots);
  if (t < kWinSums) {
    if ((t % 6) != 2 && (t % 6) != 3)
      slot_add(part_i + slot * kWinPart + t, sh.i[0][t] + sh.i[1][t] + sh.i[2][t] + sh.i[3][t]);
  } else if (t < kWinSums + 1 + nb) {
    const int i = t - kWinSums;
    slot_add(part_f + kWinPartF * slot + i, ((sh.f[0][i] + sh.f[1][i]) + sh.f[2][i]) + sh.f[3][i]);
  }
}

// The same with the sums of W * q still in fp64 (exact below 2^53).
__device__ inline void win_write_partials_int(const WinAcc& acc, int nb, int64_t bid,
                                              long long* part_i, double* part_f, WinShared& sh) {
  long long wq[kWindow];
#pragma unroll
  for (int j = 0; j < kWindow; ++j) wq[j] = exact_i64(acc.PL[j]);
  win_write_partials_wq(acc, wq, nb, bid, part_i, part_f, sh);
}

// Launch helpers shared by the streaming search and the fused C-Block.
constexpr int kFinThreads = kWinSlots;  // one wave: one slot per lane

}  // namespace fxpq
