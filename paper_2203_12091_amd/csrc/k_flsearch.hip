// Fractional-length search (Sec. "Quantization Parameters Optimization"):
// argmin over fl of the data-structure error L(fl) of Eq. 14, ties to the
// larger fl, decided EXACTLY.
//
// Pass 1 ("window", one read of the tensor, fp64 only):
//   * beta_nosat, the largest fl at which no value saturates, comes from the
//     tensor's min/max.  Below it L is non-increasing in fl (each coarser
//     grid's points are points of the finer grid, and an unsaturated value's
//     error is its distance to the infinite grid), so with ties going to the
//     larger fl the winner is >= beta_nosat.
//   * kWindow candidates from beta_nosat upward are evaluated with
//         2^(2 sigma) L(fl) = sum W^2 - 2^(d+1) sum W q + 2^(2d) sum q^2,
//     W = v * 2^sigma the value as an integer, d = sigma - fl, q its code.
//     sum W^2 is the same for every candidate, so the argmin only needs the
//     exact integers sum q^2 and sum W q.  W is split as Wh * 2^26 + Wl so
//     every per-thread partial stays an exact integer below 2^53; blocks
//     reduce in int64 and the last block compares candidates in 512-bit
//     integer arithmetic.
//   * Candidates above the window are discarded when a lower bound of their
//     error, the clipping error at the first of them (non-decreasing in fl),
//     exceeds an upper bound of the window's best error.
// Pass 2 ("general", only when pass 1 could not decide, when the caller asks
//   for every error, or for word lengths above 16): the exact error of every
//   remaining candidate in 128-bit integer arithmetic, compared exactly.
#include "fls.hpp"

namespace fxpq {

// Register sets of the window pass's packet pipeline.
constexpr int kWinSets = 4;

// 8-bit codes of the window candidates, written while the values are read
// (fused FxP-QLayer): candidate j's codes go to y[j] (none when null), as
// bytes q (signed formats) or q - 128 (unsigned formats; q ^ 0x80 for
// 0 <= q <= 255).
struct WinCodes {
  int8_t* y[kWindow];
  int qmax;
  unsigned xorw;  // 0x80808080 for unsigned formats, else 0
};

// Packs EP codes (one byte each) and stores them at y + i (4-byte aligned).
template <int EP>
__device__ inline void store_codes(int8_t* y, int64_t i, const int* c, unsigned xorw) {
  unsigned w[EP / 4];
#pragma unroll
  for (int k = 0; k < EP / 4; ++k)
    w[k] = ((unsigned)(c[4 * k] & 0xFF) | ((unsigned)(c[4 * k + 1] & 0xFF) << 8) |
            ((unsigned)(c[4 * k + 2] & 0xFF) << 16) | ((unsigned)c[4 * k + 3] << 24)) ^ xorw;
  if constexpr (EP == 16)
    *reinterpret_cast<uint4*>(y + i) = make_uint4(w[0], w[1], w[2], w[3]);
  else
    *reinterpret_cast<unsigned*>(y + i) = w[0];
}

// Main loop of the streaming window pass over this thread's values.
// MM: also the min / max of the values (predicted FxP-QLayer) into mn / mx.
template <int KIND, int DT, bool NONNEG, bool CLAMP0, int NB, bool CODES, bool MM = false>
__device__ inline void win_loop(const SrcDev& s, int64_t n, const FlsU& u, const WinSetup& ws,
                                const WinCodes& wcd, WinAcc& acc, double* mn = nullptr,
                                double* mx = nullptr) {
  const WinCtx wc = win_ctx(u, ws);
  win_acc_zero(acc);
  double lo = INFINITY, hi = -INFINITY;
  // Codes of one value: the window's codes are clamped except candidate 0
  // when it cannot saturate (beta_nosat), where a value at qmax + 1/2 rounds
  // to qmax + 1 (same error either way, but the code must be clamped).
  auto consume = [&](double W, int* cq) {
    double q[kWindow];
    win_consume<KIND == FXPQ_SRC_F32, NONNEG, CLAMP0, NB>(wc, acc, W, q);
    if constexpr (CODES) {
#pragma unroll
      for (int j = 0; j < kWindow; ++j) cq[j] = (int)q[j];
      if (!CLAMP0) cq[0] = min(cq[0], wcd.qmax);
    }
  };

  using PK = Pack<KIND, DT>;
  const int64_t gtid = (int64_t)blockIdx.x * kThreads + threadIdx.x;
  ThreadVals<PK::V> tv;
  thread_vals_init<KIND, DT>(s, (int64_t)blockIdx.x * kThreads * PK::V, tv);
  // Integer sources are searched at sigma = sv (W = v); fp32 values are
  // scaled by 2^(sigma - sv) = 2^(fl_hi + 24), exactly.
  const double post = u.wscale;
  const int64_t nfull = n - n % PK::EP;
  // backwards: the pass starts with the lines the previous kernel (the
  // conv, or the eltwise min / max pass, which reads forwards) touched last
  stream_packets<KIND, DT, false, kWinSets, true>(s, n, tv, [&](const double* v, int64_t i0, int) {
    int cq[PK::EP][kWindow];
#pragma unroll
    for (int j = 0; j < PK::EP; ++j) {
      if constexpr (MM) {
        lo = min64(lo, v[j]);
        hi = max64(hi, v[j]);
      }
      consume(KIND == FXPQ_SRC_F32 ? v[j] * post : v[j], cq[j]);
    }
    if constexpr (CODES) {
#pragma unroll
      for (int k = 0; k < kWindow; ++k) {
        if (!wcd.y[k]) continue;
        int c[PK::EP];
#pragma unroll
        for (int j = 0; j < PK::EP; ++j) c[j] = cq[j][k];
        store_codes<PK::EP>(wcd.y[k], i0, c, wcd.xorw);
      }
    }
  });
  if (gtid == 0)
    for (int64_t i = nfull; i < n; ++i) {
      int cq[kWindow];
      const double vi = load1<KIND, DT>(s, i);
      if constexpr (MM) {
        lo = min64(lo, vi);
        hi = max64(hi, vi);
      }
      consume(vi * u.wscale, cq);
      if constexpr (CODES) {
#pragma unroll
        for (int k = 0; k < kWindow; ++k)
          if (wcd.y[k]) wcd.y[k][i] = (int8_t)((cq[k] & 0xFF) ^ (wcd.xorw & 0xFF));
      }
    }
  if constexpr (MM) {
    *mn = lo;
    *mx = hi;
  }
}

// ---------------------------------------------------------------------------
// Eltwise sources through a histogram.  Every sum of the window pass (per
// candidate sum q^2 and sum W q, sum W^2, the clipping error) and the min /
// max depend on the values only through how often each integer
// W = relu(a 2^sa + b 2^sb) occurs.  With two 8-bit codes and shifts of at
// most 5 the sum before ReLU takes at most 255 * 33 + 1 values, so a block
// counts them in an LDS histogram while it streams the operands and writes
// the codes of the wanted window candidate(s) (16-bit lanes, two values per
// register), and derives its window sums from the counts at the end: a few
// instructions per value instead of the fp64 sums of every value.  The sums
// are the same exact integers as the per-value form (the code of a value
// exactly at qmax + 1/2 of the unsaturated candidate is qmax here, qmax + 1
// there: the same error term).
// ---------------------------------------------------------------------------
constexpr int kAddHistBins = 33 * 256;  // >= 255 * (2^5 + 1) + 1
constexpr int kAddHistSets = 4;         // register sets of the histogram pass

typedef short s2v __attribute__((ext_vector_type(2)));
typedef unsigned short u2v __attribute__((ext_vector_type(2)));

struct AddHist {
  int ok;
  int d0;          // sigma - b0, in [-8, 14]; candidate 1 shifts by d0 - 1 (left when negative)
  int ma, mb;      // 2^sa, 2^sb (one is 1)
  int k;           // the +128 of offset-stored codes, aligned: W = a ma + b mb + k
  int wlo, nbins;  // histogram bin i counts the sums (before ReLU) wlo + i
  int relu;
  int qmin, qmax;
  int cs;          // fl of the clipping bound less sigma
};

// The histogram form applies when the window has two candidates, both
// shifts are at most 5, the codes are 8 bits wide and a block adds at most
// 2^31 values (counts in 32 bits; every sum W q per thread below 2^53).  A
// candidate at or above sigma (d <= 0) takes the values exactly, W 2^-d:
// within the range the window was set up for (no value saturates at b0)
// these stay below 2^10 in magnitude for both candidates; beyond it (a
// predicted range that turns out wrong: the call is a miss) they wrap in
// their 16-bit lanes without effect on anything kept.
__device__ inline AddHist add_hist_setup(const SrcDev& s, const FlsU& u, const WinSetup& ws,
                                         int64_t per_thread) {
  AddHist p{};
  const int F = imax(s.fa->fl, s.fb->fl);
  const int sa = F - s.fa->fl, sb = F - s.fb->fl;
  const int d0 = u.sigma - ws.b0;
  const int cs = ws.bce - u.sigma;
  p.ok = ws.nc == 2 && u.sigma == F && sa <= 5 && sb <= 5 && d0 >= -8 && d0 <= 14 &&
         u.qmax <= 255.0 && u.qmin >= -128.0 && per_thread * kThreads <= (1ll << 31);
  if (!p.ok) return p;
  p.d0 = d0;
  p.ma = 1 << sa;
  p.mb = 1 << sb;
  // offset-stored codes hold u - 128 as a signed byte
  p.k = (code_is_off(s.dtype, s.fa) ? 128 * p.ma : 0) + (code_is_off(s.dtype2, s.fb) ? 128 * p.mb : 0);
  p.wlo = -128 * (p.ma + p.mb) + p.k;
  p.nbins = 255 * (p.ma + p.mb) + 1;
  p.relu = s.relu;
  p.qmin = (int)u.qmin;
  p.qmax = (int)u.qmax;
  p.cs = cs;
  return p;
}

// rne(W / 2^d) per 16-bit lane (1 <= d <= 14, |W| < 2^14: no overflow).
__device__ inline s2v rne_shr(s2v W, s2v dv, s2v halfm1) {
  const s2v bit = (W >> dv) & (s2v){1, 1};
  return (W + halfm1 + bit) >> dv;
}

// rne(W / 2^d) of one value (d >= 1), W 2^-d exactly for d <= 0.
__device__ inline int rne_shr1(int W, int d) {
  if (d <= 0) return (int)((unsigned)W << (-d));
  return (W + (1 << (d - 1)) - 1 + ((W >> d) & 1)) >> d;
}

// Bytes 1 and 3 of w, sign-extended, as two 16-bit lanes (permute
// selectors 8 and 9 replicate the sign bits of bytes 1 and 3).
__device__ inline s2v sext_odd_bytes(unsigned w) {
  return __builtin_bit_cast(s2v, __builtin_amdgcn_perm(0u, w, 0x09030801u));
}

// Streams the operands: counts every sum in hist and writes the codes of
// candidate 0 (2^-d0) to y0 and of candidate 1 (2^-(d0 - 1)) to y1, XOR xorw
// (Y0, Y1: the buffers exist).  DM: both candidates round (d0 >= 2), only
// candidate 0 rounds (d0 = 1), or both take the values exactly, W 2^-d
// (d0 <= 0).
enum { kHistBothRound = 2, kHistOneRounds = 1, kHistExact = 0 };

template <int DM, bool Y0, bool Y1>
__device__ __forceinline__ void add_hist_stream(const SrcDev& s, int64_t n, const AddHist& ap,
                                                int8_t* y0, int8_t* y1, unsigned xorw,
                                                unsigned* hist) {
  using PK = Pack<FXPQ_SRC_ADD, FXPQ_I8>;
  ThreadVals<PK::V> tv;  // unused by the raw callback
  const s2v ma = {(short)ap.ma, (short)ap.ma}, mb = {(short)ap.mb, (short)ap.mb};
  const s2v kv = {(short)ap.k, (short)ap.k};
  const short lo = ap.relu ? 0 : (short)ap.qmin;  // ReLU folds into the lower clamp
  const s2v lov = {lo, lo}, hiv = {(short)ap.qmax, (short)ap.qmax};
  const short d0 = (short)ap.d0, d1 = (short)(ap.d0 - 1);
  const short h0 = DM >= kHistOneRounds ? (short)((1 << (d0 - 1)) - 1) : 0;
  const short h1 = DM == kHistBothRound ? (short)((1 << (d1 - 1)) - 1) : 0;
  const s2v dv0 = {d0, d0}, dv1 = {d1, d1}, hm0 = {h0, h0}, hm1 = {h1, h1};
  const unsigned short l0 = DM == kHistExact ? (unsigned short)(-d0) : 0;
  const unsigned short l1 = DM == kHistBothRound ? 0 : (unsigned short)(-d1);
  const u2v lsh0 = {l0, l0}, lsh1 = {l1, l1};
  unsigned* hb = hist - ap.wlo;  // hb[W] is bin W - wlo
  auto clampq = [&](s2v q) {
    q = q > lov ? q : lov;
    return q < hiv ? q : hiv;
  };
  auto shl = [](s2v W, u2v sh) { return __builtin_bit_cast(s2v, __builtin_bit_cast(u2v, W) << sh); };
  auto code0 = [&](s2v W) { return clampq(DM >= kHistOneRounds ? rne_shr(W, dv0, hm0) : shl(W, lsh0)); };
  auto code1 = [&](s2v W) { return clampq(DM == kHistBothRound ? rne_shr(W, dv1, hm1) : shl(W, lsh1)); };
  auto pack = [&](s2v qe, s2v qo) {
    return __builtin_amdgcn_perm(__builtin_bit_cast(unsigned, qo), __builtin_bit_cast(unsigned, qe),
                                 0x06020400u) ^ xorw;
  };
  stream_packets<FXPQ_SRC_ADD, FXPQ_I8, false, kAddHistSets, true, true>(
      s, n, tv, [&](const Raw<FXPQ_SRC_ADD, FXPQ_I8>& r, int64_t i0, int) {
        const unsigned wa[4] = {(unsigned)r.a.x, (unsigned)r.a.y, (unsigned)r.a.z, (unsigned)r.a.w};
        const unsigned wb[4] = {(unsigned)r.b.x, (unsigned)r.b.y, (unsigned)r.b.z, (unsigned)r.b.w};
        unsigned cw0[4], cw1[4];
#pragma unroll
        for (int k = 0; k < 4; ++k) {
          // lanes: values 4k, 4k + 2 (even) and 4k + 1, 4k + 3 (odd)
          const s2v We = sext_odd_bytes(wa[k] << 8) * ma + (sext_odd_bytes(wb[k] << 8) * mb + kv);
          const s2v Wo = sext_odd_bytes(wa[k]) * ma + (sext_odd_bytes(wb[k]) * mb + kv);
          atomicAdd(hb + We.x, 1u);
          atomicAdd(hb + Wo.x, 1u);
          atomicAdd(hb + We.y, 1u);
          atomicAdd(hb + Wo.y, 1u);
          if (Y0) cw0[k] = pack(code0(We), code0(Wo));
          if (Y1) cw1[k] = pack(code1(We), code1(Wo));
        }
        if (Y0) *reinterpret_cast<uint4*>(y0 + i0) = make_uint4(cw0[0], cw0[1], cw0[2], cw0[3]);
        if (Y1) *reinterpret_cast<uint4*>(y1 + i0) = make_uint4(cw1[0], cw1[1], cw1[2], cw1[3]);
      });
}

// The histogram pass of an eltwise window (a block's share): zero the
// histogram, stream (codes of candidate 0 to y0, of candidate 1 to y1, when
// given), add the tail, then derive this thread's share of the window sums
// (nb clipping bounds) and of the min / max from the counts.
__device__ __forceinline__ void add_hist_run(const SrcDev& s, int64_t n, const AddHist& ap, int nb,
                                             int8_t* y0, int8_t* y1, unsigned xorw, unsigned* hist,
                                             WinAcc& acc, double* mn, double* mx) {
  for (int i = threadIdx.x; i < ap.nbins; i += kThreads) hist[i] = 0u;
  __syncthreads();
  const int dm = ap.d0 >= 2 ? kHistBothRound : (ap.d0 == 1 ? kHistOneRounds : kHistExact);
#define FXPQ_AHS(DM)                                                          \
  do {                                                                        \
    if (y0 && y1) add_hist_stream<DM, true, true>(s, n, ap, y0, y1, xorw, hist);   \
    else if (y0) add_hist_stream<DM, true, false>(s, n, ap, y0, y1, xorw, hist);   \
    else if (y1) add_hist_stream<DM, false, true>(s, n, ap, y0, y1, xorw, hist);   \
    else add_hist_stream<DM, false, false>(s, n, ap, y0, y1, xorw, hist);          \
  } while (0)
  if (dm == kHistBothRound) FXPQ_AHS(kHistBothRound);
  else if (dm == kHistOneRounds) FXPQ_AHS(kHistOneRounds);
  else FXPQ_AHS(kHistExact);
#undef FXPQ_AHS
  const int lo = ap.relu ? 0 : ap.qmin;
  auto clampq = [&](int q, int l) { return q < l ? l : (q > ap.qmax ? ap.qmax : q); };
  if ((int64_t)blockIdx.x * kThreads + threadIdx.x == 0) {
    const int8_t* xa = static_cast<const int8_t*>(s.x);
    const int8_t* xb = static_cast<const int8_t*>(s.x2);
    for (int64_t i = n - n % 16; i < n; ++i) {
      const int W = (int)xa[i] * ap.ma + (int)xb[i] * ap.mb + ap.k;
      atomicAdd(hist + (W - ap.wlo), 1u);
      if (y0) y0[i] = (int8_t)((clampq(rne_shr1(W, ap.d0), lo) & 0xFF) ^ (int)(xorw & 0xFF));
      if (y1) y1[i] = (int8_t)((clampq(rne_shr1(W, ap.d0 - 1), lo) & 0xFF) ^ (int)(xorw & 0xFF));
    }
  }
  __syncthreads();
  win_acc_zero(acc);
  const double cce = ldexp(1.0, ap.cs), qmx = ap.qmax, qmn = ap.qmin;
  int wmin = 0x7fffffff, wmax = -0x7fffffff - 1;
  for (int i = threadIdx.x; i < ap.nbins; i += kThreads) {
    const unsigned c = hist[i];
    if (c == 0u) continue;
    int W = ap.wlo + i;
    if (ap.relu) W = W > 0 ? W : 0;
    wmin = W < wmin ? W : wmin;
    wmax = W > wmax ? W : wmax;
    const int q0 = clampq(rne_shr1(W, ap.d0), ap.qmin);
    const int q1 = clampq(rne_shr1(W, ap.d0 - 1), ap.qmin);
    const double cd = (double)c;
    acc.A[0] = fma(cd, (double)(q0 * q0), acc.A[0]);
    acc.PL[0] = fma(cd, (double)(W * q0), acc.PL[0]);
    acc.A[1] = fma(cd, (double)(q1 * q1), acc.A[1]);
    acc.PL[1] = fma(cd, (double)(W * q1), acc.PL[1]);
    acc.V2 = fma(cd, (double)W * (double)W, acc.V2);
    // clipping errors at the first nb fl above the window: W 2^(fl - sigma)
    // doubles (exactly) from one to the next
    double t = (double)W * cce;
#pragma unroll
    for (int k = 0; k < kCeBounds; ++k) {
      if (k >= nb) break;
      if (k) t += t;
      const double e1 = max64z(t - qmx), e2 = min64z(t - qmn);
      acc.CE[k] = fma(cd, e1 * e1 + e2 * e2, acc.CE[k]);
    }
  }
  if (wmin <= wmax) {
    *mn = (double)wmin;
    *mx = (double)wmax;
  }
}

// Which window candidate's codes go to the output buffer of a fused
// FxP-QLayer: candidate 1 when the format found by the previous search into
// the same format (still in `out`) is that candidate's, else candidate 0.
// When that format is one of the window's candidates (same word length and
// sign, no error) the other candidate's codes are not written at all (a
// requantization pass follows if it wins); otherwise they go to the
// alternate buffer.
struct SpecPick {
  int pj;
  bool both;
};

__device__ inline SpecPick spec_pick(const WinSetup& ws, int wl, const fxpq_fmt* out) {
  const fxpq_fmt o = *out;
  SpecPick p;
  p.pj = (ws.nc == 2 && o.fl == ws.b0 + 1) ? 1 : 0;
  const bool known = o.wl == wl && o.status == 0 && o.sign == ws.u.sign &&
                     (o.fl == ws.b0 || o.fl == ws.b1);
  p.both = !known;
  return p;
}

// NB clipping bounds above the window (1, or kCeBounds for short word lengths).
// CODES: also writes both candidates' 8-bit codes (fused FxP-QLayer).
template <int KIND, int DT, int NB, bool CODES>
__global__ __launch_bounds__(kThreads) void k_fls_window(
    SrcDev s, int64_t n, int wl, int sign_req, int fl_lo, int fl_hi, int mode, int64_t per_thread,
    const double* mm, long long* part_i, double* part_f, FlsPlan* plan, fxpq_fmt* out,
    unsigned* flags, int8_t* y, int8_t* y_alt) {
  __shared__ WinShared wsh;
  const WinSetup ws = win_setup<KIND>(s, mm, wl, sign_req, fl_lo, fl_hi, mode, per_thread);
  const FlsU& u = ws.u;

  // Decisions every block takes identically before touching the data.
  if (ws.verdict != 0) {
    if (blockIdx.x == 0 && threadIdx.x == 0) win_verdict_write(ws, wl, fl_lo, fl_hi, plan, out, flags);
    return;
  }
  WinCodes wcd{};
  if constexpr (CODES) {
    const SpecPick sp = spec_pick(ws, wl, out);
    int8_t* other = sp.both ? y_alt : nullptr;
    wcd.y[0] = sp.pj ? other : y;
    wcd.y[1] = sp.pj ? y : other;
    wcd.qmax = (int)u.qmax;
    wcd.xorw = u.sign ? 0u : 0x80808080u;
  }
  WinAcc acc;
  if constexpr (KIND == FXPQ_SRC_ADD) {
    // eltwise sums through the histogram when it applies (uniform)
    __shared__ unsigned hist[kAddHistBins];
    const AddHist ap = add_hist_setup(s, u, ws, per_thread);
    if (ap.ok) {
      double mn, mx;  // not needed: the search has the min / max
      add_hist_run(s, n, ap, NB, wcd.y[0], wcd.y[1], wcd.xorw, hist, acc, &mn, &mx);
      win_write_partials_int(acc, NB, blockIdx.x, part_i, part_f, wsh);
      return;
    }
  }
  switch (win_variant(u, ws, mm)) {
    case 0: win_loop<KIND, DT, false, false, NB, CODES>(s, n, u, ws, wcd, acc); break;
    case 1: win_loop<KIND, DT, false, true, NB, CODES>(s, n, u, ws, wcd, acc); break;
    case 2: win_loop<KIND, DT, true, false, NB, CODES>(s, n, u, ws, wcd, acc); break;
    default: win_loop<KIND, DT, true, true, NB, CODES>(s, n, u, ws, wcd, acc); break;
  }
  if constexpr (KIND == FXPQ_SRC_F32) win_write_partials(acc, NB, blockIdx.x, part_i, part_f, wsh);
  else win_write_partials_int(acc, NB, blockIdx.x, part_i, part_f, wsh);
}

// Predicted FxP-QLayer over a streaming source: the window of the min / max
// held in mm (the previous call's values), the codes of the candidate the
// format in `out` picks (the previous call's choice) into y, and this call's
// min / max as block partials; the decision (k_pred_fin) checks the
// prediction.  verdict != 0: no window, the min / max only (a miss).
template <int KIND, int DT, int NB>
__global__ __launch_bounds__(kThreads) void k_qlayer_pred(
    SrcDev s, int64_t n, int wl, int sign_req, int fl_lo, int fl_hi, int64_t per_thread,
    double* mm, long long* part_i, double* part_f, fxpq_fmt* out, int8_t* y, PredJob* job,
    unsigned* miss) {
  __shared__ WinShared wsh;
  if (job && blockIdx.x == 0 && threadIdx.x == 0)
    *job = PredJob{s, wl, sign_req, fl_lo, fl_hi, NB, per_thread, mm, out, miss, part_i, part_f};
  const WinSetup ws = win_setup<KIND>(s, mm, wl, sign_req, fl_lo, fl_hi, MODE_SEARCH, per_thread);
  const FlsU& u = ws.u;
  double mn = INFINITY, mx = -INFINITY;
  bool counted = false;
  if constexpr (KIND == FXPQ_SRC_ADD) {
    __shared__ unsigned hist[kAddHistBins];
    if (ws.verdict == 0) {
      const AddHist ap = add_hist_setup(s, u, ws, per_thread);
      if (ap.ok) {  // uniform over the grid
        WinAcc acc;
        const int pj = pred_pick(ws, *out);
        add_hist_run(s, n, ap, NB, pj ? nullptr : y, pj ? y : nullptr, u.sign ? 0u : 0x80808080u,
                     hist, acc, &mn, &mx);
        win_write_partials_int(acc, NB, blockIdx.x, part_i, part_f, wsh);
        counted = true;
      }
    }
  }
  if (counted) {
  } else if (ws.verdict == 0) {
    WinCodes wcd{};
    const int pj = pred_pick(ws, *out);
    wcd.y[pj] = y;
    wcd.qmax = (int)u.qmax;
    wcd.xorw = u.sign ? 0u : 0x80808080u;
    WinAcc acc;
    switch (win_variant(u, ws, mm)) {
      case 0: win_loop<KIND, DT, false, false, NB, true, true>(s, n, u, ws, wcd, acc, &mn, &mx); break;
      case 1: win_loop<KIND, DT, false, true, NB, true, true>(s, n, u, ws, wcd, acc, &mn, &mx); break;
      case 2: win_loop<KIND, DT, true, false, NB, true, true>(s, n, u, ws, wcd, acc, &mn, &mx); break;
      default: win_loop<KIND, DT, true, true, NB, true, true>(s, n, u, ws, wcd, acc, &mn, &mx); break;
    }
    if constexpr (KIND == FXPQ_SRC_F32) win_write_partials(acc, NB, blockIdx.x, part_i, part_f, wsh);
    else win_write_partials_int(acc, NB, blockIdx.x, part_i, part_f, wsh);
  } else {
    using PK = Pack<KIND, DT>;
    ThreadVals<PK::V> tv;
    thread_vals_init<KIND, DT>(s, (int64_t)blockIdx.x * kThreads * PK::V, tv);
    stream_packets<KIND, DT>(s, n, tv, [&](const double* v, int64_t, int) {
#pragma unroll
      for (int j = 0; j < PK::EP; ++j) {
        mn = min64(mn, v[j]);
        mx = max64(mx, v[j]);
      }
    });
    if ((int64_t)blockIdx.x * kThreads + threadIdx.x == 0)
      for (int64_t i = n - n % PK::EP; i < n; ++i) {
        const double vi = load1<KIND, DT>(s, i);
        mn = min64(mn, vi);
        mx = max64(mx, vi);
      }
  }
  mm_slot_add(mn, mx, blockIdx.x, part_i);
}

// Bits of |v| (0 for v == 0).
__device__ inline int bitlen_i128(__int128 v) {
  unsigned __int128 m = v < 0 ? (unsigned __int128)(-v) : (unsigned __int128)v;
  unsigned long long hi = (unsigned long long)(m >> 64), lo = (unsigned long long)m;
  return hi ? 128 - __builtin_clzll(hi) : (lo ? 64 - __builtin_clzll(lo) : 0);
}

__device__ inline double i128_to_double(__int128 v) {
  return (double)(long long)(v >> 64) * 0x1p64 + (double)(unsigned long long)v;
}

// Decision of the window pass, taken by one wave from the slot sums.
struct WinResult {
  int done;     // the window's best candidate is the answer
  int fl_win;   // the window's best candidate
  int gen_hi;   // top of the candidates the exact pass still has to evaluate
};

// Lane l reads slot l of the window sums (part_i / part_f, one set), the
// wave adds them exactly, lane 0 decides (its result only is meaningful).
__device__ inline WinResult win_decide(const WinSetup& ws, int nce, int fl_hi,
                                       const long long* part_i, const double* part_f) {
  constexpr int NQ = 3 * kWindow;
  const FlsU& u = ws.u;
  const int b0 = ws.b0, b1 = ws.b1, nc = ws.nc, bce = ws.bce;
  const int lane = threadIdx.x & 63;
  // The high and low 32-bit halves of each quantity are summed separately
  // (both sums stay far below 2^63).
  const long long* p = part_i + lane * kWinPart;
  long long hi[NQ], lo[NQ];
#pragma unroll
  for (int qi = 0; qi < NQ; ++qi) {
    hi[qi] = p[2 * qi];
    lo[qi] = p[2 * qi + 1];
  }
  double f[kWinPartF];
#pragma unroll
  for (int k = 0; k < kWinPartF; ++k) f[k] = part_f[kWinPartF * lane + k];
#pragma unroll
  for (int qi = 0; qi < NQ; ++qi) {
    hi[qi] = wave_reduce(hi[qi], OpAddL());
    lo[qi] = wave_reduce(lo[qi], OpAddL());
  }
#pragma unroll
  for (int k = 0; k < kWinPartF; ++k) f[k] = wave_reduce(f[k], OpAddD());
  WinResult r{0, 0, fl_hi};
  if (lane != 0) return r;
  auto total = [&](int qi) -> __int128 { return ((__int128)hi[qi] << 32) + (__int128)lo[qi]; };
  // K_j = 2^(2d) A - 2^(d+1) P, d = sigma - beta; shifted by `off` >= 0 so all
  // exponents are non-negative (same factor for every candidate).
  int dmin = u.sigma - b1;
  int off = 0;
  if (2 * dmin < 0) off = -2 * dmin;
  if (dmin + 1 + off < 0) off = -(dmin + 1);
  // 128-bit arithmetic when both terms of every K_j stay below 2^125, else
  // 512-bit.
  __int128 Aj[kWindow], Pj[kWindow];
  bool fast = true;
#pragma unroll
  for (int j = 0; j < kWindow; ++j) {
    Aj[j] = total(3 * j);
    Pj[j] = total(3 * j + 1) * (__int128)67108864 + total(3 * j + 2);
    const int d = u.sigma - (b0 + (j < nc ? j : 0));
    fast = fast && bitlen_i128(Aj[j]) + 2 * d + off <= 125 && bitlen_i128(Pj[j]) + d + 1 + off <= 125;
  }
  int bj = -1;
  double kd = 0.0;
  if (fast) {
    __int128 best = 0;
#pragma unroll
    for (int j = 0; j < kWindow; ++j) {
      if (j >= nc) break;
      const int d = u.sigma - (b0 + j);
      const __int128 kj = (Aj[j] << (2 * d + off)) - (Pj[j] << (d + 1 + off));
      if (bj < 0 || kj <= best) {  // ties -> larger fl
        best = kj;
        bj = j;
      }
    }
    kd = ldexp(i128_to_double(best), -off);
  } else {
    Big best;
#pragma unroll
    for (int j = 0; j < kWindow; ++j) {
      if (j >= nc) break;
      const int d = u.sigma - (b0 + j);
      Big kj = big_sub(big_shl(big_from_i128(Aj[j]), 2 * d + off),
                       big_shl(big_from_i128(Pj[j]), d + 1 + off));
      if (bj < 0 || big_cmp(kj, best) <= 0) {  // ties -> larger fl
        best = kj;
        bj = j;
      }
    }
    kd = ldexp(big_to_double(best), -off);
  }
  r.fl_win = b0 + bj;
  bool done = (b1 == fl_hi);
  int gen_hi = fl_hi;
  if (!done) {
    // Upper bound of the window's best error; the clipping error at fl is a
    // lower bound of the error of every candidate >= fl (it is non-decreasing
    // in fl), so the first bound above the best error excludes the rest
    // (relative fp64 error of each sum, in any summation order, < 2^-40).
    double v2 = f[0];
    double sse_ub = (v2 * (1.0 + 0x1p-30) + kd + fabs(kd) * 0x1p-50 + v2 * 0x1p-50);
    sse_ub = ldexp(sse_ub, -2 * u.sigma) * (1.0 + 0x1p-50);
    for (int k = 0; k < nce && bce + k <= fl_hi; ++k) {
      const double ce_lb = ldexp(f[1 + k] * (1.0 - 0x1p-30), -2 * (bce + k));
      if (ce_lb > sse_ub) {
        gen_hi = bce + k - 1;
        break;
      }
    }
    done = gen_hi <= b1;
  }
  r.done = done;
  r.gen_hi = gen_hi;
  return r;
}

// Records a window decision in the plan (and the format when it is final).
// `codes`: the window pass wrote codes (fused FxP-QLayer); `out` still holds
// the previous format, which picked where they went.
__device__ inline void win_record(const WinSetup& ws, const WinResult& r, int wl, int codes,
                                  FlsPlan* plan, fxpq_fmt* out) {
  plan->sign = ws.u.sign;
  plan->status = 0;
  plan->spec = codes;
  if (codes) {
    // the window pass wrote candidate pj's codes to the output buffer (and
    // the other's to the alternate buffer when both)
    const SpecPick sp = spec_pick(ws, wl, out);
    plan->spec_fl[0] = ws.b0 + sp.pj;
    plan->spec_fl[1] = sp.both ? ws.b0 + (ws.nc == 2 ? 1 - sp.pj : 0) : INT_MIN;
  }
  if (r.done) {
    plan->need_general = 0;
    *out = fxpq_fmt{wl, r.fl_win, ws.u.sign, 0};
  } else {
    plan->need_general = 1;
    plan->gen_lo = ws.b1 + 1;
    plan->gen_hi = r.gen_hi;
    plan->gen_extra = r.fl_win;
  }
}

// Zeroes one set of window slots (the block's threads).
__device__ inline void win_slots_clear(long long* part_i, double* part_f) {
  for (int k = threadIdx.x; k < kWinSlots * kWinPart; k += blockDim.x) part_i[k] = 0;
  for (int k = threadIdx.x; k < kWinSlots * kWinPartF; k += blockDim.x) part_f[k] = 0.0;
}

// Finalize of a window pass whose decision later launches need before the
// general pass (fused conv path): one wave decides from slot set `part_*`
// and clears the other set `clr_*` (used by the search before).
template <int KIND>
__global__ __launch_bounds__(kFinThreads) void k_fls_window_fin(
    SrcDev s, int wl, int sign_req, int fl_lo, int nce, int fl_hi, int mode, int64_t per_thread,
    const double* mm, const long long* part_i, const double* part_f, long long* clr_i,
    double* clr_f, FlsPlan* plan, fxpq_fmt* out) {
  win_slots_clear(clr_i, clr_f);
  const WinSetup ws = win_setup<KIND>(s, mm, wl, sign_req, fl_lo, fl_hi, mode, per_thread);
  if (ws.verdict != 0) return;  // the pass kernel already wrote the plan
  const WinResult r = win_decide(ws, nce, fl_hi, part_i, part_f);
  if (threadIdx.x == 0) win_record(ws, r, wl, 0, plan, out);
}

// Decision of a predicted C-Block or FxP-QLayer (one wave, after the pass):
// combines the min / max keys of the slots into this call's exact min / max
// and checks that the window the pass evaluated (from the predicted min / max
// held in mm) is this call's window: same verdict 0, candidates, clipping
// bound, sign and variant.  Then the wave decides from the window sums; the
// format is recorded when the decision is final and is the candidate whose
// codes the pass wrote, else *miss is set.  mm ends with this call's
// min / max; the other slot set is cleared for the next search.
// The decision itself, by one wave.  deferred: the calls that consumed this
// call's codes have already run with the format held in *out (the
// prediction), so a hit also needs the decision to be that format; the
// slots are the call's own set, cleared afterwards for its next use.
template <int KIND>
__device__ inline void pred_decision(const SrcDev& s, int wl, int sign_req, int fl_lo, int fl_hi,
                                     int nce, int64_t per_thread, double* mm,
                                     const long long* part_i, const double* part_f, fxpq_fmt* out,
                                     unsigned* miss, bool deferred) {
  const double pred[2] = {mm[0], mm[1]};
  const long long* p = part_i + (threadIdx.x & 63) * kWinPart + kWinSums;
  const unsigned long long kmn = wave_reduce((unsigned long long)p[0], OpMaxU());
  const unsigned long long kmx = wave_reduce((unsigned long long)p[1], OpMaxU());
  const double act[2] = {kmn ? mm_unkey(~kmn) : INFINITY, kmx ? mm_unkey(kmx) : -INFINITY};
  const WinSetup wp = win_setup<KIND>(s, pred, wl, sign_req, fl_lo, fl_hi, MODE_SEARCH, per_thread);
  const WinSetup wa = win_setup<KIND>(s, act, wl, sign_req, fl_lo, fl_hi, MODE_SEARCH, per_thread);
  const bool same = wp.verdict == 0 && wa.verdict == 0 && wp.b0 == wa.b0 && wp.b1 == wa.b1 &&
                    wp.nc == wa.nc && wp.bce == wa.bce && wp.u.sign == wa.u.sign &&
                    win_variant(wp.u, wp, pred) == win_variant(wa.u, wa, act);
  const fxpq_fmt used = *out;
  bool hit = false, undecided = false;
  int fl = 0;
  if (same) {  // uniform over the wave
    const WinResult r = win_decide(wa, nce, fl_hi, part_i, part_f);
    if (threadIdx.x == 0) {
      fl = r.fl_win;
      hit = r.done && r.fl_win == wa.b0 + pred_pick(wp, used);
      if (deferred) hit = hit && used.fl == fl && used.sign == wa.u.sign && used.status == 0;
      undecided = !r.done;
    }
  }
  if (threadIdx.x == 0) {
    // miss 1: the prediction was wrong; 2: right, but the window alone
    // cannot decide (the exact search needs more candidates), so the next
    // call on the same data misses again
    if (hit) *out = fxpq_fmt{wl, fl, wa.u.sign, 0};
    else *miss = undecided ? 2u : 1u;
    mm[0] = act[0];
    mm[1] = act[1];
  }
}

// Decision of a predicted C-Block or FxP-QLayer (one wave, after the pass):
// combines the min / max keys of the slots into this call's exact min / max
// and checks that the window the pass evaluated (from the predicted min / max
// held in mm) is this call's window: same verdict 0, candidates, clipping
// bound, sign and variant.  Then the wave decides from the window sums; the
// format is recorded when the decision is final and is the candidate whose
// codes the pass wrote, else *miss is set.  mm ends with this call's
// min / max; the other slot set is cleared for the next search.
template <int KIND>
__global__ __launch_bounds__(kFinThreads) void k_pred_fin(
    SrcDev s, int wl, int sign_req, int fl_lo, int fl_hi, int nce, int64_t per_thread, double* mm,
    const long long* part_i, const double* part_f, long long* clr_i, double* clr_f, fxpq_fmt* out,
    unsigned* miss) {
  win_slots_clear(clr_i, clr_f);
  pred_decision<KIND>(s, wl, sign_req, fl_lo, fl_hi, nce, per_thread, mm, part_i, part_f, out,
                      miss, false);
}

// Deferred decisions: block b decides pending call b (recorded by the call's
// own kernel), then clears that call's slot set.
__global__ __launch_bounds__(kFinThreads) void k_pred_decide(const PredJob* jobs) {
  const PredJob& j = jobs[blockIdx.x];
  switch (j.s.kind) {
    case FXPQ_SRC_ACC:
      pred_decision<FXPQ_SRC_ACC>(j.s, j.wl, j.sign, j.fl_lo, j.fl_hi, j.nce, j.per_thread, j.mm,
                                  j.pi, j.pf, j.out, j.miss, true);
      break;
    case FXPQ_SRC_ADD:
      pred_decision<FXPQ_SRC_ADD>(j.s, j.wl, j.sign, j.fl_lo, j.fl_hi, j.nce, j.per_thread, j.mm,
                                  j.pi, j.pf, j.out, j.miss, true);
      break;
    case FXPQ_SRC_F32:
      pred_decision<FXPQ_SRC_F32>(j.s, j.wl, j.sign, j.fl_lo, j.fl_hi, j.nce, j.per_thread, j.mm,
                                  j.pi, j.pf, j.out, j.miss, true);
      break;
    default:
      pred_decision<FXPQ_SRC_INT>(j.s, j.wl, j.sign, j.fl_lo, j.fl_hi, j.nce, j.per_thread, j.mm,
                                  j.pi, j.pf, j.out, j.miss, true);
      break;
  }
  __syncthreads();
  win_slots_clear(j.pi, j.pf);
}

// ---------------------------------------------------------------------------
// Pass 2: exact general search (128-bit errors, 192-bit sums).
// ---------------------------------------------------------------------------
struct U192 {
  unsigned __int128 lo;
  unsigned long long hi;
};

__device__ inline void u192_add(U192& a, unsigned __int128 x) {
  unsigned __int128 s = a.lo + x;
  if (s < a.lo) a.hi += 1;
  a.lo = s;
}

__device__ inline void u192_add(U192& a, const U192& b) {
  unsigned __int128 s = a.lo + b.lo;
  a.hi += b.hi + (s < a.lo ? 1 : 0);
  a.lo = s;
}

__device__ inline int u192_cmp(const U192& a, const U192& b) {
  if (a.hi != b.hi) return a.hi < b.hi ? -1 : 1;
  if (a.lo != b.lo) return a.lo < b.lo ? -1 : 1;
  return 0;
}

__device__ inline double u192_to_double(const U192& a) {
  return (double)a.hi * 0x1p128 + (double)(unsigned long long)(a.lo >> 64) * 0x1p64 +
         (double)(unsigned long long)a.lo;
}

// What the exact pass has to do.
struct GenPlan {
  int need, status, sign;
  int glo, ghi, extra;  // candidates glo..ghi, plus `extra` unless INT_MIN
};

__device__ void general_decide(int wl, int fl_lo, int fl_hi, int nchunks, int sigma,
                               const GenPlan& gp, const unsigned long long* part, fxpq_fmt* out,
                               double* d_sse);

// The window pass's finalize, when the general kernel takes it: every block
// decides from the slot set (pi, pf) itself (same sums, same decision), block
// 0 records it and clears the other slot set (ci, cf).
struct WinIn {
  int decide;  // 0: the plan already holds the decision
  int sign_req, nce, mode, codes;
  int64_t per_thread;
  const long long* pi;
  const double* pf;
  long long* ci;  // may be null
  double* cf;
};

// Exact errors of the remaining candidates over (candidate, chunk) items; the
// last block to finish sums the chunk partials and decides.  Nothing runs
// unless the window pass left candidates undecided (and only then is the
// device-scope release / acquire paid).
template <int KIND, int DT>
__global__ __launch_bounds__(kThreads) void k_fls_general(
    SrcDev s, int64_t n, int wl, int fl_lo, int fl_hi, int nchunks, const double* mm, WinIn wi,
    FlsPlan* plan, unsigned long long* part, unsigned* done, fxpq_fmt* out, double* d_sse,
    unsigned* flags) {
  __shared__ unsigned long long shp[kThreads * 3];
  __shared__ int last;
  __shared__ GenPlan gp_sh;
  if (wi.ci && blockIdx.x == 0) win_slots_clear(wi.ci, wi.cf);
  bool from_plan = true;
  if (wi.decide) {
    const WinSetup ws = win_setup<KIND>(s, mm, wl, wi.sign_req, fl_lo, fl_hi, wi.mode, wi.per_thread);
    if (ws.verdict == 0) {  // else the window pass wrote the plan
      from_plan = false;
      if (threadIdx.x < 64) {
        const WinResult r = win_decide(ws, wi.nce, fl_hi, wi.pi, wi.pf);
        if (threadIdx.x == 0) {
          if (blockIdx.x == 0) win_record(ws, r, wl, wi.codes, plan, out);
          gp_sh = GenPlan{r.done ? 0 : 1, 0, ws.u.sign, ws.b1 + 1, r.gen_hi, r.fl_win};
        }
      }
    }
  }
  if (from_plan && threadIdx.x == 0)
    gp_sh = GenPlan{plan->need_general, plan->status, plan->sign, plan->gen_lo, plan->gen_hi,
                    plan->gen_extra};
  __syncthreads();
  const GenPlan gp = gp_sh;
  if (!gp.need || gp.status) return;
  const int sign = gp.sign;
  const int glo = gp.glo, ghi = gp.ghi, extra = gp.extra;
  const int nreg = ghi - glo + 1;
  const int nc = nreg + (extra != INT_MIN ? 1 : 0);
  auto cand = [&](int j) { return (extra != INT_MIN) ? (j == 0 ? extra : glo + j - 1) : glo + j; };

  const int sv = (KIND == FXPQ_SRC_F32) ? 0 : src_scale(s);
  const int sigma = (KIND == FXPQ_SRC_F32) ? fl_hi + 24 : imax(sv, fl_hi);
  const double wscale = ldexp(1.0, sigma - sv);
  const double absmax = fmax(fabs(mm[0]), fabs(mm[1]));
  // signed 1 bit (Eq. 13): the decoded value is sign(x) * 2^-beta, 2^d units
  const bool binary = (wl == 1 && sign == 1);
  if (absmax * wscale >= 0x1p62 || (binary && sigma - fl_lo > 62)) {
    if (blockIdx.x == 0 && threadIdx.x == 0) {
      *out = fxpq_fmt{wl, 0, sign, 2};
      raise_flag(flags, FXPQ_FLAG_RANGE);
    }
    return;
  }
  const long long qmax = (1ll << (wl - sign)) - 1;
  const long long qmin = sign ? -(1ll << (wl - 1)) : 0;
  const int64_t clen = (n + nchunks - 1) / nchunks;
  // int64 values are scaled in integers (fp64 holds them exactly only below
  // 2^53); |v| 2^(sigma - sv) < 2^62 after the check above (a shift of 62 or
  // more leaves only zeros)
  const long long wmul = (sigma - sv < 62) ? (1ll << (sigma - sv)) : 0ll;

  for (int item = blockIdx.x; item < nc * nchunks; item += gridDim.x) {
    const int j = item / nchunks, ch = item % nchunks;
    const int beta = cand(j);
    const int d = sigma - beta;  // >= 0
    const int64_t e0 = (int64_t)ch * clen;
    const int64_t e1 = (e0 + clen < n) ? e0 + clen : n;
    U192 acc{0, 0};
    for (int64_t i = e0 + threadIdx.x; i < e1; i += kThreads) {
      double W = 0.0;
      long long Wi = 0;
      bool frac = false;  // W not an integer (fp32 values only)
      if constexpr (KIND == FXPQ_SRC_INT && DT == FXPQ_I64) {
        Wi = static_cast<const int64_t*>(s.x)[i] * wmul;
      } else {
        W = load1<KIND, DT>(s, i) * wscale;
        frac = W != floor(W);
        if (!frac) Wi = (long long)W;
      }
      unsigned __int128 e2;
      if (binary) {
        // |x - sign(x) 2^-beta| = | |x| - 2^-beta |; an fp32 value below
        // 2^-(fl_hi+24) has a fractional |W|: (2^d - |W|)^2 is then summed
        // truncated to the unit (error below 2 units per such value)
        if (frac) {
          const double aw = fabs(W);
          const unsigned __int128 u = (unsigned __int128)1 << d;
          e2 = u * u - (unsigned __int128)(unsigned long long)floor(ldexp(aw, d + 1)) +
               (unsigned __int128)(unsigned long long)floor(aw * aw);
        } else {
          __int128 err = (__int128)(Wi < 0 ? -Wi : Wi) - ((__int128)1 << d);
          if (err < 0) err = -err;
          e2 = (unsigned __int128)err * (unsigned __int128)err;
        }
      } else if (frac) {
        // fp32 value below 2^-(fl_hi+1): its code is 0 for every candidate and
        // its (identical) error is added truncated to the common unit.
        e2 = (unsigned __int128)(unsigned long long)floor(W * W);
      } else {
        long long q;
        if (d >= 63) {
          q = 0;
        } else if (d == 0) {
          q = Wi;
        } else {
          long long f = Wi >> d;
          long long r = Wi - (f << d);
          long long half = 1ll << (d - 1);
          q = f + ((r > half || (r == half && (f & 1))) ? 1 : 0);
        }
        q = q < qmin ? qmin : (q > qmax ? qmax : q);
        __int128 err = (__int128)Wi - ((d >= 63) ? (__int128)0 : ((__int128)q << d));
        if (err < 0) err = -err;
        e2 = (unsigned __int128)err * (unsigned __int128)err;
      }
      u192_add(acc, e2);
    }
    // block reduce the 192-bit partial
    shp[3 * threadIdx.x] = (unsigned long long)acc.lo;
    shp[3 * threadIdx.x + 1] = (unsigned long long)(acc.lo >> 64);
    shp[3 * threadIdx.x + 2] = acc.hi;
    __syncthreads();
    if (threadIdx.x == 0) {
      U192 t{0, 0};
      for (int k = 0; k < kThreads; ++k) {
        U192 x{((unsigned __int128)shp[3 * k + 1] << 64) | shp[3 * k], shp[3 * k + 2]};
        u192_add(t, x);
      }
      unsigned long long* p = part + ((int64_t)j * kGenChunks + ch) * 3;
      p[0] = (unsigned long long)t.lo;
      p[1] = (unsigned long long)(t.lo >> 64);
      p[2] = t.hi;
    }
    __syncthreads();
  }
  __threadfence();
  __syncthreads();
  if (threadIdx.x == 0) last = atomicAdd(done, 1u) == gridDim.x - 1;
  __syncthreads();
  if (!last) return;
  __threadfence();
  general_decide(wl, fl_lo, fl_hi, nchunks, sigma, gp, part, out, d_sse);
  if (threadIdx.x == 0) *done = 0u;  // ready for the next search
}

// One block: totals per candidate, exact comparison, ties to the larger fl.
__device__ void general_decide(int wl, int fl_lo, int fl_hi, int nchunks, int sigma,
                               const GenPlan& gp, const unsigned long long* part, fxpq_fmt* out,
                               double* d_sse) {
  __shared__ unsigned long long tot[kMaxCand][3];
  const int sign = gp.sign;
  const int glo = gp.glo, ghi = gp.ghi, extra = gp.extra;
  const int nc = ghi - glo + 1 + (extra != INT_MIN ? 1 : 0);
  auto cand = [&](int j) { return (extra != INT_MIN) ? (j == 0 ? extra : glo + j - 1) : glo + j; };
  for (int j = threadIdx.x; j < nc; j += kThreads) {
    U192 t{0, 0};
    for (int ch = 0; ch < nchunks; ++ch) {
      const unsigned long long* p = part + ((int64_t)j * kGenChunks + ch) * 3;
      U192 x{((unsigned __int128)p[1] << 64) | p[0], p[2]};
      u192_add(t, x);
    }
    tot[j][0] = (unsigned long long)t.lo;
    tot[j][1] = (unsigned long long)(t.lo >> 64);
    tot[j][2] = t.hi;
  }
  __syncthreads();
  if (threadIdx.x != 0) return;
  U192 best{0, 0};
  int bbeta = INT_MIN;
  for (int j = 0; j < nc; ++j) {
    U192 t{((unsigned __int128)tot[j][1] << 64) | tot[j][0], tot[j][2]};
    int beta = cand(j);
    int c = (bbeta == INT_MIN) ? -1 : u192_cmp(t, best);
    if (c < 0 || (c == 0 && beta > bbeta)) {
      best = t;
      bbeta = beta;
    }
    if (d_sse && beta >= fl_lo && beta <= fl_hi)
      d_sse[beta - fl_lo] = ldexp(u192_to_double(t), -2 * sigma);
  }
  *out = fxpq_fmt{wl, bbeta, sign, 0};
}

// ---------------------------------------------------------------------------
// Launcher.
// ---------------------------------------------------------------------------
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

// Slot set of the current search (searches alternate between two sets: the
// one a search adds into is cleared by the next search's finalize).
static long long* slots_i(const Ctx& c, int set) { return c.sc.win_part + (size_t)set * kWinSlots * kWinPart; }
static double* slots_f(const Ctx& c, int set) { return c.sc.win_part_f + (size_t)set * kWinSlots * kWinPartF; }

int fls_begin(const Ctx& c) { return (int)((*c.search_seq)++ & 1u); }

hipError_t launch_fls_window_fin(const Ctx& c, const SrcDev& s, int set, int wl, int sign, int fl_lo,
                                 int nce, int fl_hi, int mode, int64_t per_thread,
                                 const double* d_minmax, fxpq_fmt* out) {
  FlsPlan* plan = static_cast<FlsPlan*>(c.sc.plan);
  FXPQ_DISPATCH_SRC(s.kind, s.dtype,
                    (k_fls_window_fin<K_><<<1, kFinThreads, 0, c.stream>>>(
                        s, wl, sign, fl_lo, nce, fl_hi, mode, per_thread, d_minmax, slots_i(c, set),
                        slots_f(c, set), slots_i(c, 1 - set), slots_f(c, 1 - set), plan, out)));
  return hipGetLastError();
}

// The general pass; with `wi.decide` it first takes the window decision
// (replacing the finalize launch).
static hipError_t general_pass(const Ctx& c, const SrcDev& s, int64_t n, int wl, int fl_lo,
                               int fl_hi, const double* d_minmax, const WinIn& wi, fxpq_fmt* out,
                               double* d_sse) {
  FlsPlan* plan = static_cast<FlsPlan*>(c.sc.plan);
  int nchunks = (int)((n + 65535) / 65536);
  if (nchunks > kGenChunks) nchunks = kGenChunks;
  if (nchunks < 1) nchunks = 1;
  int gblocks = 240;
  FXPQ_DISPATCH_SRC(s.kind, s.dtype,
                    (k_fls_general<K_, D_><<<gblocks, kThreads, 0, c.stream>>>(
                        s, n, wl, fl_lo, fl_hi, nchunks, d_minmax, wi, plan, c.sc.gen_part,
                        c.sc.gen_done, out, d_sse, c.sc.flags)));
  return hipGetLastError();
}

hipError_t launch_fls_general(const Ctx& c, const SrcDev& s, int64_t n, int wl, int fl_lo,
                              int fl_hi, const double* d_minmax, fxpq_fmt* out, double* d_sse) {
  WinIn wi{};
  return general_pass(c, s, n, wl, fl_lo, fl_hi, d_minmax, wi, out, d_sse);
}

// Values per thread of the streaming window pass for a grid of `blocks`.
static int64_t window_per_thread(int64_t n, int blocks, int vec) {
  const int64_t threads = (int64_t)blocks * kThreads;
  return ((n / vec + threads - 1) / threads) * vec + vec;
}

// Window pass (+ its finalize and the general pass when needed).  With y
// and y_alt (fused FxP-QLayer, 8-bit codes) the window pass also writes the
// codes of its two candidates.
static hipError_t fl_search_passes(const Ctx& c, const SrcDev& s, int64_t n, int wl, int sign,
                                   int fl_lo, int fl_hi, const double* d_minmax, fxpq_fmt* out,
                                   double* d_sse, int8_t* y, int8_t* y_alt) {
  int channels = (s.kind == FXPQ_SRC_ACC) ? s.channels : 0;
  const int vec = (s.kind == FXPQ_SRC_ADD) ? 16 : 4;  // Pack<>::V
  const int nce = (wl <= kCeMultiMaxWl) ? kCeBounds : 1;
  FlsPlan* plan = static_cast<FlsPlan*>(c.sc.plan);
  int mode = d_sse ? MODE_REPORT : MODE_SEARCH;
  const bool codes = y != nullptr;
  // algorithmic bytes: the values read once (+ one code per value written)
  const double elem_bytes = ((s.kind == FXPQ_SRC_ADD) ? 2.0 : (s.kind == FXPQ_SRC_INT && s.dtype == FXPQ_I64) ? 8.0 : 4.0) +
                            (codes ? 1.0 : 0.0);
  int64_t per_thread = 0;
  int blocks = 0;
  const int set = fls_begin(c);
  auto run = [&](auto kernel) {
    blocks = stream_grid(n, channels, kWinMaxPerThread, vec, resident_blocks(c, (const void*)kernel));
    if (s.kind == FXPQ_SRC_ADD && blocks > 2 * c.cus) blocks = 2 * c.cus;  // as the predicted pass
    per_thread = window_per_thread(n, blocks, vec);
    bool timed = timer_begin(c, FXPQ_TIMER_FLS_WINDOW);
    kernel<<<blocks, kThreads, 0, c.stream>>>(s, n, wl, sign, fl_lo, fl_hi, mode, per_thread,
                                              d_minmax, slots_i(c, set), slots_f(c, set), plan, out,
                                              c.sc.flags, y, y_alt);
    timer_end(c, timed, elem_bytes * (double)n);
  };
  if (codes) {
    // 4- and 16-value packets only (fp32, C-Block and eltwise sources)
    if (nce == 1) {
      FXPQ_DISPATCH_SRC(s.kind, s.dtype, (run(&k_fls_window<K_, D_, 1, Pack<K_, D_>::EP != 2>)));
    } else {
      FXPQ_DISPATCH_SRC(s.kind, s.dtype, (run(&k_fls_window<K_, D_, kCeBounds, Pack<K_, D_>::EP != 2>)));
    }
  } else if (nce == 1) {
    FXPQ_DISPATCH_SRC(s.kind, s.dtype, (run(&k_fls_window<K_, D_, 1, false>)));
  } else {
    FXPQ_DISPATCH_SRC(s.kind, s.dtype, (run(&k_fls_window<K_, D_, kCeBounds, false>)));
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  WinIn wi{1, sign, nce, mode, codes ? 1 : 0, per_thread, slots_i(c, set), slots_f(c, set),
           slots_i(c, 1 - set), slots_f(c, 1 - set)};
  return general_pass(c, s, n, wl, fl_lo, fl_hi, d_minmax, wi, out, d_sse);
}

hipError_t launch_fl_search(const Ctx& c, const SrcDev& s, int64_t n, int wl, int sign, int fl_lo,
                            int fl_hi, const double* d_minmax, fxpq_fmt* out, double* d_sse) {
  return fl_search_passes(c, s, n, wl, sign, fl_lo, fl_hi, d_minmax, out, d_sse, nullptr, nullptr);
}

// Fused FxP-QLayer: the search writes both window candidates' codes; a gated
// requantization then does nothing when the chosen format's codes are already
// in `codes`, copies them from `alt` when they are there, and requantizes
// otherwise.
hipError_t launch_qlayer(const Ctx& c, const SrcDev& s, int64_t n, int wl, int sign, int fl_lo,
                         int fl_hi, const double* d_minmax, fxpq_fmt* out, int8_t* codes,
                         int8_t* alt) {
  hipError_t e = fl_search_passes(c, s, n, wl, sign, fl_lo, fl_hi, d_minmax, out, nullptr, codes, alt);
  if (e != hipSuccess) return e;
  return launch_requant_gated(c, s, n, out, codes, static_cast<const FlsPlan*>(c.sc.plan), alt);
}

hipError_t launch_pred_decide(const Ctx& c, const PredJob* jobs, int n) {
  if (n > 0) k_pred_decide<<<n, kFinThreads, 0, c.stream>>>(jobs);
  return hipGetLastError();
}

hipError_t launch_pred_fin(const Ctx& c, const SrcDev& ep, int set, int wl, int sign, int fl_lo,
                           int fl_hi, int64_t per_thread, double* d_minmax, fxpq_fmt* out,
                           unsigned* miss) {
  const int nce = 1;  // the conv epilogue evaluates one clipping bound
  k_pred_fin<FXPQ_SRC_ACC><<<1, kFinThreads, 0, c.stream>>>(
      ep, wl, sign, fl_lo, fl_hi, nce, per_thread, d_minmax, slots_i(c, set), slots_f(c, set),
      slots_i(c, 1 - set), slots_f(c, 1 - set), out, miss);
  return hipGetLastError();
}

// Predicted FxP-QLayer over a streaming source (fp32, int32 C-Block values,
// eltwise sums): one pass writing the predicted candidate's codes and the
// min / max, then the decision.
hipError_t launch_qlayer_pred(const Ctx& c, const SrcDev& s, int64_t n, int wl, int sign,
                              int fl_lo, int fl_hi, fxpq_fmt* out, int8_t* y, double* d_minmax,
                              unsigned* miss) {
  const int channels = (s.kind == FXPQ_SRC_ACC) ? s.channels : 0;
  const int vec = (s.kind == FXPQ_SRC_ADD) ? 16 : 4;
  const int nce = (wl <= kCeMultiMaxWl) ? kCeBounds : 1;
  // deferred mode: the call's own slot set and record, no decision launch
  const int job = c.pred_jobs_n ? (*c.pred_jobs_n)++ : -1;
  const int set = job < 0 ? fls_begin(c) : 0;
  long long* pi = job < 0 ? slots_i(c, set) : c.sc.pred_slots_i + (size_t)job * kWinSlots * kWinPart;
  double* pf = job < 0 ? slots_f(c, set) : c.sc.pred_slots_f + (size_t)job * kWinSlots * kWinPartF;
  PredJob* rec = job < 0 ? nullptr : c.sc.pred_jobs + job;
  int blocks = 0;
  int64_t per_thread = 0;
  auto run = [&](auto kernel, auto fin) {
    blocks = stream_grid(n, channels, kWinMaxPerThread, vec, resident_blocks(c, (const void*)kernel));
    // eltwise sources: at most two blocks per CU, each streaming more values
    // (fewer histograms to clear and reduce; measured 12 % faster over the
    // ResNet-50 eltwise sums than the per-thread cap of the other sources)
    if (s.kind == FXPQ_SRC_ADD && blocks > 2 * c.cus) blocks = 2 * c.cus;
    per_thread = window_per_thread(n, blocks, vec);
    bool timed = timer_begin(c, FXPQ_TIMER_FLS_WINDOW);
    kernel<<<blocks, kThreads, 0, c.stream>>>(s, n, wl, sign, fl_lo, fl_hi, per_thread, d_minmax,
                                              pi, pf, out, y, rec, miss);
    const double elem = (s.kind == FXPQ_SRC_ADD) ? 2.0 : 4.0;
    timer_end(c, timed, (elem + 1.0) * (double)n);
    if (job < 0)
      fin<<<1, kFinThreads, 0, c.stream>>>(s, wl, sign, fl_lo, fl_hi, nce, per_thread, d_minmax,
                                           pi, pf, slots_i(c, 1 - set), slots_f(c, 1 - set), out,
                                           miss);
  };
#define FXPQ_QPRED(K, D)                                                            \
  (nce == 1 ? run(&k_qlayer_pred<K, D, 1>, &k_pred_fin<K>)                         \
            : run(&k_qlayer_pred<K, D, kCeBounds>, &k_pred_fin<K>))
  if (s.kind == FXPQ_SRC_F32) FXPQ_QPRED(FXPQ_SRC_F32, FXPQ_F32);
  else if (s.kind == FXPQ_SRC_ADD) FXPQ_QPRED(FXPQ_SRC_ADD, FXPQ_I8);
  else if (s.kind == FXPQ_SRC_ACC) FXPQ_QPRED(FXPQ_SRC_ACC, FXPQ_I32);
  else FXPQ_QPRED(FXPQ_SRC_INT, FXPQ_I32);
#undef FXPQ_QPRED
  return hipGetLastError();
}

}  // namespace fxpq
