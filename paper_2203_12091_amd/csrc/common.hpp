// Internal definitions shared by the libfxpq translation units (gfx950 only).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fxpq.h"

namespace fxpq {

constexpr int kThreads = 256;        // threads per block of the streaming kernels
constexpr int kMaxStreamBlocks = 2048;
constexpr int kMaxConvBlocks = 1 << 20;
constexpr int kWindow = 2;           // candidates of the first FL-search pass
constexpr int kWinSums = 6 * kWindow;  // int64 window-pass sums per slot
// int64 per slot: the sums, then the min / max keys of a predicted call
constexpr int kWinPart = kWinSums + 2;
constexpr int kWinSlots = 64;          // slots the window-pass blocks add into (block % kWinSlots)
// Clipping-error lower bounds the window pass can take above its candidates
// (at fl = b1 + 1, b1 + 2, ...), and fp64 sums per slot: sum W^2 and the bounds.
constexpr int kCeBounds = 4;
constexpr int kWinPartF = 1 + kCeBounds;
// Word lengths up to this one take all kCeBounds bounds (their best fl lies
// above the window more often); longer ones take one.
constexpr int kCeMultiMaxWl = 6;
// Values per thread of the streaming window pass (the grid grows beyond that):
// sums of W * q stay exact for max|W * q| < 2^53 / 512.
constexpr int64_t kWinMaxPerThread = 512;
constexpr int kMaxCand = 160;        // fl_hi - fl_lo + 1 upper bound (|fl| <= 64 plus slack)
constexpr int kGenChunks = 256;      // element chunks of the exact general search

// Device-resident state of one handle.  Offsets into one scratch allocation.
struct Scratch {
  unsigned* flags;          // sticky FXPQ_FLAG_* bits
  double* minmax;           // internal [2]
  double* minmax_part;      // per-block partials [kMaxConvBlocks][2]
  long long* win_part;      // window FL-search integer sums [2][kWinSlots][kWinPart]
  double* win_part_f;       // window FL-search fp64 bound sums [2][kWinSlots][kWinPartF]
                            // (two sets, see fls_begin; a set is 0 when a search starts on it)
  unsigned long long* gen_part;  // general search partials [kMaxCand][kGenChunks][3]
  unsigned* gen_done;       // blocks of the general pass finished (0 between searches)
  void* plan;               // FlsPlan
  int32_t* sink;            // target of discarded stores [64]
  // deferred decisions of predicted calls: one record and one slot set per
  // call since the last fxpq_predicted_decide (slot sets zero between uses)
  struct PredJob* pred_jobs;     // [kMaxPredJobs]
  long long* pred_slots_i;       // [kMaxPredJobs][kWinSlots][kWinPart]
  double* pred_slots_f;          // [kMaxPredJobs][kWinSlots][kWinPartF]
  // first-layer filters re-laid with every filter row padded to 8 taps
  // (kRgbWBytes; nullptr: not available, the packed RGB loader runs)
  int8_t* rgb_w;
};

constexpr size_t kRgbWBytes = 1 << 16;

// Pending decisions of predicted calls in deferred mode (at most this many
// between two fxpq_predicted_decide calls).
constexpr int kMaxPredJobs = 256;

// Everything a kernel needs to produce the value v_i of an FxP-QLayer input,
// as an exact double (integers below 2^53), plus its fractional length.
struct SrcDev {
  int kind;
  int dtype;
  const void* x;
  const void* x2;
  int dtype2;
  int relu;  // ADD
  const int32_t* d_scale;
  const fxpq_fmt* fa;
  const fxpq_fmt* fb;
  // epilogue (ACC)
  int channels;
  int fl_w;
  const fxpq_fmt* fin;
  const int32_t* bias;
  int fl_bias;
  int ep_relu;
  const int32_t* scale;
  int fl_scale;
  const int32_t* shift;
  int fl_shift;
};

// Uniform part of the C-Block epilogue: exponents of the exact alignment.
// What the decision of a predicted call needs, written by block 0 of the
// call's own kernel in deferred mode and read by the batched decision.
struct PredJob {
  SrcDev s;
  int wl, sign, fl_lo, fl_hi, nce;
  int64_t per_thread;
  double* mm;          // predicted min / max in, this call's out
  fxpq_fmt* out;       // the format the codes were written with (prediction)
  unsigned* miss;
  long long* pi;       // the call's slot set
  double* pf;
};

struct EpiU {
  int s_out;    // fractional length of the epilogue value
  int sh_acc;   // acc * 2^sh_acc ...
  int sh_bias;  // bias * 2^sh_bias (before the Scale multiply)
  int sh_mid;   // (...)*scale * 2^sh_mid
  int sh_shift; // shift * 2^sh_shift
  int u8off;    // input codes stored as u - 128: add 128 * colsum
};

__host__ __device__ inline int imax(int a, int b) { return a > b ? a : b; }

__device__ inline EpiU epi_uniform(const SrcDev& s) {
  EpiU u;
  int s_acc = s.fin->fl + s.fl_w;
  int s1 = s.bias ? imax(s_acc, s.fl_bias) : s_acc;
  u.sh_acc = s1 - s_acc;
  u.sh_bias = s.bias ? s1 - s.fl_bias : 0;
  int s2 = s.scale ? s1 + s.fl_scale : s1;
  int s3 = s.shift ? imax(s2, s.fl_shift) : s2;
  u.sh_mid = s3 - s2;
  u.sh_shift = s.shift ? s3 - s.fl_shift : 0;
  u.s_out = s3;
  u.u8off = 0;
  return u;
}

// Per-channel epilogue codes (Scale multiplier, bias, Scale addend) of channel
// c; 1 / 0 / 0 where the epilogue has none.  The loads are unconditional
// (absent operands read a constant) so that no wait follows them.
struct EpiRaw {
  int32_t sc, b, sh;
};

__device__ int32_t kEpiOne = 1;  // never written
__device__ int32_t kEpiZero = 0;  // never written

__device__ inline EpiRaw epi_channel_load(const SrcDev& s, int c) {
  EpiRaw r;
  r.sc = *(s.scale ? s.scale + c : &kEpiOne);
  r.b = *(s.bias ? s.bias + c : &kEpiZero);
  r.sh = *(s.shift ? s.shift + c : &kEpiZero);
  return r;
}

// Per-channel multiplier and addend: v = relu(acc * M + A), exact while |v| < 2^53.
__device__ inline void epi_channel_raw(const SrcDev& s, const EpiU& u, const EpiRaw& r, double& M,
                                       double& A) {
  const double sc = (double)r.sc;
  M = ldexp(sc, u.sh_acc + u.sh_mid);
  double a = s.bias ? ldexp((double)r.b, u.sh_bias + u.sh_mid) * sc : 0.0;
  if (s.shift) a += ldexp((double)r.sh, u.sh_shift);
  A = a;
}

__device__ inline void epi_channel(const SrcDev& s, const EpiU& u, int c, double& M, double& A) {
  epi_channel_raw(s, u, epi_channel_load(s, c), M, A);
}

// Fractional length of the values described by s.
__device__ inline int src_scale(const SrcDev& s) {
  switch (s.kind) {
    case FXPQ_SRC_INT: return *s.d_scale;
    case FXPQ_SRC_ACC: return epi_uniform(s).s_out;
    case FXPQ_SRC_ADD: return imax(s.fa->fl, s.fb->fl);
    default: return 0;
  }
}

// 8-bit code storage resolved against a format: 1 when stored as u - 128.
__device__ inline int code_is_off(int dtype, const fxpq_fmt* f) {
  if (dtype == FXPQ_U8OFF) return 1;
  if (dtype == 6 /* C8 */) return f && f->sign == 0;
  return 0;
}

// ---- kernel timing (measurement only) ------------------------------------------
struct Timer {
  int kind = 0;           // fxpq_timer_kind being timed
  int capacity = 0;       // event pairs available
  int used = 0;
  double work = 0.0;      // summed algorithmic bytes or operations
  hipEvent_t* ev = nullptr;  // 2 * capacity events
};

// ---- launchers implemented in the kernel translation units -------------------
struct Ctx {
  hipStream_t stream;
  Scratch sc;
  Timer* timer;
  int cus;                  // compute units of the handle's device
  unsigned* search_seq;     // FL searches enqueued on the handle (host counter)
  int conv_tiling;          // fxpq_conv_tiling
  int* pred_jobs_n;         // deferred mode: pending predicted calls (host counter), else null
};

// Brackets one launch with events when `kind` is being timed.
inline bool timer_begin(const Ctx& c, int kind) {
  Timer* t = c.timer;
  if (!t || t->kind != kind || t->used >= t->capacity) return false;
  return hipEventRecord(t->ev[2 * t->used], c.stream) == hipSuccess;
}
inline void timer_end(const Ctx& c, bool started, double work) {
  if (!started) return;
  Timer* t = c.timer;
  if (hipEventRecord(t->ev[2 * t->used + 1], c.stream) == hipSuccess) {
    t->used += 1;
    t->work += work;
  }
}

// Blocks of `kernel` (kThreads threads, no dynamic LDS) resident on the
// handle's device at once; 0 if unknown.  Cached per kernel.
int resident_blocks(const Ctx& c, const void* kernel);
// Grid of a streaming launch over n values, `vec` per thread per iteration.
int stream_grid(int64_t n, int channels, int64_t max_per_thread, int vec, int resident);
hipError_t launch_minmax(const Ctx& c, const SrcDev& s, int64_t n, double* out);
int minmax_blocks(const Ctx& c, const SrcDev& s, int64_t n);
hipError_t launch_minmax_fin(const Ctx& c, const double* part, int nb, double* out);
hipError_t launch_requant(const Ctx& c, const SrcDev& s, int64_t n, const fxpq_fmt* fmt, void* codes,
                          int code_type);
hipError_t launch_requant_addmm(const Ctx& c, const SrcDev& s, int64_t n, const fxpq_fmt* fmt,
                                void* codes, int code_type, const int8_t* b, int b_type,
                                const fxpq_fmt* fmt_b, int relu, double* d_add_minmax);
hipError_t launch_fl_search(const Ctx& c, const SrcDev& s, int64_t n, int wl, int sign, int fl_lo,
                            int fl_hi, const double* d_minmax, fxpq_fmt* out, double* d_sse);
// FL searches alternate between two sets of window slots: returns this
// search's set (the next search's finalize clears it).
int fls_begin(const Ctx& c);
hipError_t launch_fls_window_fin(const Ctx& c, const SrcDev& s, int set, int wl, int sign, int fl_lo,
                                 int nce, int fl_hi, int mode, int64_t per_thread,
                                 const double* d_minmax, fxpq_fmt* out);
struct FlsPlan;
// FL search + requantization to 8-bit codes (fused FxP-QLayer; C8 storage).
hipError_t launch_qlayer(const Ctx& c, const SrcDev& s, int64_t n, int wl, int sign, int fl_lo,
                         int fl_hi, const double* d_minmax, fxpq_fmt* out, int8_t* codes,
                         int8_t* alt);
// Requantization to C8 codes gated by a fused search's plan: nothing when
// `codes` already holds the chosen format's codes, a copy from `alt` when it
// holds them, else requantization.
hipError_t launch_requant_gated(const Ctx& c, const SrcDev& s, int64_t n, const fxpq_fmt* fmt,
                                int8_t* codes, const FlsPlan* plan, const int8_t* alt);
hipError_t launch_fls_general(const Ctx& c, const SrcDev& s, int64_t n, int wl, int fl_lo,
                              int fl_hi, const double* d_minmax, fxpq_fmt* out, double* d_sse);
hipError_t launch_conv(const Ctx& c, const fxpq_conv_desc& d, const void* x, int x_type,
                       const int8_t* w, const int32_t* colsum, const SrcDev* ep, int32_t* acc,
                       double* d_minmax);
// Blocks of the fused / predicted C-Block launch; -1 when it does not apply
// (the padded RGB layout: the predicted C-Block only, rgb_ok).
int conv_fused_blocks(const fxpq_conv_desc& d, int cus, bool rgb_ok = false);
hipError_t launch_conv_pred(const Ctx& c, const fxpq_conv_desc& d, const void* x, int x_type,
                            const int8_t* w, const int32_t* colsum, const SrcDev& ep, int wl,
                            int sign, int fl_lo, int fl_hi, fxpq_fmt* out, int8_t* y,
                            double* d_minmax, unsigned* miss);
hipError_t launch_pred_fin(const Ctx& c, const SrcDev& ep, int set, int wl, int sign, int fl_lo,
                           int fl_hi, int64_t per_thread, double* d_minmax, fxpq_fmt* out,
                           unsigned* miss);
hipError_t launch_qlayer_pred(const Ctx& c, const SrcDev& s, int64_t n, int wl, int sign,
                              int fl_lo, int fl_hi, fxpq_fmt* out, int8_t* y, double* d_minmax,
                              unsigned* miss);
// One launch deciding the n pending predicted calls recorded in jobs.
hipError_t launch_pred_decide(const Ctx& c, const PredJob* jobs, int n);
hipError_t launch_conv_fused(const Ctx& c, const fxpq_conv_desc& d, const void* x, int x_type,
                             const int8_t* w, const int32_t* colsum, const SrcDev& ep, int wl,
                             int sign, int fl_lo, int fl_hi, fxpq_fmt* out, int8_t* y, int y_type,
                             double* d_minmax);
hipError_t launch_dequant(const Ctx& c, const void* codes, int code_type, const fxpq_fmt* fmt,
                          int64_t n, float* out);
hipError_t launch_logit_ties(const Ctx& c, const void* scores, int dtype, int rows, int cols,
                             long long* out);
hipError_t launch_preprocess(const Ctx& c, const SrcDev& s, const double* d_minmax, int wl,
                             int strategy, int rule, int fl_lo, int fl_hi, fxpq_fmt* out);
hipError_t launch_colsum(const Ctx& c, const int8_t* w, int64_t k, int64_t len, int32_t* out);
// Wide C-Blocks (k_wide.hip): digit planes of int32 codes, and the exact
// combination of the plane contractions with the epilogue.
// One fused wide C-Block contraction (see k_wide_fused).
struct WideFusedArgs {
  const int8_t* px;   // np_x input byte planes (NHWC), plane stride xs
  int64_t xs;
  const int8_t* pw;   // np_w weight digit planes [K][wrow], plane stride ws
  int64_t ws;
  const int32_t* cs;  // column sums of the weight planes [np_w][K]
  int np_x, np_w, sign_x;
  int N, H, W, C, K, R, S, stride, pad, Ho, Wo, M, kdepth, wrow;
  SrcDev ep;
  int64_t* v;
  int32_t* d_scale;
  unsigned* flags;
};
hipError_t launch_wide_fused(const Ctx& c, const WideFusedArgs& a, bool wide);
hipError_t launch_wide_split_x(const Ctx& c, const int32_t* x, int64_t n, int np, int sign,
                               int64_t plane_stride, int8_t* planes);
hipError_t launch_wide_split_w(const Ctx& c, const int32_t* w, int64_t n, int np, int sign,
                               int64_t plane_stride, int8_t* planes);
hipError_t launch_wide_combine(const Ctx& c, const int32_t* acc, int64_t mk, int np_x, int np_w,
                               const SrcDev& ep, int64_t* v, int32_t* d_scale);
hipError_t launch_acc_overflow(const Ctx& c, const int32_t* acc, int64_t n, int bits,
                               int64_t* count);
hipError_t launch_maxpool(const Ctx& c, const int8_t* x, int n, int h, int w, int ch, int ks,
                          int stride, int pad, int8_t* y);
hipError_t launch_avgpool(const Ctx& c, const int8_t* x, int dtype, const fxpq_fmt* fmt, int n,
                          int hw, int ch, int64_t recip, int64_t* y);
hipError_t launch_layer_error(const Ctx& c, const float* ref, const void* codes, int code_type,
                              const fxpq_fmt* fmt, int64_t n, double* out);
hipError_t launch_epi_scale(const Ctx& c, const SrcDev& s, int32_t* out);
hipError_t launch_teacher_conv(const Ctx& c, const fxpq_conv_desc& d, const float* x,
                               const float* w, float* y);
hipError_t launch_teacher_affine(const Ctx& c, const float* t, int64_t n, int channels,
                                 const float* a1, const float* a2, const float* bias, int relu,
                                 float* y);
hipError_t launch_teacher_add(const Ctx& c, const float* a, const float* b, int64_t n, int relu,
                              float* y);
hipError_t launch_teacher_maxpool(const Ctx& c, const float* x, int n, int h, int w, int ch,
                                  int ks, int stride, int pad, float* y);
hipError_t launch_teacher_avgpool(const Ctx& c, const float* x, int n, int hw, int ch, float* y);

}  // namespace fxpq
