// libfxpq C ABI: handle management, host-side argument checks and dispatch to
// the kernels.  Every function is extern "C"; no exception or C++ type crosses
// the boundary.
#include <stdint.h>
#include <string.h>

#include <mutex>
#include <new>

#include "common.hpp"

using namespace fxpq;

struct fxpq_handle_s {
  int device;
  int cus;  // compute units
  hipStream_t stream;
  void* scratch;
  size_t scratch_bytes;
  Scratch sc;
  Timer timer;
  unsigned search_seq = 0;
  int conv_tiling = FXPQ_TILING_AUTO;
  int pred_defer = 0;  // predicted calls defer their decisions
  int pred_n = 0;      // pending deferred decisions
};

constexpr int kTimerPairs = 16384;

namespace {

constexpr int64_t kMaxFlsBlocks = 1 << 16;

size_t align_up(size_t v, size_t a) { return (v + a - 1) / a * a; }

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

bool is_code8(int t) { return t == FXPQ_I8 || t == FXPQ_U8OFF || t == FXPQ_C8; }

bool is_code(int t) { return is_code8(t) || t == FXPQ_I16 || t == FXPQ_I32 || t == FXPQ_U32; }

size_t code_align(int t) { (void)t; return 16; }

Ctx ctx(fxpq_handle h) {
  return Ctx{h->stream, h->sc, &h->timer, h->cus, &h->search_seq, h->conv_tiling,
             h->pred_defer ? &h->pred_n : nullptr};
}

fxpq_status hip_status(hipError_t e) { return e == hipSuccess ? FXPQ_OK : FXPQ_ERR_HIP; }

// Device context guard: calls run on the handle's device.
struct DeviceGuard {
  int prev = -1;
  explicit DeviceGuard(int dev) {
    (void)hipGetDevice(&prev);
    if (prev != dev) (void)hipSetDevice(dev);
  }
  ~DeviceGuard() {
    int cur = -1;
    (void)hipGetDevice(&cur);
    if (prev >= 0 && cur != prev) (void)hipSetDevice(prev);
  }
};

fxpq_status to_dev(const fxpq_src* s, int64_t n, SrcDev* d) {
  if (!s || !s->x) return FXPQ_ERR_INVALID_ARG;
  memset(d, 0, sizeof(*d));
  d->kind = s->kind;
  d->dtype = s->dtype;
  d->x = s->x;
  switch (s->kind) {
    case FXPQ_SRC_F32:
      if (!aligned(s->x, 16)) return FXPQ_ERR_INVALID_ARG;
      d->dtype = FXPQ_F32;
      break;
    case FXPQ_SRC_INT:
      if (s->dtype != FXPQ_I32 && s->dtype != FXPQ_I64) return FXPQ_ERR_INVALID_ARG;
      if (!s->d_scale || !aligned(s->x, 16)) return FXPQ_ERR_INVALID_ARG;
      d->d_scale = s->d_scale;
      break;
    case FXPQ_SRC_ACC: {
      const fxpq_epilogue* e = s->ep;
      if (!e || !e->d_fmt_in || e->channels < 1 || !aligned(s->x, 16)) return FXPQ_ERR_INVALID_ARG;
      if (n % e->channels != 0) return FXPQ_ERR_INVALID_ARG;
      d->dtype = FXPQ_I32;
      d->channels = e->channels;
      d->fl_w = e->fl_w;
      d->fin = e->d_fmt_in;
      d->bias = e->bias;
      d->fl_bias = e->fl_bias;
      d->ep_relu = e->relu ? 1 : 0;
      d->scale = e->scale;
      d->fl_scale = e->fl_scale;
      d->shift = e->shift;
      d->fl_shift = e->fl_shift;
      break;
    }
    case FXPQ_SRC_ADD:
      if (!s->x2 || !s->d_fmt_a || !s->d_fmt_b) return FXPQ_ERR_INVALID_ARG;
      if (!is_code8(s->dtype) || !is_code8(s->dtype2)) return FXPQ_ERR_INVALID_ARG;
      if (!aligned(s->x, 16) || !aligned(s->x2, 16)) return FXPQ_ERR_INVALID_ARG;
      d->x2 = s->x2;
      d->dtype2 = s->dtype2;
      d->fa = s->d_fmt_a;
      d->fb = s->d_fmt_b;
      d->relu = s->relu ? 1 : 0;
      break;
    default:
      return FXPQ_ERR_INVALID_ARG;
  }
  return FXPQ_OK;
}

void epi_to_dev(const fxpq_epilogue* e, SrcDev* d) {
  memset(d, 0, sizeof(*d));
  d->kind = FXPQ_SRC_ACC;
  d->dtype = FXPQ_I32;
  d->channels = e->channels;
  d->fl_w = e->fl_w;
  d->fin = e->d_fmt_in;
  d->bias = e->bias;
  d->fl_bias = e->fl_bias;
  d->ep_relu = e->relu ? 1 : 0;
  d->scale = e->scale;
  d->fl_scale = e->fl_scale;
  d->shift = e->shift;
  d->fl_shift = e->fl_shift;
}

}  // namespace

// ---------------------------------------------------------------------------
// FL search that allocates nothing: its scratch is a fixed array in the
// library's device memory (one copy per device, held until the process
// ends), addressed through hipGetSymbolAddress.
// ---------------------------------------------------------------------------
namespace {

constexpr size_t a256(size_t v) { return (v + 255) / 256 * 256; }
constexpr int kStaticMmBlocks = 16384;  // min / max partials the array holds
constexpr int kStaticDevices = 64;
// Layout (bytes).  [0, kSoClearEnd) is cleared by every call: the sticky
// flags, the general pass's block counter and both window slot sets.
constexpr size_t kSoFlags = 0;
constexpr size_t kSoMinmax = 256;
constexpr size_t kSoGenDone = 512;
constexpr size_t kSoWin = 768;
constexpr size_t kSoWinF = kSoWin + a256((size_t)2 * kWinSlots * kWinPart * sizeof(long long));
constexpr size_t kSoClearEnd = kSoWinF + a256((size_t)2 * kWinSlots * kWinPartF * sizeof(double));
constexpr size_t kSoMmPart = kSoClearEnd;
constexpr size_t kSoGen = kSoMmPart + a256((size_t)kStaticMmBlocks * 2 * sizeof(double));
constexpr size_t kSoPlan = kSoGen + a256((size_t)(kMaxCand + 1) * kGenChunks * 3 * sizeof(unsigned long long));
constexpr size_t kStaticBytes = kSoPlan + 256;
static_assert(kStaticBytes == FXPQ_STATIC_SCRATCH_BYTES, "static scratch size in fxpq.h");
static_assert(kSoClearEnd % sizeof(unsigned) == 0, "cleared in 32-bit words");

struct StaticDev {
  void* ptr = nullptr;  // device address of `scratch` on this device
  int cus = 0;
};
std::mutex g_static_mu;
StaticDev g_static[kStaticDevices];

}  // namespace

static __device__ __align__(256) unsigned char scratch[kStaticBytes];

__global__ __launch_bounds__(256) void k_static_clear(unsigned* p, int words) {
  for (int i = threadIdx.x; i < words; i += 256) p[i] = 0u;
}

extern "C" {

const char* fxpq_status_string(fxpq_status s) {
  switch (s) {
    case FXPQ_OK: return "ok";
    case FXPQ_ERR_INVALID_ARG: return "invalid argument";
    case FXPQ_ERR_UNSUPPORTED: return "unsupported";
    case FXPQ_ERR_NONFINITE: return "non-finite input";
    case FXPQ_ERR_OVERFLOW: return "int32 accumulator overflow possible";
    case FXPQ_ERR_HIP: return "HIP runtime error";
    case FXPQ_ERR_ALLOC: return "allocation failed";
  }
  return "unknown status";
}

fxpq_status fxpq_create(fxpq_handle* out, int device) {
  if (!out) return FXPQ_ERR_INVALID_ARG;
  *out = nullptr;
  int count = 0;
  if (hipGetDeviceCount(&count) != hipSuccess || device < 0 || device >= count)
    return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(device);
  fxpq_handle h = new (std::nothrow) fxpq_handle_s();
  if (!h) return FXPQ_ERR_ALLOC;
  h->device = device;
  h->stream = nullptr;
  if (hipDeviceGetAttribute(&h->cus, hipDeviceAttributeMultiprocessorCount, device) != hipSuccess ||
      h->cus < 1) {
    delete h;
    return FXPQ_ERR_HIP;
  }
  size_t off = 0;
  auto take = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  size_t o_flags = take(4);
  size_t o_mm = take(2 * sizeof(double));
  size_t o_gd = take(4);
  size_t o_wp = take((size_t)2 * kWinSlots * kWinPart * sizeof(long long));
  size_t o_wpf = take((size_t)2 * kWinSlots * kWinPartF * sizeof(double));
  size_t o_psi = take((size_t)kMaxPredJobs * kWinSlots * kWinPart * sizeof(long long));
  size_t o_psf = take((size_t)kMaxPredJobs * kWinSlots * kWinPartF * sizeof(double));
  size_t o_mmp = take((size_t)kMaxConvBlocks * 2 * sizeof(double));
  size_t o_gp = take((size_t)(kMaxCand + 1) * kGenChunks * 3 * sizeof(unsigned long long));
  size_t o_plan = take(256);
  size_t o_sink = take(64 * sizeof(int32_t));
  size_t o_jobs = take((size_t)kMaxPredJobs * sizeof(PredJob));
  size_t o_rgbw = take(kRgbWBytes);
  if (hipMalloc(&h->scratch, off) != hipSuccess) {
    delete h;
    return FXPQ_ERR_ALLOC;
  }
  h->scratch_bytes = off;
  char* base = static_cast<char*>(h->scratch);
  h->sc.flags = reinterpret_cast<unsigned*>(base + o_flags);
  h->sc.minmax = reinterpret_cast<double*>(base + o_mm);
  h->sc.minmax_part = reinterpret_cast<double*>(base + o_mmp);
  h->sc.win_part = reinterpret_cast<long long*>(base + o_wp);
  h->sc.win_part_f = reinterpret_cast<double*>(base + o_wpf);
  h->sc.gen_part = reinterpret_cast<unsigned long long*>(base + o_gp);
  h->sc.gen_done = reinterpret_cast<unsigned*>(base + o_gd);
  h->sc.plan = base + o_plan;
  h->sc.sink = reinterpret_cast<int32_t*>(base + o_sink);
  h->sc.pred_jobs = reinterpret_cast<PredJob*>(base + o_jobs);
  h->sc.pred_slots_i = reinterpret_cast<long long*>(base + o_psi);
  h->sc.pred_slots_f = reinterpret_cast<double*>(base + o_psf);
  h->sc.rgb_w = reinterpret_cast<int8_t*>(base + o_rgbw);
  if (hipMemset(h->scratch, 0, o_mmp) != hipSuccess || hipDeviceSynchronize() != hipSuccess) {
    (void)hipFree(h->scratch);
    delete h;
    return FXPQ_ERR_HIP;
  }
  *out = h;
  return FXPQ_OK;
}

fxpq_status fxpq_destroy(fxpq_handle h) {
  if (!h) return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(h->device);
  (void)hipStreamSynchronize(h->stream);
  (void)hipFree(h->scratch);
  if (h->timer.ev) {
    for (int i = 0; i < 2 * h->timer.capacity; ++i) (void)hipEventDestroy(h->timer.ev[i]);
    delete[] h->timer.ev;
  }
  delete h;
  return FXPQ_OK;
}

fxpq_status fxpq_set_stream(fxpq_handle h, void* stream) {
  if (!h) return FXPQ_ERR_INVALID_ARG;
  h->stream = static_cast<hipStream_t>(stream);
  return FXPQ_OK;
}

fxpq_status fxpq_sync_status(fxpq_handle h, uint32_t* flags) {
  if (!h) return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(h->device);
  if (hipStreamSynchronize(h->stream) != hipSuccess) return FXPQ_ERR_HIP;
  uint32_t f = 0;
  if (hipMemcpy(&f, h->sc.flags, 4, hipMemcpyDeviceToHost) != hipSuccess) return FXPQ_ERR_HIP;
  if (hipMemset(h->sc.flags, 0, 4) != hipSuccess) return FXPQ_ERR_HIP;
  if (hipDeviceSynchronize() != hipSuccess) return FXPQ_ERR_HIP;
  if (flags) *flags = f;
  return FXPQ_OK;
}

fxpq_status fxpq_quantize(fxpq_handle h, const float* x, int64_t n, const fxpq_fmt* d_fmt,
                          void* codes, fxpq_dtype code_type) {
  if (!h || n < 0 || !d_fmt) return FXPQ_ERR_INVALID_ARG;
  if (n == 0) return FXPQ_OK;
  if (!x || !codes || !is_code(code_type)) return FXPQ_ERR_INVALID_ARG;
  if (!aligned(x, 16) || !aligned(codes, code_align(code_type))) return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(h->device);
  SrcDev s;
  memset(&s, 0, sizeof(s));
  s.kind = FXPQ_SRC_F32;
  s.dtype = FXPQ_F32;
  s.x = x;
  return hip_status(launch_requant(ctx(h), s, n, d_fmt, codes, code_type));
}

fxpq_status fxpq_requant(fxpq_handle h, const fxpq_src* src, int64_t n, const fxpq_fmt* d_fmt,
                         void* codes, fxpq_dtype code_type) {
  if (!h || n < 0 || !d_fmt) return FXPQ_ERR_INVALID_ARG;
  if (n == 0) return FXPQ_OK;
  if (!codes || !is_code(code_type) || !aligned(codes, code_align(code_type)))
    return FXPQ_ERR_INVALID_ARG;
  SrcDev s;
  fxpq_status st = to_dev(src, n, &s);
  if (st) return st;
  DeviceGuard g(h->device);
  return hip_status(launch_requant(ctx(h), s, n, d_fmt, codes, code_type));
}

fxpq_status fxpq_requant_addmm(fxpq_handle h, const fxpq_src* src, int64_t n,
                               const fxpq_fmt* d_fmt, void* codes, fxpq_dtype code_type,
                               const void* b, fxpq_dtype b_type, const fxpq_fmt* d_fmt_b,
                               int32_t relu, double* d_add_minmax) {
  if (!h || !src || n < 1 || !d_fmt || !codes || !b || !d_fmt_b || !d_add_minmax)
    return FXPQ_ERR_INVALID_ARG;
  if (!is_code8(code_type) || !is_code8(b_type)) return FXPQ_ERR_INVALID_ARG;
  if (src->kind != FXPQ_SRC_ACC) return FXPQ_ERR_UNSUPPORTED;
  if (!aligned(codes, 16) || !aligned(b, 16)) return FXPQ_ERR_INVALID_ARG;
  SrcDev s;
  fxpq_status st = to_dev(src, n, &s);
  if (st) return st;
  DeviceGuard g(h->device);
  return hip_status(launch_requant_addmm(ctx(h), s, n, d_fmt, codes, code_type,
                                         static_cast<const int8_t*>(b), b_type, d_fmt_b,
                                         relu ? 1 : 0, d_add_minmax));
}

fxpq_status fxpq_fl_search(fxpq_handle h, const fxpq_src* src, int64_t n, int32_t wl,
                           int32_t sign, int32_t fl_lo, int32_t fl_hi, fxpq_fmt* d_fmt_out,
                           double* d_sse) {
  if (!h || n < 1 || !d_fmt_out) return FXPQ_ERR_INVALID_ARG;
  if (wl < 1 || wl > 32) return FXPQ_ERR_INVALID_ARG;
  if (sign != 0 && sign != 1 && sign != FXPQ_SIGN_AUTO) return FXPQ_ERR_INVALID_ARG;
  if (fl_lo > fl_hi || fl_lo < -64 || fl_hi > 64) return FXPQ_ERR_INVALID_ARG;
  if (fl_hi - fl_lo + 1 > kMaxCand - 1) return FXPQ_ERR_INVALID_ARG;
  SrcDev s;
  fxpq_status st = to_dev(src, n, &s);
  if (st) return st;
  if (n / ((int64_t)kThreads * kWinMaxPerThread) + 1 > kMaxFlsBlocks - 4096) return FXPQ_ERR_UNSUPPORTED;
  DeviceGuard g(h->device);
  Ctx c = ctx(h);
  const double* mm = src->d_minmax;
  if (!mm) {
    hipError_t e = launch_minmax(c, s, n, h->sc.minmax);
    if (e != hipSuccess) return FXPQ_ERR_HIP;
    mm = h->sc.minmax;
  }
  return hip_status(launch_fl_search(c, s, n, wl, sign, fl_lo, fl_hi, mm, d_fmt_out, d_sse));
}

fxpq_status fxpq_fl_search_static(const fxpq_src* src, int64_t n, int32_t wl, int32_t sign,
                                  int32_t fl_lo, int32_t fl_hi, fxpq_fmt* d_fmt_out,
                                  double* d_sse, void* hip_stream) {
  if (n < 1 || !d_fmt_out) return FXPQ_ERR_INVALID_ARG;
  if (wl < 1 || wl > 32) return FXPQ_ERR_INVALID_ARG;
  if (sign != 0 && sign != 1 && sign != FXPQ_SIGN_AUTO) return FXPQ_ERR_INVALID_ARG;
  if (fl_lo > fl_hi || fl_lo < -64 || fl_hi > 64) return FXPQ_ERR_INVALID_ARG;
  if (fl_hi - fl_lo + 1 > kMaxCand - 1) return FXPQ_ERR_INVALID_ARG;
  SrcDev s;
  fxpq_status st = to_dev(src, n, &s);
  if (st) return st;
  if (n / ((int64_t)kThreads * kWinMaxPerThread) + 1 > kMaxFlsBlocks - 4096) return FXPQ_ERR_UNSUPPORTED;
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0) return FXPQ_ERR_HIP;
  if (dev >= kStaticDevices) return FXPQ_ERR_UNSUPPORTED;
  StaticDev sd;
  {
    // set-up once per device, with that device current: the array's device
    // address (the host-side name `scratch` is not one) and its CU count
    std::lock_guard<std::mutex> lock(g_static_mu);
    if (!g_static[dev].ptr) {
      void* ptr = nullptr;
      int cus = 0;
      if (hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)) != hipSuccess || !ptr) return FXPQ_ERR_HIP;
      if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
          cus < 1)
        return FXPQ_ERR_HIP;
      g_static[dev].cus = cus;
      g_static[dev].ptr = ptr;
    }
    sd = g_static[dev];
  }
  char* base = static_cast<char*>(sd.ptr);
  Scratch sc{};
  sc.flags = reinterpret_cast<unsigned*>(base + kSoFlags);
  sc.minmax = reinterpret_cast<double*>(base + kSoMinmax);
  sc.gen_done = reinterpret_cast<unsigned*>(base + kSoGenDone);
  sc.win_part = reinterpret_cast<long long*>(base + kSoWin);
  sc.win_part_f = reinterpret_cast<double*>(base + kSoWinF);
  sc.minmax_part = reinterpret_cast<double*>(base + kSoMmPart);
  sc.gen_part = reinterpret_cast<unsigned long long*>(base + kSoGen);
  sc.plan = base + kSoPlan;
  sc.sink = nullptr;  // not used by the search
  unsigned seq = 0;   // both slot sets are cleared below: any set will do
  Ctx c{static_cast<hipStream_t>(hip_stream), sc, nullptr, sd.cus, &seq, FXPQ_TILING_AUTO};
  if (!src->d_minmax && minmax_blocks(c, s, n) > kStaticMmBlocks) return FXPQ_ERR_UNSUPPORTED;
  // the array keeps the previous call's contents: zero what a search
  // expects at zero (a fill kernel, not a memset, so the call can be captured)
  k_static_clear<<<1, 256, 0, c.stream>>>(reinterpret_cast<unsigned*>(base),
                                          (int)(kSoClearEnd / sizeof(unsigned)));
  if (hipGetLastError() != hipSuccess) return FXPQ_ERR_HIP;
  const double* mm = src->d_minmax;
  if (!mm) {
    hipError_t e = launch_minmax(c, s, n, sc.minmax);
    if (e != hipSuccess) return FXPQ_ERR_HIP;
    mm = sc.minmax;
  }
  return hip_status(launch_fl_search(c, s, n, wl, sign, fl_lo, fl_hi, mm, d_fmt_out, d_sse));
}

fxpq_status fxpq_preprocess(fxpq_handle h, const fxpq_src* src, int64_t n, int32_t wl,
                            int32_t strategy, int32_t psi_rule, int32_t fl_lo, int32_t fl_hi,
                            fxpq_fmt* d_fmt_out) {
  if (!h || n < 1 || !d_fmt_out) return FXPQ_ERR_INVALID_ARG;
  if (wl < 2 || wl > 32) return wl == 1 ? FXPQ_ERR_UNSUPPORTED : FXPQ_ERR_INVALID_ARG;
  if (strategy < FXPQ_ROUND_CONSERVATIVE || strategy > FXPQ_ROUND_AGGRESSIVE) return FXPQ_ERR_INVALID_ARG;
  if (psi_rule != FXPQ_PSI_PRINTED && psi_rule != FXPQ_PSI_MAX) return FXPQ_ERR_INVALID_ARG;
  if (fl_lo > fl_hi || fl_lo < -64 || fl_hi > 64) return FXPQ_ERR_INVALID_ARG;
  SrcDev s;
  fxpq_status st = to_dev(src, n, &s);
  if (st) return st;
  DeviceGuard g(h->device);
  Ctx c = ctx(h);
  const double* mm = src->d_minmax;
  if (!mm) {
    hipError_t e = launch_minmax(c, s, n, h->sc.minmax);
    if (e != hipSuccess) return FXPQ_ERR_HIP;
    mm = h->sc.minmax;
  }
  return hip_status(launch_preprocess(c, s, mm, wl, strategy, psi_rule, fl_lo, fl_hi, d_fmt_out));
}

fxpq_status fxpq_set_conv_tiling(fxpq_handle h, int32_t mode) {
  if (!h || mode < FXPQ_TILING_AUTO || mode > FXPQ_TILING_HALO) return FXPQ_ERR_INVALID_ARG;
  h->conv_tiling = mode;
  return FXPQ_OK;
}

fxpq_status fxpq_qlayer(fxpq_handle h, const fxpq_src* src, int64_t n, int32_t wl, int32_t sign,
                        int32_t fl_lo, int32_t fl_hi, fxpq_fmt* d_fmt_out, void* codes,
                        fxpq_dtype code_type, void* codes_alt) {
  if (!h || n < 1 || !d_fmt_out || !codes || !codes_alt) return FXPQ_ERR_INVALID_ARG;
  if (code_type != FXPQ_C8) return FXPQ_ERR_INVALID_ARG;
  if (wl < 1 || wl > 8) return FXPQ_ERR_INVALID_ARG;
  if (sign != 0 && sign != 1 && sign != FXPQ_SIGN_AUTO) return FXPQ_ERR_INVALID_ARG;
  if (fl_lo > fl_hi || fl_lo < -64 || fl_hi > 64) return FXPQ_ERR_INVALID_ARG;
  if (fl_hi - fl_lo + 1 > kMaxCand - 1) return FXPQ_ERR_INVALID_ARG;
  if (!aligned(codes, 16) || !aligned(codes_alt, 16)) return FXPQ_ERR_INVALID_ARG;
  SrcDev s;
  fxpq_status st = to_dev(src, n, &s);
  if (st) return st;
  if (n / ((int64_t)kThreads * kWinMaxPerThread) + 1 > kMaxFlsBlocks - 4096) return FXPQ_ERR_UNSUPPORTED;
  DeviceGuard g(h->device);
  Ctx c = ctx(h);
  const double* mm = src->d_minmax;
  if (!mm) {
    hipError_t e = launch_minmax(c, s, n, h->sc.minmax);
    if (e != hipSuccess) return FXPQ_ERR_HIP;
    mm = h->sc.minmax;
  }
  if (s.kind == FXPQ_SRC_INT && s.dtype == FXPQ_I64) {
    // 2-value packets: the search and the requantization run as two passes
    hipError_t e = launch_fl_search(c, s, n, wl, sign, fl_lo, fl_hi, mm, d_fmt_out, nullptr);
    if (e != hipSuccess) return hip_status(e);
    return hip_status(launch_requant(c, s, n, d_fmt_out, codes, code_type));
  }
  return hip_status(launch_qlayer(c, s, n, wl, sign, fl_lo, fl_hi, mm, d_fmt_out,
                                  static_cast<int8_t*>(codes), static_cast<int8_t*>(codes_alt)));
}

fxpq_status fxpq_qlayer_predicted(fxpq_handle h, const fxpq_src* src, int64_t n, int32_t wl,
                                  int32_t sign, int32_t fl_lo, int32_t fl_hi, fxpq_fmt* d_fmt_out,
                                  void* codes, fxpq_dtype code_type, double* d_minmax,
                                  uint32_t* d_miss) {
  if (!h || n < 1 || !d_fmt_out || !codes || !d_minmax || !d_miss) return FXPQ_ERR_INVALID_ARG;
  if (code_type != FXPQ_C8 || !aligned(codes, 16)) return FXPQ_ERR_INVALID_ARG;
  if (wl < 2 || wl > 8) return wl == 1 ? FXPQ_ERR_UNSUPPORTED : FXPQ_ERR_INVALID_ARG;
  if (sign != 0 && sign != 1 && sign != FXPQ_SIGN_AUTO) return FXPQ_ERR_INVALID_ARG;
  if (fl_lo > fl_hi || fl_lo < -64 || fl_hi > 64) return FXPQ_ERR_INVALID_ARG;
  if (fl_hi - fl_lo + 1 > kMaxCand - 1) return FXPQ_ERR_INVALID_ARG;
  SrcDev s;
  fxpq_status st = to_dev(src, n, &s);
  if (st) return st;
  if (s.kind == FXPQ_SRC_INT && s.dtype == FXPQ_I64) return FXPQ_ERR_UNSUPPORTED;
  if (n / ((int64_t)kThreads * kWinMaxPerThread) + 1 > kMaxFlsBlocks - 4096) return FXPQ_ERR_UNSUPPORTED;
  if (h->pred_defer && h->pred_n >= kMaxPredJobs) return FXPQ_ERR_UNSUPPORTED;
  DeviceGuard g(h->device);
  return hip_status(launch_qlayer_pred(ctx(h), s, n, wl, sign, fl_lo, fl_hi, d_fmt_out,
                                       static_cast<int8_t*>(codes), d_minmax, d_miss));
}

// acc_used: the call writes int32 accumulators to acc (else acc is ignored).
static fxpq_status conv_check(const fxpq_conv_desc* d, const void* x, fxpq_dtype x_type,
                              const int8_t* w, const int32_t* w_colsum, const fxpq_epilogue* ep,
                              const int32_t* acc, bool acc_used = true) {
  if (!d || !x || !w || (acc_used && !acc)) return FXPQ_ERR_INVALID_ARG;
  if (d->n < 1 || d->h < 1 || d->w < 1 || d->c < 1 || d->k < 1 || d->r < 1 || d->s < 1 ||
      d->stride < 1 || d->pad < 0)
    return FXPQ_ERR_INVALID_ARG;
  if (!is_code8(x_type)) return FXPQ_ERR_INVALID_ARG;
  if (x_type == FXPQ_C8 && (!ep || !ep->d_fmt_in)) return FXPQ_ERR_INVALID_ARG;
  if ((x_type == FXPQ_U8OFF || x_type == FXPQ_C8) && !w_colsum) return FXPQ_ERR_INVALID_ARG;
  if (ep && (ep->channels != d->k || !ep->d_fmt_in)) return FXPQ_ERR_INVALID_ARG;
  if (!(d->c % 16 == 0 || (d->c == 4 && d->r * d->s <= 128))) return FXPQ_ERR_UNSUPPORTED;
  int64_t ho = (d->h + 2 * (int64_t)d->pad - d->r) / d->stride + 1;
  int64_t wo = (d->w + 2 * (int64_t)d->pad - d->s) / d->stride + 1;
  if (ho < 1 || wo < 1) return FXPQ_ERR_INVALID_ARG;
  int64_t M = (int64_t)d->n * ho * wo;
  if (M >= INT32_MAX || (int64_t)d->n * d->h * d->w * d->c >= ((int64_t)1 << 40))
    return FXPQ_ERR_UNSUPPORTED;
  int64_t depth = (int64_t)d->r * d->s * d->c;
  if (depth * 128 * 256 >= ((int64_t)1 << 31)) return FXPQ_ERR_OVERFLOW;
  int64_t blocks = (d->k <= 64) ? ((M + 255) / 256) * ((d->k + 63) / 64)
                                : ((M + 127) / 128) * ((d->k + 127) / 128);
  if (blocks > kMaxConvBlocks) return FXPQ_ERR_UNSUPPORTED;
  if (!aligned(w, 16) || (acc_used && !aligned(acc, 4)) || !aligned(x, d->c == 4 ? 4 : 16))
    return FXPQ_ERR_INVALID_ARG;
  return FXPQ_OK;
}

static fxpq_status conv_common(fxpq_handle h, const fxpq_conv_desc* d, const void* x,
                               fxpq_dtype x_type, const int8_t* w, const int32_t* w_colsum,
                               const fxpq_epilogue* ep, int32_t* acc, double* d_minmax) {
  if (!h) return FXPQ_ERR_INVALID_ARG;
  fxpq_status st = conv_check(d, x, x_type, w, w_colsum, ep, acc);
  if (st) return st;
  SrcDev e;
  if (ep) epi_to_dev(ep, &e);
  DeviceGuard g(h->device);
  return hip_status(launch_conv(ctx(h), *d, x, x_type, w, w_colsum, ep ? &e : nullptr, acc,
                                ep ? d_minmax : nullptr));
}

fxpq_status fxpq_cblock(fxpq_handle h, const fxpq_conv_desc* d, const void* x, fxpq_dtype x_type,
                        const int8_t* w, const int32_t* w_colsum, const fxpq_epilogue* ep,
                        int32_t wl, int32_t sign, int32_t fl_lo, int32_t fl_hi,
                        fxpq_fmt* d_fmt_out, void* y, fxpq_dtype y_type, int32_t* acc,
                        double* d_minmax) {
  if (!h || !ep || !d_fmt_out || !y || !d_minmax) return FXPQ_ERR_INVALID_ARG;
  fxpq_status st = conv_check(d, x, x_type, w, w_colsum, ep, acc);
  if (st) return st;
  if (y_type != FXPQ_C8 && y_type != FXPQ_I8 && y_type != FXPQ_U8OFF) return FXPQ_ERR_INVALID_ARG;
  if (wl < 1 || wl > 32) return FXPQ_ERR_INVALID_ARG;
  if (wl == 1) return FXPQ_ERR_UNSUPPORTED;
  if (sign != 0 && sign != 1 && sign != FXPQ_SIGN_AUTO) return FXPQ_ERR_INVALID_ARG;
  if (fl_lo > fl_hi || fl_lo < -64 || fl_hi > 64) return FXPQ_ERR_INVALID_ARG;
  if (fl_hi - fl_lo + 1 > kMaxCand - 1) return FXPQ_ERR_INVALID_ARG;
  if (d->c % 16 != 0) return FXPQ_ERR_UNSUPPORTED;
  const int nb = conv_fused_blocks(*d, h->cus);
  if (nb < 1 || nb > kMaxFlsBlocks - 4096) return FXPQ_ERR_UNSUPPORTED;
  SrcDev e;
  epi_to_dev(ep, &e);
  e.kind = FXPQ_SRC_ACC;
  e.dtype = FXPQ_I32;
  e.x = acc;
  DeviceGuard g(h->device);
  return hip_status(launch_conv_fused(ctx(h), *d, x, x_type, w, w_colsum, e, wl, sign, fl_lo,
                                      fl_hi, d_fmt_out, static_cast<int8_t*>(y), y_type, d_minmax));
}

fxpq_status fxpq_cblock_predicted(fxpq_handle h, const fxpq_conv_desc* d, const void* x,
                                  fxpq_dtype x_type, const int8_t* w, const int32_t* w_colsum,
                                  const fxpq_epilogue* ep, int32_t wl, int32_t sign, int32_t fl_lo,
                                  int32_t fl_hi, fxpq_fmt* d_fmt_out, void* y, fxpq_dtype y_type,
                                  double* d_minmax, uint32_t* d_miss) {
  if (!h || !ep || !d_fmt_out || !y || !d_minmax || !d_miss) return FXPQ_ERR_INVALID_ARG;
  fxpq_status st = conv_check(d, x, x_type, w, w_colsum, ep, nullptr, false);
  if (st) return st;
  if (y_type != FXPQ_C8 || !aligned(y, 16)) return FXPQ_ERR_INVALID_ARG;
  if (wl < 2 || wl > 8) return wl == 1 ? FXPQ_ERR_UNSUPPORTED : FXPQ_ERR_INVALID_ARG;
  if (sign != 0 && sign != 1 && sign != FXPQ_SIGN_AUTO) return FXPQ_ERR_INVALID_ARG;
  if (fl_lo > fl_hi || fl_lo < -64 || fl_hi > 64) return FXPQ_ERR_INVALID_ARG;
  // channel multiples of 16, or the padded RGB layout (conv_check)
  if (d->k % 4 != 0) return FXPQ_ERR_UNSUPPORTED;
  const int nb = conv_fused_blocks(*d, h->cus, true);
  if (nb < 1 || nb > kMaxConvBlocks) return FXPQ_ERR_UNSUPPORTED;
  if (h->pred_defer && h->pred_n >= kMaxPredJobs) return FXPQ_ERR_UNSUPPORTED;
  SrcDev e;
  epi_to_dev(ep, &e);
  e.kind = FXPQ_SRC_ACC;
  e.dtype = FXPQ_I32;
  e.x = nullptr;
  DeviceGuard g(h->device);
  return hip_status(launch_conv_pred(ctx(h), *d, x, x_type, w, w_colsum, e, wl, sign, fl_lo, fl_hi,
                                     d_fmt_out, static_cast<int8_t*>(y), d_minmax, d_miss));
}

fxpq_status fxpq_predicted_defer(fxpq_handle h, int32_t on) {
  if (!h || (on != 0 && on != 1)) return FXPQ_ERR_INVALID_ARG;
  if (h->pred_n != 0) return FXPQ_ERR_INVALID_ARG;  // decisions pending: decide first
  h->pred_defer = on;
  return FXPQ_OK;
}

fxpq_status fxpq_predicted_decide(fxpq_handle h) {
  if (!h) return FXPQ_ERR_INVALID_ARG;
  const int n = h->pred_n;
  if (n == 0) return FXPQ_OK;
  h->pred_n = 0;
  DeviceGuard g(h->device);
  return hip_status(launch_pred_decide(ctx(h), h->sc.pred_jobs, n));
}

fxpq_status fxpq_qconv(fxpq_handle h, const fxpq_conv_desc* d, const void* x, fxpq_dtype x_type,
                       const int8_t* w, const int32_t* w_colsum, const fxpq_epilogue* ep,
                       int32_t* acc, double* d_minmax) {
  return conv_common(h, d, x, x_type, w, w_colsum, ep, acc, d_minmax);
}

}  // extern "C"

namespace {

// Plane counts and workspace layout of a wide C-Block.
struct WideLayout {
  int np_x = 0, np_w = 0;
  bool fused = false;  // one contraction (no per-pair int32 tensors)
  int64_t n_in = 0, wrow = 0, M = 0, mk = 0;
  int64_t xs = 0, ws = 0;                  // bytes per input / weight plane (256-aligned)
  int64_t off_w = 0, off_cs = 0, off_acc = 0, total = 0;
};

int64_t align256(int64_t b) { return (b + 255) / 256 * 256; }

// Balanced base-256 digits needed for the code range of (wl, sign).
int wide_weight_planes(int wl, int sign) {
  const int64_t qmin = sign ? -((int64_t)1 << (wl - 1)) : 0;
  const int64_t qmax = sign ? ((int64_t)1 << (wl - 1)) - 1 : ((int64_t)1 << wl) - 1;
  for (int n = 1; n <= 5; ++n) {
    const int64_t m = (((int64_t)1 << (8 * n)) - 1) / 255;  // 1 + 256 + ... + 256^(n-1)
    if (qmin >= -128 * m && qmax <= 127 * m) return n;
  }
  return 5;
}

// Bits bounding the exact contraction of a wide C-Block: each plane pair's
// int32 sum (< 2^31) times 256^(p+q), summed over the pairs.
int wide_sum_bits(int np_x, int np_w) {
  const int pairs = np_x * np_w;
  const int lg = pairs <= 1 ? 0 : 32 - __builtin_clz((unsigned)(pairs - 1));  // ceil(log2 pairs)
  return 31 + 8 * (np_x + np_w - 2) + lg;
}

bool wide_layout(const fxpq_conv_desc* d, int wl_x, int sign_x, int wl_w, int sign_w,
                 WideLayout* L) {
  if (!d || wl_x < 1 || wl_x > 32 || wl_w < 1 || wl_w > 32) return false;
  if ((sign_x != 0 && sign_x != 1) || (sign_w != 0 && sign_w != 1)) return false;
  if (d->n < 1 || d->h < 1 || d->w < 1 || d->c < 1 || d->k < 1 || d->r < 1 || d->s < 1 ||
      d->stride < 1 || d->pad < 0)
    return false;
  const int64_t ho = (d->h + 2 * (int64_t)d->pad - d->r) / d->stride + 1;
  const int64_t wo = (d->w + 2 * (int64_t)d->pad - d->s) / d->stride + 1;
  if (ho < 1 || wo < 1) return false;
  L->np_x = (wl_x + 7) / 8;
  L->np_w = wide_weight_planes(wl_w, sign_w);
  L->n_in = (int64_t)d->n * d->h * d->w * d->c;
  const int64_t depth = (int64_t)d->r * d->s * d->c;
  L->wrow = d->c == 4 ? (depth + 63) / 64 * 64 : depth;
  L->M = (int64_t)d->n * ho * wo;
  L->mk = L->M * d->k;
  L->xs = align256(L->n_in);
  L->ws = align256((int64_t)d->k * L->wrow);
  L->off_w = L->np_x * L->xs;
  L->off_cs = L->off_w + L->np_w * L->ws;
  L->off_acc = L->off_cs + align256((int64_t)L->np_w * d->k * 4);
  // the fused contraction sums up to min(np_x, np_w) plane pairs of one
  // shift in int32: |sum| <= pairs * padded depth * 2^14 < 2^31
  const int64_t kpad = (L->wrow + 63) / 64 * 64;
  const int gp = L->np_x < L->np_w ? L->np_x : L->np_w;
  L->fused = (int64_t)gp * kpad < ((int64_t)1 << 17);
  L->total = L->fused ? L->off_acc : L->off_acc + (int64_t)L->np_x * L->np_w * L->mk * 4;
  return true;
}

}  // namespace

extern "C" {

fxpq_status fxpq_qconv_wide_workspace(const fxpq_conv_desc* d, int32_t wl_x, int32_t sign_x,
                                      int32_t wl_w, int32_t sign_w, int64_t* bytes) {
  WideLayout L;
  if (!bytes || !wide_layout(d, wl_x, sign_x, wl_w, sign_w, &L)) return FXPQ_ERR_INVALID_ARG;
  *bytes = L.total;
  return FXPQ_OK;
}

fxpq_status fxpq_qconv_wide(fxpq_handle h, const fxpq_conv_desc* d, const int32_t* x,
                            int32_t wl_x, int32_t sign_x, const int32_t* w, int32_t wl_w,
                            int32_t sign_w, const fxpq_epilogue* ep, int64_t* v,
                            int32_t* d_scale, void* workspace, int64_t workspace_bytes) {
  WideLayout L;
  if (!h || !x || !w || !ep || !v || !d_scale || !workspace) return FXPQ_ERR_INVALID_ARG;
  if (!wide_layout(d, wl_x, sign_x, wl_w, sign_w, &L)) return FXPQ_ERR_INVALID_ARG;
  if (workspace_bytes < L.total || !aligned(workspace, 256) || !aligned(x, 4) ||
      !aligned(w, 4) || !aligned(v, 8) || !aligned(d_scale, 4))
    return FXPQ_ERR_INVALID_ARG;
  if (ep->channels != d->k || !ep->d_fmt_in) return FXPQ_ERR_INVALID_ARG;
  char* ws = static_cast<char*>(workspace);
  int8_t* px = reinterpret_cast<int8_t*>(ws);
  int8_t* pw = reinterpret_cast<int8_t*>(ws + L.off_w);
  int32_t* cs = reinterpret_cast<int32_t*>(ws + L.off_cs);
  int32_t* acc = reinterpret_cast<int32_t*>(ws + L.off_acc);
  // every plane contraction must be one fxpq_qconv accepts
  for (int p = 0; p < L.np_x; ++p) {
    const fxpq_dtype t = (p < L.np_x - 1 || !sign_x) ? FXPQ_U8OFF : FXPQ_I8;
    fxpq_status st = conv_check(d, px + p * L.xs, t, pw, cs, nullptr, acc);
    if (st) return st;
  }
  SrcDev e;
  epi_to_dev(ep, &e);
  DeviceGuard g(h->device);
  const Ctx c = ctx(h);
  hipError_t err = launch_wide_split_x(c, x, L.n_in, L.np_x, sign_x, L.xs, px);
  if (err == hipSuccess)
    err = launch_wide_split_w(c, w, (int64_t)d->k * L.wrow, L.np_w, sign_w, L.ws, pw);
  for (int q = 0; q < L.np_w && err == hipSuccess; ++q)
    err = launch_colsum(c, pw + q * L.ws, d->k, L.wrow, cs + (int64_t)q * d->k);
  if (L.fused && err == hipSuccess) {
    WideFusedArgs fa{};
    fa.px = px;
    fa.xs = L.xs;
    fa.pw = pw;
    fa.ws = L.ws;
    fa.cs = cs;
    fa.np_x = L.np_x;
    fa.np_w = L.np_w;
    fa.sign_x = sign_x;
    fa.N = d->n; fa.H = d->h; fa.W = d->w; fa.C = d->c; fa.K = d->k; fa.R = d->r; fa.S = d->s;
    fa.stride = d->stride; fa.pad = d->pad;
    fa.Ho = (d->h + 2 * d->pad - d->r) / d->stride + 1;
    fa.Wo = (d->w + 2 * d->pad - d->s) / d->stride + 1;
    fa.M = (int)L.M;
    fa.kdepth = d->r * d->s * d->c;
    fa.wrow = (int)L.wrow;
    fa.ep = e;
    fa.v = v;
    fa.d_scale = d_scale;
    fa.flags = h->sc.flags;
    return hip_status(launch_wide_fused(c, fa, wide_sum_bits(L.np_x, L.np_w) >= 62));
  }
  for (int p = 0; p < L.np_x && err == hipSuccess; ++p) {
    const int t = (p < L.np_x - 1 || !sign_x) ? FXPQ_U8OFF : FXPQ_I8;
    for (int q = 0; q < L.np_w && err == hipSuccess; ++q)
      err = launch_conv(c, *d, px + p * L.xs, t, pw + q * L.ws, cs + (int64_t)q * d->k, nullptr,
                        acc + (int64_t)(p * L.np_w + q) * L.mk, nullptr);
  }
  if (err == hipSuccess) err = launch_wide_combine(c, acc, L.mk, L.np_x, L.np_w, e, v, d_scale);
  return hip_status(err);
}

fxpq_status fxpq_acc_overflow(fxpq_handle h, const int32_t* acc, int64_t n, int32_t bits,
                              int64_t* d_count) {
  if (!h || !acc || !d_count || n < 0 || bits < 2 || bits > 32) return FXPQ_ERR_INVALID_ARG;
  if (!aligned(acc, 4) || !aligned(d_count, 8)) return FXPQ_ERR_INVALID_ARG;
  if (n == 0) return FXPQ_OK;
  DeviceGuard g(h->device);
  return hip_status(launch_acc_overflow(ctx(h), acc, n, bits, d_count));
}

fxpq_status fxpq_qgemm(fxpq_handle h, int64_t M, int64_t N, int64_t K, const void* A,
                       fxpq_dtype a_type, const int8_t* B, const int32_t* b_colsum,
                       const fxpq_epilogue* ep, int32_t* C, double* d_minmax) {
  if (M < 1 || N < 1 || K < 1 || M >= INT32_MAX || N >= INT32_MAX || K >= INT32_MAX)
    return FXPQ_ERR_INVALID_ARG;
  if (K % 16 != 0) return FXPQ_ERR_UNSUPPORTED;
  fxpq_conv_desc d{(int32_t)M, 1, 1, (int32_t)K, (int32_t)N, 1, 1, 1, 0};
  return conv_common(h, &d, A, a_type, B, b_colsum, ep, C, d_minmax);
}

fxpq_status fxpq_weight_colsum(fxpq_handle h, const int8_t* w, int64_t k, int64_t len,
                               int32_t* colsum) {
  if (!h || !w || !colsum || k < 1 || len < 1 || k >= INT32_MAX) return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(h->device);
  return hip_status(launch_colsum(ctx(h), w, k, len, colsum));
}

fxpq_status fxpq_maxpool(fxpq_handle h, const void* x, fxpq_dtype type, int32_t n, int32_t hgt,
                         int32_t wid, int32_t c, int32_t ksize, int32_t stride, int32_t pad,
                         void* y) {
  if (!h || !x || !y || !is_code8(type)) return FXPQ_ERR_INVALID_ARG;
  if (n < 1 || hgt < 1 || wid < 1 || c < 1 || ksize < 1 || stride < 1 || pad < 0 || pad >= ksize)
    return FXPQ_ERR_INVALID_ARG;
  if (c % 4 != 0 || !aligned(x, 4) || !aligned(y, 4)) return FXPQ_ERR_UNSUPPORTED;
  if ((hgt + 2 * pad - ksize) < 0 || (wid + 2 * pad - ksize) < 0) return FXPQ_ERR_INVALID_ARG;
  if (c % 16 == 0 && (!aligned(x, 16) || !aligned(y, 16))) return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(h->device);
  return hip_status(launch_maxpool(ctx(h), static_cast<const int8_t*>(x), n, hgt, wid, c, ksize,
                                   stride, pad, static_cast<int8_t*>(y)));
}

fxpq_status fxpq_avgpool_global(fxpq_handle h, const void* x, fxpq_dtype type,
                                const fxpq_fmt* d_fmt, int32_t n, int32_t hw, int32_t c,
                                int64_t recip, int64_t* y) {
  if (!h || !x || !y || !is_code8(type) || n < 1 || hw < 1 || c < 1) return FXPQ_ERR_INVALID_ARG;
  if (type == FXPQ_C8 && !d_fmt) return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(h->device);
  return hip_status(launch_avgpool(ctx(h), static_cast<const int8_t*>(x), type, d_fmt, n, hw, c,
                                   recip, y));
}

fxpq_status fxpq_layer_error(fxpq_handle h, const float* ref, const void* codes,
                             fxpq_dtype code_type, const fxpq_fmt* d_fmt, int64_t n,
                             double* d_out) {
  if (!h || !ref || !codes || !d_out || n < 1) return FXPQ_ERR_INVALID_ARG;
  if (code_type != FXPQ_F32 && (!is_code(code_type) || !d_fmt)) return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(h->device);
  return hip_status(launch_layer_error(ctx(h), ref, codes, code_type, d_fmt, n, d_out));
}

fxpq_status fxpq_dequantize(fxpq_handle h, const void* codes, fxpq_dtype code_type,
                            const fxpq_fmt* d_fmt, int64_t n, float* out) {
  if (!h || !codes || !d_fmt || !out || n < 0 || !is_code(code_type)) return FXPQ_ERR_INVALID_ARG;
  if (n == 0) return FXPQ_OK;
  DeviceGuard g(h->device);
  return hip_status(launch_dequant(ctx(h), codes, code_type, d_fmt, n, out));
}

fxpq_status fxpq_prediction_ties(fxpq_handle h, const void* scores, fxpq_dtype dtype, int32_t rows,
                                 int32_t cols, int64_t* d_out) {
  if (!h || !scores || !d_out || rows < 1 || cols < 1) return FXPQ_ERR_INVALID_ARG;
  if (dtype != FXPQ_F32 && dtype != FXPQ_I32) return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(h->device);
  return hip_status(launch_logit_ties(ctx(h), scores, dtype, rows, cols,
                                      reinterpret_cast<long long*>(d_out)));
}

fxpq_status fxpq_teacher_conv(fxpq_handle h, const fxpq_conv_desc* d, const float* x,
                              const float* w_rsck, float* y) {
  if (!h || !d || !x || !w_rsck || !y) return FXPQ_ERR_INVALID_ARG;
  if (d->n < 1 || d->h < 1 || d->w < 1 || d->c < 1 || d->k < 1 || d->r < 1 || d->s < 1 ||
      d->stride < 1 || d->pad < 0)
    return FXPQ_ERR_INVALID_ARG;
  if (d->h + 2 * d->pad < d->r || d->w + 2 * d->pad < d->s) return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(h->device);
  return hip_status(launch_teacher_conv(ctx(h), *d, x, w_rsck, y));
}

fxpq_status fxpq_teacher_affine(fxpq_handle h, const float* t, int64_t n, int32_t channels,
                                const float* a1, const float* a2, const float* bias,
                                int32_t relu, float* y) {
  if (!h || !t || !y || n < 0 || channels < 1 || n % channels != 0 || (a1 && !a2))
    return FXPQ_ERR_INVALID_ARG;
  if (n == 0) return FXPQ_OK;
  DeviceGuard g(h->device);
  return hip_status(launch_teacher_affine(ctx(h), t, n, channels, a1, a2, bias, relu ? 1 : 0, y));
}

fxpq_status fxpq_teacher_add(fxpq_handle h, const float* a, const float* b, int64_t n,
                             int32_t relu, float* y) {
  if (!h || !a || !b || !y || n < 0) return FXPQ_ERR_INVALID_ARG;
  if (n == 0) return FXPQ_OK;
  DeviceGuard g(h->device);
  return hip_status(launch_teacher_add(ctx(h), a, b, n, relu ? 1 : 0, y));
}

fxpq_status fxpq_teacher_maxpool(fxpq_handle h, const float* x, int32_t n, int32_t hgt,
                                 int32_t wid, int32_t c, int32_t ksize, int32_t stride,
                                 int32_t pad, float* y) {
  if (!h || !x || !y || n < 1 || hgt < 1 || wid < 1 || c < 1 || ksize < 1 || stride < 1 ||
      pad < 0 || pad >= ksize || hgt + 2 * pad < ksize || wid + 2 * pad < ksize)
    return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(h->device);
  return hip_status(launch_teacher_maxpool(ctx(h), x, n, hgt, wid, c, ksize, stride, pad, y));
}

fxpq_status fxpq_teacher_avgpool(fxpq_handle h, const float* x, int32_t n, int32_t hw, int32_t c,
                                 float* y) {
  if (!h || !x || !y || n < 1 || hw < 1 || c < 1) return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(h->device);
  return hip_status(launch_teacher_avgpool(ctx(h), x, n, hw, c, y));
}

fxpq_status fxpq_timer_start(fxpq_handle h, fxpq_timer_kind kind) {
  if (!h || kind < FXPQ_TIMER_OFF || kind > FXPQ_TIMER_CBLOCK_PRED) return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(h->device);
  Timer& t = h->timer;
  if (kind != FXPQ_TIMER_OFF && !t.ev) {
    t.ev = new (std::nothrow) hipEvent_t[2 * kTimerPairs];
    if (!t.ev) return FXPQ_ERR_ALLOC;
    for (int i = 0; i < 2 * kTimerPairs; ++i) {
      if (hipEventCreate(&t.ev[i]) != hipSuccess) {
        for (int j = 0; j < i; ++j) (void)hipEventDestroy(t.ev[j]);
        delete[] t.ev;
        t.ev = nullptr;
        return FXPQ_ERR_HIP;
      }
    }
    t.capacity = kTimerPairs;
  }
  if (hipStreamSynchronize(h->stream) != hipSuccess) return FXPQ_ERR_HIP;
  t.kind = kind;
  t.used = 0;
  t.work = 0.0;
  return FXPQ_OK;
}

fxpq_status fxpq_timer_read(fxpq_handle h, double* total_ms, int64_t* launches, double* work) {
  if (!h || !total_ms || !launches || !work) return FXPQ_ERR_INVALID_ARG;
  DeviceGuard g(h->device);
  if (hipStreamSynchronize(h->stream) != hipSuccess) return FXPQ_ERR_HIP;
  Timer& t = h->timer;
  double sum = 0.0;
  for (int i = 0; i < t.used; ++i) {
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, t.ev[2 * i], t.ev[2 * i + 1]) != hipSuccess) return FXPQ_ERR_HIP;
    sum += ms;
  }
  *total_ms = sum;
  *launches = t.used;
  *work = t.work;
  return FXPQ_OK;
}

fxpq_status fxpq_epilogue_scale(fxpq_handle h, const fxpq_epilogue* ep, int32_t* d_scale) {
  if (!h || !ep || !ep->d_fmt_in || !d_scale) return FXPQ_ERR_INVALID_ARG;
  SrcDev e;
  epi_to_dev(ep, &e);
  DeviceGuard g(h->device);
  return hip_status(launch_epi_scale(ctx(h), e, d_scale));
}

}  // extern "C"
