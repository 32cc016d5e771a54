/*
 * fxpq.h -- C ABI of libfxpq, the MI355X (gfx950) hot path of FxP-QNet's
 * post-training quantizer (Shawahna et al., "FxP-QNet: A Post-Training
 * Quantizer for the Design of Mixed Low-Precision DNNs with Dynamic Fixed-Point
 * Representation", IEEE Access 2022).
 *
 * The hot path is the calibration forward under dynamic fixed-point (DFX)
 * quantization: quantize a tensor (Eq. 10-12), search its fractional length
 * by the data-structure error (Eq. 14), run each integer C-Block (conv/FC +
 * bias + Scale + ReLU, Sec. "Integer-Only Inference") and requantize its
 * output in the FxP-QLayer (Sec. "FxP-QLayer").
 *
 * Conventions shared by every call:
 *  - A k-bit code X with fractional length fl stands for X * 2^-fl (Eq. 1).
 *    Signed codes lie in [-2^(k-1), 2^(k-1)-1], unsigned in [0, 2^k-1] (Eq. 12).
 *  - All tensor pointers are caller-owned DEVICE memory on the handle's device;
 *    the library never frees them.  Scalars that later kernels consume (chosen
 *    formats, value scales, min/max) also live in device memory, so a whole
 *    calibration forward runs without a host round trip.
 *  - Every call is asynchronous on the handle's stream.  Argument errors that
 *    the host can see are returned at once and nothing is launched.  Conditions
 *    only the device can see (non-finite input, a value outside the exact
 *    range) set sticky flags that fxpq_sync_status() returns.
 *  - A handle owns its scratch memory (allocated once in fxpq_create); calls do
 *    not allocate.  A handle is not thread-safe: use one per host thread.
 *  - Code dtype FXPQ_U8OFF stores an unsigned 8-bit code u as the signed byte
 *    u - 128 (bit pattern u ^ 0x80), so that it feeds the signed int8 matrix
 *    cores; every call that reads it adds the 128 back exactly.  FXPQ_C8 lets
 *    the device pick I8 or U8OFF from the sign of the format it was written
 *    with; a call reading FXPQ_C8 codes needs that format (device pointer).
 */
#ifndef FXPQ_H
#define FXPQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  FXPQ_OK = 0,
  FXPQ_ERR_INVALID_ARG = 1, /* null pointer, bad size, bad word length, ... */
  FXPQ_ERR_UNSUPPORTED = 2, /* a valid combination this build does not implement */
  FXPQ_ERR_NONFINITE = 3,   /* reported through fxpq_sync_status flags */
  FXPQ_ERR_OVERFLOW = 4,    /* int32 accumulator could overflow for this shape */
  FXPQ_ERR_HIP = 5,         /* a HIP runtime call failed */
  FXPQ_ERR_ALLOC = 6        /* fxpq_create could not allocate its scratch */
} fxpq_status;

typedef enum {
  FXPQ_I8 = 0,    /* signed 8-bit codes */
  FXPQ_U8OFF = 1, /* unsigned 8-bit codes stored as u - 128 */
  FXPQ_I16 = 2,
  FXPQ_I32 = 3,
  FXPQ_I64 = 4,
  FXPQ_F32 = 5,
  FXPQ_C8 = 6,    /* 8-bit code whose storage follows the device format: I8 when
                     the format is signed, U8OFF when it is unsigned */
  FXPQ_U32 = 7    /* unsigned codes of up to 32 bits stored as uint32 (the only
                     storage an unsigned 32-bit format's codes fit) */
} fxpq_dtype;

#define FXPQ_SIGN_AUTO (-1) /* Eq. 6: signed iff the smallest value is negative */

/* Sticky device flags returned by fxpq_sync_status. */
#define FXPQ_FLAG_NONFINITE 0x1u /* NaN or Inf in an fp32 input */
#define FXPQ_FLAG_RANGE 0x2u     /* a value left the exactly handled range (see fxpq_fl_search) */
#define FXPQ_FLAG_CODE 0x4u      /* a code did not fit the requested code dtype */

/*
 * A DFX format in device memory: word length k, fractional length fl, sign
 * strategy (0 unsigned, 1 signed).  status is 0 when the format is valid;
 * fxpq_fl_search writes a nonzero status when it could not choose one.
 */
typedef struct {
  int32_t wl;
  int32_t fl;
  int32_t sign;
  int32_t status;
} fxpq_fmt;

/*
 * Integer C-Block epilogue (Sec. "Integer-Only Inference", text under Fig.
 * "FxP-QNet hardware").  The accumulator of a conv/FC with input codes at
 * fractional length fl_in (read from d_fmt_in on the device) and weights at
 * fl_w has scale s = fl_in + fl_w.  The C-Block value is, per output channel c:
 *     v = acc                                   (scale s)
 *     v = v + bias[c]        if bias            both aligned to max(s, fl_bias)
 *     v = v * scale[c]       if scale           scale += fl_scale (BN->Scale, Eq. 4-5)
 *     v = v + shift[c]       if shift           both aligned to max(., fl_shift)
 *     v = max(v, 0)          if relu
 * Alignment is an exact left shift of the coarser operand, so v is the exact
 * value of the C-Block; only the following FxP-QLayer rounds.  bias, scale and
 * shift are per-channel integer codes (device, int32: word lengths up to 32) or NULL.  `channels` is
 * the number of output channels, the innermost dimension of the accumulators.
 */
typedef struct {
  int32_t channels;
  int32_t fl_w;
  const fxpq_fmt* d_fmt_in;
  const int32_t* bias;
  int32_t fl_bias;
  int32_t relu;
  const int32_t* scale;
  int32_t fl_scale;
  int32_t pad0;
  const int32_t* shift;
  int32_t fl_shift;
  int32_t pad1;
} fxpq_epilogue;

/*
 * The values an FxP-QLayer quantizes (Sec. "FxP-QLayer"), described without
 * materializing them:
 *   FXPQ_SRC_F32  x is float[n]; the values are x.
 *   FXPQ_SRC_INT  x is int32[n] (dtype FXPQ_I32) or int64[n] (FXPQ_I64); the
 *                 values are x * 2^-s with s read from d_scale (device int32).
 *   FXPQ_SRC_ACC  x is int32[n] conv/FC accumulators laid out [rows][channels];
 *                 the values are the C-Block epilogue `ep` applied to them.
 *   FXPQ_SRC_ADD  Eltwise C-Block: x and x2 are code tensors (dtype / dtype2 in
 *                 {FXPQ_I8, FXPQ_U8OFF}) in the formats d_fmt_a / d_fmt_b; the
 *                 values are a + b, aligned to the finer fractional length,
 *                 followed by ReLU when relu != 0.
 * d_minmax (nullable) is a device double[2] holding the exact min and max of
 * the values when the caller already has them (fxpq_qconv writes it); when
 * NULL the library computes it.
 */
typedef enum { FXPQ_SRC_F32 = 0, FXPQ_SRC_INT = 1, FXPQ_SRC_ACC = 2, FXPQ_SRC_ADD = 3 } fxpq_src_kind;

typedef struct {
  int32_t kind;
  int32_t dtype;
  const void* x;
  const void* x2;
  int32_t dtype2;
  int32_t relu;
  const int32_t* d_scale;
  const fxpq_fmt* d_fmt_a;
  const fxpq_fmt* d_fmt_b;
  const fxpq_epilogue* ep;
  const double* d_minmax;
} fxpq_src;

/* Convolution shape: input NHWC codes, weights KRSC int8 codes, output NHWK. */
typedef struct {
  int32_t n, h, w, c; /* input batch, height, width, channels */
  int32_t k, r, s;    /* output channels, kernel height, kernel width */
  int32_t stride, pad;
} fxpq_conv_desc;

typedef struct fxpq_handle_s* fxpq_handle;

/* ---- handle and status --------------------------------------------------- */

/* Creates a handle on HIP device `device` using the default stream. */
fxpq_status fxpq_create(fxpq_handle* h, int device);
fxpq_status fxpq_destroy(fxpq_handle h);
/* Sets the stream (a hipStream_t, NULL = default stream) for later calls. */
fxpq_status fxpq_set_stream(fxpq_handle h, void* hip_stream);
const char* fxpq_status_string(fxpq_status s);
/* Waits for the handle's stream, returns and clears the sticky FXPQ_FLAG_* bits. */
fxpq_status fxpq_sync_status(fxpq_handle h, uint32_t* flags);

/* ---- hot path -------------------------------------------------------------- */

/*
 * Quantize (Eq. 10-12): codes[i] = clip(rne(x[i] * 2^fl), Qmin, Qmax) with the
 * format read from d_fmt (device).  rne rounds half to even.  code_type is
 * FXPQ_I8, FXPQ_U8OFF (unsigned 8-bit formats only), FXPQ_I16, FXPQ_I32 or
 * FXPQ_U32 (unsigned formats only) and must hold the format's code range (a
 * range it cannot hold raises FXPQ_FLAG_CODE and the codes saturate to it).  n >= 0; n == 0 launches nothing.
 * Word lengths 1..32.  A signed 1-bit format follows Eq. 13 (code -1 for
 * x < 0, code 0 otherwise, decoded as +1) and is stored decoded: -1 or +1,
 * so that a C-Block consumes it as it is; the same holds for every call that
 * writes codes.  A NaN or Inf in x has no code: it raises the sticky
 * FXPQ_FLAG_NONFINITE (read by fxpq_sync_status) and its code is unspecified.
 */
fxpq_status fxpq_quantize(fxpq_handle h, const float* x, int64_t n, const fxpq_fmt* d_fmt,
                          void* codes, fxpq_dtype code_type);

/*
 * FxP-QLayer requantization (Sec. "FxP-QLayer"; Eq. 10-12 applied to the exact
 * C-Block values): codes[i] = clip(rne(v[i] * 2^fl), Qmin, Qmax) for the values
 * v described by src and the format in d_fmt.  Computed exactly: the result is
 * the same as quantizing the exact rational value.  code_type as above.
 */
fxpq_status fxpq_requant(fxpq_handle h, const fxpq_src* src, int64_t n, const fxpq_fmt* d_fmt,
                         void* codes, fxpq_dtype code_type);

/*
 * fxpq_requant of C-Block values (src of kind FXPQ_SRC_ACC, code_type
 * FXPQ_C8, FXPQ_I8 or FXPQ_U8OFF), plus the min and max of the residual sum
 * (Sec. "FxP-QLayer": eltwise ADD of two FxP-QLayer outputs, aligned to the
 * finer fractional length, optionally followed by ReLU) that will consume the
 * codes written here and the 8-bit codes b (type b_type, format d_fmt_b, n
 * values, device):
 *     s_i = relu?(codes_i * 2^-fl + b_i * 2^-fl_b).
 * d_add_minmax (device double[2]) receives min and max of s_i * 2^F, F =
 * max(fl, fl_b): the d_minmax an FXPQ_SRC_ADD source over (codes, b) takes,
 * so that its FL search needs no min / max pass of its own.  codes and b must
 * be 16-byte aligned.
 */
fxpq_status fxpq_requant_addmm(fxpq_handle h, const fxpq_src* src, int64_t n,
                               const fxpq_fmt* d_fmt, void* codes, fxpq_dtype code_type,
                               const void* b, fxpq_dtype b_type, const fxpq_fmt* d_fmt_b,
                               int32_t relu, double* d_add_minmax);

/*
 * Fractional-length search (Sec. "Quantization Parameters Optimization"): for
 * every fl in [fl_lo, fl_hi] the data-structure error of Eq. 14,
 *     L(fl) = sum_i (v_i - Q(v_i; wl, fl, S) * 2^-fl)^2,
 * and the fl with the smallest error; equal errors go to the LARGER fl.  The
 * comparison is exact.  sign is 0, 1 or FXPQ_SIGN_AUTO (Eq. 6).  The chosen
 * format {wl, fl, sign, 0} is written to d_fmt_out (device).  When d_sse is not
 * NULL it receives fl_hi - fl_lo + 1 errors (device doubles; fp64 sums whose
 * relative error is far below 1e-9); otherwise candidates that provably cannot
 * win are skipped.  Requirements: 1 <= wl <= 32, -64 <= fl_lo <= fl_hi <= 64,
 * n >= 1.  Exact range: |v| * 2^(fl_hi+24) < 2^52 for fp32 values and
 * |v * 2^s| < 2^52 for integer values when wl <= 16; |v * 2^max(s, fl_hi)| <
 * 2^62 when wl > 16.  Outside it FXPQ_FLAG_RANGE is raised and d_fmt_out gets a
 * nonzero status.  Word length 1 with a signed format evaluates every
 * candidate with the Eq. 13 values (+-2^-fl) exactly; fp32 values below
 * 2^-(fl_hi+24) in magnitude enter its errors truncated to that unit.
 */
fxpq_status fxpq_fl_search(fxpq_handle h, const fxpq_src* src, int64_t n, int32_t wl, int32_t sign,
                           int32_t fl_lo, int32_t fl_hi, fxpq_fmt* d_fmt_out, double* d_sse);

/*
 * For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the search
 * of fxpq_fl_search without a handle, with the same arguments, requirements
 * and results (d_fmt_out, and d_sse when not NULL).  It runs on hip_stream
 * (NULL: the default stream) of the calling thread's current device and
 * allocates nothing: its scratch is a fixed array of
 * FXPQ_STATIC_SCRATCH_BYTES in the library's device memory, one copy per
 * device (devices 0..63), held until the process ends.  The first call on a
 * device looks up that copy's address (hipGetSymbolAddress).  Every call
 * clears the parts of the array a search needs at zero with a small kernel
 * (no memset); calls that overlap on one device race on the array and must
 * be serialized (e.g. one stream).  There are no sticky flags to read:
 * non-finite or out-of-range data give d_fmt_out a nonzero status.  Returns
 * FXPQ_ERR_UNSUPPORTED when the tensor needs more min / max partials than the
 * array holds (n * sizeof(value) beyond what 16384 blocks stream; never for
 * resident-capped grids on one MI355X), or more than 2^16 - 4096 window
 * blocks (the limit of fxpq_fl_search).
 */
#define FXPQ_STATIC_SCRATCH_BYTES 1271808
fxpq_status fxpq_fl_search_static(const fxpq_src* src, int64_t n, int32_t wl, int32_t sign,
                                  int32_t fl_lo, int32_t fl_hi, fxpq_fmt* d_fmt_out,
                                  double* d_sse, void* hip_stream);

/*
 * FxP-QLayer in one call (Sec. "FxP-QLayer" with the search of Sec.
 * "Quantization Parameters Optimization"): the chosen format in d_fmt_out
 * and the codes are bit for bit those of
 *     fxpq_fl_search(h, src, n, wl, sign, fl_lo, fl_hi, d_fmt_out, NULL);
 *     fxpq_requant(h, src, n, d_fmt_out, codes, FXPQ_C8);
 * but the search's read of the values also writes the codes of its two
 * likeliest formats (fl = beta_nosat, the largest fl at which no value
 * saturates, and beta_nosat + 1): one set to `codes`, the other to
 * `codes_alt`, so the values are normally read once.  Afterwards nothing more
 * runs when the chosen format's codes are in `codes`, a copy of n bytes when
 * they are in `codes_alt`, and a requantization pass otherwise.  The format
 * d_fmt_out holds on entry (e.g. this layer's format from the previous
 * batch) picks which candidate goes to `codes`; when it is one of the two
 * candidates (same wl and sign, status 0) the other candidate's codes are not
 * written, and should it win, the requantization pass produces them.  Any
 * content of d_fmt_out on entry is valid.
 * codes_alt: device, n bytes, caller-owned scratch, contents unspecified
 * afterwards.  Requirements: code_type FXPQ_C8, 1 <= wl <= 8, codes and
 * codes_alt 16-byte aligned, the rest as fxpq_fl_search.  Sources with 8-byte
 * values (FXPQ_SRC_INT over int64) run the two calls above.
 */
fxpq_status fxpq_qlayer(fxpq_handle h, const fxpq_src* src, int64_t n, int32_t wl, int32_t sign,
                        int32_t fl_lo, int32_t fl_hi, fxpq_fmt* d_fmt_out, void* codes,
                        fxpq_dtype code_type, void* codes_alt);

/*
 * Predicted FxP-QLayer (Sec. "FxP-QLayer"; Eq. 10-14) for a layer evaluated
 * again on data like its previous call's: ONE read of the values evaluates
 * the FL search's window for the min / max held in d_minmax on entry (the
 * previous call's values), writes the codes of the window candidate that the
 * format in d_fmt_out on entry picks (as fxpq_cblock_predicted), and reduces
 * this call's min / max (no separate min / max pass, no alternate buffer).
 * A one-block decision then checks the prediction: when this call's min /
 * max give the same window and the window decides, exactly, on the written
 * candidate, d_fmt_out and codes hold what fxpq_qlayer writes (bit for bit);
 * otherwise *d_miss is set to 1 or 2 (as fxpq_cblock_predicted) and both
 * are unspecified (the caller runs fxpq_qlayer, and every layer fed by it,
 * again).  d_minmax always ends with
 * this call's min / max (NaN in it predicts nothing).  src->d_minmax is not
 * used.  Sources: fp32, int32 values, C-Block values (FXPQ_SRC_ACC) and
 * eltwise sums; 2 <= wl <= 8; code_type FXPQ_C8; codes 16-byte aligned.
 */
fxpq_status fxpq_qlayer_predicted(fxpq_handle h, const fxpq_src* src, int64_t n, int32_t wl,
                                  int32_t sign, int32_t fl_lo, int32_t fl_hi, fxpq_fmt* d_fmt_out,
                                  void* codes, fxpq_dtype code_type, double* d_minmax,
                                  uint32_t* d_miss);

/*
 * Preprocessor initial format (Sec. "Initial Design Generation", Eq. 6-9):
 *   S = 1 when the smallest value is negative (Eq. 6);
 *   psi = X_max / (2^k - 1) for S = 0, and for S = 1
 *   psi = min(X_min / -2^(k-1), X_max / (2^(k-1) - 1)) (Eq. 7 as printed,
 *   FXPQ_PSI_PRINTED) or the max of the two (FXPQ_PSI_MAX);
 *   fl = floor, nearest or ceil of -log2(psi) (Eq. 8-9) for the conservative,
 *   neutral or aggressive strategy, clamped to [fl_lo, fl_hi].
 * The integer length is wl - fl.  Decided exactly from the exact min / max of
 * the values described by src (src->d_minmax when given, else a min / max
 * pass).  Readings: all-zero data takes fl_hi; signed data without a positive
 * value takes the negative side alone.  d_fmt_out (device) receives
 * {wl, fl, S, 0}; non-finite data gives status 1 and FXPQ_FLAG_RANGE.
 * Requirements: 2 <= wl <= 32 (Eq. 7 has no scale for 1 bit), -64 <= fl_lo <=
 * fl_hi <= 64, n >= 1.
 */
typedef enum { FXPQ_ROUND_CONSERVATIVE = 0, FXPQ_ROUND_NEUTRAL = 1, FXPQ_ROUND_AGGRESSIVE = 2 } fxpq_round_strategy;
typedef enum { FXPQ_PSI_PRINTED = 0, FXPQ_PSI_MAX = 1 } fxpq_psi_rule;
fxpq_status fxpq_preprocess(fxpq_handle h, const fxpq_src* src, int64_t n, int32_t wl,
                            int32_t strategy, int32_t psi_rule, int32_t fl_lo, int32_t fl_hi,
                            fxpq_fmt* d_fmt_out);

/*
 * Quantized convolution (C-Block contraction, Sec. "Integer-Only Inference"):
 * acc[n][oh][ow][k] = sum_{r,s,c} x[n][oh*stride-pad+r][ow*stride-pad+s][c] * w[k][r][s][c]
 * with zero padding (value 0 in either code dtype), int32 accumulation on the
 * int8 matrix cores.  x_type is FXPQ_I8 or FXPQ_U8OFF.  Layout requirements:
 * c % 16 == 0, or c == 4 (first layer, padded RGB).  For FXPQ_U8OFF inputs
 * w_colsum (device int32[k], sum of each filter's codes) must be given.  When
 * ep and d_minmax are both non-NULL the exact min and max of the epilogue
 * values are written to d_minmax (device double[2]) for the FxP-QLayer that
 * follows.  Returns FXPQ_ERR_OVERFLOW when r*s*c*128*256 >= 2^31.
 */
fxpq_status fxpq_qconv(fxpq_handle h, const fxpq_conv_desc* d, const void* x, fxpq_dtype x_type,
                       const int8_t* w, const int32_t* w_colsum, const fxpq_epilogue* ep,
                       int32_t* acc, double* d_minmax);

/*
 * Quantized FC layer: C[m][n] = sum_k A[m][k] * B[n][k], int32 accumulation;
 * same contract as fxpq_qconv with a 1x1 kernel (K % 16 == 0).
 */
fxpq_status fxpq_qgemm(fxpq_handle h, int64_t M, int64_t N, int64_t K, const void* A,
                       fxpq_dtype a_type, const int8_t* B, const int32_t* b_colsum,
                       const fxpq_epilogue* ep, int32_t* C, double* d_minmax);

/*
 * C-Block followed by its FxP-QLayer in one call (Sec. "Integer-Only
 * Inference" and "FxP-QLayer"), for shallow contractions with wide outputs.
 * Results are bit for bit those of
 *     fxpq_qconv(h, d, x, x_type, w, w_colsum, ep, acc, d_minmax);
 *     fxpq_fl_search(h, &src, M * d->k, wl, sign, fl_lo, fl_hi, d_fmt_out, NULL);
 *     fxpq_requant(h, &src, M * d->k, d_fmt_out, y, y_type);
 * with src the FXPQ_SRC_ACC source over acc with epilogue ep (M = n * Ho *
 * Wo), but the int32 accumulators are recomputed by three passes of the
 * contraction (min / max, window sums of the search, codes) instead of being
 * stored and read back.  acc (device int32[M * k], caller-owned) is written
 * only when the search needs its exact general pass; its contents are
 * unspecified afterwards.  d_minmax (device double[2]) receives the min and max
 * of the C-Block values.  y (device, M x k codes, NHWC) has y_type FXPQ_C8,
 * FXPQ_I8 or FXPQ_U8OFF.  Requirements: those of fxpq_qconv, ep != NULL,
 * c % 16 == 0, 2 <= wl <= 32, fl range as fxpq_fl_search, and at most 61440
 * output tiles (of 128 x 128, or 256 x 64 when k <= 64); FXPQ_ERR_UNSUPPORTED
 * otherwise.  Errors of the search are reported as by fxpq_fl_search.
 */
fxpq_status fxpq_cblock(fxpq_handle h, const fxpq_conv_desc* d, const void* x, fxpq_dtype x_type,
                        const int8_t* w, const int32_t* w_colsum, const fxpq_epilogue* ep,
                        int32_t wl, int32_t sign, int32_t fl_lo, int32_t fl_hi,
                        fxpq_fmt* d_fmt_out, void* y, fxpq_dtype y_type, int32_t* acc,
                        double* d_minmax);

/*
 * Predicted C-Block (Sec. "FxP-QLayer"; Eq. 10-14): the C-Block of
 * fxpq_cblock and its FxP-QLayer in ONE contraction, without int32
 * accumulators, for a layer evaluated again on data like its previous call's
 * (the calibration loop re-runs the network on the same batch).  The
 * epilogue evaluates the FL search's window (the two candidates from
 * beta_nosat up, Eq. 14 sums and the clipping bound) for the min / max held
 * in d_minmax on entry, i.e. the previous call's C-Block values, and writes
 * the 8-bit codes of the window candidate that the format held in d_fmt_out
 * on entry picks (the previous call's choice: the second candidate when its
 * fl is that one, else the first).  A one-block decision then reduces this
 * call's exact min / max and checks the prediction: when those give the same
 * window (same beta_nosat, sign and variant) and the window decides, exactly,
 * on the candidate whose codes were written, d_fmt_out and y hold what
 * fxpq_qconv + fxpq_qlayer would write (bit for bit) and *d_miss is left
 * unchanged; otherwise *d_miss is set to 1 (2 when the prediction was right
 * but the window alone cannot decide, so that the same data miss again) and
 * d_fmt_out / y are unspecified: the caller runs the layer again with
 * fxpq_qconv + fxpq_qlayer (and every layer fed by it).  In both cases d_minmax ends with this call's min / max,
 * the next call's prediction; NaN in d_minmax predicts nothing (a miss).
 * d_minmax: device double[2], caller-owned, in units of 2^-s of the C-Block
 * value (as fxpq_qconv writes it); d_miss: device uint32, caller-owned.
 * Requirements: as fxpq_qconv (C % 16 == 0, or the padded RGB layout C == 4),
 * K % 4 == 0, 2 <= wl <= 8, y_type FXPQ_C8, y 16-byte aligned.
 */
fxpq_status fxpq_cblock_predicted(fxpq_handle h, const fxpq_conv_desc* d, const void* x,
                                  fxpq_dtype x_type, const int8_t* w, const int32_t* w_colsum,
                                  const fxpq_epilogue* ep, int32_t wl, int32_t sign, int32_t fl_lo,
                                  int32_t fl_hi, fxpq_fmt* d_fmt_out, void* y, fxpq_dtype y_type,
                                  double* d_minmax, uint32_t* d_miss);

/*
 * Deferred decisions of the predicted calls (fxpq_cblock_predicted,
 * fxpq_qlayer_predicted; the same decisions of Eq. 14's FL search, taken
 * later).  With on = 1 a predicted call launches only its pass: the pass
 * records what its decision needs (in the handle) and its window sums go to
 * the call's own slot set; fxpq_predicted_decide then decides every call
 * recorded since the last decide in ONE launch, in call order.  Because the
 * calls after a predicted call already consumed its codes with the format
 * held in d_fmt_out on entry (the prediction), a deferred decision is a hit
 * only when the searched format is that one (and the window conditions of
 * fxpq_cblock_predicted hold); otherwise *d_miss is set as there and the
 * caller reruns with the standard calls from the first call that missed.
 * d_minmax gets each call's min / max at the decision.  Up to 256 calls may
 * be pending (more: FXPQ_ERR_UNSUPPORTED from the predicted call).  The
 * mode can change only with no decision pending (else FXPQ_ERR_INVALID_ARG).
 * fxpq_predicted_decide with none pending does nothing.  The caller must
 * keep every buffer a pending call names alive until its decision ran.
 */
fxpq_status fxpq_predicted_defer(fxpq_handle h, int32_t on);
fxpq_status fxpq_predicted_decide(fxpq_handle h);

/*
 * C-Block contraction over codes of up to 32 bits (Sec. "Integer-Only
 * Inference"; the first and last layers start at 32-bit activations and
 * weights, Sec. "Initial Design Generation"), followed by its epilogue:
 *     v[m][k] = epilogue(sum_{r,s,c} x[..][c] * w[k][r][s][c])     (exact)
 * with the shapes, zero padding and layout of fxpq_qconv (NHWC input, KRSC
 * weights; c % 16 == 0, or c == 4 with each weight row padded with zeros to
 * a multiple of 64; an FC layer is the 1x1 convolution of a 1x1 image).
 * x (device int32[n*h*w*c]) holds codes of the format (wl_x, sign_x),
 * w (device int32[k * row]) codes of (wl_w, sign_w): int32 codes for signed
 * formats, uint32 codes (FXPQ_U32 storage) for unsigned ones; a signed 1-bit
 * format holds its decoded codes (-1 / +1).  ep (required) is the epilogue, with
 * ep->d_fmt_in the input's format on the device (its fl sets the scale).
 * The result v (device int64[M * k], M = n * Ho * Wo, channels innermost) is
 * the exact C-Block value times 2^s, s written to d_scale (device int32):
 * FXPQ_SRC_INT with dtype FXPQ_I64 and this d_scale describes the values
 * for fxpq_fl_search / fxpq_requant / fxpq_qlayer.
 * Computed on the int8 matrix cores: x splits into ceil(wl_x / 8) base-256
 * planes (unsigned low bytes, the top byte signed for signed formats), w into
 * balanced base-256 digits in [-128, 127] (up to 5 for 32-bit weights); one
 * contraction walks the plane pairs by shift 256^(p+q), sums each shift's
 * pairs in int32 and folds them exactly into a 128-bit (or, when provably
 * enough, 64-bit) accumulator per value, then applies the epilogue.  When
 * min(planes of x, digits of w) * (r * s * c rounded up to 64) reaches 2^17
 * the int32 group sums could overflow: one int8 contraction per plane pair
 * into an int32 tensor and an exact combination pass instead.
 * workspace (device, 256-byte aligned, caller-owned) must hold at least the
 * bytes fxpq_qconv_wide_workspace reports for the same arguments; its
 * contents are unspecified afterwards.  Codes outside their format's range
 * raise FXPQ_FLAG_CODE; values of magnitude 2^62 or more raise
 * FXPQ_FLAG_RANGE and are written as 0.  Requirements: 1 <= wl <= 32, and
 * every plane contraction within the limits of fxpq_qconv (else its error).
 */
fxpq_status fxpq_qconv_wide_workspace(const fxpq_conv_desc* d, int32_t wl_x, int32_t sign_x,
                                      int32_t wl_w, int32_t sign_w, int64_t* bytes);
fxpq_status fxpq_qconv_wide(fxpq_handle h, const fxpq_conv_desc* d, const int32_t* x,
                            int32_t wl_x, int32_t sign_x, const int32_t* w, int32_t wl_w,
                            int32_t sign_w, const fxpq_epilogue* ep, int64_t* v,
                            int32_t* d_scale, void* workspace, int64_t workspace_bytes);

/*
 * Accumulator overflow accounting (Sec. "Integer-Only Inference": the MAC
 * results of the layers between the first and the last are kept in 16 bits).
 * Adds to *d_count (device int64, caller-initialized) the number of int32
 * accumulators acc[0..n) (device) outside the two's-complement range of
 * `bits` bits, [-2^(bits-1), 2^(bits-1) - 1]: the outputs a MAC of that
 * width cannot hold (with wrap-around arithmetic, partial sums may leave the
 * range harmlessly as long as the result is inside).  2 <= bits <= 32.
 */
fxpq_status fxpq_acc_overflow(fxpq_handle h, const int32_t* acc, int64_t n, int32_t bits,
                              int64_t* d_count);

/*
 * Tile family of fxpq_qconv (results are the same integers either way):
 * FXPQ_TILING_AUTO (default) and FXPQ_TILING_GEMM use implicit-GEMM tiles;
 * FXPQ_TILING_HALO uses halo tiles where the shape allows them (3x3 filters,
 * stride 1 or 2, c % 64 == 0, k % 256 == 0, r*s*c >= 1024, an input patch of
 * at most 512 pixels per tile): whole output-image rows per tile, the input
 * patch loaded into LDS once per channel chunk for all nine taps.
 */
typedef enum { FXPQ_TILING_AUTO = 0, FXPQ_TILING_GEMM = 1, FXPQ_TILING_HALO = 2 } fxpq_conv_tiling;
fxpq_status fxpq_set_conv_tiling(fxpq_handle h, int32_t mode);

/* Sum of each filter's codes: colsum[k] = sum_j w[k][j] for w[k][len] (device). */
fxpq_status fxpq_weight_colsum(fxpq_handle h, const int8_t* w, int64_t k, int64_t len,
                               int32_t* colsum);

/* MAX-POOL on NHWC codes (no FxP-QLayer needed, Sec. "FxP-QLayer"); taps
 * outside the input are skipped. */
fxpq_status fxpq_maxpool(fxpq_handle h, const void* x, fxpq_dtype type, int32_t n, int32_t hgt,
                         int32_t wid, int32_t c, int32_t ksize, int32_t stride, int32_t pad,
                         void* y);

/* Global AVG-POOL on NHWC codes x[n][hw][c]: y[n][c] = recip * sum_hw code
 * (exact, int64), the reciprocal of the window being quantized like a
 * parameter (Sec. "FxP-QLayer").  The value scale of y is the input fl plus the
 * reciprocal's fl.  d_fmt (device) is the codes' format, needed for FXPQ_C8. */
fxpq_status fxpq_avgpool_global(fxpq_handle h, const void* x, fxpq_dtype type,
                                const fxpq_fmt* d_fmt, int32_t n, int32_t hw, int32_t c,
                                int64_t recip, int64_t* y);

/*
 * Layer error (Eq. 14 against a full-precision reference, with the statistics
 * of Eq. 16 and Eq. 18): d_out[0] = sum_i (ref_i - code_i * 2^-fl)^2,
 * d_out[1] = min(ref), d_out[2] = max(ref), d_out[3] = population standard
 * deviation of ref.  fp64 accumulation.  d_out is a device double[4].
 * code_type FXPQ_F32 compares two fp32 tensors (codes holds fp32 values,
 * d_fmt unused and may be NULL).
 */
fxpq_status fxpq_layer_error(fxpq_handle h, const float* ref, const void* codes,
                             fxpq_dtype code_type, const fxpq_fmt* d_fmt, int64_t n,
                             double* d_out);

/*
 * Dequantization (Eq. 1): out[i] = code_i * 2^-fl (codes stored as u - 128
 * restored), exact in fp32 for codes below 2^24 in magnitude.  code_type any
 * code dtype; d_fmt (device) the codes' format; out device float[n].
 */
fxpq_status fxpq_dequantize(fxpq_handle h, const void* codes, fxpq_dtype code_type,
                            const fxpq_fmt* d_fmt, int64_t n, float* out);

/*
 * Prediction ties of a classifier (Sec. "Quantization Parameters
 * Optimization", Eq. 19-20): for each of `rows` rows of `cols` scores
 * (FXPQ_F32 or FXPQ_I32, row-major, device), c = the number of classes
 * sharing the highest score (exact comparison).  d_out (device int64[2]):
 * d_out[0] = rows with c > 1 (UnClass = d_out[0] / rows), d_out[1] = sum of
 * c - 1 (MisPred = d_out[1] / (rows * cols)).
 */
fxpq_status fxpq_prediction_ties(fxpq_handle h, const void* scores, fxpq_dtype dtype, int32_t rows,
                                 int32_t cols, int64_t* d_out);

/* Sets d_scale[0] = fl_in + fl_w + ... as the C-Block output scale of `ep`
 * (device int32), for consumers that need it as a plain FXPQ_SRC_INT scale. */
fxpq_status fxpq_epilogue_scale(fxpq_handle h, const fxpq_epilogue* ep, int32_t* d_scale);

/* ---- FP32 teacher ---------------------------------------------------------
 * The full-precision network whose activations are the reference of the
 * layer error in the per-layer sensitivity sweep (Sec. "Data-Structures
 * Sensitivity to Quantization"; the full-precision model as teacher, Sec.
 * "Quantization Parameters Optimization").  Reference data, not the DFX hot
 * path.  The arithmetic is fixed so that every implementation gets the same
 * bits: a conv / FC output is the fp64 sum of the fp32 x fp32 products (exact
 * in fp64) in the order r, s, c with padded taps skipped, rounded once to
 * fp32; the BN-as-Scale affine is one fp32 fma; a bias one fp32 add; ReLU maps
 * every value <= 0 to +0.  All tensors are device fp32, activations NHWC.
 */

/* y[n][oh][ow][k] from x (NHWC) and w_rsck ([r][s][c][k]). */
fxpq_status fxpq_teacher_conv(fxpq_handle h, const fxpq_conv_desc* d, const float* x,
                              const float* w_rsck, float* y);
/* Per channel c = i % channels: y = relu?(fmaf(t, a1[c], a2[c])) when a1 is
 * given, else relu?(t + bias[c]) when bias is given, else relu?(t).  In place
 * allowed.  n % channels == 0. */
fxpq_status fxpq_teacher_affine(fxpq_handle h, const float* t, int64_t n, int32_t channels,
                                const float* a1, const float* a2, const float* bias,
                                int32_t relu, float* y);
/* y = relu?(a + b), one fp32 add (residual connection). */
fxpq_status fxpq_teacher_add(fxpq_handle h, const float* a, const float* b, int64_t n,
                             int32_t relu, float* y);
/* NHWC max-pool; out-of-range taps are skipped. */
fxpq_status fxpq_teacher_maxpool(fxpq_handle h, const float* x, int32_t n, int32_t hgt,
                                 int32_t wid, int32_t c, int32_t ksize, int32_t stride,
                                 int32_t pad, float* y);
/* Global average of x[n][hw][c]: y[n][c] = (float)(fp64 sum in pixel order / hw). */
fxpq_status fxpq_teacher_avgpool(fxpq_handle h, const float* x, int32_t n, int32_t hw, int32_t c,
                                 float* y);

/* ---- measurement --------------------------------------------------------- */

/* Kernels the handle can time with HIP events on its stream. */
typedef enum {
  FXPQ_TIMER_OFF = 0,
  FXPQ_TIMER_FLS_WINDOW = 1, /* the one-read window pass of fxpq_fl_search */
  FXPQ_TIMER_QCONV = 2,      /* the contraction kernel of fxpq_qconv / fxpq_qgemm */
  FXPQ_TIMER_REQUANT = 3,    /* the kernel of fxpq_requant / fxpq_quantize */
  FXPQ_TIMER_CBLOCK_PASS = 4, /* each contraction pass of fxpq_cblock */
  FXPQ_TIMER_CBLOCK_PRED = 5  /* the contraction of fxpq_cblock_predicted */
} fxpq_timer_kind;

/*
 * Starts timing every launch of one kernel: the handle brackets each launch
 * with a pair of pre-created HIP events on its stream (at most 16384 launches
 * per session; later launches run untimed).  Resets earlier totals.
 * FXPQ_TIMER_OFF stops timing.
 */
fxpq_status fxpq_timer_start(fxpq_handle h, fxpq_timer_kind kind);

/*
 * Waits for the stream and returns, over the launches timed since
 * fxpq_timer_start: the summed kernel time in ms, the number of launches, and
 * the summed algorithmic work (HBM bytes the kernel must move: 4 B per int32
 * value read, 2 B per eltwise element, 8 B per int64 value, 4 + 1 B per
 * quantized fp32 value; or int8 operations 2*M*N*K for the contraction, per
 * pass for fxpq_cblock, per call for fxpq_cblock_predicted).
 */
fxpq_status fxpq_timer_read(fxpq_handle h, double* total_ms, int64_t* launches, double* work);

#ifdef __cplusplus
}
#endif
#endif /* FXPQ_H */
