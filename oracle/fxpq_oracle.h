/*
 * fxpq_oracle.h -- the CPU oracle of the DFX calibration hot path.
 *
 * TEST INFRASTRUCTURE ONLY.  This header and fxpq_oracle.c are a plain, slow,
 * exact CPU implementation of what the FxP-QNet quantizer computes (Shawahna
 * et al., "FxP-QNet", IEEE Access 2022).  Only the tests, the smoke check and
 * the CPU-baseline leg of the benchmark may load it.  It shares no code, header
 * or table with the GPU library.
 *
 * Number format (Sec. "Dynamic Fixed-Point Representation", Eq. 1): a k-bit
 * integer code X with fractional length fl (beta) stands for X * 2^-fl.
 * Code range (Eq. 12): Qmin = -S * 2^(k-S), Qmax = 2^(k-S) - 1.
 * Quantizer (Eq. 10, 11): X = clip(rne(x * 2^fl), Qmin, Qmax), rne = round
 * half to even.  k = 1 with S = 1 is the binary quantizer of Eq. 13.
 * Data-structure error (Eq. 14): L = sum_i (x_i - X_i * 2^-fl)^2.
 *
 * Every result here is exact: quantization is done on dyadic rationals
 * (m * 2^e with integer m), errors are exact integers scaled by a power of
 * two, and sums of squares go into a wide fixed-point (Kulisch) accumulator,
 * so the outcome does not depend on summation order or thread count.
 *
 * Status codes: 0 ok, 1 invalid argument, 2 a value is outside the range in
 * which the exact arithmetic below is implemented (|error| * 2^scale >= 2^62).
 */
#ifndef FXPQ_ORACLE_H
#define FXPQ_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define ORC_OK 0
#define ORC_EINVAL 1
#define ORC_ERANGE 2
#define ORC_SIGN_AUTO (-1)

/* Eq. 12. */
int orc_qrange(int k, int sign, int64_t* qmin, int64_t* qmax);

/* Eq. 6: sign strategy from the smallest value (-0.0 counts as non-negative). */
int orc_sign_f32(const float* x, int64_t n);
int orc_sign_i64(const int64_t* v, int64_t n);

/* Eq. 10-13 on fp32 data: codes[i] = Q(x[i]; k, fl, sign). */
int orc_quantize_f32(const float* x, int64_t n, int k, int fl, int sign, int32_t* codes);
/* Eq. 10-13 on the exact values v[i] * 2^-s (the FxP-QLayer on a C-Block result). */
int orc_quantize_i64(const int64_t* v, int64_t n, int s, int k, int fl, int sign, int32_t* codes);

/* Eq. 14, exact, returned rounded to double. */
int orc_sse_f32(const float* x, int64_t n, int k, int fl, int sign, double* sse);
int orc_sse_i64(const int64_t* v, int64_t n, int s, int k, int fl, int sign, double* sse);

/*
 * Exhaustive fractional-length search: for every fl in [fl_lo, fl_hi] the exact
 * Eq. 14 error at word length k; the winner is the smallest error, ties going
 * to the largest fl.  sign may be ORC_SIGN_AUTO (Eq. 6).  sse (nullable) gets
 * fl_hi - fl_lo + 1 errors rounded to double.
 */
int orc_fl_search_f32(const float* x, int64_t n, int k, int sign, int fl_lo, int fl_hi,
                      int* fl_best, int* sign_used, double* sse);
int orc_fl_search_i64(const int64_t* v, int64_t n, int s, int k, int sign, int fl_lo, int fl_hi,
                      int* fl_best, int* sign_used, double* sse);

/* Integer contraction: C[m][n] = sum_k A[m][k] * B[n][k] (codes as plain
 * integers, any format up to 32 bits: Eq. 12 puts signed codes in
 * [-2^31, 2^31 - 1] and unsigned ones in [0, 2^32 - 1]).  Summed exactly in
 * 128 bits; a result outside int64 is ORC_ERANGE. */
int orc_gemm(const int64_t* A, const int64_t* B, int64_t M, int64_t N, int64_t K, int64_t* C);

/* Direct convolution, NCHW input, KCRS weights, zero padding (code 0 = value 0);
 * codes and range as orc_gemm. */
int orc_conv2d(const int64_t* x, int N, int C, int H, int W, const int64_t* w, int K, int R,
               int S, int stride, int pad, int64_t* y);
/* One output y[n][k][oh][ow] of the same convolution into *y. */
int orc_conv2d_point(const int64_t* x, int N, int C, int H, int W, const int64_t* w, int K,
                     int R, int S, int stride, int pad, int n, int k, int oh, int ow, int64_t* y);

/*
 * C-Block epilogue on the accumulators acc (NCHW, `channels` channels, `hw`
 * pixels per channel) at fractional length s_acc:
 *   bias (codes at fl_b) is added after aligning both operands to the finer
 *   of the two scales by exact left shifts; the Scale layer multiplies by the
 *   per-channel code a1 (fl_a1) and adds a2 (fl_a2), again aligned exactly;
 *   then ReLU.  Any pointer may be NULL.  v gets the exact result, *s_out its
 *   fractional length.
 */
int orc_epilogue(const int64_t* acc, int n_img, int channels, int64_t hw, int s_acc,
                 const int64_t* bias, int fl_b, const int64_t* a1, int fl_a1,
                 const int64_t* a2, int fl_a2, int relu, int64_t* v, int* s_out);

/* MAX-POOL on codes (NCHW); out-of-range window taps are skipped. */
int orc_maxpool(const int32_t* x, int N, int C, int H, int W, int k, int stride, int pad,
                int32_t* y);
/* Global AVG-POOL: y[n][c] = recip * sum_{h,w} x[n][c][h][w] (exact integer). */
int orc_avgpool_global(const int32_t* x, int N, int C, int HW, int64_t recip, int64_t* y);
/* Eltwise sum of two code tensors aligned to the finer scale, optional ReLU. */
int orc_eltwise_add(const int32_t* a, int fa, const int32_t* b, int fb, int64_t n, int relu,
                    int64_t* v, int* s_out);

/* Layer error: out[0] = exact sum (ref - X*2^-fl)^2, out[1] = min(ref),
 * out[2] = max(ref), out[3] = population standard deviation of ref (Eq. 16). */
int orc_layer_error(const float* ref, const int32_t* codes, int64_t n, int k, int fl, int sign,
                    double out[4]);

/* ---- FP32 teacher ----------------------------------------------------------
 * The full-precision network whose activations are the reference of the
 * layer error in the per-layer sensitivity sweep (Sec. "Data-Structures
 * Sensitivity to Quantization": one layer quantized, the others intact; the
 * full-precision model as teacher, Sec. "Quantization Parameters
 * Optimization").  Its arithmetic is fixed so that any implementation gets
 * the same bits: a conv / FC output is the fp64 sum of the fp32 x fp32
 * products (exact in fp64) taken in the order r, s, c with padded taps
 * skipped, rounded once to fp32; the BN-as-Scale affine is one fp32 fma; the
 * bias one fp32 add; ReLU maps every value <= 0 to +0. */

/* NCHW x KCRS -> NKHW fp32. */
int orc_teacher_conv2d(const float* x, int N, int C, int H, int W, const float* w, int K, int R,
                       int S, int stride, int pad, float* y);
/* Per channel c of NCHW t (hw pixels per channel): y = relu?(fmaf(t, a1[c], a2[c]))
 * when a1 is given, else relu?(t + bias[c]) when bias is given, else relu?(t). */
int orc_teacher_affine(const float* t, int N, int C, int64_t hw, const float* a1,
                       const float* a2, const float* bias, int relu, float* y);
/* Global average: y[n][c] = (float)(sequential fp64 sum over hw / hw). */
int orc_teacher_avgpool(const float* x, int N, int C, int64_t hw, float* y);

#ifdef __cplusplus
}
#endif
#endif
