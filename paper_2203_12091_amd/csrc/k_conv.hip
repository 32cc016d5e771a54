// Quantized convolution / FC (the C-Block contraction, Sec. "Integer-Only
// Inference"): implicit GEMM over NHWC int8 codes and KRSC int8 weights with
// int32 accumulation on the gfx950 int8 matrix cores (v_mfma_i32_32x32x32_i8).
//
//   rows    m = (n, oh, ow)          M = N * Ho * Wo
//   columns j = output channel       N = K
//   depth   k = (r, s, c), c fastest K = R * S * C
//
// A block computes a BM x BN tile with 4 waves of 64 x 64 (2 x 2 MFMA tiles),
// stepping through depth in 64-byte slabs staged in LDS (double buffered, the
// next slab's global loads in flight during the current slab's MFMAs).  No
// im2col buffer: each thread gathers its rows' 16-byte chunks straight from
// the NHWC tensor, with zero padding (code 0, or -128 for codes stored as
// u - 128, both meaning the value 0).
//
// Epilogue: for inputs stored as u - 128 the exact accumulator is restored by
// adding 128 * (sum of the filter's codes).  Then, by mode:
//   EPI_ACC  store the int32 accumulators; optionally reduce the exact min /
//            max of the C-Block values (bias, Scale, ReLU applied in fp64,
//            exact below 2^53) for the FxP-QLayer;
//   EPI_MM   only the min / max;
//   EPI_WIN  the window partial sums of the exact FL search over the C-Block
//            values (the same sums the streaming window pass forms);
//   EPI_REQ  the C-Block values requantized to the searched format (Eq. 1-2);
//   EPI_PRED the predicted FxP-QLayer in one pass: the window partial sums at
//            the window the previous call's min / max give, the codes of the
//            candidate the previous call chose, and this call's min / max (no
//            int32 accumulators); a one-block decision checks the prediction.
// A C-Block whose contraction is shallow (R * S * C small next to the output)
// is cheaper to recompute three times than to write, and read twice, as
// int32: the fused launcher runs EPI_MM, EPI_WIN and EPI_REQ over the same
// operands, and stores int32 accumulators only when the window pass cannot
// decide and the exact general pass needs them.
#include <limits.h>
#include <math.h>

#include <type_traits>

#include "fls.hpp"

namespace fxpq {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v4i_a4 __attribute__((ext_vector_type(4), aligned(4)));  // dword-aligned 16 bytes
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr int BK = 64;
// Cache policy of the int32 accumulator stores: non-temporal (the tensor is
// read once, by the FL search that follows, not by this kernel).
constexpr int kAccPolicy = 2;

// LDS slab layout: rows of 64 bytes (four 16-byte chunks), no padding; chunk
// c of row r sits at chunk position c ^ f(r) with f(r) = (r >> 2) & 3.  The
// MFMA operand reads (lane l: row l % 32, one chunk) then run at the full
// ds_read_b128 rate on gfx950 (measured: 1.5x slower with f = (r >> 1) ^
// (r >> 3), 3x without a swizzle); the 16-byte stores of whole rows are
// insensitive to it.
__device__ inline int lds_swz(int row) { return (row >> 2) & 3; }
__device__ inline int lds_off(int row, int chunk) {
  return row * 64 + ((chunk ^ lds_swz(row)) & 3) * 16;
}

// FAST64: C % 64 == 0, register-staged slabs; GEN16: C % 16 == 0; RGB4: the
// 4-channel padded input; DMA64: C % 64 == 0, slabs loaded straight into a
// three-stage LDS ring (global_load_lds), two slabs in flight.  HALO4 /
// HALO8: C % 64 == 0, tiles of whole output-image rows whose input patch
// (up to 256 / 512 pixels per channel chunk) is loaded into LDS once and read
// by every filter tap, weights through the DMA ring.
enum Loader { LD_FAST64 = 0, LD_GEN16 = 1, LD_RGB4 = 2, LD_DMA64 = 3, LD_HALO4 = 4, LD_HALO8 = 5,
              LD_RGB8 = 6 };

constexpr bool is_halo(int loader) { return loader == LD_HALO4 || loader == LD_HALO8; }

// Weight stages of the halo tiles' LDS ring (HD - 1 slabs in flight).
constexpr int kHaloStages = 3;

// 16-byte padding sources of the LDS-ring loader: code 0, and code -128 for
// inputs stored as u - 128 (both the value 0).
__device__ int4 kPadVec[2] = {{0, 0, 0, 0},
                              {(int)0x80808080, (int)0x80808080, (int)0x80808080, (int)0x80808080}};

// s_waitcnt immediate that waits until at most n vector memory operations are
// outstanding (gfx9 encoding: vmcnt split over bits 3:0 and 15:14; expcnt and
// lgkmcnt left at their maxima, i.e. not waited for).
template <int N>
__device__ inline void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// One 16-byte global -> LDS load per lane (global_load_lds_dwordx4): lane l's
// bytes land at lds + 16 l.  Issued as inline asm so that the compiler does
// not add its own conservative wait for these LDS writes before later LDS
// reads (it cannot tell the ring stages apart); the ring waits explicitly
// (wait_vmcnt) and orders with ring_barrier().  M0 holds the wave-uniform LDS
// address; the s_nop separates its write from the load.
__device__ inline void dma16(const int8_t* g, int8_t* lds) {
  const uint32_t l = __builtin_amdgcn_readfirstlane((uint32_t)(uintptr_t)lds);
  asm volatile("s_nop 0\n\tglobal_load_lds_dwordx4 %0, off" ::"v"(g), "{m0}"(l) : "memory");
}

// Workgroup barrier without the memory fence __syncthreads() adds: that fence
// would wait for every outstanding LDS-ring load.  The empty asm statements
// keep the compiler from moving memory accesses across it.
__device__ inline void ring_barrier() {
  asm volatile("" ::: "memory");
  __builtin_amdgcn_s_barrier();
  asm volatile("" ::: "memory");
}
enum Epi { EPI_ACC = 0, EPI_MM = 1, EPI_WIN = 2, EPI_REQ = 3, EPI_PRED = 4 };

struct ConvArgs {
  const int8_t* x;
  const int8_t* w;
  const int32_t* colsum;
  int32_t* acc;
  int N, H, W, C, K, R, S, stride, pad, Ho, Wo;
  int M;        // rows
  int kdepth;   // R * S * C
  int wrow;     // bytes per weight row (kdepth, or padded to 64 for RGB4)
  int x_type;
  int want_mm;  // reduce min / max of the epilogue values
  SrcDev ep;    // kind == FXPQ_SRC_ACC when an epilogue is given
  int has_ep;
  double* mm_part;
  // EPI_ACC: store only when the FL-search plan asks for the general pass
  int only_if_general;
  const FlsPlan* plan_in;
  // EPI_WIN
  int wl, sign_req, fl_lo, fl_hi;
  const double* mm;      // min / max of the C-Block values
  long long* part_i;
  double* part_f;
  FlsPlan* plan;
  fxpq_fmt* fmt_win;
  unsigned* flags;
  // EPI_REQ
  const fxpq_fmt* fmt_req;
  int8_t* y;
  int y_type;
  // EPI_PRED in deferred mode: block (0, 0) records the decision's inputs
  PredJob* job;
  unsigned* job_miss;
  int64_t job_per_thread;
  // halo tiles: hG images of hTH output rows each (hG > 1 only with hTH ==
  // Ho), hTPI tiles per image (hG == 1), input patch hPH x hPW per image;
  // stores of rows that do not exist go to `sink` (32 int32)
  int hG, hTH, hTPI, hPH, hPW;
  int32_t* sink;
};

// Tile configurations: block BM x BN, four waves of (32 TM) x (32 TN), MINW
// waves per SIMD requested from the register allocator.
enum TileCfg { TC_256x64 = 0, TC_128x128 = 1, TC_256x128 = 2, TC_H224x256 = 3, TC_H128x256 = 4 };

// Accumulators per thread of a configuration (the per-thread bound of the
// fused window epilogue).
constexpr int conv_per_thread(int cfg) { return cfg == TC_256x128 ? 128 : 64; }

template <int BM, int BN, int TM, int TN, int MINW, int LOADER, int EPI>
__global__ __launch_bounds__(256, MINW) void k_qconv(ConvArgs a) {
  constexpr int WGN = BN / (32 * TN);  // waves along N
  static_assert((BM / (32 * TM)) * WGN == 4, "four waves per block");
  constexpr int WROWS = 32 * TM, WCOLS = 32 * TN;
  constexpr int PER_THREAD = TM * TN * 16;
  constexpr int ACH = BM / 64;  // A chunks (16 B) per thread per slab
  constexpr int BCH = BN / 64;
  // LDS slabs: two stages for the register-staged loaders; the ring of the
  // DMA loader is declared with it (one array per stage, so that the compiler
  // sees which stage a read touches and does not wait for the other stages'
  // loads in flight).
  constexpr int NST = (LOADER == LD_DMA64) ? 1 : 2;
  __shared__ __attribute__((aligned(16))) int8_t As[NST][BM * 64];
  __shared__ __attribute__((aligned(16))) int8_t Bs[NST][BN * 64];
  __shared__ int rs_tab[128];
  __shared__ double shd[8];
  __shared__ WinShared wsh;

  // Decisions every block takes identically before any load.
  WinSetup ws;
  QFmt qf;
  if constexpr (EPI == EPI_ACC) {
    if (a.only_if_general && (!a.plan_in->need_general || a.plan_in->status)) return;
  } else if constexpr (EPI == EPI_WIN) {
    ws = win_setup<FXPQ_SRC_ACC>(a.ep, a.mm, a.wl, a.sign_req, a.fl_lo, a.fl_hi, MODE_SEARCH,
                                 PER_THREAD);
    if (ws.verdict != 0) {
      if (blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0)
        win_verdict_write(ws, a.wl, a.fl_lo, a.fl_hi, a.plan, a.fmt_win, a.flags);
      return;
    }
  } else if constexpr (EPI == EPI_PRED) {
    // the window of the predicted min / max (verdict != 0: none to evaluate,
    // the decision counts the call a miss; the min / max still go out)
    ws = win_setup<FXPQ_SRC_ACC>(a.ep, a.mm, a.wl, a.sign_req, a.fl_lo, a.fl_hi, MODE_SEARCH,
                                 PER_THREAD);
    if (a.job && blockIdx.x == 0 && blockIdx.y == 0 && threadIdx.x == 0)
      *a.job = PredJob{a.ep, a.wl, a.sign_req, a.fl_lo, a.fl_hi, 1, a.job_per_thread,
                       const_cast<double*>(a.mm), a.fmt_win, a.job_miss, a.part_i, a.part_f};
  } else if constexpr (EPI == EPI_REQ) {
    const int sv = src_scale(a.ep);
    if (a.y_type == FXPQ_I8) qf = qfmt_setup<FXPQ_I8>(a.fmt_req, sv, a.flags);
    else if (a.y_type == FXPQ_U8OFF) qf = qfmt_setup<FXPQ_U8OFF>(a.fmt_req, sv, a.flags);
    else qf = qfmt_setup<FXPQ_C8>(a.fmt_req, sv, a.flags);
    if (!qf.ok) return;
  }

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform per wave
  const int wm = wave / WGN, wn = wave % WGN;
  // Tile of this block.  Blocks are dealt to the 8 XCDs round-robin by linear
  // id; remapped so that each XCD takes a contiguous run of tiles in
  // row-block-major order, i.e. the column tiles of one row block run on the
  // same XCD and share its L2 copy of the input rows.
  int tm = blockIdx.x, tn = blockIdx.y;
  {
    const int T = gridDim.x * gridDim.y;
    if (T % 8 == 0) {
      const int L = blockIdx.y * gridDim.x + blockIdx.x;
      const int t = (L % 8) * (T / 8) + L / 8;
      tm = t / gridDim.y;
      tn = t - tm * gridDim.y;
    }
  }
  int m0 = tm * BM;
  const int n0 = tn * BN;
  const int kc = tid & 3;
  // Halo tiles: output rows oh0 .. oh0 + hTH - 1 (all columns) of images
  // img0 .. img0 + hG - 1; vrows of the BM rows exist.
  int img0 = 0, oh0 = 0, vrows = BM;
  if constexpr (is_halo(LOADER)) {
    if (a.hG > 1) {
      img0 = tm * a.hG;
      vrows = min(a.hG, a.N - img0) * a.Ho * a.Wo;
    } else {
      img0 = tm / a.hTPI;
      oh0 = (tm - img0 * a.hTPI) * a.hTH;
      vrows = min(a.hTH, a.Ho - oh0) * a.Wo;
    }
    m0 = (img0 * a.Ho + oh0) * a.Wo;
  }

  // Inputs stored as u - 128 (branch-free, so the operand loads need not wait
  // for the format).
  const int fin_sign = *(a.has_ep ? &a.ep.fin->sign : &kEpiOne);
  const int a_off = (a.x_type == FXPQ_U8OFF) || (a.x_type == FXPQ_C8 && fin_sign == 0);
  const int padw = a_off ? (int)0x80808080 : 0;
  const v4i padv = {padw, padw, padw, padw};

  if (LOADER == LD_RGB4) {
    for (int i = tid; i < 128; i += 256) rs_tab[i] = (i < a.R * a.S) ? ((i / a.S) << 16) | (i % a.S) : -1;
    __syncthreads();
  }

  v16i acc[TM][TN];
#pragma unroll
  for (int mi = 0; mi < TM; ++mi)
#pragma unroll
    for (int ni = 0; ni < TN; ++ni)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[mi][ni][e] = 0;

  // MFMAs of one staged slab: two 32-deep steps over this wave's tile.
  auto compute = [&](const int8_t* sa, const int8_t* sb) {
    // All fragments of the slab are read first, then the MFMAs run: the LDS
    // latency is paid once per slab (interleaving reads and MFMAs on a few
    // reused registers paid it before every pair of MFMAs).
    v4i af[2][TM], bf[2][TN];
#pragma unroll
    for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
      for (int mi = 0; mi < TM; ++mi)
        af[kk][mi] = *reinterpret_cast<const v4i*>(
            &sa[lds_off(wm * WROWS + mi * 32 + (lane & 31), kk * 2 + (lane >> 5))]);
#pragma unroll
      for (int ni = 0; ni < TN; ++ni)
        bf[kk][ni] = *reinterpret_cast<const v4i*>(
            &sb[lds_off(wn * WCOLS + ni * 32 + (lane & 31), kk * 2 + (lane >> 5))]);
    }
    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
    for (int kk = 0; kk < 2; ++kk)
#pragma unroll
      for (int mi = 0; mi < TM; ++mi)
#pragma unroll
        for (int ni = 0; ni < TN; ++ni)
          acc[mi][ni] =
              __builtin_amdgcn_mfma_i32_32x32x32_i8(af[kk][mi], bf[kk][ni], acc[mi][ni], 0, 0, 0);
  };

  // Per-channel epilogue operands of this thread's output columns, loaded
  // before the main loop so that their latency overlaps it.
  const bool want_vals = (EPI != EPI_ACC) || a.want_mm;
  int csum[TN];
  EpiRaw eraw[TN];
  auto epi_loads = [&]() {
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) {
      const int col = n0 + wn * WCOLS + ni * 32 + (lane & 31);
      const int cc = col < a.K ? col : a.K - 1;
      csum[ni] = *(a_off ? a.colsum + cc : &kEpiZero);
      if (want_vals) eraw[ni] = epi_channel_load(a.ep, cc);
    }
  };
  // EPI_PRED: the accumulators start at the restoring term 128 * (sum of
  // the filter's codes) of inputs stored as u - 128 (zero otherwise), so the
  // matrix cores return the restored accumulator (exact in int32 like it)
  auto acc_start = [&]() {
    if constexpr (EPI == EPI_PRED) {
#pragma unroll
      for (int ni = 0; ni < TN; ++ni)
#pragma unroll
        for (int mi = 0; mi < TM; ++mi)
#pragma unroll
          for (int e = 0; e < 16; ++e) acc[mi][ni][e] = 128 * csum[ni];
    }
  };
  const int ktiles = (a.kdepth + BK - 1) / BK;
  const int hw_out = a.Ho * a.Wo;
  const int taps = a.R * a.S;

  if constexpr (LOADER == LD_DMA64) {
    // Each wave fills 1 KB pieces of a stage (16 rows of 64 bytes): piece
    // q = 4 j + wave, lane l -> row 16 q + l / 4, physical chunk l % 4, which
    // holds logical chunk (l % 4) ^ f(row) of the swizzled layout.  The
    // channel chunks are walked outermost and the filter taps innermost.
    constexpr int AJ = BM / 64, BJ = BN / 64;
    const int8_t* asrc[AJ];
    int aih[AJ], aiw[AJ], acoff[AJ];
    bool aok[AJ];
#pragma unroll
    for (int j = 0; j < AJ; ++j) {
      const int row = 16 * (4 * j + wave) + (lane >> 2);
      const int grow = m0 + row;
      aok[j] = grow < a.M;
      const int rr = aok[j] ? grow : a.M - 1;
      const int n = rr / hw_out, rem = rr - n * hw_out;
      const int oh = rem / a.Wo, ow = rem - oh * a.Wo;
      aih[j] = oh * a.stride - a.pad;
      aiw[j] = ow * a.stride - a.pad;
      asrc[j] = a.x + (int64_t)n * a.H * a.W * a.C;
      acoff[j] = (((lane & 3) ^ lds_swz(row)) & 3) * 16;
    }
    const int8_t* bsrc[BJ];
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
      const int row = 16 * (4 * j + wave) + (lane >> 2);
      const int col = n0 + row;
      const int cc = col < a.K ? col : a.K - 1;
      bsrc[j] = a.w + (int64_t)cc * a.wrow + (((lane & 3) ^ lds_swz(row)) & 3) * 16;
    }
    const int8_t* padp = reinterpret_cast<const int8_t*>(&kPadVec[a_off]);
    __shared__ __attribute__((aligned(16))) int8_t A0[BM * 64], A1[BM * 64], A2[BM * 64];
    __shared__ __attribute__((aligned(16))) int8_t B0[BN * 64], B1[BN * 64], B2[BN * 64];
    auto issue = [&](int kt, int8_t* sa, int8_t* sb) {
      const int cchunk = kt / taps;
      const int rs = kt - cchunk * taps;
      const int r = rs / a.S, sx = rs - r * a.S;
      const int c0 = cchunk * BK;
      const int k0 = rs * a.C + c0;
#pragma unroll
      for (int j = 0; j < AJ; ++j) {
        const int ih = aih[j] + r, iw = aiw[j] + sx;
        const bool ok = aok[j] && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
        const int8_t* p = ok ? asrc[j] + ((int64_t)ih * a.W + iw) * a.C + c0 + acoff[j] : padp;
        dma16(p, &sa[(4 * j + wave) * 1024]);
      }
#pragma unroll
      for (int j = 0; j < BJ; ++j) {
        dma16(bsrc[j] + k0, &sb[(4 * j + wave) * 1024]);
      }
    };
    // One ring step: slab kt from stage (ca, cb); slab kt + 2 into the stage
    // (ia, ib) that slab kt - 1 used.  Waiting: this wave's pieces of slab kt
    // have landed (the next slab's may still be in flight); after the barrier
    // every wave's have, and every wave has finished reading stage (ia, ib).
    auto step = [&](int kt, const int8_t* ca, const int8_t* cb, int8_t* ia, int8_t* ib) {
      if (kt + 1 < ktiles) wait_vmcnt<AJ + BJ>();
      else wait_vmcnt<0>();
      ring_barrier();
      if (kt + 2 < ktiles) issue(kt + 2, ia, ib);
      compute(ca, cb);
    };
    epi_loads();
    issue(0, A0, B0);
    if (ktiles > 1) issue(1, A1, B1);
    acc_start();
    for (int kt = 0; kt < ktiles; kt += 3) {
      step(kt, A0, B0, A2, B2);
      if (kt + 1 < ktiles) step(kt + 1, A1, B1, A0, B0);
      if (kt + 2 < ktiles) step(kt + 2, A2, B2, A1, B1);
    }
  } else if constexpr (is_halo(LOADER)) {
    // Patch row R (pixel of the padded input patch) of a chunk sits at LDS row
    // R of a patch buffer; the DMA pieces of 16 rows are dealt to the waves as
    // in LD_DMA64.  Filter tap (r, s) of output row p reads patch row
    // pbase(p) + r * hPW + s.  Weights: one 64-byte slab per (chunk, tap).
    static_assert(WGN == 4, "halo tiles split the block's columns over the four waves");
    constexpr int AJ = (LOADER == LD_HALO8) ? 8 : 4, BJ = BN / 64;
    constexpr int NPR = 64 * AJ;  // patch rows per buffer
    constexpr int HD = kHaloStages;
    __shared__ __attribute__((aligned(16))) int8_t P0[NPR * 64], P1[NPR * 64];
    __shared__ __attribute__((aligned(16))) int8_t Bst[HD][BN * 64];
    const int ppx = a.hPH * a.hPW;
    const int npx = a.hG * ppx;
    const int8_t* psrc[AJ];
    bool pok[AJ];
#pragma unroll
    for (int j = 0; j < AJ; ++j) {
      const int R = 16 * (4 * j + wave) + (lane >> 2);
      const int g = R / ppx, rem = R - g * ppx;
      const int py = rem / a.hPW, px = rem - py * a.hPW;
      const int ih = oh0 * a.stride - a.pad + py, iw = px - a.pad, img = img0 + g;
      pok[j] = R < npx && img < a.N && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
      const int lch = ((lane & 3) ^ lds_swz(R)) & 3;
      psrc[j] = a.x + (pok[j] ? (((int64_t)img * a.H + ih) * a.W + iw) * a.C + lch * 16 : 0);
    }
    const int8_t* bsrc[BJ];
#pragma unroll
    for (int j = 0; j < BJ; ++j) {
      const int row = 16 * (4 * j + wave) + (lane >> 2);
      const int col = n0 + row;
      const int cc = col < a.K ? col : a.K - 1;
      bsrc[j] = a.w + (int64_t)cc * a.wrow + (((lane & 3) ^ lds_swz(row)) & 3) * 16;
    }
    // patch row of tap (0, 0) for each of this lane's output rows
    int pbase[TM];
    const int rows_img = a.hTH * a.Wo;
#pragma unroll
    for (int mi = 0; mi < TM; ++mi) {
      const int p = mi * 32 + (lane & 31);
      const int g = p / rows_img, q = p - g * rows_img;
      const int ohl = q / a.Wo, ow = q - ohl * a.Wo;
      pbase[mi] = (p < vrows) ? g * ppx + ohl * a.stride * a.hPW + ow * a.stride : 0;
    }
    const int8_t* padp = reinterpret_cast<const int8_t*>(&kPadVec[a_off]);
    auto issue = [&](int kt, int8_t* sb) {
      const int cchunk = kt / taps;
      const int rs = kt - cchunk * taps;
      const int c0 = cchunk * BK;
      if (rs == 0) {
        int8_t* pb = (cchunk & 1) ? P1 : P0;
#pragma unroll
        for (int j = 0; j < AJ; ++j) dma16(pok[j] ? psrc[j] + c0 : padp, &pb[(4 * j + wave) * 1024]);
      }
      const int k0 = rs * a.C + c0;
#pragma unroll
      for (int j = 0; j < BJ; ++j) dma16(bsrc[j] + k0, &sb[(4 * j + wave) * 1024]);
    };
    auto compute_tap = [&](int kt, const int8_t* sb) {
      const int cchunk = kt / taps;
      const int rs = kt - cchunk * taps;
      const int r = rs / a.S, sx = rs - r * a.S;
      const int toff = r * a.hPW + sx;
      const int8_t* pb = (cchunk & 1) ? P1 : P0;
      v4i af[2][TM], bf[2][TN];
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
        for (int mi = 0; mi < TM; ++mi)
          af[kk][mi] = *reinterpret_cast<const v4i*>(&pb[lds_off(pbase[mi] + toff, kk * 2 + (lane >> 5))]);
#pragma unroll
        for (int ni = 0; ni < TN; ++ni)
          bf[kk][ni] = *reinterpret_cast<const v4i*>(
              &sb[lds_off(wn * WCOLS + ni * 32 + (lane & 31), kk * 2 + (lane >> 5))]);
      }
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int kk = 0; kk < 2; ++kk)
#pragma unroll
        for (int mi = 0; mi < TM; ++mi)
#pragma unroll
          for (int ni = 0; ni < TN; ++ni)
            acc[mi][ni] =
                __builtin_amdgcn_mfma_i32_32x32x32_i8(af[kk][mi], bf[kk][ni], acc[mi][ni], 0, 0, 0);
    };
    // Ring of HD weight stages: slab kt + HD - 1 is issued at step kt into
    // the stage slab kt - 1 used.  Waiting at step kt: slab kt's loads have
    // landed while the (up to HD - 2) later slabs' may be in flight; at most
    // one of those carries a chunk's patch (a chunk has taps >= HD - 1 slabs).
    auto wait_slab = [&](int kt) {
      const int later = min(HD - 2, ktiles - 1 - kt);
      bool patch = false;
      for (int j = 1; j <= later; ++j) patch = patch || (kt + j) % taps == 0;
      switch (later * 2 + (patch ? 1 : 0)) {
        case 0: wait_vmcnt<0>(); break;
        case 2: wait_vmcnt<BJ>(); break;
        case 3: wait_vmcnt<BJ + AJ>(); break;
        case 4: wait_vmcnt<2 * BJ>(); break;
        case 5: wait_vmcnt<2 * BJ + AJ>(); break;
        case 6: wait_vmcnt<3 * BJ>(); break;
        default: wait_vmcnt<3 * BJ + AJ>(); break;
      }
    };
    static_assert(HD >= 3 && HD <= 5, "ring depth");
    epi_loads();
#pragma unroll
    for (int j = 0; j < HD - 1; ++j)
      if (j < ktiles) issue(j, Bst[j]);
    for (int kt0 = 0; kt0 < ktiles; kt0 += HD) {
#pragma unroll
      for (int j = 0; j < HD; ++j) {
        const int kt = kt0 + j;
        if (kt < ktiles) {
          wait_slab(kt);
          ring_barrier();
          if (kt + HD - 1 < ktiles) issue(kt + HD - 1, Bst[(j + HD - 1) % HD]);
          compute_tap(kt, Bst[j]);
        }
      }
    }
  } else {
    // Rows owned by this thread for A loads.
    const int8_t* abase[ACH];
    int ih0[ACH], iw0[ACH];
    bool aval[ACH];
#pragma unroll
    for (int i = 0; i < ACH; ++i) {
      int row = m0 + (tid >> 2) + 64 * i;
      aval[i] = row < a.M;
      int rr = aval[i] ? row : a.M - 1;
      int n = rr / hw_out, rem = rr - n * hw_out;
      int oh = rem / a.Wo, ow = rem - oh * a.Wo;
      ih0[i] = oh * a.stride - a.pad;
      iw0[i] = ow * a.stride - a.pad;
      abase[i] = a.x + (int64_t)n * a.H * a.W * a.C;
    }
    const int8_t* bptr[BCH];
#pragma unroll
    for (int i = 0; i < BCH; ++i) {
      int col = n0 + (tid >> 2) + 64 * i;
      int cc = col < a.K ? col : a.K - 1;
      bptr[i] = a.w + (int64_t)cc * a.wrow;
    }
    // Loads are unconditional (from a valid address when the element does
    // not exist); the pad / zero value replaces them at the LDS store.  A
    // select right after the load would let the compiler branch around the
    // load and then wait at the join for the loads just issued, i.e. for
    // the next slab before this slab's MFMAs.
    v4i regA[ACH], regB[BCH];
    bool aok[ACH], bok[BCH];
    int rgb_d[ACH];  // LD_RGB8: dword shift of the loaded pixels (0 inside)
    auto gload = [&](int kt) {
      // FAST64 walks the depth channel chunk by channel chunk with the filter
      // taps innermost, so that consecutive slabs read neighbouring pixels of
      // the same channels (cache reuse); the integer sums do not depend on the
      // order.
      const int cchunk = (LOADER == LD_FAST64) ? kt / taps : 0;
      const int rs = (LOADER == LD_FAST64) ? kt - cchunk * taps : 0;
      const int k0 = (LOADER == LD_FAST64) ? rs * a.C + cchunk * BK : kt * BK;
      if constexpr (LOADER == LD_FAST64) {
        const int c0 = cchunk * BK;
        int r = rs / a.S, s = rs - r * a.S;
#pragma unroll
        for (int i = 0; i < ACH; ++i) {
          int ih = ih0[i] + r, iw = iw0[i] + s;
          bool ok = aval[i] && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
          const int8_t* p = abase[i] + (ok ? ((int64_t)ih * a.W + iw) * a.C + c0 + kc * 16 : 0);
          regA[i] = *reinterpret_cast<const v4i*>(p);
          aok[i] = ok;
        }
      } else if constexpr (LOADER == LD_GEN16) {
        int k = k0 + kc * 16;
        int rs = k / a.C, c0 = k - rs * a.C;
        int r = rs / a.S, s = rs - r * a.S;
        bool kin = k < a.kdepth;
#pragma unroll
        for (int i = 0; i < ACH; ++i) {
          int ih = ih0[i] + r, iw = iw0[i] + s;
          bool ok = kin && aval[i] && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
          const int8_t* p = abase[i] + (ok ? ((int64_t)ih * a.W + iw) * a.C + c0 : 0);
          regA[i] = *reinterpret_cast<const v4i*>(p);
          aok[i] = ok;
        }
      } else if constexpr (LOADER == LD_RGB8) {
        // filters re-laid as [r][s < 8][c]: chunk q = 4 kt + kc is filter
        // row q / 2, taps 4 (q % 2) .. + 3, i.e. four neighbouring pixels of
        // one input row: one 16-byte load of the four pixels from column
        // iw clamped to [0, W - 4] (W >= 4); at the image borders the LDS
        // store shifts them by d = iw - that column and pads the pixels
        // outside the row (the taps past S have zero weights: their pixels
        // only need to be readable).  Rows past R are zero filter rows; a
        // row outside the image is all padding (d = 8).
        const int q = kt * 4 + kc;
        const int r = q >> 1, s0 = (q & 1) * 4;
#pragma unroll
        for (int i = 0; i < ACH; ++i) {
          const int ih = ih0[i] + r, iw = iw0[i] + s0;
          const bool rowok = aval[i] && r < a.R && ih >= 0 && ih < a.H;
          const int iwc = min(max(iw, 0), a.W - 4);
          const int64_t off = rowok ? ((int64_t)ih * a.W + iwc) * 4 : 0;
          regA[i] = *reinterpret_cast<const v4i_a4*>(abase[i] + off);
          rgb_d[i] = rowok ? iw - iwc : 8;
          aok[i] = true;
        }
      } else {  // LD_RGB4: four 4-byte pixels per 16-byte chunk
#pragma unroll
        for (int i = 0; i < ACH; ++i) {
          v4i v;
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            int rs = (k0 + kc * 16 + 4 * j) >> 2;
            int t = (rs < 128) ? rs_tab[rs] : -1;
            int word = padw;
            if (t >= 0 && aval[i]) {
              int ih = ih0[i] + (t >> 16), iw = iw0[i] + (t & 0xFFFF);
              if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W)
                word = *reinterpret_cast<const int*>(abase[i] + ((int64_t)ih * a.W + iw) * 4);
            }
            v[j] = word;
          }
          regA[i] = v;
          aok[i] = true;
        }
      }
#pragma unroll
      for (int i = 0; i < BCH; ++i) {
        const int k = k0 + kc * 16;
        const bool kin = LOADER != LD_GEN16 || k < a.kdepth;
        regB[i] = *reinterpret_cast<const v4i*>(bptr[i] + (kin ? k : 0));
        bok[i] = kin;
      }
    };
    auto lstore = [&](int buf) {
#pragma unroll
      for (int i = 0; i < ACH; ++i) {
        v4i v = aok[i] ? regA[i] : padv;
        if constexpr (LOADER == LD_RGB8) {
          const int d = rgb_d[i];
          if (d != 0) {  // image border or missing row (no loads in here)
            v4i o;
#pragma unroll
            for (int j = 0; j < 4; ++j) {
              const int m = j + d;
              const int pk = m <= 0 ? v[0] : (m == 1 ? v[1] : (m == 2 ? v[2] : v[3]));
              o[j] = (m >= 0 && m < 4) ? pk : padw;
            }
            v = o;
          }
        }
        *reinterpret_cast<v4i*>(&As[buf][lds_off((tid >> 2) + 64 * i, kc)]) = v;
      }
#pragma unroll
      for (int i = 0; i < BCH; ++i)
        *reinterpret_cast<v4i*>(&Bs[buf][lds_off((tid >> 2) + 64 * i, kc)]) =
            bok[i] ? regB[i] : v4i{0, 0, 0, 0};
    };
    gload(0);
    epi_loads();
    lstore(0);
    acc_start();
    __syncthreads();
    for (int kt = 0; kt < ktiles; ++kt) {
      const int buf = kt & 1;
      if (kt + 1 < ktiles) gload(kt + 1);
      compute(As[buf], Bs[buf]);
      if (kt + 1 < ktiles) lstore(buf ^ 1);
      __syncthreads();
    }
  }

  // ---- epilogue ----
  // Visits this thread's in-range accumulators (restored for u - 128 inputs)
  // with the channel's epilogue constants.
  EpiU eu;
  if (want_vals) eu = epi_uniform(a.ep);
  const bool full = m0 + BM <= a.M && n0 + BN <= a.K;
  auto visit = [&](auto&& f) {
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) {
      const int col = n0 + wn * WCOLS + ni * 32 + (lane & 31);
      const int corr = 128 * csum[ni];
      double Mc = 1.0, Ac = 0.0;
      if (want_vals) epi_channel_raw(a.ep, eu, eraw[ni], Mc, Ac);
#pragma unroll
      for (int mi = 0; mi < TM; ++mi) {
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const int row = m0 + wm * WROWS + mi * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
          if (full || (row < a.M && col < a.K)) f(acc[mi][ni][e] + corr, Mc, Ac, row, col);
        }
      }
    }
  };
  const double relo = a.ep.ep_relu ? 0.0 : -INFINITY;  // ReLU as max(v, relo)
  const int bid = blockIdx.y * gridDim.x + blockIdx.x;

  if constexpr (EPI == EPI_ACC || EPI == EPI_MM) {
    // The epilogue value is a monotonic function of the accumulator within a
    // channel (v = relu(acc * M + A), rounding included), so the min / max of
    // the values are those of the channel's extreme accumulators: track the
    // integer extremes per column, evaluate the epilogue on them only.
    int lo[TN], hi[TN];
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) {
      lo[ni] = INT_MAX;
      hi[ni] = INT_MIN;
    }
    if constexpr (is_halo(LOADER)) {
      // Rows past vrows do not exist (padding of the last MFMA row tile, or a
      // partial tile): their stores go to a scratch sink, their values are not
      // counted (branch-free selects).
#pragma unroll
      for (int ni = 0; ni < TN; ++ni) {
        const int col = n0 + wn * WCOLS + ni * 32 + (lane & 31);
        const int corr = 128 * csum[ni];
        int32_t* dst = a.acc + (int64_t)m0 * a.K + col;
        int32_t* sink = a.sink + (lane & 31);
#pragma unroll
        for (int mi = 0; mi < TM; ++mi) {
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int lr = mi * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
            const bool ok = lr < vrows;
            const int v = acc[mi][ni][e];
            if constexpr (EPI == EPI_ACC)
              __builtin_nontemporal_store(v + corr, ok ? dst + (int64_t)lr * a.K : sink);
            lo[ni] = min(lo[ni], ok ? v : INT_MAX);
            hi[ni] = max(hi[ni], ok ? v : INT_MIN);
          }
        }
      }
    } else if (full) {
      // Full tile: buffer stores with the row offset in a scalar register.
      __amdgpu_buffer_rsrc_t rs;
      int vo[TN];
      if constexpr (EPI == EPI_ACC) {
        rs = __builtin_amdgcn_make_buffer_rsrc(a.acc + (int64_t)(m0 + wm * WROWS) * a.K, (short)0,
                                               0x7fffffff, 0x00020000);
#pragma unroll
        for (int ni = 0; ni < TN; ++ni)
          vo[ni] = (4 * (lane >> 5) * a.K + n0 + wn * WCOLS + ni * 32 + (lane & 31)) * 4;
      }
#pragma unroll
      for (int ni = 0; ni < TN; ++ni) {
        const int corr = 128 * csum[ni];
#pragma unroll
        for (int mi = 0; mi < TM; ++mi) {
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int v = acc[mi][ni][e];
            if constexpr (EPI == EPI_ACC)
              __builtin_amdgcn_raw_buffer_store_b32(
                  v + corr, rs, vo[ni], (mi * 32 + 8 * (e >> 2) + (e & 3)) * a.K * 4, kAccPolicy);
            lo[ni] = min(lo[ni], v);
            hi[ni] = max(hi[ni], v);
          }
        }
      }
    } else {
#pragma unroll
      for (int ni = 0; ni < TN; ++ni) {
        const int col = n0 + wn * WCOLS + ni * 32 + (lane & 31);
        const int corr = 128 * csum[ni];
#pragma unroll
        for (int mi = 0; mi < TM; ++mi) {
#pragma unroll
          for (int e = 0; e < 16; ++e) {
            const int row = m0 + wm * WROWS + mi * 32 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
            if (row < a.M && col < a.K) {
              const int v = acc[mi][ni][e];
              if constexpr (EPI == EPI_ACC)
                __builtin_nontemporal_store(v + corr, a.acc + (int64_t)row * a.K + col);
              lo[ni] = min(lo[ni], v);
              hi[ni] = max(hi[ni], v);
            }
          }
        }
      }
    }
    if (!want_vals) return;
    double mn = INFINITY, mx = -INFINITY;
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) {
      if (lo[ni] > hi[ni]) continue;  // no in-range value in this column
      double Mc, Ac;
      epi_channel_raw(a.ep, eu, eraw[ni], Mc, Ac);
      const int corr = 128 * csum[ni];
      const double f0 = fmax(fma((double)(lo[ni] + corr), Mc, Ac), relo);
      const double f1 = fmax(fma((double)(hi[ni] + corr), Mc, Ac), relo);
      mn = fmin(mn, fmin(f0, f1));
      mx = fmax(mx, fmax(f0, f1));
    }
    mn = block_reduce(mn, OpMin(), shd);
    mx = block_reduce(mx, OpMax(), shd);
    if (tid == 0) {
      a.mm_part[2 * bid] = mn;
      a.mm_part[2 * bid + 1] = mx;
    }
  } else if constexpr (EPI == EPI_WIN) {
    const FlsU& u = ws.u;
    const WinCtx wc = win_ctx(u, ws);
    WinAcc wa;
    win_acc_zero(wa);
    // W = v * 2^(sigma - sv): fold the integer scaling into the constants.
    const double wsc = u.wscale;
#define FXPQ_WIN_VISIT(NN, C0)                                              \
  visit([&](int v, double Mc, double Ac, int, int) {                        \
    const double W = fmax(fma((double)v, Mc * wsc, Ac * wsc), relo);       \
    win_consume<false, NN, C0>(wc, wa, W);                                  \
  })
    switch (win_variant(u, ws, a.mm)) {
      case 0: FXPQ_WIN_VISIT(false, false); break;
      case 1: FXPQ_WIN_VISIT(false, true); break;
      case 2: FXPQ_WIN_VISIT(true, false); break;
      default: FXPQ_WIN_VISIT(true, true); break;
    }
#undef FXPQ_WIN_VISIT
    win_write_partials_int(wa, 1, bid, a.part_i, a.part_f, wsh);
  } else if constexpr (EPI == EPI_PRED) {
    // Every value: W = the C-Block value (exact; at the source's own scale,
    // so W is also what the min / max report), its min / max, and when the
    // predicted window exists its window sums and the code of candidate pj
    // (the previous call's choice) as a byte (q - 128 when unsigned).  The
    // codes leave as dwords: a lane holds one column at 4 consecutive rows
    // (e = 4g .. 4g + 3), and a 4 x 4 byte transpose inside each lane quad
    // (two DPP exchanges) gives lane 4k + j row j at 4 consecutive columns.
    // Full tiles run straight-line code without checks; partial tiles check
    // every value (as straight-line selects their 64 compare masks would not
    // fit the registers).
    const FlsU& u = ws.u;
    const bool win = ws.verdict == 0;
    const int pj = pred_pick(ws, *a.fmt_win);
    const int qmax = (int)u.qmax, qmin = (int)u.qmin;
    const unsigned xorw = u.sign ? 0u : 0x80808080u;
    WinCtx wc;
    if (win) wc = win_ctx(u, ws);
    WinAcc wa;
    win_acc_zero(wa);
    // The window sums are formed from x = W 2^(b0 - sigma), the value in
    // units of the first candidate's step, straight from the accumulator
    // (multiplier and addend scaled by that power of two): its code is
    // rne(x), the second candidate's rne(2 x), the clipping bound's
    // argument x 2^(bce - b0).  Sums of x q and x^2 are those of W q and W^2
    // scaled by 2^(b0 - sigma) and its square, exactly (every term keeps its
    // bits); they are scaled back before the block reduction.  In windows
    // with negative values whose first candidate cannot saturate, the second
    // candidate's code comes from the low bits of x plus a rounding
    // constant, clamped as an integer by one median-of-three, then converted
    // back (as measured, this form does not pay in the non-negative windows,
    // whose clamps are one-sided).
    const double xs = win ? wc.cj[0] : 1.0;      // 2^(b0 - sigma)
    const double xce = win ? wc.cce / xs : 1.0;  // 2^(bce - b0)
    const double xce_hi = win ? wc.qmax / xce : 0.0, xce_lo = win ? wc.qmin / xce : 0.0;
    // byte selectors of the two transpose steps (v_perm: bytes 0-3 this
    // lane's dword, 4-7 the partner's): step 1 pairs lanes j, j ^ 1 (even
    // lanes keep bytes 0 and 2 of both, odd lanes bytes 1 and 3), step 2
    // lanes j, j ^ 2 (the low or high halves of both)
    const int qj = lane & 3;
    const unsigned s1 = (qj & 1) ? 0x03070105u : 0x06020400u;
    const unsigned s2 = (qj & 2) ? 0x03020706u : 0x05040100u;
    // min / max from the integer extremes of each column (the epilogue is
    // monotonic in the accumulator within a channel), as EPI_ACC does
    int lo[TN], hi[TN];
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) {
      lo[ni] = INT_MAX;
      hi[ni] = INT_MIN;
    }
    auto tile = [&](auto nn, auto c0, auto wn_, auto pj_, auto full_) {
      constexpr bool NN = decltype(nn)::value, C0 = decltype(c0)::value;
      constexpr bool WIN = decltype(wn_)::value, FULL = decltype(full_)::value;
      constexpr int PJ = decltype(pj_)::value ? 1 : 0;
#pragma unroll
      for (int ni = 0; ni < TN; ++ni) {
        const int col = n0 + wn * WCOLS + ni * 32 + (lane & 31);
        double Mc, Ac;
        epi_channel_raw(a.ep, eu, eraw[ni], Mc, Ac);
        Mc *= xs;
        Ac *= xs;
        const int scol = n0 + wn * WCOLS + ni * 32 + ((lane & 31) & ~3);
#pragma unroll
        for (int mi = 0; mi < TM; ++mi) {
#pragma unroll
          for (int g = 0; g < 4; ++g) {
            const int rbase = m0 + wm * WROWS + mi * 32 + 8 * g + 4 * (lane >> 5);
            int c[4];
#pragma unroll
            for (int jj = 0; jj < 4; ++jj) {
              const int v = acc[mi][ni][4 * g + jj];
              const bool ok = FULL || (rbase + jj < a.M && col < a.K);
              lo[ni] = min(lo[ni], ok ? v : INT_MAX);
              hi[ni] = max(hi[ni], ok ? v : INT_MIN);
              c[jj] = 0;
              if constexpr (WIN) {
                if (ok) {
                  static_assert(kWindow == 2, "two window candidates");
                  if constexpr (NN) {
                    double x = fma((double)v, Mc, Ac);
                    x = max64s(x, relo);
                    wa.V2 = fma(x, x, wa.V2);
                    double q0 = rint(x);
                    if (C0) q0 = min64(q0, wc.qmax);
                    wa.A[0] = fma(q0, q0, wa.A[0]);
                    wa.PL[0] = fma(x, q0, wa.PL[0]);
                    const double q1 = min64(rint(x + x), wc.qmax);
                    wa.A[1] = fma(q1, q1, wa.A[1]);
                    wa.PL[1] = fma(x, q1, wa.PL[1]);
                    // clipping error at bce: (x - x clamped to its range
                    // [qmin, qmax] 2^(b0 - bce))^2, in units scaled by
                    // 2^(2 (b0 - bce)) (exactly those of (t - qmax)^+ and
                    // (t - qmin)^- with t = x 2^(bce - b0), scaled back
                    // below); one-sided here
                    const double e = x - min64(x, xce_hi);
                    wa.CE[0] = fma(e, e, wa.CE[0]);
                    int c0 = (int)q0;
                    const int c1 = (int)q1;
                    if (PJ == 0 && !C0) c0 = min(c0, qmax);
                    c[jj] = PJ ? c1 : c0;
                  } else {
                    // a window with negative values is never a ReLU layer's
                    // (its values are >= 0, so is the previous call's
                    // minimum): no max with the ReLU bound here; a prediction
                    // that says otherwise is a miss anyway (its window's
                    // variant differs from the actual one)
                    const double x = fma((double)v, Mc, Ac);
                    wa.V2 = fma(x, x, wa.V2);
                    double q0, q1;
                    int c0 = 0, c1;
                    if (C0) {
                      // the first candidate saturates: x is not bounded by
                      // the codes' range (the rounding constant's int view
                      // needs |2 x| < 2^31), so both codes are clamped in fp64
                      q0 = max64(min64(rint(x), wc.qmax), wc.qmin);
                      q1 = max64(min64(rint(x + x), wc.qmax), wc.qmin);
                      c0 = (int)q0;
                      c1 = (int)q1;
                    } else {
                      // every value of a hit lies within [qmin - 1/2,
                      // qmax + 1/2] at the first candidate's step
                      q0 = rint(x);
                      if (PJ == 0) c0 = min((int)q0, qmax);
                      c1 = med3i(rne_lo(x + kRne1), qmin, qmax);
                      q1 = (double)c1;
                    }
                    wa.A[0] = fma(q0, q0, wa.A[0]);
                    wa.PL[0] = fma(x, q0, wa.PL[0]);
                    wa.A[1] = fma(q1, q1, wa.A[1]);
                    wa.PL[1] = fma(x, q1, wa.PL[1]);
                    // clipping error at bce, two-sided
                    const double xcl = max64(min64(x, xce_hi), xce_lo);
                    const double e = x - xcl;
                    wa.CE[0] = fma(e, e, wa.CE[0]);
                    c[jj] = PJ ? c1 : c0;
                  }
                }
              }
            }
            if constexpr (WIN) {
              // the four codes' low bytes into one dword (row jj in byte jj)
              const unsigned p01 = __builtin_amdgcn_perm((unsigned)c[1], (unsigned)c[0], 0x0C0C0400u);
              const unsigned p23 = __builtin_amdgcn_perm((unsigned)c[3], (unsigned)c[2], 0x0C0C0400u);
              unsigned w4 = __builtin_amdgcn_perm(p23, p01, 0x05040100u);
              // lane j of the quad holds rows 0..3 of column j: transpose
              // with one partner exchange and one per-lane byte permute per step
              w4 = __builtin_amdgcn_perm((unsigned)__builtin_amdgcn_mov_dpp((int)w4, 0xB1, 0xF, 0xF, false),
                                         w4, s1);
              w4 = __builtin_amdgcn_perm((unsigned)__builtin_amdgcn_mov_dpp((int)w4, 0x4E, 0xF, 0xF, false),
                                         w4, s2);
              const int srow = rbase + qj;
              if (FULL || (srow < a.M && scol < a.K))
                *reinterpret_cast<unsigned*>(a.y + (int64_t)srow * a.K + scol) = w4 ^ xorw;
            }
          }
        }
      }
    };
    using F = std::false_type;
    using T = std::true_type;
    if (!win) {
      if (full) tile(F(), F(), F(), F(), T());
      else tile(F(), F(), F(), F(), F());
    } else {
      const int var = win_variant(u, ws, a.mm);
#define FXPQ_PRED_TILE(NN, C0)                                                                  \
  (full ? (pj ? tile(NN(), C0(), T(), T(), T()) : tile(NN(), C0(), T(), F(), T()))              \
        : (pj ? tile(NN(), C0(), T(), T(), F()) : tile(NN(), C0(), T(), F(), F())))
      switch (var) {
        case 0: FXPQ_PRED_TILE(F, F); break;
        case 1: FXPQ_PRED_TILE(F, T); break;
        case 2: FXPQ_PRED_TILE(T, F); break;
        default: FXPQ_PRED_TILE(T, T); break;
      }
#undef FXPQ_PRED_TILE
      // back to the units of W: sum W q = 2^(sigma - b0) sum x q, sum W^2 =
      // 2^(2 (sigma - b0)) sum x^2 (exact powers of two)
      const double up = 1.0 / xs;
      wa.PL[0] *= up;
      wa.PL[1] *= up;
      wa.V2 *= up * up;
      wa.CE[0] *= xce * xce;
      win_write_partials_int(wa, 1, bid, a.part_i, a.part_f, wsh);
    }
    double mn = INFINITY, mx = -INFINITY;
#pragma unroll
    for (int ni = 0; ni < TN; ++ni) {
      if (lo[ni] > hi[ni]) continue;  // no in-range value in this column
      double Mc, Ac;
      epi_channel_raw(a.ep, eu, eraw[ni], Mc, Ac);
      const double f0 = fmax(fma((double)lo[ni], Mc, Ac), relo);
      const double f1 = fmax(fma((double)hi[ni], Mc, Ac), relo);
      mn = fmin(mn, fmin(f0, f1));
      mx = fmax(mx, fmax(f0, f1));
    }
    // into the slots, beside the window sums (no per-block partials to finish)
    mm_slot_add(mn, mx, bid, a.part_i);
  } else {  // EPI_REQ
    visit([&](int v, double Mc, double Ac, int row, int col) {
      const double val = fmax(fma((double)v, Mc, Ac), relo);
      a.y[(int64_t)row * a.K + col] = (int8_t)quant_one(val, qf);
    });
  }
}

template <int BM, int BN, int TM, int TN, int MINW, int EPI>
static void conv_dispatch_loader(int loader, dim3 grid, hipStream_t st, const ConvArgs& a) {
  if (loader == LD_FAST64)
    k_qconv<BM, BN, TM, TN, MINW, LD_FAST64, EPI><<<grid, 256, 0, st>>>(a);
  else if (loader == LD_DMA64)
    k_qconv<BM, BN, TM, TN, MINW, LD_DMA64, EPI><<<grid, 256, 0, st>>>(a);
  else if (loader == LD_GEN16)
    k_qconv<BM, BN, TM, TN, MINW, LD_GEN16, EPI><<<grid, 256, 0, st>>>(a);
  else if (loader == LD_HALO4 || loader == LD_HALO8)
    return;  // halo tiles have their own configurations
  else if constexpr ((EPI == EPI_ACC || EPI == EPI_PRED) && BN == 64) {
    if (loader == LD_RGB8) k_qconv<BM, BN, TM, TN, MINW, LD_RGB8, EPI><<<grid, 256, 0, st>>>(a);
    else k_qconv<BM, BN, TM, TN, MINW, LD_RGB4, EPI><<<grid, 256, 0, st>>>(a);
  }
}

// First-layer filters [k][(r S + s) 4 + c] (rows of wrow bytes) re-laid as
// [k][r][s < 8][c] (rows of wrow8 bytes, zeros past R, S).
__global__ void k_rgb8_weights(const int8_t* w, int K, int R, int S, int wrow, int8_t* out,
                               int wrow8) {
  const int64_t n = (int64_t)K * wrow8;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    const int k = (int)(i / wrow8), b = (int)(i - (int64_t)k * wrow8);
    const int r = b >> 5, s = (b >> 2) & 7, c = b & 3;
    out[i] = (r < R && s < S) ? w[(int64_t)k * wrow + (r * S + s) * 4 + c] : (int8_t)0;
  }
}

// The padded RGB layout with filter rows of at most 8 taps: re-lay the
// filters into the handle's buffer and switch to the 16-byte pixel loader.
static void rgb8_setup(const Ctx& c, const fxpq_conv_desc& d, ConvArgs& a, int& loader) {
  if (loader != LD_RGB4 || d.s > 8 || d.w < 4 || !c.sc.rgb_w) return;
  const int wrow8 = (d.r * 32 + 63) / 64 * 64;
  if ((size_t)d.k * wrow8 > kRgbWBytes) return;
  const int64_t n = (int64_t)d.k * wrow8;
  k_rgb8_weights<<<(int)((n + 255) / 256), 256, 0, c.stream>>>(a.w, d.k, d.r, d.s, a.wrow, c.sc.rgb_w,
                                                               wrow8);
  a.w = c.sc.rgb_w;
  a.wrow = wrow8;
  a.kdepth = wrow8;
  loader = LD_RGB8;
}

// Convolutions the halo tiles take: 3x3 filters (stride 1 or 2), 64-channel
// multiples in, 256-channel multiples out, contraction deep enough to be
// bound by the matrix cores.
static bool ep_halo_ok(const fxpq_conv_desc& d) {
  return d.r == 3 && d.s == 3 && (d.stride == 1 || d.stride == 2) && d.pad <= 2 && d.c % 64 == 0 &&
         d.k % 256 == 0 && d.r * d.s * d.c >= 1024;
}

// Tile shape and grid of a conv; loader choice and the geometry in `a`.
static dim3 conv_setup(const fxpq_conv_desc& d, const void* x, int x_type, const int8_t* w,
                       const int32_t* colsum, const SrcDev* ep, ConvArgs& a, int& loader,
                       int& cfg, int cus, int halo = FXPQ_TILING_GEMM, bool wide_ok = true) {
  a.x = static_cast<const int8_t*>(x);
  a.w = w;
  a.colsum = colsum;
  a.N = d.n; a.H = d.h; a.W = d.w; a.C = d.c; a.K = d.k; a.R = d.r; a.S = d.s;
  a.stride = d.stride; a.pad = d.pad;
  a.Ho = (d.h + 2 * d.pad - d.r) / d.stride + 1;
  a.Wo = (d.w + 2 * d.pad - d.s) / d.stride + 1;
  a.M = d.n * a.Ho * a.Wo;
  a.kdepth = d.r * d.s * d.c;
  loader = (d.c % 64 == 0) ? LD_FAST64 : (d.c == 4 ? LD_RGB4 : LD_GEN16);
  a.wrow = (loader == LD_RGB4) ? (a.kdepth + 63) / 64 * 64 : a.kdepth;
  if (loader == LD_RGB4) a.kdepth = a.wrow;
  a.x_type = x_type;
  a.has_ep = ep != nullptr;
  if (ep) a.ep = *ep;
  // 256 x 64 tiles for narrow outputs; 256 x 128 (128 x 64 per wave: fewer LDS
  // bytes per MFMA, two blocks per CU) for deep contractions with enough tiles
  // to fill the chip; else 128 x 128 (three blocks per CU).
  const int64_t tiles_256x128 = (int64_t)((a.M + 255) / 256) * ((d.k + 127) / 128);
  if (d.k <= 64 || loader == LD_RGB4) cfg = TC_256x64;
  else if (wide_ok && loader == LD_FAST64 && a.kdepth >= 512 && 2 * tiles_256x128 >= 3 * (int64_t)cus)
    cfg = TC_256x128;
  else cfg = TC_128x128;
  // channel multiples of 64 outside the narrow tiles: slabs through the LDS ring
  if (loader == LD_FAST64 && cfg != TC_256x64) loader = LD_DMA64;
  // 3x3 filters over small images with 256-channel multiples, on request:
  // halo tiles of whole output rows (224 rows in 7 MFMA row tiles, else 128
  // in 4) when the patch fits 512 LDS rows and, first choice, the tiles fill
  // the chip.  (Measured slower than the implicit-GEMM tiles on ResNet-50's
  // 14x14 and 7x7 layers: one block per CU cannot hide the LDS and barrier
  // latency of each slab.)
  if (halo == FXPQ_TILING_HALO && loader == LD_DMA64 && ep_halo_ok(d)) {
    for (int opt = 0; opt < 2; ++opt) {
      const int bm = opt == 0 ? 224 : 128;
      const int howo = a.Ho * a.Wo;
      int G, TH;
      if (howo <= bm) {
        G = bm / howo;
        TH = a.Ho;
      } else {
        G = 1;
        TH = bm / a.Wo;
        if (TH < 1) continue;
      }
      const int PH = (TH - 1) * d.stride + d.r, PW = (a.Wo - 1) * d.stride + d.s;
      const int npx = G * PH * PW;
      if (npx > 512) continue;
      const int tpi = (a.Ho + TH - 1) / TH;
      const int64_t tm = (G > 1) ? (d.n + G - 1) / G : (int64_t)d.n * tpi;
      const int64_t tiles = tm * (d.k / 256);
      if (opt == 0 && tiles < cus) continue;
      a.hG = G;
      a.hTH = TH;
      a.hTPI = tpi;
      a.hPH = PH;
      a.hPW = PW;
      loader = npx <= 256 ? LD_HALO4 : LD_HALO8;
      cfg = opt == 0 ? TC_H224x256 : TC_H128x256;
      return dim3((unsigned)tm, d.k / 256);
    }
  }
  switch (cfg) {
    case TC_256x64: return dim3((a.M + 255) / 256, (d.k + 63) / 64);
    case TC_256x128: return dim3((a.M + 255) / 256, (d.k + 127) / 128);
    default: return dim3((a.M + 127) / 128, (d.k + 127) / 128);
  }
}

template <int EPI>
static void conv_run(const ConvArgs& a, int loader, int cfg, dim3 grid, hipStream_t st) {
  if constexpr (EPI == EPI_ACC) {
    if (cfg == TC_H224x256) {
      if (loader == LD_HALO4) k_qconv<224, 256, 7, 2, 1, LD_HALO4, EPI><<<grid, 256, 0, st>>>(a);
      else k_qconv<224, 256, 7, 2, 1, LD_HALO8, EPI><<<grid, 256, 0, st>>>(a);
      return;
    }
    if (cfg == TC_H128x256) {
      if (loader == LD_HALO4) k_qconv<128, 256, 4, 2, 1, LD_HALO4, EPI><<<grid, 256, 0, st>>>(a);
      else k_qconv<128, 256, 4, 2, 1, LD_HALO8, EPI><<<grid, 256, 0, st>>>(a);
      return;
    }
  }
  constexpr int W3 = 3;
  if (cfg == TC_256x64)
    conv_dispatch_loader<256, 64, 2, 2, W3, EPI>(loader, grid, st, a);
  else if (cfg == TC_256x128) {
    if constexpr (EPI != EPI_PRED) conv_dispatch_loader<256, 128, 4, 2, 2, EPI>(loader, grid, st, a);
  } else
    conv_dispatch_loader<128, 128, 2, 2, W3, EPI>(loader, grid, st, a);
}

hipError_t launch_conv(const Ctx& c, const fxpq_conv_desc& d, const void* x, int x_type,
                       const int8_t* w, const int32_t* colsum, const SrcDev* ep, int32_t* acc,
                       double* d_minmax) {
  ConvArgs a{};
  int loader;
  int cfg;
  const dim3 grid = conv_setup(d, x, x_type, w, colsum, ep, a, loader, cfg, c.cus, c.conv_tiling);
  a.acc = acc;
  a.sink = c.sc.sink;
  a.want_mm = (ep != nullptr && d_minmax != nullptr);
  a.mm_part = c.sc.minmax_part;
  bool timed = timer_begin(c, FXPQ_TIMER_QCONV);
  rgb8_setup(c, d, a, loader);
  conv_run<EPI_ACC>(a, loader, cfg, grid, c.stream);
  timer_end(c, timed, 2.0 * (double)a.M * (double)d.k * (double)(d.r * d.s * d.c));
  if (a.want_mm) return launch_minmax_fin(c, a.mm_part, (int)(grid.x * grid.y), d_minmax);
  return hipGetLastError();
}

int conv_fused_blocks(const fxpq_conv_desc& d, int cus, bool rgb_ok) {
  ConvArgs a{};
  int loader;
  int cfg;
  const dim3 grid = conv_setup(d, nullptr, 0, nullptr, nullptr, nullptr, a, loader, cfg, cus);
  if (loader == LD_RGB4 && !rgb_ok) return -1;
  return (int)(grid.x * grid.y);
}

// Conv + epilogue + FxP-QLayer (FL search, requantization) with the int32
// accumulators recomputed instead of stored.  `ep` is the ACC source of the
// C-Block values, its x pointing at the fallback int32 buffer.
hipError_t launch_conv_fused(const Ctx& c, const fxpq_conv_desc& d, const void* x, int x_type,
                             const int8_t* w, const int32_t* colsum, const SrcDev& ep, int wl,
                             int sign, int fl_lo, int fl_hi, fxpq_fmt* out, int8_t* y, int y_type,
                             double* d_minmax) {
  ConvArgs a{};
  int loader;
  int cfg;
  const dim3 grid = conv_setup(d, x, x_type, w, colsum, &ep, a, loader, cfg, c.cus);
  const int nb = (int)(grid.x * grid.y);
  const double ops = 2.0 * (double)a.M * (double)d.k * (double)(d.r * d.s * d.c);
  const int64_t n = (int64_t)a.M * d.k;
  // 1. min / max of the C-Block values
  a.want_mm = 1;
  a.mm_part = c.sc.minmax_part;
  bool timed = timer_begin(c, FXPQ_TIMER_CBLOCK_PASS);
  conv_run<EPI_MM>(a, loader, cfg, grid, c.stream);
  timer_end(c, timed, ops);
  hipError_t e = launch_minmax_fin(c, a.mm_part, nb, d_minmax);
  if (e != hipSuccess) return e;
  // 2. window partial sums, then the exact decision
  a.wl = wl;
  a.sign_req = sign;
  a.fl_lo = fl_lo;
  a.fl_hi = fl_hi;
  a.mm = d_minmax;
  const int set = fls_begin(c);
  a.part_i = c.sc.win_part + (size_t)set * kWinSlots * kWinPart;
  a.part_f = c.sc.win_part_f + (size_t)set * kWinSlots * kWinPartF;
  a.plan = static_cast<FlsPlan*>(c.sc.plan);
  a.fmt_win = out;
  a.flags = c.sc.flags;
  timed = timer_begin(c, FXPQ_TIMER_CBLOCK_PASS);
  conv_run<EPI_WIN>(a, loader, cfg, grid, c.stream);
  timer_end(c, timed, ops);
  e = launch_fls_window_fin(c, ep, set, wl, sign, fl_lo, 1, fl_hi, MODE_SEARCH, conv_per_thread(cfg),
                            d_minmax, out);
  if (e != hipSuccess) return e;
  // 3. only when the plan asks for the general pass: int32 accumulators, then
  //    the exact search over every remaining candidate
  ConvArgs g = a;
  g.acc = static_cast<int32_t*>(const_cast<void*>(ep.x));
  g.want_mm = 0;
  g.only_if_general = 1;
  g.plan_in = static_cast<const FlsPlan*>(c.sc.plan);
  conv_run<EPI_ACC>(g, loader, cfg, grid, c.stream);
  e = launch_fls_general(c, ep, n, wl, fl_lo, fl_hi, d_minmax, out, nullptr);
  if (e != hipSuccess) return e;
  // 4. codes in the searched format
  a.fmt_req = out;
  a.y = y;
  a.y_type = y_type;
  timed = timer_begin(c, FXPQ_TIMER_CBLOCK_PASS);
  conv_run<EPI_REQ>(a, loader, cfg, grid, c.stream);
  timer_end(c, timed, ops);
  return hipGetLastError();
}

// Predicted C-Block (conv + epilogue + FxP-QLayer in one contraction): the
// epilogue evaluates the window of the min / max in d_minmax (the previous
// call's) and writes the codes of the candidate the format in `out` picks;
// the decision checks the prediction and sets *miss when it fails.
hipError_t launch_conv_pred(const Ctx& c, const fxpq_conv_desc& d, const void* x, int x_type,
                            const int8_t* w, const int32_t* colsum, const SrcDev& ep, int wl,
                            int sign, int fl_lo, int fl_hi, fxpq_fmt* out, int8_t* y,
                            double* d_minmax, unsigned* miss) {
  ConvArgs a{};
  int loader;
  int cfg;
  // no 256 x 128 tiles: their 128 accumulators per thread and the window
  // state of this epilogue do not fit the registers of two blocks per CU
  const dim3 grid = conv_setup(d, x, x_type, w, colsum, &ep, a, loader, cfg, c.cus,
                               FXPQ_TILING_GEMM, false);
  a.want_mm = 1;
  a.wl = wl;
  a.sign_req = sign;
  a.fl_lo = fl_lo;
  a.fl_hi = fl_hi;
  a.mm = d_minmax;
  // deferred mode: the call's own slot set and record, no decision launch
  const int job = c.pred_jobs_n ? (*c.pred_jobs_n)++ : -1;
  const int set = job < 0 ? fls_begin(c) : 0;
  if (job < 0) {
    a.part_i = c.sc.win_part + (size_t)set * kWinSlots * kWinPart;
    a.part_f = c.sc.win_part_f + (size_t)set * kWinSlots * kWinPartF;
  } else {
    a.part_i = c.sc.pred_slots_i + (size_t)job * kWinSlots * kWinPart;
    a.part_f = c.sc.pred_slots_f + (size_t)job * kWinSlots * kWinPartF;
    a.job = c.sc.pred_jobs + job;
    a.job_miss = miss;
    a.job_per_thread = conv_per_thread(cfg);
  }
  a.fmt_win = out;
  a.y = y;
  a.y_type = FXPQ_C8;
  a.flags = c.sc.flags;
  bool timed = timer_begin(c, FXPQ_TIMER_CBLOCK_PRED);
  rgb8_setup(c, d, a, loader);
  conv_run<EPI_PRED>(a, loader, cfg, grid, c.stream);
  timer_end(c, timed, 2.0 * (double)a.M * (double)d.k * (double)(d.r * d.s * d.c));
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || job >= 0) return e;
  return launch_pred_fin(c, ep, set, wl, sign, fl_lo, fl_hi, conv_per_thread(cfg), d_minmax, out,
                         miss);
}

}  // namespace fxpq
