/*
 * fcm_oracle.c -- TEST INFRASTRUCTURE ONLY.
 *
 * A plain, slow, obviously correct CPU reference for the fused depthwise (DW) /
 * pointwise (PW) convolution modules of Qararyah et al., "Fusing Depthwise and
 * Pointwise Convolutions for Efficient Inference on GPUs" (arXiv 2404.19331).
 *
 * Fusion only moves data; it does not change what is computed (Sec. III-A: an FCM
 * evaluates the same convolution-normalisation-activation layers, keeping the
 * intermediate on chip). So this oracle is the plain definition of each layer
 * (Sec. II-B): a depthwise KxK convolution applies one filter per channel over the
 * spatial dimensions, a pointwise convolution is a 1x1 filter spanning all channels.
 * Modules are plain compositions of those stages:
 *   DW->PW      depthwise separable convolution        (Sec. II-B, Sec. III-A "DWPW")
 *   PW->DW      first two layers of an inverted residual (Sec. III-A "PWDW")
 *   PW->DW->PW  the inverted residual block              (Sec. II-B)
 *
 * Every stage is "convolution -> + bias (folded normalisation) -> activation ->
 * cast to the storage precision" (Sec. III-A: an FCM combines each convolution with
 * the normalisation and activation following it). Accumulation is exact: double for
 * the float paths, int64 for int8 (whose intermediate is requantised to int8 before
 * the next stage, Sec. III-B: INT8 results are packed before being written to any
 * buffer). int8 tensors may be asymmetric: a code q stands for scale * (q - zero point),
 * and every stage convolves codes minus their zero point, so padding is real 0.
 *
 * Who may use this file: the test-suite, the smoke check and the CPU-baseline leg of
 * the benchmark. The product path (the HIP library) never loads or calls it, and this
 * file shares no code, header or table with it.
 *
 * Canonical internal layout is NCHW; NHWC inputs/outputs are converted at the edges.
 */
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <math.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { ORC_F32 = 0, ORC_BF16 = 1, ORC_I8 = 2, ORC_F64 = 3 };
enum { ORC_NCHW = 0, ORC_NHWC = 1 };
enum { ORC_ACT_NONE = 0, ORC_ACT_RELU = 1, ORC_ACT_RELU6 = 2 };
enum { ORC_OK = 0, ORC_EINVAL = 1, ORC_EUNSUPPORTED = 2, ORC_EOVERFLOW = 3 };

/* int8 requantisation of a stage's output. zero_point is the code of real 0 in that
 * output (asymmetric quantisation: a code q stands for scale * (q - zero_point)). */
typedef struct {
  int32_t mult, shift, qmin, qmax, zero_point;
} orc_rq;

typedef struct {
  int32_t n, h, w;
  int32_t c_in, c_mid, c_out;
  int32_t k, stride, pad;
  int32_t dtype, layout;
  int32_t act[3];
  orc_rq rq[3];
  /* int8 per-channel requantisation of stage i (NULL = per-tensor rq[i]): host array of
   * 2 x (the stage's output channels), the multipliers then the shifts; qmin/qmax stay
   * those of rq[i] */
  const int32_t* rqc[3];
  /* int8 zero point of the input x; stage i > 0 takes its input's from rq[i-1] */
  int32_t zp_in;
} orc_desc;

/* ------------------------------------------------------------------------- */
/* Scalar helpers                                                             */
/* ------------------------------------------------------------------------- */

/* bfloat16 = the upper 16 bits of an IEEE binary32; conversion rounds to nearest,
 * ties to even, on the 16 discarded bits. NaN stays NaN (quiet). */
uint16_t orc_bf16_from_f32(float f) {
  uint32_t u;
  memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u && (u & 0x007fffffu) != 0)
    return (uint16_t)((u >> 16) | 0x0040u);
  uint32_t lsb = (u >> 16) & 1u;
  uint32_t rounded = u + 0x7fffu + lsb;
  return (uint16_t)(rounded >> 16);
}

float orc_f32_from_bf16(uint16_t b) {
  uint32_t u = ((uint32_t)b) << 16;
  float f;
  memcpy(&f, &u, 4);
  return f;
}

/* Requantisation of an integer accumulator by the per-tensor scale mult * 2^-shift:
 * q = round_half_to_even(acc * mult / 2^shift), then saturated to [qmin, qmax].
 * Written on integers only, so it is exact. */
int64_t orc_requant(int64_t acc, int32_t mult, int32_t shift, int32_t qmin, int32_t qmax) {
  int64_t t = acc * (int64_t)mult;
  int64_t q;
  if (shift <= 0) {
    q = t;
  } else {
    q = t >> shift;                      /* floor division (arithmetic shift) */
    int64_t r = t - (q << shift);         /* remainder in [0, 2^shift) */
    int64_t half = (int64_t)1 << (shift - 1);
    if (r > half || (r == half && (q & 1))) q += 1;
  }
  if (q < qmin) q = qmin;
  if (q > qmax) q = qmax;
  return q;
}

static double act_f(double v, int act) {
  if (act == ORC_ACT_RELU) return v > 0.0 ? v : 0.0;
  if (act == ORC_ACT_RELU6) return v < 0.0 ? 0.0 : (v > 6.0 ? 6.0 : v);
  return v;
}

/* Cast an exactly accumulated value to the storage precision of the dtype. */
static double cast_f(double v, int dtype) {
  if (dtype == ORC_F32) return (double)(float)v;
  if (dtype == ORC_BF16) return (double)orc_f32_from_bf16(orc_bf16_from_f32((float)v));
  return v; /* ORC_F64: no rounding at all */
}

/* ------------------------------------------------------------------------- */
/* Conversions between storage formats and the canonical NCHW work arrays      */
/* ------------------------------------------------------------------------- */

static double load_elem_f(const void* p, int dtype, size_t i) {
  if (dtype == ORC_F32) return (double)((const float*)p)[i];
  if (dtype == ORC_BF16) return (double)orc_f32_from_bf16(((const uint16_t*)p)[i]);
  return ((const double*)p)[i];
}

static void store_elem_f(void* p, int dtype, size_t i, double v) {
  if (dtype == ORC_F32) ((float*)p)[i] = (float)v;
  else if (dtype == ORC_BF16) ((uint16_t*)p)[i] = orc_bf16_from_f32((float)v);
  else ((double*)p)[i] = v;
}

/* index of (n,c,h,w) in a tensor of the given layout */
static size_t idx(int layout, int N, int C, int H, int W, int n, int c, int h, int w) {
  (void)N;
  if (layout == ORC_NHWC) return (((size_t)n * H + h) * W + w) * C + c;
  return (((size_t)n * C + c) * H + h) * W + w;
}

static double* load_fmap_f(const void* src, int dtype, int layout, int N, int C, int H, int W) {
  size_t cnt = (size_t)N * C * H * W;
  double* d = (double*)malloc(cnt * sizeof(double));
  for (int n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c)
      for (int h = 0; h < H; ++h)
        for (int w = 0; w < W; ++w)
          d[idx(ORC_NCHW, N, C, H, W, n, c, h, w)] =
              load_elem_f(src, dtype, idx(layout, N, C, H, W, n, c, h, w));
  return d;
}

static int64_t* load_fmap_i(const int8_t* src, int layout, int N, int C, int H, int W) {
  size_t cnt = (size_t)N * C * H * W;
  int64_t* d = (int64_t*)malloc(cnt * sizeof(int64_t));
  for (int n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c)
      for (int h = 0; h < H; ++h)
        for (int w = 0; w < W; ++w)
          d[idx(ORC_NCHW, N, C, H, W, n, c, h, w)] = src[idx(layout, N, C, H, W, n, c, h, w)];
  return d;
}

static void store_fmap_f(const double* d, int dtype, int layout, int N, int C, int H, int W, void* dst) {
  for (int n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c)
      for (int h = 0; h < H; ++h)
        for (int w = 0; w < W; ++w)
          store_elem_f(dst, dtype, idx(layout, N, C, H, W, n, c, h, w),
                       d[idx(ORC_NCHW, N, C, H, W, n, c, h, w)]);
}

static void store_fmap_i(const int64_t* d, int layout, int N, int C, int H, int W, int8_t* dst) {
  for (int n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c)
      for (int h = 0; h < H; ++h)
        for (int w = 0; w < W; ++w)
          dst[idx(layout, N, C, H, W, n, c, h, w)] = (int8_t)d[idx(ORC_NCHW, N, C, H, W, n, c, h, w)];
}

static double* load_vec_f(const void* src, int dtype, size_t cnt) {
  double* d = (double*)malloc((cnt ? cnt : 1) * sizeof(double));
  for (size_t i = 0; i < cnt; ++i) d[i] = load_elem_f(src, dtype, i);
  return d;
}

static int64_t* load_vec_i(const int8_t* src, size_t cnt) {
  int64_t* d = (int64_t*)malloc((cnt ? cnt : 1) * sizeof(int64_t));
  for (size_t i = 0; i < cnt; ++i) d[i] = src[i];
  return d;
}

/* Bias of a float path: float for F32/BF16, double for F64. NULL means zero. */
static double bias_f(const void* b, int dtype, int i) {
  if (!b) return 0.0;
  if (dtype == ORC_F64) return ((const double*)b)[i];
  return (double)((const float*)b)[i];
}

static int64_t bias_i(const int32_t* b, int i) { return b ? (int64_t)b[i] : 0; }

/* ------------------------------------------------------------------------- */
/* The two convolution stages, exact accumulation, canonical NCHW             */
/* ------------------------------------------------------------------------- */

/* Depthwise KxK, channel multiplier 1, symmetric zero padding P, stride S:
 *   y[n,c,i,j] = sum_{u,v<K} wd[c,u,v] * xpad[n,c,i*S-P+u, j*S-P+v] + bd[c]
 * where xpad is x extended by zeros outside [0,H)x[0,W). */
static void dw_stage_f(const double* x, int N, int C, int H, int W, const double* wd, const void* bd,
                       int bdtype, int K, int S, int P, int Ho, int Wo, double* y) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c)
      for (int i = 0; i < Ho; ++i)
        for (int j = 0; j < Wo; ++j) {
          double s = 0.0;
          for (int u = 0; u < K; ++u)
            for (int v = 0; v < K; ++v) {
              int r = i * S - P + u, q = j * S - P + v;
              if (r < 0 || r >= H || q < 0 || q >= W) continue;
              s += wd[((size_t)c * K + u) * K + v] * x[(((size_t)n * C + c) * H + r) * W + q];
            }
          y[(((size_t)n * C + c) * Ho + i) * Wo + j] = s + bias_f(bd, bdtype, c);
        }
}

static void dw_stage_i(const int64_t* x, int N, int C, int H, int W, const int64_t* wd, const int32_t* bd,
                       int K, int S, int P, int Ho, int Wo, int64_t* y) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int n = 0; n < N; ++n)
    for (int c = 0; c < C; ++c)
      for (int i = 0; i < Ho; ++i)
        for (int j = 0; j < Wo; ++j) {
          int64_t s = 0;
          for (int u = 0; u < K; ++u)
            for (int v = 0; v < K; ++v) {
              int r = i * S - P + u, q = j * S - P + v;
              if (r < 0 || r >= H || q < 0 || q >= W) continue;
              s += wd[((size_t)c * K + u) * K + v] * x[(((size_t)n * C + c) * H + r) * W + q];
            }
          y[(((size_t)n * C + c) * Ho + i) * Wo + j] = s + bias_i(bd, c);
        }
}

/* Pointwise 1x1: y[n,o,i,j] = sum_{c<C} wp[o,c] * x[n,c,i,j] + bp[o] */
static void pw_stage_f(const double* x, int N, int C, int H, int W, const double* wp, const void* bp,
                       int bdtype, int Co, double* y) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int n = 0; n < N; ++n)
    for (int o = 0; o < Co; ++o)
      for (int i = 0; i < H; ++i)
        for (int j = 0; j < W; ++j) {
          double s = 0.0;
          for (int c = 0; c < C; ++c)
            s += wp[(size_t)o * C + c] * x[(((size_t)n * C + c) * H + i) * W + j];
          y[(((size_t)n * Co + o) * H + i) * W + j] = s + bias_f(bp, bdtype, o);
        }
}

static void pw_stage_i(const int64_t* x, int N, int C, int H, int W, const int64_t* wp, const int32_t* bp,
                       int Co, int64_t* y) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int n = 0; n < N; ++n)
    for (int o = 0; o < Co; ++o)
      for (int i = 0; i < H; ++i)
        for (int j = 0; j < W; ++j) {
          int64_t s = 0;
          for (int c = 0; c < C; ++c)
            s += wp[(size_t)o * C + c] * x[(((size_t)n * C + c) * H + i) * W + j];
          y[(((size_t)n * Co + o) * H + i) * W + j] = s + bias_i(bp, o);
        }
}

/* Normalisation is folded into weights/bias, so the per-stage tail is activation then
 * cast. The float path applies the activation to the exact value and rounds once. */
static void finish_f(double* v, size_t cnt, int act, int dtype) {
  for (size_t i = 0; i < cnt; ++i) v[i] = cast_f(act_f(v[i], act), dtype);
}

/* int8 tail: requantise (RNE), add the output zero point, saturate to [qmin, qmax], then
 * ReLU, which in the quantised domain clamps below at the zero point (the code of real 0).
 * With a zero point of 0 both maps are monotone and fix zero, so the order of ReLU and
 * requantisation does not change the result. ReLU6 is the quantised clamp: below at the
 * zero point, above at qmax, which carries 6.0 in the output's quantised units (the upper
 * clamp is the requantisation's own saturation).
 * Returns ORC_EOVERFLOW when an accumulator does not fit the 32-bit accumulator
 * the method prescribes (Sec. III-B: four-way dot product with 32-bit accumulate). */
static int finish_i(int64_t* v, size_t cnt, int C, size_t HW, int act, orc_rq rq, const int32_t* rqc) {
  for (size_t i = 0; i < cnt; ++i) {
    if (v[i] > INT32_MAX || v[i] < INT32_MIN) return ORC_EOVERFLOW;
    int32_t mult = rq.mult, shift = rq.shift;
    if (rqc) {  /* canonical [n][c][h][w]: channel of element i */
      const int c = (int)((i / HW) % (size_t)C);
      mult = rqc[c];
      shift = rqc[C + c];
      if (shift < 0 || shift > 62) return ORC_EINVAL;
    }
    /* rounding only (int32-wide clamp: the int8 clamp below makes it immaterial) */
    int64_t q = orc_requant(v[i], mult, shift, INT32_MIN, INT32_MAX) + rq.zero_point;
    if (q < rq.qmin) q = rq.qmin;
    if (q > rq.qmax) q = rq.qmax;
    if (act != ORC_ACT_NONE && q < rq.zero_point) q = rq.zero_point;
    v[i] = q;
  }
  return ORC_OK;
}

/* The value a stage convolves is the real one up to the scale: code minus zero point.
 * So a zero-padded position (real 0) contributes nothing, whatever the zero point. */
static void center_i(int64_t* v, size_t cnt, int32_t zero_point) {
  for (size_t i = 0; i < cnt; ++i) v[i] -= zero_point;
}

/* ------------------------------------------------------------------------- */
/* Validation                                                                 */
/* ------------------------------------------------------------------------- */

static int out_dim(int in, int K, int S, int P) { return (in + 2 * P - K) / S + 1; }

static int check_common(const orc_desc* d) {
  if (!d) return ORC_EINVAL;
  if (d->n <= 0 || d->h <= 0 || d->w <= 0) return ORC_EINVAL;
  if (d->dtype < ORC_F32 || d->dtype > ORC_F64) return ORC_EINVAL;
  if (d->layout != ORC_NCHW && d->layout != ORC_NHWC) return ORC_EINVAL;
  for (int i = 0; i < 3; ++i) {
    if (d->act[i] < ORC_ACT_NONE || d->act[i] > ORC_ACT_RELU6) return ORC_EINVAL;
    if (d->dtype == ORC_I8) {
      if (d->rq[i].shift < 0 || d->rq[i].shift > 62) return ORC_EINVAL;
      if (d->rq[i].qmin > d->rq[i].qmax || d->rq[i].qmin < -128 || d->rq[i].qmax > 127) return ORC_EINVAL;
      if (d->rq[i].zero_point < -128 || d->rq[i].zero_point > 127) return ORC_EINVAL;
    }
  }
  if (d->dtype == ORC_I8 && (d->zp_in < -128 || d->zp_in > 127)) return ORC_EINVAL;
  return ORC_OK;
}

static int check_dw_geom(const orc_desc* d, int H, int W) {
  if (d->k <= 0 || d->stride <= 0 || d->pad < 0) return ORC_EINVAL;
  if (H + 2 * d->pad < d->k || W + 2 * d->pad < d->k) return ORC_EINVAL;
  return ORC_OK;
}

/* ------------------------------------------------------------------------- */
/* Public entry points                                                        */
/* ------------------------------------------------------------------------- */

int orc_num_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}

/* Threads of the following calls' parallel loops (for timing: 1 = single-threaded). */
void orc_set_num_threads(int n) {
#ifdef _OPENMP
  if (n > 0) omp_set_num_threads(n);
#else
  (void)n;
#endif
}

/* Single depthwise layer: channels c_in, stage 0 activation/requant. */
int orc_dw(const orc_desc* d, const void* x, const void* wd, const void* bd, void* y) {
  int st = check_common(d);
  if (st) return st;
  if (d->c_in <= 0 || !x || !wd || !y) return ORC_EINVAL;
  if ((st = check_dw_geom(d, d->h, d->w))) return st;
  int N = d->n, C = d->c_in, H = d->h, W = d->w, K = d->k, S = d->stride, P = d->pad;
  int Ho = out_dim(H, K, S, P), Wo = out_dim(W, K, S, P);
  size_t no = (size_t)N * C * Ho * Wo;
  if (d->dtype == ORC_I8) {
    int64_t* xi = load_fmap_i((const int8_t*)x, d->layout, N, C, H, W);
    center_i(xi, (size_t)N * C * H * W, d->zp_in);
    int64_t* wi = load_vec_i((const int8_t*)wd, (size_t)C * K * K);
    int64_t* yi = (int64_t*)malloc(no * sizeof(int64_t));
    dw_stage_i(xi, N, C, H, W, wi, (const int32_t*)bd, K, S, P, Ho, Wo, yi);
    st = finish_i(yi, no, C, (size_t)Ho * Wo, d->act[0], d->rq[0], d->rqc[0]);
    if (!st) store_fmap_i(yi, d->layout, N, C, Ho, Wo, (int8_t*)y);
    free(xi); free(wi); free(yi);
    return st;
  }
  double* xf = load_fmap_f(x, d->dtype, d->layout, N, C, H, W);
  double* wf = load_vec_f(wd, d->dtype, (size_t)C * K * K);
  double* yf = (double*)malloc(no * sizeof(double));
  dw_stage_f(xf, N, C, H, W, wf, bd, d->dtype, K, S, P, Ho, Wo, yf);
  finish_f(yf, no, d->act[0], d->dtype);
  store_fmap_f(yf, d->dtype, d->layout, N, C, Ho, Wo, y);
  free(xf); free(wf); free(yf);
  return ORC_OK;
}

/* Single pointwise layer: c_in -> c_out on the h x w grid, stage 0 activation. */
int orc_pw(const orc_desc* d, const void* x, const void* wp, const void* bp, void* y) {
  int st = check_common(d);
  if (st) return st;
  if (d->c_in <= 0 || d->c_out <= 0 || !x || !wp || !y) return ORC_EINVAL;
  int N = d->n, C = d->c_in, Co = d->c_out, H = d->h, W = d->w;
  size_t no = (size_t)N * Co * H * W;
  if (d->dtype == ORC_I8) {
    int64_t* xi = load_fmap_i((const int8_t*)x, d->layout, N, C, H, W);
    center_i(xi, (size_t)N * C * H * W, d->zp_in);
    int64_t* wi = load_vec_i((const int8_t*)wp, (size_t)Co * C);
    int64_t* yi = (int64_t*)malloc(no * sizeof(int64_t));
    pw_stage_i(xi, N, C, H, W, wi, (const int32_t*)bp, Co, yi);
    st = finish_i(yi, no, Co, (size_t)H * W, d->act[0], d->rq[0], d->rqc[0]);
    if (!st) store_fmap_i(yi, d->layout, N, Co, H, W, (int8_t*)y);
    free(xi); free(wi); free(yi);
    return st;
  }
  double* xf = load_fmap_f(x, d->dtype, d->layout, N, C, H, W);
  double* wf = load_vec_f(wp, d->dtype, (size_t)Co * C);
  double* yf = (double*)malloc(no * sizeof(double));
  pw_stage_f(xf, N, C, H, W, wf, bp, d->dtype, Co, yf);
  finish_f(yf, no, d->act[0], d->dtype);
  store_fmap_f(yf, d->dtype, d->layout, N, Co, H, W, y);
  free(xf); free(wf); free(yf);
  return ORC_OK;
}

/* DW -> PW (depthwise separable convolution). c_mid must equal c_in. */
int orc_dw_pw(const orc_desc* d, const void* x, const void* wd, const void* bd, const void* wp,
              const void* bp, void* y) {
  int st = check_common(d);
  if (st) return st;
  if (d->c_in <= 0 || d->c_out <= 0 || d->c_mid != d->c_in || !x || !wd || !wp || !y) return ORC_EINVAL;
  if ((st = check_dw_geom(d, d->h, d->w))) return st;
  int N = d->n, C = d->c_in, Co = d->c_out, H = d->h, W = d->w, K = d->k, S = d->stride, P = d->pad;
  int Ho = out_dim(H, K, S, P), Wo = out_dim(W, K, S, P);
  size_t nm = (size_t)N * C * Ho * Wo, no = (size_t)N * Co * Ho * Wo;
  if (d->dtype == ORC_I8) {
    int64_t* xi = load_fmap_i((const int8_t*)x, d->layout, N, C, H, W);
    center_i(xi, (size_t)N * C * H * W, d->zp_in);
    int64_t* wdi = load_vec_i((const int8_t*)wd, (size_t)C * K * K);
    int64_t* wpi = load_vec_i((const int8_t*)wp, (size_t)Co * C);
    int64_t* mi = (int64_t*)malloc(nm * sizeof(int64_t));
    int64_t* yi = (int64_t*)malloc(no * sizeof(int64_t));
    dw_stage_i(xi, N, C, H, W, wdi, (const int32_t*)bd, K, S, P, Ho, Wo, mi);
    st = finish_i(mi, nm, C, (size_t)Ho * Wo, d->act[0], d->rq[0], d->rqc[0]);
    if (!st) center_i(mi, nm, d->rq[0].zero_point);
    if (!st) {
      pw_stage_i(mi, N, C, Ho, Wo, wpi, (const int32_t*)bp, Co, yi);
      st = finish_i(yi, no, Co, (size_t)Ho * Wo, d->act[1], d->rq[1], d->rqc[1]);
    }
    if (!st) store_fmap_i(yi, d->layout, N, Co, Ho, Wo, (int8_t*)y);
    free(xi); free(wdi); free(wpi); free(mi); free(yi);
    return st;
  }
  double* xf = load_fmap_f(x, d->dtype, d->layout, N, C, H, W);
  double* wdf = load_vec_f(wd, d->dtype, (size_t)C * K * K);
  double* wpf = load_vec_f(wp, d->dtype, (size_t)Co * C);
  double* mf = (double*)malloc(nm * sizeof(double));
  double* yf = (double*)malloc(no * sizeof(double));
  dw_stage_f(xf, N, C, H, W, wdf, bd, d->dtype, K, S, P, Ho, Wo, mf);
  finish_f(mf, nm, d->act[0], d->dtype);
  pw_stage_f(mf, N, C, Ho, Wo, wpf, bp, d->dtype, Co, yf);
  finish_f(yf, no, d->act[1], d->dtype);
  store_fmap_f(yf, d->dtype, d->layout, N, Co, Ho, Wo, y);
  free(xf); free(wdf); free(wpf); free(mf); free(yf);
  return ORC_OK;
}

/* PW -> DW. The PW output (c_mid channels, h x w) is the DW input, zero padded by the
 * DW like any other input: positions outside the image are real 0, never act(bias)
 * (for int8, the code of real 0 is the intermediate's zero point).
 * c_out must equal c_mid. */
int orc_pw_dw(const orc_desc* d, const void* x, const void* wp, const void* bp, const void* wd,
              const void* bd, void* y) {
  int st = check_common(d);
  if (st) return st;
  if (d->c_in <= 0 || d->c_mid <= 0 || d->c_out != d->c_mid || !x || !wd || !wp || !y) return ORC_EINVAL;
  if ((st = check_dw_geom(d, d->h, d->w))) return st;
  int N = d->n, Ci = d->c_in, Cm = d->c_mid, H = d->h, W = d->w, K = d->k, S = d->stride, P = d->pad;
  int Ho = out_dim(H, K, S, P), Wo = out_dim(W, K, S, P);
  size_t nm = (size_t)N * Cm * H * W, no = (size_t)N * Cm * Ho * Wo;
  if (d->dtype == ORC_I8) {
    int64_t* xi = load_fmap_i((const int8_t*)x, d->layout, N, Ci, H, W);
    center_i(xi, (size_t)N * Ci * H * W, d->zp_in);
    int64_t* wpi = load_vec_i((const int8_t*)wp, (size_t)Cm * Ci);
    int64_t* wdi = load_vec_i((const int8_t*)wd, (size_t)Cm * K * K);
    int64_t* mi = (int64_t*)malloc(nm * sizeof(int64_t));
    int64_t* yi = (int64_t*)malloc(no * sizeof(int64_t));
    pw_stage_i(xi, N, Ci, H, W, wpi, (const int32_t*)bp, Cm, mi);
    st = finish_i(mi, nm, Cm, (size_t)H * W, d->act[0], d->rq[0], d->rqc[0]);
    if (!st) center_i(mi, nm, d->rq[0].zero_point);
    if (!st) {
      dw_stage_i(mi, N, Cm, H, W, wdi, (const int32_t*)bd, K, S, P, Ho, Wo, yi);
      st = finish_i(yi, no, Cm, (size_t)Ho * Wo, d->act[1], d->rq[1], d->rqc[1]);
    }
    if (!st) store_fmap_i(yi, d->layout, N, Cm, Ho, Wo, (int8_t*)y);
    free(xi); free(wpi); free(wdi); free(mi); free(yi);
    return st;
  }
  double* xf = load_fmap_f(x, d->dtype, d->layout, N, Ci, H, W);
  double* wpf = load_vec_f(wp, d->dtype, (size_t)Cm * Ci);
  double* wdf = load_vec_f(wd, d->dtype, (size_t)Cm * K * K);
  double* mf = (double*)malloc(nm * sizeof(double));
  double* yf = (double*)malloc(no * sizeof(double));
  pw_stage_f(xf, N, Ci, H, W, wpf, bp, d->dtype, Cm, mf);
  finish_f(mf, nm, d->act[0], d->dtype);
  dw_stage_f(mf, N, Cm, H, W, wdf, bd, d->dtype, K, S, P, Ho, Wo, yf);
  finish_f(yf, no, d->act[1], d->dtype);
  store_fmap_f(yf, d->dtype, d->layout, N, Cm, Ho, Wo, y);
  free(xf); free(wpf); free(wdf); free(mf); free(yf);
  return ORC_OK;
}

/* PW -> PW: two pointwise convolutions, c_in -> c_mid -> c_out, spatial size unchanged
 * (the paper's PwPw module; k, stride and pad are ignored). */
int orc_pw_pw(const orc_desc* d, const void* x, const void* wp1, const void* bp1, const void* wp2,
              const void* bp2, void* y) {
  int st = check_common(d);
  if (st) return st;
  if (d->c_in <= 0 || d->c_mid <= 0 || d->c_out <= 0 || !x || !wp1 || !wp2 || !y) return ORC_EINVAL;
  int N = d->n, Ci = d->c_in, Cm = d->c_mid, Co = d->c_out, H = d->h, W = d->w;
  size_t nm = (size_t)N * Cm * H * W, no = (size_t)N * Co * H * W;
  if (d->dtype == ORC_I8) {
    int64_t* xi = load_fmap_i((const int8_t*)x, d->layout, N, Ci, H, W);
    center_i(xi, (size_t)N * Ci * H * W, d->zp_in);
    int64_t* w1 = load_vec_i((const int8_t*)wp1, (size_t)Cm * Ci);
    int64_t* w2 = load_vec_i((const int8_t*)wp2, (size_t)Co * Cm);
    int64_t* mi = (int64_t*)malloc(nm * sizeof(int64_t));
    int64_t* yi = (int64_t*)malloc(no * sizeof(int64_t));
    pw_stage_i(xi, N, Ci, H, W, w1, (const int32_t*)bp1, Cm, mi);
    st = finish_i(mi, nm, Cm, (size_t)H * W, d->act[0], d->rq[0], d->rqc[0]);
    if (!st) center_i(mi, nm, d->rq[0].zero_point);
    if (!st) {
      pw_stage_i(mi, N, Cm, H, W, w2, (const int32_t*)bp2, Co, yi);
      st = finish_i(yi, no, Co, (size_t)H * W, d->act[1], d->rq[1], d->rqc[1]);
    }
    if (!st) store_fmap_i(yi, d->layout, N, Co, H, W, (int8_t*)y);
    free(xi); free(w1); free(w2); free(mi); free(yi);
    return st;
  }
  double* xf = load_fmap_f(x, d->dtype, d->layout, N, Ci, H, W);
  double* w1 = load_vec_f(wp1, d->dtype, (size_t)Cm * Ci);
  double* w2 = load_vec_f(wp2, d->dtype, (size_t)Co * Cm);
  double* mf = (double*)malloc(nm * sizeof(double));
  double* yf = (double*)malloc(no * sizeof(double));
  pw_stage_f(xf, N, Ci, H, W, w1, bp1, d->dtype, Cm, mf);
  finish_f(mf, nm, d->act[0], d->dtype);
  pw_stage_f(mf, N, Cm, H, W, w2, bp2, d->dtype, Co, yf);
  finish_f(yf, no, d->act[1], d->dtype);
  store_fmap_f(yf, d->dtype, d->layout, N, Co, H, W, y);
  free(xf); free(w1); free(w2); free(mf); free(yf);
  return ORC_OK;
}

/* PW -> DW -> PW (inverted residual without the skip connection). */
int orc_pw_dw_pw(const orc_desc* d, const void* x, const void* wp1, const void* bp1, const void* wd,
                 const void* bd, const void* wp2, const void* bp2, void* y) {
  int st = check_common(d);
  if (st) return st;
  if (d->c_in <= 0 || d->c_mid <= 0 || d->c_out <= 0 || !x || !wp1 || !wd || !wp2 || !y) return ORC_EINVAL;
  if ((st = check_dw_geom(d, d->h, d->w))) return st;
  int N = d->n, Ci = d->c_in, Cm = d->c_mid, Co = d->c_out, H = d->h, W = d->w;
  int K = d->k, S = d->stride, P = d->pad;
  int Ho = out_dim(H, K, S, P), Wo = out_dim(W, K, S, P);
  size_t n1 = (size_t)N * Cm * H * W, n2 = (size_t)N * Cm * Ho * Wo, no = (size_t)N * Co * Ho * Wo;
  if (d->dtype == ORC_I8) {
    int64_t* xi = load_fmap_i((const int8_t*)x, d->layout, N, Ci, H, W);
    center_i(xi, (size_t)N * Ci * H * W, d->zp_in);
    int64_t* w1 = load_vec_i((const int8_t*)wp1, (size_t)Cm * Ci);
    int64_t* wdi = load_vec_i((const int8_t*)wd, (size_t)Cm * K * K);
    int64_t* w2 = load_vec_i((const int8_t*)wp2, (size_t)Co * Cm);
    int64_t* m1 = (int64_t*)malloc(n1 * sizeof(int64_t));
    int64_t* m2 = (int64_t*)malloc(n2 * sizeof(int64_t));
    int64_t* yi = (int64_t*)malloc(no * sizeof(int64_t));
    pw_stage_i(xi, N, Ci, H, W, w1, (const int32_t*)bp1, Cm, m1);
    st = finish_i(m1, n1, Cm, (size_t)H * W, d->act[0], d->rq[0], d->rqc[0]);
    if (!st) center_i(m1, n1, d->rq[0].zero_point);
    if (!st) {
      dw_stage_i(m1, N, Cm, H, W, wdi, (const int32_t*)bd, K, S, P, Ho, Wo, m2);
      st = finish_i(m2, n2, Cm, (size_t)Ho * Wo, d->act[1], d->rq[1], d->rqc[1]);
    if (!st) center_i(m2, n2, d->rq[1].zero_point);
    }
    if (!st) {
      pw_stage_i(m2, N, Cm, Ho, Wo, w2, (const int32_t*)bp2, Co, yi);
      st = finish_i(yi, no, Co, (size_t)Ho * Wo, d->act[2], d->rq[2], d->rqc[2]);
    }
    if (!st) store_fmap_i(yi, d->layout, N, Co, Ho, Wo, (int8_t*)y);
    free(xi); free(w1); free(wdi); free(w2); free(m1); free(m2); free(yi);
    return st;
  }
  double* xf = load_fmap_f(x, d->dtype, d->layout, N, Ci, H, W);
  double* w1 = load_vec_f(wp1, d->dtype, (size_t)Cm * Ci);
  double* wdf = load_vec_f(wd, d->dtype, (size_t)Cm * K * K);
  double* w2 = load_vec_f(wp2, d->dtype, (size_t)Co * Cm);
  double* m1 = (double*)malloc(n1 * sizeof(double));
  double* m2 = (double*)malloc(n2 * sizeof(double));
  double* yf = (double*)malloc(no * sizeof(double));
  pw_stage_f(xf, N, Ci, H, W, w1, bp1, d->dtype, Cm, m1);
  finish_f(m1, n1, d->act[0], d->dtype);
  dw_stage_f(m1, N, Cm, H, W, wdf, bd, d->dtype, K, S, P, Ho, Wo, m2);
  finish_f(m2, n2, d->act[1], d->dtype);
  pw_stage_f(m2, N, Cm, Ho, Wo, w2, bp2, d->dtype, Co, yf);
  finish_f(yf, no, d->act[2], d->dtype);
  store_fmap_f(yf, d->dtype, d->layout, N, Co, Ho, Wo, y);
  free(xf); free(w1); free(wdf); free(w2); free(m1); free(m2); free(yf);
  return ORC_OK;
}
