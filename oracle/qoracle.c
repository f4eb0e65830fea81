/*
 * qoracle.c -- plain, slow CPU oracle for the MINW-Net inference path.
 *
 * TEST INFRASTRUCTURE ONLY.  The test suite, the smoke check and the CPU
 * baseline leg of the benchmark are the only callers.  The GPU library never
 * links, loads or calls anything here, and this file includes nothing from the
 * GPU library: the two implementations share no code.
 *
 * Source: Chen, Liu, Zhang, Hou, Yang, "Propagating Asymptotic-Estimated
 * Gradients for Low Bitwidth Quantized Neural Networks".
 *
 *   - inference quantizers h(.) (Sec. III-C, Eq. 20): sign (Eq. 4, with the
 *     tie rule of Sec. II-A: +1 only for a positive input), ternary (Eq. 21),
 *     power-of-two 3-bit (Eq. 22; level set listed in Sec. IV-C);
 *   - the layer product a^q_{l-1} W^q_l of Algorithm 1 (inference branch),
 *     written as a direct convolution over integer level codes;
 *   - the layer constructs of Sec. III-E ({QConv-pool-BN-HardTanh} and
 *     {QConv-BN-HardTanh}) as separate, unfused steps;
 *   - full-precision support layers (first conv, last FC, pooling).
 *
 * Integer level codes (one int8 per value):
 *   1 bit : {-1, +1}
 *   2 bits: {-1, 0, +1}
 *   3 bits: {0, +-1, +-2, +-4} = 4 x the paper's levels {0, +-1/4, +-1/2, +-1},
 *           so every product is an integer; the real value of a convolution
 *           is acc * 2^-(2[a_bits==3] + 2[w_bits==3]).
 *
 * Floating point: no fast-math, no contraction (build with
 * -ffp-contract=off); every fused multiply-add is an explicit fmaf/fma.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define ORACLE_OK 0
#define ORACLE_EINVAL -1
#define ORACLE_EOVERFLOW -4

/* ------------------------------------------------------------------------ */
/* Quantizers (Sec. III-C)                                                   */
/* ------------------------------------------------------------------------ */

/* Eq. 4: sign(a) is +1 for a positive input and -1 otherwise (Sec. II-A),
 * so 0, -0 and NaN all give -1. */
static int8_t q_sign(float x) { return (x > 0.0f) ? (int8_t)1 : (int8_t)-1; }

/* Eq. 21: 0 when |a| <= delta, sign(a) otherwise. */
static int8_t q_ternary(float x, float delta) {
  if (fabsf(x) <= delta) return 0;
  return q_sign(x);
}

/* Eq. 22 for n = 3: q = 2^(n-1) - 1 = 3 non-zero magnitudes 2^-p, p = 2, 1, 0,
 * tested in that order against thresholds t[0] < t[1] < t[2]; beyond the last
 * threshold the magnitude is 2^0 (the scan ends at p = 0).  Codes are 4x the
 * level: 2^-2 -> 1, 2^-1 -> 2, 2^0 -> 4. */
static int8_t q_pow2(float x, const float t[3]) {
  float ax = fabsf(x);
  int8_t mag;
  if (ax <= t[0]) return 0;
  if (ax <= t[1]) mag = 1;
  else if (ax <= t[2]) mag = 2;
  else mag = 4;
  return (x > 0.0f) ? mag : (int8_t)-mag;
}

static int8_t q_level(float x, int bits, const float* thr) {
  if (bits == 1) return q_sign(x);
  if (bits == 2) return q_ternary(x, thr[0]);
  return q_pow2(x, thr);
}

/* Quantize n activations with one threshold set (thr: 2 bits {delta},
 * 3 bits {t1, t2, t3}; ignored for 1 bit). */
int oracle_quantize(const float* x, int64_t n, int bits, const float* thr, int8_t* out) {
  if (bits < 1 || bits > 3 || (bits > 1 && thr == NULL)) return ORACLE_EINVAL;
  for (int64_t i = 0; i < n; ++i) out[i] = q_level(x[i], bits, thr);
  return ORACLE_OK;
}

/* Per-output-channel weight scale s_c = mean |W_c| over the k = Cin*Kh*Kw
 * weights of channel c, in double with a fixed summation order, then
 * rounded once to float: 256 partial sums P_j (j = 0..255), P_j adding
 * |w_i| for the storage indices i = j, j + 256, j + 512, ... in turn; the
 * partial sums are then added pairwise (P_0 + P_1, P_2 + P_3, ..., then
 * those sums pairwise, and so on up to one sum); s_c = (float)(sum / k). */
void oracle_weight_scale(const float* w, int cout, int64_t k, float* s) {
  for (int c = 0; c < cout; ++c) {
    const float* wc = w + (int64_t)c * k;
    double part[256];
    for (int j = 0; j < 256; ++j) {
      part[j] = 0.0;
      for (int64_t i = j; i < k; i += 256) part[j] += fabs((double)wc[i]);
    }
    for (int step = 1; step < 256; step *= 2)
      for (int j = 0; j < 256; j += 2 * step) part[j] = part[j] + part[j + step];
    s[c] = (float)(part[0] / (double)k);
  }
}

/* Quantize weights of cout channels (k each).  Channel c uses thresholds
 * (float)(base_thr[j] * s_c), computed in double. */
int oracle_quantize_weights(const float* w, int cout, int64_t k, int bits, const float* s,
                            const float* base_thr, int8_t* out) {
  if (bits < 1 || bits > 3 || (bits > 1 && (s == NULL || base_thr == NULL))) return ORACLE_EINVAL;
  for (int c = 0; c < cout; ++c) {
    float thr[3] = {0.0f, 0.0f, 0.0f};
    if (bits == 2) thr[0] = (float)((double)base_thr[0] * (double)s[c]);
    if (bits == 3)
      for (int j = 0; j < 3; ++j) thr[j] = (float)((double)base_thr[j] * (double)s[c]);
    for (int64_t i = 0; i < k; ++i)
      out[(int64_t)c * k + i] = q_level(w[(int64_t)c * k + i], bits, thr);
  }
  return ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Quantized layer product (Algorithm 1, inference branch)                   */
/* ------------------------------------------------------------------------ */

static int out_dim(int in, int k, int stride, int pad) { return (in + 2 * pad - k) / stride + 1; }

/* One output of the direct convolution over level codes.
 * a: [n][cin][h][w], wt: [cout][cin][kh][kw]; taps outside the input take
 * the level pad_level.  Accumulates in int64. */
static int64_t conv_one(const int8_t* a, const int8_t* wt, int cin, int h, int w, int kh, int kw,
                        int stride, int pad, int pad_level, int n, int co, int oh, int ow) {
  int64_t acc = 0;
  for (int ci = 0; ci < cin; ++ci)
    for (int y = 0; y < kh; ++y)
      for (int x = 0; x < kw; ++x) {
        int ih = oh * stride - pad + y;
        int iw = ow * stride - pad + x;
        int64_t av;
        if (ih < 0 || ih >= h || iw < 0 || iw >= w)
          av = pad_level;
        else
          av = a[(((int64_t)n * cin + ci) * h + ih) * w + iw];
        int64_t wv = wt[(((int64_t)co * cin + ci) * kh + y) * kw + x];
        acc += av * wv;
      }
  return acc;
}

/* acc[n][cout][ho][wo] = sum_{ci,y,x} a[n][ci][oh*s-p+y][ow*s-p+x] * wt[co][ci][y][x].
 * Returns ORACLE_EOVERFLOW (after finishing) if any result does not fit int32. */
int oracle_conv_levels(const int8_t* a, const int8_t* wt, int n, int cin, int h, int w, int cout,
                       int kh, int kw, int stride, int pad, int pad_level, int32_t* acc) {
  if (n < 0 || cin < 1 || h < 1 || w < 1 || cout < 1 || kh < 1 || kw < 1 || stride < 1 || pad < 0)
    return ORACLE_EINVAL;
  int ho = out_dim(h, kh, stride, pad), wo = out_dim(w, kw, stride, pad);
  if (ho < 1 || wo < 1) return ORACLE_EINVAL;
  int overflow = 0;
#pragma omp parallel for collapse(2) schedule(static) reduction(| : overflow)
  for (int b = 0; b < n; ++b)
    for (int co = 0; co < cout; ++co)
      for (int oh = 0; oh < ho; ++oh)
        for (int ow = 0; ow < wo; ++ow) {
          int64_t v = conv_one(a, wt, cin, h, w, kh, kw, stride, pad, pad_level, b, co, oh, ow);
          if (v > INT32_MAX || v < INT32_MIN) overflow = 1;
          acc[(((int64_t)b * cout + co) * ho + oh) * wo + ow] = (int32_t)v;
        }
  return overflow ? ORACLE_EOVERFLOW : ORACLE_OK;
}

/* The same product at a list of flat NCHW output indices only (for sampled
 * checks at full size). */
int oracle_conv_levels_at(const int8_t* a, const int8_t* wt, int n, int cin, int h, int w, int cout,
                          int kh, int kw, int stride, int pad, int pad_level, const int64_t* idx,
                          int64_t nidx, int32_t* out) {
  int ho = out_dim(h, kh, stride, pad), wo = out_dim(w, kw, stride, pad);
  if (ho < 1 || wo < 1) return ORACLE_EINVAL;
  int bad = 0;
#pragma omp parallel for schedule(static) reduction(| : bad)
  for (int64_t i = 0; i < nidx; ++i) {
    int64_t f = idx[i];
    int ow = (int)(f % wo);
    f /= wo;
    int oh = (int)(f % ho);
    f /= ho;
    int co = (int)(f % cout);
    int b = (int)(f / cout);
    if (b < 0 || b >= n) {
      bad = 1;
      continue;
    }
    int64_t v = conv_one(a, wt, cin, h, w, kh, kw, stride, pad, pad_level, b, co, oh, ow);
    if (v > INT32_MAX || v < INT32_MIN) bad = 1;
    out[i] = (int32_t)v;
  }
  return bad ? ORACLE_EOVERFLOW : ORACLE_OK;
}

/* ------------------------------------------------------------------------ */
/* Epilogue steps (Sec. III-E layer constructs), each its own pass            */
/* ------------------------------------------------------------------------ */

/* Real value of an accumulator: acc * 2^-shift (exact in float for |acc| < 2^24). */
static float acc_real(int32_t acc, int shift) { return ldexpf((float)acc, -shift); }

/* y[n][c][hw] = fl32(s_c * acc_real): one rounding. */
void oracle_epi_scale(const int32_t* acc, int n, int c, int64_t hw, int shift, const float* s,
                      float* y) {
  for (int b = 0; b < n; ++b)
    for (int ch = 0; ch < c; ++ch)
      for (int64_t i = 0; i < hw; ++i) {
        int64_t f = ((int64_t)b * c + ch) * hw + i;
        y[f] = s[ch] * acc_real(acc[f], shift);
      }
}

/* Batch normalisation folded to z = fmaf(k_c, acc_real, b_c). */
void oracle_epi_bn(const int32_t* acc, int n, int c, int64_t hw, int shift, const float* k,
                   const float* bb, float* z) {
  for (int b = 0; b < n; ++b)
    for (int ch = 0; ch < c; ++ch)
      for (int64_t i = 0; i < hw; ++i) {
        int64_t f = ((int64_t)b * c + ch) * hw + i;
        z[f] = fmaf(k[ch], acc_real(acc[f], shift), bb[ch]);
      }
}

/* Batch normalisation of an fp32 activation: z = fmaf(k_c, x, b_c). */
void oracle_bn_f32(const float* x, int n, int c, int64_t hw, const float* k, const float* bb,
                   float* z) {
  for (int b = 0; b < n; ++b)
    for (int ch = 0; ch < c; ++ch)
      for (int64_t i = 0; i < hw; ++i) {
        int64_t f = ((int64_t)b * c + ch) * hw + i;
        z[f] = fmaf(k[ch], x[f], bb[ch]);
      }
}

/* BN folding in double: k = gamma / sqrt(var + eps), b = beta - k * mean,
 * each rounded once to float (b uses the double k). */
void oracle_bn_fold(const float* gamma, const float* beta, const float* mean, const float* var,
                    double eps, int c, float* k, float* b) {
  for (int i = 0; i < c; ++i) {
    double kd = (double)gamma[i] / sqrt((double)var[i] + eps);
    k[i] = (float)kd;
    b[i] = (float)((double)beta[i] - kd * (double)mean[i]);
  }
}

/* 2x2 / stride-2 max pooling on integer accumulators (pooling sits before BN
 * in {QConv-pool-BN-HardTanh}).  Output [n][c][h/2][w/2], floor sizes. */
void oracle_maxpool2_int(const int32_t* x, int n, int c, int h, int w, int32_t* y) {
  int ho = h / 2, wo = w / 2;
  for (int b = 0; b < n; ++b)
    for (int ch = 0; ch < c; ++ch)
      for (int oh = 0; oh < ho; ++oh)
        for (int ow = 0; ow < wo; ++ow) {
          const int32_t* p = x + ((int64_t)b * c + ch) * h * w;
          int32_t m = p[(2 * oh) * w + 2 * ow];
          for (int dy = 0; dy < 2; ++dy)
            for (int dx = 0; dx < 2; ++dx) {
              int32_t v = p[(2 * oh + dy) * w + 2 * ow + dx];
              if (v > m) m = v;
            }
          y[(((int64_t)b * c + ch) * ho + oh) * wo + ow] = m;
        }
}

/* HardTanh max(-1, min(1, x)) (Sec. III-E). */
void oracle_hardtanh(const float* x, int64_t n, float* y) {
  for (int64_t i = 0; i < n; ++i) {
    float v = x[i];
    if (v > 1.0f) v = 1.0f;
    if (v < -1.0f) v = -1.0f;
    y[i] = v;
  }
}

void oracle_relu(const float* x, int64_t n, float* y) {
  for (int64_t i = 0; i < n; ++i) y[i] = (x[i] > 0.0f) ? x[i] : 0.0f;
}

/* y = fl32(x + r) elementwise (residual add). */
void oracle_add(const float* x, const float* r, int64_t n, float* y) {
  for (int64_t i = 0; i < n; ++i) y[i] = x[i] + r[i];
}

/* ------------------------------------------------------------------------ */
/* Full-precision support layers                                             */
/* ------------------------------------------------------------------------ */

/* fp32 convolution, zero padding, no bias.  Each output is one chain of
 * single-rounding fused multiply-adds over (ci, kh, kw) in that order,
 * starting from +0. */
int oracle_conv_f32(const float* x, const float* wt, int n, int cin, int h, int w, int cout, int kh,
                    int kw, int stride, int pad, float* y) {
  int ho = out_dim(h, kh, stride, pad), wo = out_dim(w, kw, stride, pad);
  if (ho < 1 || wo < 1) return ORACLE_EINVAL;
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < n; ++b)
    for (int co = 0; co < cout; ++co)
      for (int oh = 0; oh < ho; ++oh)
        for (int ow = 0; ow < wo; ++ow) {
          float acc = 0.0f;
          for (int ci = 0; ci < cin; ++ci)
            for (int yy = 0; yy < kh; ++yy)
              for (int xx = 0; xx < kw; ++xx) {
                int ih = oh * stride - pad + yy, iw = ow * stride - pad + xx;
                if (ih < 0 || ih >= h || iw < 0 || iw >= w) continue;
                acc = fmaf(x[(((int64_t)b * cin + ci) * h + ih) * w + iw],
                           wt[(((int64_t)co * cin + ci) * kh + yy) * kw + xx], acc);
              }
          y[(((int64_t)b * cout + co) * ho + oh) * wo + ow] = acc;
        }
  return ORACLE_OK;
}

/* Same convolution in double (used only to bound the fp32 rounding). */
int oracle_conv_f64(const double* x, const double* wt, int n, int cin, int h, int w, int cout,
                    int kh, int kw, int stride, int pad, double* y) {
  int ho = out_dim(h, kh, stride, pad), wo = out_dim(w, kw, stride, pad);
  if (ho < 1 || wo < 1) return ORACLE_EINVAL;
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < n; ++b)
    for (int co = 0; co < cout; ++co)
      for (int oh = 0; oh < ho; ++oh)
        for (int ow = 0; ow < wo; ++ow) {
          double acc = 0.0;
          for (int ci = 0; ci < cin; ++ci)
            for (int yy = 0; yy < kh; ++yy)
              for (int xx = 0; xx < kw; ++xx) {
                int ih = oh * stride - pad + yy, iw = ow * stride - pad + xx;
                if (ih < 0 || ih >= h || iw < 0 || iw >= w) continue;
                acc += x[(((int64_t)b * cin + ci) * h + ih) * w + iw] *
                       wt[(((int64_t)co * cin + ci) * kh + yy) * kw + xx];
              }
          y[(((int64_t)b * cout + co) * ho + oh) * wo + ow] = acc;
        }
  return ORACLE_OK;
}

/* Fully connected fp32 layer: y[b][o] = fl32(chain_i fmaf(x[b][i], W[o][i], .) + bias[o]),
 * the chain in index order starting from +0; bias may be NULL (0). */
void oracle_fc_f32(const float* x, const float* wt, const float* bias, int n, int in, int out,
                   float* y) {
#pragma omp parallel for collapse(2) schedule(static)
  for (int b = 0; b < n; ++b)
    for (int o = 0; o < out; ++o) {
      float acc = 0.0f;
      for (int i = 0; i < in; ++i)
        acc = fmaf(x[(int64_t)b * in + i], wt[(int64_t)o * in + i], acc);
      y[(int64_t)b * out + o] = acc + (bias ? bias[o] : 0.0f);
    }
}

/* k x k / stride s max pooling with padding p (padding never wins). */
void oracle_maxpool_f32(const float* x, int n, int c, int h, int w, int k, int s, int p, float* y) {
  int ho = out_dim(h, k, s, p), wo = out_dim(w, k, s, p);
  for (int b = 0; b < n; ++b)
    for (int ch = 0; ch < c; ++ch)
      for (int oh = 0; oh < ho; ++oh)
        for (int ow = 0; ow < wo; ++ow) {
          float m = -INFINITY;
          for (int dy = 0; dy < k; ++dy)
            for (int dx = 0; dx < k; ++dx) {
              int ih = oh * s - p + dy, iw = ow * s - p + dx;
              if (ih < 0 || ih >= h || iw < 0 || iw >= w) continue;
              float v = x[(((int64_t)b * c + ch) * h + ih) * w + iw];
              if (v > m) m = v;
            }
          y[(((int64_t)b * c + ch) * ho + oh) * wo + ow] = m;
        }
}

/* Global average pooling: fp32 sum in (h, w) order from +0, then one
 * division by h*w. */
void oracle_avgpool_f32(const float* x, int n, int c, int h, int w, float* y) {
  for (int b = 0; b < n; ++b)
    for (int ch = 0; ch < c; ++ch) {
      float s = 0.0f;
      const float* p = x + ((int64_t)b * c + ch) * h * w;
      for (int i = 0; i < h * w; ++i) s += p[i];
      y[(int64_t)b * c + ch] = s / (float)(h * w);
    }
}

int oracle_num_threads(void) {
#ifdef _OPENMP
  extern int omp_get_max_threads(void);
  return omp_get_max_threads();
#else
  return 1;
#endif
}
