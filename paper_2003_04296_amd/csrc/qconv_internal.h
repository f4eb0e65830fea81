// qconv_internal.h -- device helpers and launcher declarations shared by the
// library's HIP translation units (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "../../include/qconv.h"

namespace qc {

// Bitplanes per bitwidth: sign (+ nonzero mask for 2 bits, + three one-hot
// magnitude planes |l| = 1, 1/2, 1/4 for 3 bits).
__host__ __device__ constexpr int planes_of(int bits) { return bits == 1 ? 1 : (bits == 2 ? 2 : 4); }

// Exponent (in code units) of magnitude plane j (1-based) of a `bits`-wide
// operand: 3-bit codes are 4 x level, so plane 1 (|l| = 1) weighs 4 = 2^2.
__host__ __device__ constexpr int plane_exp(int planes, int j) { return planes == 4 ? 3 - j : 0; }

struct Thr {
  float t0, t1, t2;
};

// Inference quantizer h(.) of Sec. III-C returning the bitplane pattern of
// the level: bit 0 = sign (level > 0), bit p = magnitude plane p.
//  1 bit : sign (Eq. 4), +1 only for x > 0.
//  2 bits: 0 when |x| <= t0, else sign (Eq. 21).
//  3 bits: 0 when |x| <= t0, 1/4 when <= t1, 1/2 when <= t2, else 1 (Eq. 22).
template <int BITS>
__device__ __forceinline__ uint32_t quant_planes(float x, Thr t) {
  const uint32_t s = (x > 0.0f) ? 1u : 0u;
  if constexpr (BITS == 1) {
    return s;
  } else if constexpr (BITS == 2) {
    return (fabsf(x) <= t.t0) ? 0u : (s | 2u);
  } else {
    const float ax = fabsf(x);
    if (ax <= t.t0) return 0u;
    if (ax <= t.t1) return s | 8u;  // |l| = 1/4 -> plane 3
    if (ax <= t.t2) return s | 4u;  // |l| = 1/2 -> plane 2
    return s | 2u;                  // |l| = 1   -> plane 1
  }
}

// HardTanh max(-1, min(1, x)) written as two compares (a NaN passes through).
__device__ __forceinline__ float hardtanh(float v) {
  if (v > 1.0f) v = 1.0f;
  if (v < -1.0f) v = -1.0f;
  return v;
}

__host__ __device__ inline int ceil_div(int a, int b) { return (a + b - 1) / b; }
inline int cout_pad(int cout) { return ceil_div(cout, 64) * 64; }

// ---------------------------------------------------------------------------
// Launchers (each returns a qconv_status; inputs already validated).
// ---------------------------------------------------------------------------
int launch_pack_act(const float* x, int n, int c, int h, int w, int bits, Thr t, uint32_t* out,
                    hipStream_t s);
int launch_pack_weight(const float* w, int cout, int cin, int kh, int kw, int bits,
                       const float* base_thr, uint32_t* out, float* scale, hipStream_t s);

struct ConvArgs {
  const uint32_t* act;
  const uint32_t* wt;
  int n, h, w, cw;        // input; cw = 32-bit words per plane per pixel
  int cout, cop;          // cop = padded output channels of the weight layout
  int kh, kw, stride, pad;
  int ho, wo;             // conv output size
  int oh_out, ow_out;     // output size after optional 2x2 pooling
  int kreal;              // cin * kh * kw
  int shift;              // acc_real = acc * 2^-shift
  int a_bits, w_bits;
  // epilogue
  int mode, pool, residual_on;
  const float* scale;
  const float* bn_k;
  const float* bn_b;
  const float* residual;
  void* out;
  uint32_t* out_packed;
  int out_bits, out_cw;
  Thr othr;
};
int launch_conv_bitplane(const ConvArgs& a, hipStream_t s);
int launch_conv_mfma(const ConvArgs& a, hipStream_t s);
bool mfma_supports(const ConvArgs& a);

int launch_conv_f32(const float* x, const float* wt_t /* [cin][k][k][cout_pad32] */, int n, int cin,
                    int h, int w, int cout, int k, int stride, int pad, const float* bn_k,
                    const float* bn_b, int relu, int out_bits, Thr othr, float* out_f32,
                    uint32_t* out_packed, hipStream_t s);
int launch_transpose_conv_weight(const float* w, int cout, int cin, int k, float* wt_t,
                                 hipStream_t s);
int launch_maxpool_f32(const float* x, int n, int c, int h, int w, int k, int stride, int pad,
                       float* y, hipStream_t s);
int launch_avgpool_f32(const float* x, int n, int c, int h, int w, float* y, hipStream_t s);
int launch_fc_f32(const void* x, int x_bits, int n, int in, const float* w, const float* bias,
                  int out, float* y, hipStream_t s);

inline int hip_status() {
  return hipGetLastError() == hipSuccess ? QCONV_OK : QCONV_EHIP;
}

}  // namespace qc
