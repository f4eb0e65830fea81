// qconv_internal.h -- device helpers and launcher declarations shared by the
// library's HIP translation units (not part of the public ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <type_traits>

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

// Workgroup barrier that orders LDS accesses only.  __syncthreads() also
// waits for every outstanding global load and store of the wave (its
// release fence covers global memory), which stalls a barrier that a
// prefetch of the next tile or the previous tile's output stores are still
// in flight across; this one leaves them in flight.  For blocks that share
// data through LDS alone.
__device__ __forceinline__ void lds_barrier() {
  __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
  __builtin_amdgcn_s_barrier();
  __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

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

// The bitplane compares may take z itself instead of HardTanh(z) unless a
// threshold reaches 1: below 1, |HardTanh(z)| <= t exactly when |z| <= t, and
// the sign is kept.
inline bool hardtanh_needed(int bits, Thr t) {
  return (bits == 2 && t.t0 >= 1.0f) || (bits == 3 && t.t2 >= 1.0f);
}

// n / d by a multiply-high, exact whenever n * d < 2^32 (checked on the host
// against the largest dividend of each use).
struct FastDiv {
  uint32_t d, m;
};
inline FastDiv make_fastdiv(uint32_t d) {
  FastDiv f;
  f.d = d;
  f.m = d <= 1 ? 0u : (uint32_t)(0xFFFFFFFFu / d + 1u);
  return f;
}
__device__ __forceinline__ uint32_t fdiv(uint32_t n, FastDiv f) { return f.m ? __umulhi(n, f.m) : n; }

// Thresholds that give the compares on |z| the results of those on
// |HardTanh(z)| = min(|z|, 1) for every z, NaN included: one below 1 is
// kept, one at or above 1 (which |HardTanh(z)| never exceeds) becomes +inf.
inline Thr thr_unclamped(Thr t) {
  auto f = [](float v) { return v >= 1.0f ? __builtin_inff() : v; };
  return Thr{f(t.t0), f(t.t1), f(t.t2)};
}

// Compile-time loop: f(integral_constant<I>) for I in [B, E), so that the
// accumulator tiles are only ever indexed with constants.
template <int B, int E>
struct Unroll {
  template <class F>
  __device__ __forceinline__ static void run(F&& f) {
    f(std::integral_constant<int, B>{});
    Unroll<B + 1, E>::run(f);
  }
};
template <int E>
struct Unroll<E, E> {
  template <class F>
  __device__ __forceinline__ static void run(F&&) {}
};

// Ballots of the bitplanes of Q(HardTanh(z)) over the wave (Eqs. 4, 21, 22):
// the same compares as the quantizer, one ballot each, combined with scalar
// bit operations.  `ok` = the lane's channel and unit exist; its ballot is
// taken once and masks the others, so that each compare's lane mask is the
// ballot itself.
template <int OB>
__device__ __forceinline__ void plane_ballots(float z, bool ok, Thr t, uint64_t* b) {
  const uint64_t om = __builtin_amdgcn_ballot_w64(ok);
  const uint64_t s = __builtin_amdgcn_ballot_w64(z > 0.0f) & om;
  if constexpr (OB == 1) {
    b[0] = s;
  } else if constexpr (OB == 2) {
    const uint64_t nz = __builtin_amdgcn_ballot_w64(!(fabsf(z) <= t.t0)) & om;
    b[0] = s & nz;
    b[1] = nz;
  } else {
    const float az = fabsf(z);
    const uint64_t a1 = __builtin_amdgcn_ballot_w64(!(az <= t.t0)) & om;
    const uint64_t a2 = __builtin_amdgcn_ballot_w64(!(az <= t.t1)) & om;
    const uint64_t a3 = __builtin_amdgcn_ballot_w64(!(az <= t.t2)) & om;
    b[0] = s & a1;
    b[1] = a3;
    b[2] = a2 & ~a3;
    b[3] = a1 & ~a2;
  }
}

// Eight v_writelane_b32: lanes L0..L3 of w take lo0..lo3, lanes H0..H3 take
// hi0..hi3 (wave-uniform values).  The lanes are inline constants, so the
// value is the instruction's only scalar operand.  The values usually come
// straight from a VALU compare; s_nop 4 provides the wait states a VALU
// write of an SGPR needs before v_writelane reads it, which the compiler does
// not insert across inline assembly.
template <int L0, int L1, int L2, int L3, int H0, int H1, int H2, int H3>
__device__ __forceinline__ uint32_t writelanes8(uint32_t w, uint32_t lo0, uint32_t lo1, uint32_t lo2,
                                                uint32_t lo3, uint32_t hi0, uint32_t hi1, uint32_t hi2,
                                                uint32_t hi3) {
  asm("s_nop 4\n\t"
      "v_writelane_b32 %0, %1, %9\n\t"
      "v_writelane_b32 %0, %2, %10\n\t"
      "v_writelane_b32 %0, %3, %11\n\t"
      "v_writelane_b32 %0, %4, %12\n\t"
      "v_writelane_b32 %0, %5, %13\n\t"
      "v_writelane_b32 %0, %6, %14\n\t"
      "v_writelane_b32 %0, %7, %15\n\t"
      "v_writelane_b32 %0, %8, %16"
      : "+v"(w)
      : "s"(lo0), "s"(lo1), "s"(lo2), "s"(lo3), "s"(hi0), "s"(hi1), "s"(hi2), "s"(hi3), "i"(L0), "i"(L1),
        "i"(L2), "i"(L3), "i"(H0), "i"(H1), "i"(H2), "i"(H3));
  return w;
}

__host__ __device__ inline int ceil_div(int a, int b) { return (a + b - 1) / b; }
inline int cout_pad(int cout) { return ceil_div(cout, 128) * 128; }

// ---------------------------------------------------------------------------
// Bitplanes -> matrix-core operands.  One 32-channel word of `P` planes is
// turned into the level codes of its channels.  `valid` marks the channels
// that exist (bits past cin give 0; only needed for 1-bit operands, whose
// sign plane alone cannot express 0).
// ---------------------------------------------------------------------------

// Nibble -> one bit per byte: bit j of `nib` (j < 4) lands in bit 0 of byte j.
// The four shifted copies of the nibble (offsets 0, 7, 14, 21) never overlap,
// so the product has no carries.
__device__ __forceinline__ uint32_t spread4(uint32_t nib) {
  return __umul24(nib, 0x00204081u) & 0x01010101u;
}

// int8 codes of channels [4q, 4q+4) as 4 bytes, by a byte lookup (v_perm_b32)
// with index = S + 2*M for 1/2-bit operands (M = nonzero mask) and
// index = B0 + 2*B1 + 4*S for 3-bit ones (B0 = |l| in {1,4}, B1 = |l| in {2,4}).
template <int P>
__device__ __forceinline__ void expand_i8_word(const uint32_t* pl, uint32_t valid, uint32_t out[8]) {
  if constexpr (P <= 2) {
    const uint32_t S = pl[0];
    const uint32_t M = (P == 1) ? valid : pl[1];
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const uint32_t idx = spread4((S >> (4 * q)) & 0xFu) | (spread4((M >> (4 * q)) & 0xFu) << 1);
      // idx 0/1 -> 0, 2 -> -1, 3 -> +1
      out[q] = __builtin_amdgcn_perm(0u, 0x01FF0000u, idx);
    }
  } else {
    const uint32_t S = pl[0], E1 = pl[1], E2 = pl[2], E3 = pl[3];
    const uint32_t B0 = E1 | E3, B1 = E1 | E2;
#pragma unroll
    for (int q = 0; q < 8; ++q) {
      const uint32_t idx = spread4((B0 >> (4 * q)) & 0xFu) | (spread4((B1 >> (4 * q)) & 0xFu) << 1) |
                           (spread4((S >> (4 * q)) & 0xFu) << 2);
      // idx 0..3 -> 0, -1, -2, -4 ; idx 4..7 -> 0, +1, +2, +4
      out[q] = __builtin_amdgcn_perm(0x04020100u, 0xFCFEFF00u, idx);
    }
  }
}

// E2M1 (fp4) codes of 32 channels as 4 words: +1 = 0x2, +2 = 0x4, +4 = 0x6,
// sign bit 0x8, zero = 0x0.  Word q holds channels q, q + 4, ..., q + 28 in
// nibbles 0..7, so each word takes one shift and one mask per plane: bit
// q + 4k of a plane lands in bit 4k.  Any fixed channel order works for the
// product as long as both operands use it (weights and activations are
// expanded by this one function).
template <int P>
__device__ __forceinline__ void expand_fp4_word(const uint32_t* pl, uint32_t valid, uint32_t out[4]) {
  constexpr uint32_t K = 0x11111111u;
  if constexpr (P <= 2) {
    const uint32_t M = (P == 1) ? valid : pl[1];
    const uint32_t N = M & ~pl[0];
#pragma unroll
    for (int q = 0; q < 4; ++q) out[q] = (((M >> q) & K) << 1) | (((N >> q) & K) << 3);
  } else {
    const uint32_t E1 = pl[1], E2 = pl[2], E3 = pl[3];
    const uint32_t B1 = E1 | E3, B2 = E1 | E2, N = (E1 | E2 | E3) & ~pl[0];
#pragma unroll
    for (int q = 0; q < 4; ++q)
      out[q] = (((B1 >> q) & K) << 1) | (((B2 >> q) & K) << 2) | (((N >> q) & K) << 3);
  }
}

// fp16 bits of a float, rounded to nearest even.
__device__ __forceinline__ uint32_t f16_bits(float v) {
  return (uint32_t)__builtin_bit_cast(uint16_t, (_Float16)v);
}

// fp16 codes of the four int8 codes of `word` as two words (channel 2i in
// the low half; exact: the codes are 0, +-1, +-2, +-4).
__device__ __forceinline__ void i8_word_to_f16(uint32_t word, uint32_t* lo, uint32_t* hi) {
  *lo = f16_bits((float)(int8_t)word) | (f16_bits((float)(int8_t)(word >> 8)) << 16);
  *hi = f16_bits((float)(int8_t)(word >> 16)) | (f16_bits((float)(int8_t)(word >> 24)) << 16);
}

// Byte sizes of the four parts of a packed weight buffer.
inline size_t wbytes_planes(int cout, int cin, int kh, int kw, int bits) {
  return (size_t)kh * kw * ceil_div(cin, 32) * cout_pad(cout) * planes_of(bits) * 4;
}
inline size_t wbytes_i8(int cout, int cin, int kh, int kw) {
  return (size_t)kh * kw * ceil_div(cin, 32) * cout_pad(cout) * 32;
}
inline size_t wbytes_fp4(int cout, int cin, int kh, int kw) {
  return (size_t)kh * kw * ceil_div(ceil_div(cin, 32), 2) * cout_pad(cout) * 32;
}
// fp16 codes, 16 channels (32 bytes) per (tap, k-step, output channel).
inline size_t wbytes_f16(int cout, int cin, int kh, int kw) {
  return (size_t)kh * kw * 2 * ceil_div(cin, 32) * cout_pad(cout) * 32;
}

// 32-bit words per (pixel, 32-channel word) of an activation tensor: the
// bitplanes of 1..3-bit levels, or 32 fp16 values of a 16-bit input.
__host__ __device__ constexpr int act_words(int bits) { return bits == 16 ? 16 : planes_of(bits); }

// ---------------------------------------------------------------------------
// Launchers (each returns a qconv_status; inputs already validated).
// ---------------------------------------------------------------------------
int launch_pack_act(const float* x, int n, int c, int h, int w, int bits, Thr t, uint32_t* out,
                    hipStream_t s);
int launch_pack_act_f16(const float* x, int n, int c, int h, int w, uint32_t* out, hipStream_t s);
int launch_pack_weight(const float* w, int cout, int cin, int kh, int kw, int bits,
                       const float* base_thr, uint32_t* out, float* scale, hipStream_t s);
int launch_pack_weight_f16(const float* w, int cout, int cin, int kh, int kw, uint32_t* out, float* scale,
                           hipStream_t s);

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
  int a_bits, w_bits;     // a_bits 16: fp16 activations [n][h][w][cw * 32]; w_bits 16: fp16 weights
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
  // matrix-core operand copies of the weights (parts of the packed buffer)
  int cin;
  const uint8_t* w_i8;
  const uint8_t* w_fp4;
  const uint8_t* w_f16;
  int mfma_op;  // MfmaOp: the operand format of the matrix-core kernel
};
enum MfmaOp { OP_I8 = 0, OP_FP4 = 1, OP_F16 = 2 };
int launch_conv_bitplane(const ConvArgs& a, hipStream_t s);
// The LDS-tiled XNOR kernel (1-2 bit operands, 1x1 / 3x3, stride 1-2,
// unpacked unpooled outputs); launch_conv_bitplane runs it when it applies.
bool xnor_supports(const ConvArgs& a);
int launch_conv_xnor(const ConvArgs& a, hipStream_t s);
int xnor_kernel_name(const ConvArgs& a, char* buf, int len);
int launch_conv_mfma(const ConvArgs& a, hipStream_t s);
bool mfma_supports(const ConvArgs& a);
// Name of the kernel instantiation each launcher would run (template
// arguments as the profiler prints them); returns the name's length.
int bitplane_kernel_name(const ConvArgs& a, char* buf, int len);
int mfma_kernel_name(const ConvArgs& a, char* buf, int len);

int launch_conv_f32(const float* x, const float* wt_t /* [cin][k][k][cout_pad64] */, int n, int cin,
                    int h, int w, int cout, int k, int stride, int pad, const float* bn_k,
                    const float* bn_b, int relu, int out_bits, Thr othr, float* out_f32,
                    uint32_t* out_packed, hipStream_t s);
// fp32 conv on the matrix cores with BN, ReLU, optional 3x3 / 2 max pooling
// (pad 1) and an optional packed Q(HardTanh(.)) copy (conv_f32_mfma.hip).
// alg 0: fp32 matrix cores; alg 1: exact bf16 splits, six partial products
// on the bf16 matrix cores (pooled 7 x 7 / 2 layers with cin <= 3 only).
bool conv_f32_mfma_supports(int n, int cin, int h, int w, int cout, int k, int stride, int pad, int pool, int alg);
int launch_conv_f32_mfma(const float* x, const float* w, int n, int cin, int h, int wd, int cout, int k, int stride,
                         int pad, const float* bn_k, const float* bn_b, int relu, int pool, float* out,
                         uint32_t* out_packed, int out_bits, Thr othr, int alg, hipStream_t s);
int launch_transpose_conv_weight(const float* w, int cout, int cin, int k, float* wt_t,
                                 hipStream_t s);
int launch_maxpool_f32(const float* x, int n, int c, int h, int w, int k, int stride, int pad,
                       float* y, hipStream_t s);
int launch_avgpool_f32(const float* x, int n, int c, int h, int w, float* y, hipStream_t s);
int launch_fc_f32(const void* x, int x_bits, int n, int in, const float* w, const float* bias,
                  int out, float* y, hipStream_t s);

int launch_aqe_forward(const float* x, int64_t n, int bits, float alpha, Thr base, const float* scale,
                       int64_t group, float* y, hipStream_t s);
int launch_aqe_backward(const float* x, const float* gy, int64_t n, float alpha, float* gx, hipStream_t s);
int launch_aqe_sgd_clip(float* w, const float* g, int64_t n, float lr, hipStream_t s);

inline int hip_status() {
  return hipGetLastError() == hipSuccess ? QCONV_OK : QCONV_EHIP;
}

}  // namespace qc
