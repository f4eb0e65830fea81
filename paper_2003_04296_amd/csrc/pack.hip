// pack.hip -- quantize-and-pack kernels (Sec. III-C, Eq. 20 with the
// quantizers of Eqs. 4, 21, 22).
//
// Activations: fp32 NCHW -> bitplanes [n][h][w][cw][P].  One thread owns one
// (image, 32-channel word, pixel); consecutive lanes take consecutive pixels,
// so each of the 32 channel reads of a wave is one contiguous 256-byte run
// (HBM-bound: 4 bytes read per channel, P/8 bytes written).
//
// 16-bit inputs: fp32 NCHW -> fp16 [n][h][w][cw * 32] (round to nearest
// even; channels past c are +0), with the same thread mapping.
//
// Weights: fp32 OIHW -> per-channel scale s_c = mean|W_c| (double, storage
// order) -> thresholds scaled by s_c -> bitplanes [kh][kw][cw][cout_pad][P],
// then the int8, fp4 and fp16 matrix-core operand copies of the same codes.
#include "qconv_internal.h"

namespace qc {

namespace {

template <int BITS>
__global__ __launch_bounds__(256) void pack_act_kernel(const float* __restrict__ x, int c,
                                                       int hw, int cwn, int64_t total, Thr t,
                                                       uint32_t* __restrict__ out) {
  constexpr int P = planes_of(BITS);
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= total) return;
  const int pix = (int)(tid % hw);
  const int64_t r = tid / hw;
  const int cw = (int)(r % cwn);
  const int64_t b = r / cwn;
  const int c0 = cw * 32;
  const int nch = min(32, c - c0);
  const float* src = x + (b * c + c0) * (int64_t)hw + pix;
  uint32_t word[P];
#pragma unroll
  for (int p = 0; p < P; ++p) word[p] = 0u;
  if (nch == 32) {
#pragma unroll 8
    for (int j = 0; j < 32; ++j) {
      const uint32_t pl = quant_planes<BITS>(src[(int64_t)j * hw], t);
#pragma unroll
      for (int p = 0; p < P; ++p) word[p] |= ((pl >> p) & 1u) << j;
    }
  } else {
    for (int j = 0; j < nch; ++j) {
      const uint32_t pl = quant_planes<BITS>(src[(int64_t)j * hw], t);
#pragma unroll
      for (int p = 0; p < P; ++p) word[p] |= ((pl >> p) & 1u) << j;
    }
  }
  uint32_t* dst = out + ((b * hw + pix) * cwn + cw) * P;
#pragma unroll
  for (int p = 0; p < P; ++p) dst[p] = word[p];
}

// The same quantizer with the packed words staged in LDS: a block owns 64
// pixels of one image and every word of them; wave w computes words w,
// w + 4, ... with lanes along the pixels (each channel read one contiguous
// 256-byte run), then the block writes the 64 pixels' words as one
// contiguous run (the per-thread stores of pack_act_kernel land 4 * P bytes
// apart and write each HBM sector twice).
constexpr int PACK_PIX = 64;
template <int BITS>
__global__ __launch_bounds__(256) void pack_act_lds_kernel(const float* __restrict__ x, int c, int hw, int cwn,
                                                           int chunks, Thr t, uint32_t* __restrict__ out) {
  constexpr int P = planes_of(BITS);
  extern __shared__ uint32_t tile[];  // [PACK_PIX][cwn][P]
  const int b = blockIdx.x / chunks;
  const int pix0 = (blockIdx.x - b * chunks) * PACK_PIX;
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int pix = pix0 + lane;
  const bool pok = pix < hw;
  for (int cw = wave; cw < cwn; cw += 4) {
    const int c0 = cw * 32;
    const int nch = min(32, c - c0);
    const float* src = x + ((int64_t)b * c + c0) * hw + (pok ? pix : 0);
    uint32_t word[P];
#pragma unroll
    for (int p = 0; p < P; ++p) word[p] = 0u;
    if (nch == 32) {
#pragma unroll 8
      for (int j = 0; j < 32; ++j) {
        const uint32_t pl = quant_planes<BITS>(src[(int64_t)j * hw], t);
#pragma unroll
        for (int p = 0; p < P; ++p) word[p] |= ((pl >> p) & 1u) << j;
      }
    } else {
      for (int j = 0; j < nch; ++j) {
        const uint32_t pl = quant_planes<BITS>(src[(int64_t)j * hw], t);
#pragma unroll
        for (int p = 0; p < P; ++p) word[p] |= ((pl >> p) & 1u) << j;
      }
    }
#pragma unroll
    for (int p = 0; p < P; ++p) tile[(lane * cwn + cw) * P + p] = word[p];
  }
  __syncthreads();
  const int npix = min(PACK_PIX, hw - pix0);
  const int nwords = npix * cwn * P;
  uint32_t* dst = out + ((int64_t)b * hw + pix0) * cwn * P;
  for (int i = threadIdx.x; i < nwords; i += 256) dst[i] = tile[i];
}

__global__ __launch_bounds__(256) void pack_act_f16_kernel(const float* __restrict__ x, int c, int hw, int cwn,
                                                           int64_t total, uint32_t* __restrict__ out) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (tid >= total) return;
  const int pix = (int)(tid % hw);
  const int64_t r = tid / hw;
  const int cw = (int)(r % cwn);
  const int64_t b = r / cwn;
  const int c0 = cw * 32;
  const int nch = min(32, c - c0);
  const float* src = x + (b * c + c0) * (int64_t)hw + pix;
  uint32_t h[16];
  if (nch == 32) {
#pragma unroll
    for (int j = 0; j < 16; ++j)
      h[j] = f16_bits(src[(int64_t)(2 * j) * hw]) | (f16_bits(src[(int64_t)(2 * j + 1) * hw]) << 16);
  } else {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const uint32_t lo = 2 * j < nch ? f16_bits(src[(int64_t)(2 * j) * hw]) : 0u;
      const uint32_t hi = 2 * j + 1 < nch ? f16_bits(src[(int64_t)(2 * j + 1) * hw]) : 0u;
      h[j] = lo | (hi << 16);
    }
  }
  uint4* dst = reinterpret_cast<uint4*>(out + ((b * hw + pix) * cwn + cw) * 16);
#pragma unroll
  for (int q = 0; q < 4; ++q) dst[q] = make_uint4(h[4 * q], h[4 * q + 1], h[4 * q + 2], h[4 * q + 3]);
}

// s_c = (float)(sum_k |W_ck| / K), the sum in double in storage order.
// s_c = mean |W_c| (Eq. 20's scale of a channel's weights), one block per
// output channel.  The sum is taken in double in a fixed order, so the
// result does not depend on the launch: thread j adds |w_i| for i = j,
// j + 256, ... in turn (coalesced reads, up to 32 loads in flight), then the
// 256 partial sums are added pairwise: lanes exchange with lane l ^ 1, l ^ 2,
// ... l ^ 32 (every lane of a pair forms the same sum, IEEE addition being
// commutative), and the four wave sums are added (w0 + w1) + (w2 + w3).  One
// rounding to float at the end.
__global__ __launch_bounds__(256) void weight_scale_kernel(const float* __restrict__ w, int k,
                                                          float* __restrict__ scale) {
  __shared__ double wsum[4];
  const int co = blockIdx.x;
  const float* p = w + (int64_t)co * k;
  double acc = 0.0;
  constexpr int B = 32;
  for (int i0 = threadIdx.x; i0 < k; i0 += 256 * B) {
    // unguarded loads (indices clamped into the channel) so that all of them
    // issue before the first addition; only in-range values are added
    float v[B];
#pragma unroll
    for (int u = 0; u < B; ++u) v[u] = p[min(i0 + 256 * u, k - 1)];
#pragma unroll
    for (int u = 0; u < B; ++u) {
      const double t = fabs((double)v[u]);
      if (i0 + 256 * u < k) acc += t;
    }
  }
#pragma unroll
  for (int m = 1; m < 64; m *= 2) acc = acc + __shfl_xor(acc, m);
  if ((threadIdx.x & 63) == 0) wsum[threadIdx.x >> 6] = acc;
  __syncthreads();
  if (threadIdx.x == 0) scale[co] = (float)(((wsum[0] + wsum[1]) + (wsum[2] + wsum[3])) / (double)k);
}

template <int BITS>
__global__ __launch_bounds__(256) void pack_weight_kernel(const float* __restrict__ w, int cout,
                                                          int cin, int kh, int kw, int cwn,
                                                          int cop, Thr base,
                                                          const float* __restrict__ scale,
                                                          uint32_t* __restrict__ out) {
  constexpr int P = planes_of(BITS);
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)kh * kw * cwn * cop;
  if (tid >= total) return;
  const int co = (int)(tid % cop);
  int64_t r = tid / cop;
  const int cw = (int)(r % cwn);
  r /= cwn;
  const int x = (int)(r % kw);
  const int y = (int)(r / kw);
  uint32_t word[P];
#pragma unroll
  for (int p = 0; p < P; ++p) word[p] = 0u;
  if (co < cout) {
    Thr t = {0.0f, 0.0f, 0.0f};
    if constexpr (BITS > 1) {
      const double s = (double)scale[co];
      t.t0 = (float)((double)base.t0 * s);
      t.t1 = (float)((double)base.t1 * s);
      t.t2 = (float)((double)base.t2 * s);
    }
    const int c0 = cw * 32;
    const int nch = min(32, cin - c0);
    for (int j = 0; j < nch; ++j) {
      const float v = w[(((int64_t)co * cin + c0 + j) * kh + y) * kw + x];
      const uint32_t pl = quant_planes<BITS>(v, t);
#pragma unroll
      for (int p = 0; p < P; ++p) word[p] |= ((pl >> p) & 1u) << j;
    }
  }
  uint32_t* dst = out + tid * P;
#pragma unroll
  for (int p = 0; p < P; ++p) dst[p] = word[p];
}

// Channels of a 32-channel word that exist, given how many remain (>= 1).
__device__ __forceinline__ uint32_t chan_mask(int remaining) {
  return remaining >= 32 ? 0xFFFFFFFFu : ((1u << remaining) - 1u);
}

// Matrix-core operand copies of packed weights: one thread per
// (tap, word, output channel) for int8 (32 bytes), per (tap, word pair,
// output channel) for fp4 (32 bytes = 64 nibbles), per (tap, 16-channel
// k-step, output channel) for fp16 (32 bytes = 16 halves).  Channels past
// cin and padding output channels get code 0 (a 1-bit sign plane alone
// would read as -1 there).
template <int P>
__global__ __launch_bounds__(256) void expand_weight_kernel(const uint32_t* __restrict__ planes,
                                                            int taps, int cwn, int cout, int cop, int cin,
                                                            uint8_t* __restrict__ w_i8,
                                                            uint8_t* __restrict__ w_fp4,
                                                            uint8_t* __restrict__ w_f16) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int cwp = (cwn + 1) / 2;
  const int64_t n_i8 = (int64_t)taps * cwn * cop;
  const int64_t n_fp4 = (int64_t)taps * cwp * cop;
  const int64_t n_f16 = (int64_t)taps * 2 * cwn * cop;
  if (tid >= n_i8 + n_fp4 && tid < n_i8 + n_fp4 + n_f16) {
    const int64_t u = tid - n_i8 - n_fp4;
    const int co = (int)(u % cop);
    const int64_t r = u / cop;
    const int ks = (int)(r % (2 * cwn));
    const int tap = (int)(r / (2 * cwn));
    const int cw = ks >> 1, half = ks & 1;
    const uint32_t* src = planes + (((int64_t)tap * cwn + cw) * cop + co) * P;
    const uint32_t valid = co < cout ? chan_mask(cin - cw * 32) : 0u;
    uint32_t pl[P];
#pragma unroll
    for (int p = 0; p < P; ++p) pl[p] = src[p];
    uint32_t o[8];
    expand_i8_word<P>(pl, valid, o);
    uint32_t hv[8];  // channels 16 half .. 16 half + 15 as fp16 pairs
#pragma unroll
    for (int q = 0; q < 4; ++q) i8_word_to_f16(o[4 * half + q], &hv[2 * q], &hv[2 * q + 1]);
    uint4* dst = reinterpret_cast<uint4*>(w_f16 + u * 32);
    dst[0] = make_uint4(hv[0], hv[1], hv[2], hv[3]);
    dst[1] = make_uint4(hv[4], hv[5], hv[6], hv[7]);
  } else if (tid < n_i8) {
    const int co = (int)(tid % cop);
    const int64_t r = tid / cop;
    const int cw = (int)(r % cwn);
    const int tap = (int)(r / cwn);
    const uint32_t* src = planes + (((int64_t)tap * cwn + cw) * cop + co) * P;
    const uint32_t valid = co < cout ? chan_mask(cin - cw * 32) : 0u;
    uint32_t pl[P];
#pragma unroll
    for (int p = 0; p < P; ++p) pl[p] = src[p];
    uint32_t o[8];
    expand_i8_word<P>(pl, valid, o);
    uint4* dst = reinterpret_cast<uint4*>(w_i8 + tid * 32);
    dst[0] = make_uint4(o[0], o[1], o[2], o[3]);
    dst[1] = make_uint4(o[4], o[5], o[6], o[7]);
  } else if (tid < n_i8 + n_fp4) {
    const int64_t u = tid - n_i8;
    const int co = (int)(u % cop);
    const int64_t r = u / cop;
    const int kp = (int)(r % cwp);
    const int tap = (int)(r / cwp);
    uint32_t o[8];
#pragma unroll
    for (int half = 0; half < 2; ++half) {
      const int cw = 2 * kp + half;
      uint32_t pl[P];
      uint32_t valid = 0u;
#pragma unroll
      for (int p = 0; p < P; ++p) pl[p] = 0u;
      if (cw < cwn) {
        const uint32_t* src = planes + (((int64_t)tap * cwn + cw) * cop + co) * P;
#pragma unroll
        for (int p = 0; p < P; ++p) pl[p] = src[p];
        valid = co < cout ? chan_mask(cin - cw * 32) : 0u;
      }
      expand_fp4_word<P>(pl, valid, o + 4 * half);
    }
    uint4* dst = reinterpret_cast<uint4*>(w_fp4 + u * 32);
    dst[0] = make_uint4(o[0], o[1], o[2], o[3]);
    dst[1] = make_uint4(o[4], o[5], o[6], o[7]);
  }
}

// 16-bit weights (Table I rows with 1..3-bit inputs and 16-bit weights):
// fp32 OIHW -> fp16 [kh][kw][2 cw][cout_pad][16 halves], the layout of the
// fp16 operand copy, rounded to nearest even; channels past cin and padding
// output channels are +0.  One thread per 32-byte record.
__global__ __launch_bounds__(256) void pack_weight_f16_kernel(const float* __restrict__ w, int cout, int cin,
                                                              int kh, int kw, int cwn, int cop,
                                                              uint32_t* __restrict__ out) {
  const int64_t tid = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)kh * kw * 2 * cwn * cop;
  if (tid >= total) return;
  const int co = (int)(tid % cop);
  const int64_t r = tid / cop;
  const int ks = (int)(r % (2 * cwn));
  const int tap = (int)(r / (2 * cwn));
  const int y = tap / kw, x = tap - (tap / kw) * kw;
  uint32_t hv[8];
#pragma unroll
  for (int q = 0; q < 8; ++q) {
    uint32_t pair = 0u;
#pragma unroll
    for (int e = 0; e < 2; ++e) {
      const int ci = 16 * ks + 2 * q + e;
      if (co < cout && ci < cin) pair |= f16_bits(w[(((int64_t)co * cin + ci) * kh + y) * kw + x]) << (16 * e);
    }
    hv[q] = pair;
  }
  uint4* dst = reinterpret_cast<uint4*>(out + tid * 8);
  dst[0] = make_uint4(hv[0], hv[1], hv[2], hv[3]);
  dst[1] = make_uint4(hv[4], hv[5], hv[6], hv[7]);
}

}  // namespace

int launch_pack_act(const float* x, int n, int c, int h, int w, int bits, Thr t, uint32_t* out,
                    hipStream_t s) {
  const int hw = h * w;
  const int cwn = ceil_div(c, 32);
  const int64_t total = (int64_t)n * cwn * hw;
  if (total == 0) return QCONV_OK;
  const size_t lds = (size_t)PACK_PIX * cwn * planes_of(bits) * sizeof(uint32_t);
  if (lds <= 32 * 1024) {
    const int chunks = ceil_div(hw, PACK_PIX);
    const dim3 g((unsigned)((int64_t)n * chunks));
    switch (bits) {
      case 1: pack_act_lds_kernel<1><<<g, 256, lds, s>>>(x, c, hw, cwn, chunks, t, out); break;
      case 2: pack_act_lds_kernel<2><<<g, 256, lds, s>>>(x, c, hw, cwn, chunks, t, out); break;
      default: pack_act_lds_kernel<3><<<g, 256, lds, s>>>(x, c, hw, cwn, chunks, t, out); break;
    }
    return hip_status();
  }
  // very wide tensors (more than 32 KB of words per 64 pixels): one thread per word
  const dim3 grid((unsigned)((total + 255) / 256));
  switch (bits) {
    case 1: pack_act_kernel<1><<<grid, 256, 0, s>>>(x, c, hw, cwn, total, t, out); break;
    case 2: pack_act_kernel<2><<<grid, 256, 0, s>>>(x, c, hw, cwn, total, t, out); break;
    default: pack_act_kernel<3><<<grid, 256, 0, s>>>(x, c, hw, cwn, total, t, out); break;
  }
  return hip_status();
}

int launch_pack_act_f16(const float* x, int n, int c, int h, int w, uint32_t* out, hipStream_t s) {
  const int hw = h * w;
  const int cwn = ceil_div(c, 32);
  const int64_t total = (int64_t)n * cwn * hw;
  if (total == 0) return QCONV_OK;
  pack_act_f16_kernel<<<dim3((unsigned)((total + 255) / 256)), 256, 0, s>>>(x, c, hw, cwn, total, out);
  return hip_status();
}

int launch_pack_weight_f16(const float* w, int cout, int cin, int kh, int kw, uint32_t* out, float* scale,
                           hipStream_t s) {
  weight_scale_kernel<<<cout, 256, 0, s>>>(w, cin * kh * kw, scale);
  const int cwn = ceil_div(cin, 32);
  const int64_t total = (int64_t)kh * kw * 2 * cwn * cout_pad(cout);
  pack_weight_f16_kernel<<<dim3((unsigned)((total + 255) / 256)), 256, 0, s>>>(w, cout, cin, kh, kw, cwn,
                                                                                cout_pad(cout), out);
  return hip_status();
}

int launch_pack_weight(const float* w, int cout, int cin, int kh, int kw, int bits,
                       const float* base_thr, uint32_t* out, float* scale, hipStream_t s) {
  const int k = cin * kh * kw;
  weight_scale_kernel<<<cout, 256, 0, s>>>(w, k, scale);
  const int cwn = ceil_div(cin, 32);
  const int cop = cout_pad(cout);
  const int64_t total = (int64_t)kh * kw * cwn * cop;
  const dim3 grid((unsigned)((total + 255) / 256));
  Thr b = {base_thr[0], base_thr[1], base_thr[2]};
  switch (bits) {
    case 1: pack_weight_kernel<1><<<grid, 256, 0, s>>>(w, cout, cin, kh, kw, cwn, cop, b, scale, out); break;
    case 2: pack_weight_kernel<2><<<grid, 256, 0, s>>>(w, cout, cin, kh, kw, cwn, cop, b, scale, out); break;
    default: pack_weight_kernel<3><<<grid, 256, 0, s>>>(w, cout, cin, kh, kw, cwn, cop, b, scale, out); break;
  }
  uint8_t* w_i8 = reinterpret_cast<uint8_t*>(out) + wbytes_planes(cout, cin, kh, kw, bits);
  uint8_t* w_fp4 = w_i8 + wbytes_i8(cout, cin, kh, kw);
  uint8_t* w_f16 = w_fp4 + wbytes_fp4(cout, cin, kh, kw);
  const int taps = kh * kw;
  const int64_t items =
      (int64_t)taps * cwn * cop + (int64_t)taps * ((cwn + 1) / 2) * cop + (int64_t)taps * 2 * cwn * cop;
  const dim3 g2((unsigned)((items + 255) / 256));
  switch (bits) {
    case 1: expand_weight_kernel<1><<<g2, 256, 0, s>>>(out, taps, cwn, cout, cop, cin, w_i8, w_fp4, w_f16); break;
    case 2: expand_weight_kernel<2><<<g2, 256, 0, s>>>(out, taps, cwn, cout, cop, cin, w_i8, w_fp4, w_f16); break;
    default: expand_weight_kernel<4><<<g2, 256, 0, s>>>(out, taps, cwn, cout, cop, cin, w_i8, w_fp4, w_f16); break;
  }
  return hip_status();
}

}  // namespace qc
