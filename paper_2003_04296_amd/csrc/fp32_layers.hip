// fp32_layers.hip -- full-precision support layers around the quantized
// layers: the first convolution (its input is the image, which the paper
// leaves unquantized, Sec. III-E), max/average pooling and the last FC.
//
// Every output of the first conv and of the FC is one chain of
// single-rounding fused multiply-adds in a fixed input order, started from
// +0, so the result does not depend on the launch configuration.  That makes
// the binarisation after the first layer reproducible bit for bit.
#include "qconv_internal.h"

namespace qc {

namespace {

// Output channels per thread: 32 when the output is packed (one word per
// plane), 64 for fp32 outputs (each tap's scalar weight loads then feed 64
// fmaf).  The transposed weights are padded to a multiple of CONV_PAD.
constexpr int CONV_TN = 32;
constexpr int CONV_PAD = 64;

// OIHW -> [cin][k][k][cout_pad64] so that the TN weights of one tap are one
// contiguous, wave-uniform run.
__global__ void transpose_weight_kernel(const float* __restrict__ w, int cout, int cin, int kk,
                                        int cop, float* __restrict__ wt) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)cin * kk * cop;
  if (i >= total) return;
  const int co = (int)(i % cop);
  const int64_t tap = i / cop;  // ci * kk + (ky * k + kx)
  wt[i] = (co < cout) ? w[(int64_t)co * cin * kk + tap] : 0.0f;
}

template <int OUT_BITS, int TN>
__global__ __launch_bounds__(256) void conv_f32_kernel(const float* __restrict__ x,
                                                       const float* __restrict__ wt, int n, int cin,
                                                       int h, int w, int cout, int cop, int k,
                                                       int stride, int pad, int ho, int wo,
                                                       const float* __restrict__ bn_k,
                                                       const float* __restrict__ bn_b, int relu,
                                                       Thr othr, float* __restrict__ out,
                                                       uint32_t* __restrict__ out_packed) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t total = (int64_t)n * ho * wo;
  if (g >= total) return;
  const int co0 = blockIdx.y * TN;
  const int ow = (int)(g % wo);
  const int64_t r = g / wo;
  const int oh = (int)(r % ho);
  const int b = (int)(r / ho);
  float acc[TN];
#pragma unroll
  for (int j = 0; j < TN; ++j) acc[j] = 0.0f;
  const float* xb = x + (int64_t)b * cin * h * w;
  for (int ci = 0; ci < cin; ++ci) {
    for (int ky = 0; ky < k; ++ky) {
      const int ih = oh * stride - pad + ky;
      if (ih < 0 || ih >= h) continue;
      for (int kx = 0; kx < k; ++kx) {
        const int iw = ow * stride - pad + kx;
        if (iw < 0 || iw >= w) continue;
        const float xv = xb[((int64_t)ci * h + ih) * w + iw];
        const float* wp = wt + ((int64_t)(ci * k + ky) * k + kx) * cop + co0;
#pragma unroll
        for (int j = 0; j < TN; ++j) acc[j] = fmaf(xv, wp[j], acc[j]);
      }
    }
  }
  const int64_t plane = (int64_t)ho * wo;
  uint32_t words[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int j = 0; j < TN; ++j) {
    const int co = co0 + j;
    if (co >= cout) break;
    float z = fmaf(bn_k[co], acc[j], bn_b[co]);
    if (relu) z = (z > 0.0f) ? z : 0.0f;
    if constexpr (OUT_BITS == 0) {
      out[((int64_t)b * cout + co) * plane + (int64_t)oh * wo + ow] = z;
    } else {
      const uint32_t pl = quant_planes<OUT_BITS>(hardtanh(z), othr);
#pragma unroll
      for (int p = 0; p < 4; ++p) words[p] |= ((pl >> p) & 1u) << j;
    }
  }
  if constexpr (OUT_BITS != 0) {
    constexpr int P = planes_of(OUT_BITS);
    const int cwn = ceil_div(cout, 32);
    uint32_t* dst = out_packed + ((((int64_t)b * ho + oh) * wo + ow) * cwn + (co0 >> 5)) * P;
#pragma unroll
    for (int p = 0; p < P; ++p) dst[p] = words[p];
  }
}

// k x k / stride max pooling, one output per thread.  Planes (image, channel)
// come from blockIdx.y plus a loop over plane groups, positions inside a
// plane from a 32-bit division.  The window is scanned in (dy, dx) order from
// -inf with "v > m": padding never wins, a NaN never replaces the running
// maximum, and of equal values the first stays.  KC > 0: the window size is
// KC and all its loads are issued before the first compare (taps outside the
// image read the plane's first element and are masked out).
template <int KC>
__global__ __launch_bounds__(256) void maxpool_f32_kernel(const float* __restrict__ x, int64_t planes,
                                                          int h, int w, int k, int stride, int pad,
                                                          int ho, int wo, float* __restrict__ y) {
  const int pos = blockIdx.x * blockDim.x + threadIdx.x;
  if (pos >= ho * wo) return;
  const int oh = pos / wo, ow = pos - (pos / wo) * wo;
  const int ih0 = oh * stride - pad, iw0 = ow * stride - pad;
  for (int64_t bc = blockIdx.y; bc < planes; bc += gridDim.y) {
    const float* p = x + bc * h * w;
    float m = -INFINITY;
    if constexpr (KC > 0) {
      float v[KC * KC];
      bool ok[KC * KC];
#pragma unroll
      for (int dy = 0; dy < KC; ++dy)
#pragma unroll
        for (int dx = 0; dx < KC; ++dx) {
          const int ih = ih0 + dy, iw = iw0 + dx;
          ok[dy * KC + dx] = ih >= 0 && ih < h && iw >= 0 && iw < w;
          v[dy * KC + dx] = p[ok[dy * KC + dx] ? ih * w + iw : 0];
        }
#pragma unroll
      for (int t = 0; t < KC * KC; ++t)
        if (ok[t] && v[t] > m) m = v[t];
    } else {
      for (int dy = 0; dy < k; ++dy) {
        const int ih = ih0 + dy;
        if (ih < 0 || ih >= h) continue;
        for (int dx = 0; dx < k; ++dx) {
          const int iw = iw0 + dx;
          if (iw < 0 || iw >= w) continue;
          const float v = p[ih * w + iw];
          if (v > m) m = v;
        }
      }
    }
    y[bc * ho * wo + pos] = m;
  }
}

// 3 x 3 / 2 max pooling with padding 1 over rows of even width (the stem of
// ResNet-18): the lane holding output column ow reads input columns 2ow and
// 2ow + 1 of each window row as one aligned 8-byte load and takes column
// 2ow - 1 from the lane holding ow - 1 (the previous lane, in the same output
// row whenever ow > 0; a wave's first lane loads it itself), so a wave
// issues three loads per output instead of nine.  The scan order and the
// compares are those of maxpool_f32_kernel, so the results are identical.
__global__ __launch_bounds__(256) void maxpool3s2_f32_kernel(const float* __restrict__ x, int64_t planes, int h,
                                                            int w, int ho, int wo, float* __restrict__ y) {
  const int pos = blockIdx.x * blockDim.x + threadIdx.x;
  const bool live = pos < ho * wo;
  const int p = live ? pos : ho * wo - 1;  // every lane takes part in the exchange
  const int oh = p / wo, ow = p - (p / wo) * wo;
  const bool first_lane = (threadIdx.x & 63) == 0;
  for (int64_t bc = blockIdx.y; bc < planes; bc += gridDim.y) {
    const float* pl = x + bc * h * w;
    float2 v[3];
    float left[3];
    bool rok[3];
#pragma unroll
    for (int dy = 0; dy < 3; ++dy) {
      const int ih = 2 * oh - 1 + dy;
      rok[dy] = ih >= 0 && ih < h;
      const int row = rok[dy] ? ih : 0;
      v[dy] = *reinterpret_cast<const float2*>(pl + row * w + 2 * ow);
    }
#pragma unroll
    for (int dy = 0; dy < 3; ++dy) {
      left[dy] = __shfl_up(v[dy].y, 1);
      if (first_lane && ow > 0) left[dy] = pl[(rok[dy] ? 2 * oh - 1 + dy : 0) * w + 2 * ow - 1];
    }
    float m = -INFINITY;
#pragma unroll
    for (int dy = 0; dy < 3; ++dy) {
      if (!rok[dy]) continue;
      if (ow > 0 && left[dy] > m) m = left[dy];
      if (v[dy].x > m) m = v[dy].x;
      if (v[dy].y > m) m = v[dy].y;
    }
    if (live) y[bc * ho * wo + pos] = m;
  }
}

__global__ __launch_bounds__(256) void avgpool_f32_kernel(const float* __restrict__ x,
                                                          int64_t nc, int hw,
                                                          float* __restrict__ y) {
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (i >= nc) return;
  const float* p = x + i * hw;
  float s = 0.0f;
  for (int j = 0; j < hw; ++j) s += p[j];
  y[i] = s / (float)hw;
}

// The same sums for small maps (hw <= AVG_LDS_HW): a block's 64 planes are
// contiguous in memory, so its 256 threads first copy them into LDS with
// coalesced loads (all of a thread's loads issued before its first store);
// one thread per plane then sums it in order from LDS (a plane's values are
// hw words apart, odd for the odd hw of the pooled maps in use, so the 64
// lanes' reads fall in distinct banks).
constexpr int AVG_LDS_HW = 60;
constexpr int AVG_PLANES = 64;
__global__ __launch_bounds__(256) void avgpool_lds_kernel(const float* __restrict__ x, int64_t nc, int hw,
                                                          float* __restrict__ y) {
  constexpr int PER = AVG_PLANES * AVG_LDS_HW / 256;  // values per thread at most
  __shared__ float t[AVG_PLANES * AVG_LDS_HW];
  const int64_t p0 = (int64_t)blockIdx.x * AVG_PLANES;
  const int np = (int)min((int64_t)AVG_PLANES, nc - p0);
  const int total = np * hw;
  const float* src = x + p0 * hw;
  float v[PER];
#pragma unroll
  for (int u = 0; u < PER; ++u) v[u] = src[min((int)threadIdx.x + 256 * u, total - 1)];
#pragma unroll
  for (int u = 0; u < PER; ++u) {
    const int e = (int)threadIdx.x + 256 * u;
    if (e < total) t[e] = v[u];
  }
  __syncthreads();
  if ((int)threadIdx.x >= np) return;
  const float* r = t + threadIdx.x * hw;
  float s = 0.0f;
  for (int j = 0; j < hw; ++j) s += r[j];
  y[p0 + threadIdx.x] = s / (float)hw;
}

// Last FC.  Each output of each image is one sequential fmaf chain over the
// inputs, so the run time is set by the chain length, not by the flops: a
// wave owns ONE output for 64 images (lane = image) and a block of 4 waves
// owns 4 consecutive outputs.  Per chunk of inputs the block stages, with
// all of its loads in flight at once, the 64 images' inputs and the 4 weight
// rows in LDS; lanes then read their own input row (16-byte reads, padded
// rows) and the wave's weight row as a broadcast.
//
// x_bits = 0: x is fp32 [n][in].  x_bits = 1: x is the packed sign plane
// [n][ceil(in/32)] of {-1,+1} inputs (a 1x1 map), and fmaf(+-1, w, acc) is
// computed as the single-rounding add acc + (+-w).
constexpr int FC_CI_F32 = 192;           // fp32 inputs per chunk
constexpr int FC_XLD = FC_CI_F32 + 4;    // padded LDS row (floats)
constexpr int FC_CW_BIN = 32;            // packed words per chunk (1024 inputs)
constexpr int FC_XLD_BIN = FC_CW_BIN + 1;

template <int X_BITS>
__global__ __launch_bounds__(256) void fc_f32_kernel(const void* __restrict__ xin, int n, int in,
                                                    const float* __restrict__ w,
                                                    const float* __restrict__ bias, int out,
                                                    float* __restrict__ y) {
  constexpr int CI = X_BITS ? FC_CW_BIN * 32 : FC_CI_F32;
  constexpr int XWORDS = X_BITS ? 64 * FC_XLD_BIN : 64 * FC_XLD;
  __shared__ __attribute__((aligned(16))) float ws[4 * CI];
  __shared__ __attribute__((aligned(16))) uint32_t xs[XWORDS];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int b0 = blockIdx.x * 64;
  const int nb = min(64, n - b0);
  const int o = blockIdx.y * 4 + wave;
  const int oc = min(o, out - 1);
  const int ob = blockIdx.y * 4;
  float acc = 0.0f;
  // Every load of a chunk is issued before the first LDS store, and the
  // loads of chunk c + 1 are issued before the chain over chunk c, so they
  // arrive under it.  Indices are clamped into the chunk (and the batch), so
  // no load is guarded; values staged past L (or past the batch) are never
  // read.  Weights: thread -> row tid / 64 (rows past out repeat the last
  // one), columns tid % 64 + 64 u.  Inputs: thread -> row tid / 4, columns
  // tid % 4 + 4 u.
  constexpr int WU = CI / 64;
  constexpr int XCOLS = X_BITS ? FC_CW_BIN : CI;
  constexpr int XU = XCOLS / 4;
  constexpr int XLD = X_BITS ? FC_XLD_BIN : FC_XLD;
  float wv[WU];
  uint32_t xv[XU];
  auto load = [&](int c0) __attribute__((always_inline)) {
    const int L = min(CI, in - c0);
    const int xl = X_BITS ? ((L + 31) >> 5) : L;  // valid columns of the input tile
    const float* wrow = w + (int64_t)min(ob + (tid >> 6), out - 1) * in + c0;
#pragma unroll
    for (int u = 0; u < WU; ++u) wv[u] = wrow[min((tid & 63) + 64 * u, L - 1)];
    const int r = min(tid >> 2, nb - 1);
    const uint32_t* xrow;
    if constexpr (X_BITS == 0)
      xrow = static_cast<const uint32_t*>(xin) + (int64_t)(b0 + r) * in + c0;
    else
      xrow = static_cast<const uint32_t*>(xin) + (int64_t)(b0 + r) * ((in + 31) >> 5) + (c0 >> 5);
#pragma unroll
    for (int u = 0; u < XU; ++u) xv[u] = xrow[min((tid & 3) + 4 * u, xl - 1)];
  };
  load(0);
  for (int c0 = 0; c0 < in; c0 += CI) {
    const int L = min(CI, in - c0);  // inputs in this chunk
    __syncthreads();
#pragma unroll
    for (int u = 0; u < WU; ++u) ws[(tid >> 6) * CI + (tid & 63) + 64 * u] = wv[u];
#pragma unroll
    for (int u = 0; u < XU; ++u) xs[(tid >> 2) * XLD + (tid & 3) + 4 * u] = xv[u];
    __syncthreads();
    if (c0 + CI < in) load(c0 + CI);
    const float* wr = ws + wave * CI;
    if constexpr (X_BITS == 0) {
      const float* xr = reinterpret_cast<const float*>(xs) + lane * FC_XLD;
      const int L4 = L & ~3;
#pragma unroll 4
      for (int k = 0; k < L4; k += 4) {
        const float4 xv = *reinterpret_cast<const float4*>(xr + k);
        const float4 wv = *reinterpret_cast<const float4*>(wr + k);
        acc = fmaf(xv.x, wv.x, acc);
        acc = fmaf(xv.y, wv.y, acc);
        acc = fmaf(xv.z, wv.z, acc);
        acc = fmaf(xv.w, wv.w, acc);
      }
      for (int k = L4; k < L; ++k) acc = fmaf(xr[k], wr[k], acc);
    } else {
      const uint32_t* xr = xs + lane * FC_XLD_BIN;
      const int full = L >> 5;
      for (int c = 0; c < full; ++c) {
        const uint32_t neg = ~xr[c];  // bit set <=> input -1
#pragma unroll
        for (int k0 = 0; k0 < 32; k0 += 4) {
          const float4 wv = *reinterpret_cast<const float4*>(wr + 32 * c + k0);
          const float wk[4] = {wv.x, wv.y, wv.z, wv.w};
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const uint32_t sgn = (neg << (31 - k0 - k)) & 0x80000000u;
            acc = acc + __uint_as_float(__float_as_uint(wk[k]) ^ sgn);
          }
        }
      }
      if (L & 31) {
        const uint32_t neg = ~xr[full];
        for (int k = 0; k < (L & 31); ++k) {
          const uint32_t sgn = (neg << (31 - k)) & 0x80000000u;
          acc = acc + __uint_as_float(__float_as_uint(wr[32 * full + k]) ^ sgn);
        }
      }
    }
  }
  if (o < out && lane < nb) y[(int64_t)(b0 + lane) * out + o] = acc + (bias ? bias[oc] : 0.0f);
}

}  // namespace

int launch_transpose_conv_weight(const float* w, int cout, int cin, int k, float* wt,
                                 hipStream_t s) {
  const int cop = ceil_div(cout, CONV_PAD) * CONV_PAD;
  const int64_t total = (int64_t)cin * k * k * cop;
  transpose_weight_kernel<<<(unsigned)((total + 255) / 256), 256, 0, s>>>(w, cout, cin, k * k, cop,
                                                                           wt);
  return hip_status();
}

int launch_conv_f32(const float* x, const float* wt, int n, int cin, int h, int w, int cout, int k,
                    int stride, int pad, const float* bn_k, const float* bn_b, int relu,
                    int out_bits, Thr othr, float* out_f32, uint32_t* out_packed, hipStream_t s) {
  const int ho = (h + 2 * pad - k) / stride + 1, wo = (w + 2 * pad - k) / stride + 1;
  const int cop = ceil_div(cout, CONV_PAD) * CONV_PAD;
  const int64_t total = (int64_t)n * ho * wo;
  if (total == 0) return QCONV_OK;
  const unsigned gx = (unsigned)((total + 255) / 256);
#define QC_F32(B, TN)                                                                                        \
  conv_f32_kernel<B, TN><<<dim3(gx, (unsigned)ceil_div(cout, TN)), 256, 0, s>>>(                            \
      x, wt, n, cin, h, w, cout, cop, k, stride, pad, ho, wo, bn_k, bn_b, relu, othr, out_f32, out_packed)
  switch (out_bits) {
    case 0:
      if (cout > CONV_TN) QC_F32(0, 64); else QC_F32(0, 32);
      break;
    case 1: QC_F32(1, 32); break;
    case 2: QC_F32(2, 32); break;
    default: QC_F32(3, 32); break;
  }
#undef QC_F32
  return hip_status();
}

int launch_maxpool_f32(const float* x, int n, int c, int h, int w, int k, int stride, int pad,
                       float* y, hipStream_t s) {
  const int ho = (h + 2 * pad - k) / stride + 1, wo = (w + 2 * pad - k) / stride + 1;
  const int64_t planes = (int64_t)n * c;
  if ((int64_t)h * w >= ((int64_t)1 << 31)) return QCONV_EUNSUPPORTED;
  if (planes == 0 || ho < 1 || wo < 1) return QCONV_OK;
  const dim3 grid((unsigned)ceil_div(ho * wo, 256), (unsigned)(planes < 65535 ? planes : 65535));
  if (k == 3 && stride == 2 && pad == 1 && w % 2 == 0 && ((uintptr_t)x & 7u) == 0)
    maxpool3s2_f32_kernel<<<grid, 256, 0, s>>>(x, planes, h, w, ho, wo, y);
  else if (k == 3)
    maxpool_f32_kernel<3><<<grid, 256, 0, s>>>(x, planes, h, w, k, stride, pad, ho, wo, y);
  else if (k == 2)
    maxpool_f32_kernel<2><<<grid, 256, 0, s>>>(x, planes, h, w, k, stride, pad, ho, wo, y);
  else
    maxpool_f32_kernel<0><<<grid, 256, 0, s>>>(x, planes, h, w, k, stride, pad, ho, wo, y);
  return hip_status();
}

int launch_avgpool_f32(const float* x, int n, int c, int h, int w, float* y, hipStream_t s) {
  const int64_t nc = (int64_t)n * c;
  if (nc == 0) return QCONV_OK;
  if (h * w <= AVG_LDS_HW)
    avgpool_lds_kernel<<<(unsigned)((nc + AVG_PLANES - 1) / AVG_PLANES), 256, 0, s>>>(x, nc, h * w, y);
  else
    avgpool_f32_kernel<<<(unsigned)((nc + 255) / 256), 256, 0, s>>>(x, nc, h * w, y);
  return hip_status();
}

int launch_fc_f32(const void* x, int x_bits, int n, int in, const float* w, const float* bias,
                  int out, float* y, hipStream_t s) {
  if (n == 0) return QCONV_OK;
  const dim3 grid((unsigned)ceil_div(n, 64), (unsigned)ceil_div(out, 4));
  if (x_bits == 0)
    fc_f32_kernel<0><<<grid, 256, 0, s>>>(x, n, in, w, bias, out, y);
  else
    fc_f32_kernel<1><<<grid, 256, 0, s>>>(x, n, in, w, bias, out, y);
  return hip_status();
}

}  // namespace qc
