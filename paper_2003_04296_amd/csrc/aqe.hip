// aqe.hip -- the elementwise steps of training with the asymptotic-quantized
// estimator (Sec. III-B and III-D; Eqs. activation and weight; Algorithm 1,
// training branch):
//   forward   y  = alpha h(x) + (1 - alpha) x      (h: the level of Q_bits)
//   backward  gx = 2 alpha gy 1{|x| <= 1}
//   update    w  = clip(w - lr g, -1, 1)           (plain SGD, then the clip)
// Each is one pass over HBM; four values per thread when every pointer is
// 16-byte aligned.
#include "qconv_internal.h"

namespace qc {

namespace {

// Level of Q_bits(x) as a float: +-1, 0, +-1/2, +-1/4 (the same compares and
// tie rules as the packing kernels).
template <int BITS>
__device__ __forceinline__ float level_of(float x, Thr t) {
  const uint32_t pl = quant_planes<BITS>(x, t);
  const float sgn = (pl & 1u) ? 1.0f : -1.0f;
  if constexpr (BITS == 1) {
    return sgn;
  } else if constexpr (BITS == 2) {
    return (pl & 2u) ? sgn : 0.0f;
  } else {
    if (pl & 2u) return sgn;
    if (pl & 4u) return 0.5f * sgn;
    if (pl & 8u) return 0.25f * sgn;
    return 0.0f;
  }
}

// Thresholds of group g: the activation set, or the weight base set scaled
// by s_g in double with one rounding (as the weight packing does).
__device__ __forceinline__ Thr group_thr(Thr base, const float* scale, int64_t i, int64_t group) {
  if (!scale) return base;
  const double s = (double)scale[i / group];
  Thr t;
  t.t0 = (float)((double)base.t0 * s);
  t.t1 = (float)((double)base.t1 * s);
  t.t2 = (float)((double)base.t2 * s);
  return t;
}

template <int BITS>
__device__ __forceinline__ float aqe_value(float x, Thr t, float alpha, float om) {
  const float a = alpha * level_of<BITS>(x, t);
  const float b = om * x;
  return a + b;
}

template <int BITS, int VEC>
__global__ __launch_bounds__(256) void aqe_forward_kernel(const float* __restrict__ x, int64_t n, Thr base,
                                                          const float* __restrict__ scale, int64_t group,
                                                          float alpha, float om, float* __restrict__ y) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i * VEC < n; i += stride) {
    if constexpr (VEC == 4) {
      if (i * 4 + 3 < n) {
        const float4 v = reinterpret_cast<const float4*>(x)[i];
        float4 o;
        o.x = aqe_value<BITS>(v.x, group_thr(base, scale, 4 * i, group), alpha, om);
        o.y = aqe_value<BITS>(v.y, group_thr(base, scale, 4 * i + 1, group), alpha, om);
        o.z = aqe_value<BITS>(v.z, group_thr(base, scale, 4 * i + 2, group), alpha, om);
        o.w = aqe_value<BITS>(v.w, group_thr(base, scale, 4 * i + 3, group), alpha, om);
        reinterpret_cast<float4*>(y)[i] = o;
        continue;
      }
      for (int64_t j = 4 * i; j < n; ++j) y[j] = aqe_value<BITS>(x[j], group_thr(base, scale, j, group), alpha, om);
    } else {
      y[i] = aqe_value<BITS>(x[i], group_thr(base, scale, i, group), alpha, om);
    }
  }
}

__device__ __forceinline__ float aqe_grad(float x, float g, float twoa) {
  return fabsf(x) <= 1.0f ? twoa * g : 0.0f;
}

template <int VEC>
__global__ __launch_bounds__(256) void aqe_backward_kernel(const float* __restrict__ x, const float* __restrict__ gy,
                                                           int64_t n, float twoa, float* __restrict__ gx) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i * VEC < n; i += stride) {
    if constexpr (VEC == 4) {
      if (i * 4 + 3 < n) {
        const float4 v = reinterpret_cast<const float4*>(x)[i];
        const float4 g = reinterpret_cast<const float4*>(gy)[i];
        reinterpret_cast<float4*>(gx)[i] =
            make_float4(aqe_grad(v.x, g.x, twoa), aqe_grad(v.y, g.y, twoa), aqe_grad(v.z, g.z, twoa),
                        aqe_grad(v.w, g.w, twoa));
        continue;
      }
      for (int64_t j = 4 * i; j < n; ++j) gx[j] = aqe_grad(x[j], gy[j], twoa);
    } else {
      gx[i] = aqe_grad(x[i], gy[i], twoa);
    }
  }
}

// w - lr g, then clipped to [-1, 1] with two compares (a NaN passes through).
__device__ __forceinline__ float sgd_clip(float w, float g, float lr) {
  float v = w - lr * g;
  if (v > 1.0f) v = 1.0f;
  if (v < -1.0f) v = -1.0f;
  return v;
}

template <int VEC>
__global__ __launch_bounds__(256) void aqe_sgd_clip_kernel(float* __restrict__ w, const float* __restrict__ g,
                                                           int64_t n, float lr) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i * VEC < n; i += stride) {
    if constexpr (VEC == 4) {
      if (i * 4 + 3 < n) {
        const float4 v = reinterpret_cast<const float4*>(w)[i];
        const float4 d = reinterpret_cast<const float4*>(g)[i];
        reinterpret_cast<float4*>(w)[i] =
            make_float4(sgd_clip(v.x, d.x, lr), sgd_clip(v.y, d.y, lr), sgd_clip(v.z, d.z, lr), sgd_clip(v.w, d.w, lr));
        continue;
      }
      for (int64_t j = 4 * i; j < n; ++j) w[j] = sgd_clip(w[j], g[j], lr);
    } else {
      w[i] = sgd_clip(w[i], g[i], lr);
    }
  }
}

bool aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

// Blocks of a grid-stride launch over `units` work units: enough to fill the
// chip several times over, never more than the units.
unsigned grid_for(int64_t units) {
  const int64_t b = (units + 255) / 256;
  return (unsigned)(b < 8192 ? b : 8192);
}

}  // namespace

int launch_aqe_forward(const float* x, int64_t n, int bits, float alpha, Thr base, const float* scale,
                       int64_t group, float* y, hipStream_t s) {
  if (n == 0) return QCONV_OK;
  const float om = 1.0f - alpha;
  const bool vec = aligned16(x) && aligned16(y);
  const int64_t units = vec ? (n + 3) / 4 : n;
#define QC_AQE(B)                                                                                         \
  do {                                                                                                    \
    if (vec)                                                                                              \
      aqe_forward_kernel<B, 4><<<grid_for(units), 256, 0, s>>>(x, n, base, scale, group, alpha, om, y);  \
    else                                                                                                  \
      aqe_forward_kernel<B, 1><<<grid_for(units), 256, 0, s>>>(x, n, base, scale, group, alpha, om, y);  \
  } while (0)
  if (bits == 1) QC_AQE(1);
  else if (bits == 2) QC_AQE(2);
  else QC_AQE(3);
#undef QC_AQE
  return hip_status();
}

int launch_aqe_backward(const float* x, const float* gy, int64_t n, float alpha, float* gx, hipStream_t s) {
  if (n == 0) return QCONV_OK;
  const float twoa = 2.0f * alpha;
  if (aligned16(x) && aligned16(gy) && aligned16(gx))
    aqe_backward_kernel<4><<<grid_for((n + 3) / 4), 256, 0, s>>>(x, gy, n, twoa, gx);
  else
    aqe_backward_kernel<1><<<grid_for(n), 256, 0, s>>>(x, gy, n, twoa, gx);
  return hip_status();
}

int launch_aqe_sgd_clip(float* w, const float* g, int64_t n, float lr, hipStream_t s) {
  if (n == 0) return QCONV_OK;
  if (aligned16(w) && aligned16(g))
    aqe_sgd_clip_kernel<4><<<grid_for((n + 3) / 4), 256, 0, s>>>(w, g, n, lr);
  else
    aqe_sgd_clip_kernel<1><<<grid_for(n), 256, 0, s>>>(w, g, n, lr);
  return hip_status();
}

}  // namespace qc
