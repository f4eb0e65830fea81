// conv_bitplane.hip -- the layer product of Algorithm 1 (inference branch)
// on channel-packed bitplanes with VALU bit operations (Sec. III-C: the
// multiplies become XNOR for 1-2 bit operands and SHIFT for 3-bit ones;
// Sec. IV-C gives the choice by bitwidth).
//
// A level is l = (2S - 1) * sum_j 2^e_j E_j with sign plane S and one-hot
// magnitude planes E_j (implicitly all ones for 1 bit).  For one 32-channel
// word of activation a and weight w, with X = S_a xor S_w and M_jr = E_j^a & E_r^w:
//     sum_c a_c w_c = sum_{j,r} 2^(e_j+e_r) (pc(M_jr) - 2 pc(M_jr & X)).
// For 1W1A this is K - 2 pc(X) summed over the receptive field.  For 3W3A
// the pairs with equal e_j + e_r are merged first (the masks are disjoint
// because magnitudes are one-hot), which gives five shift classes.
//
// This kernel serves every bitplane layer the LDS-tiled XNOR kernel
// (conv_xnor.hip) does not: 3-bit operands (SHIFT), packed or pooled
// outputs, other kernel sizes and strides.
//
// Work mapping: one lane = one output pixel (or one 2x2 pooling window,
// walked pixel by pixel), one wave = TN consecutive output channels, so the
// weight words of a (tap, word) step are wave-uniform and come in through
// the scalar cache into SGPRs; activation words are per-lane vector loads
// (L1/L2 cached; neighbouring taps and channel tiles re-read the same lines).
// The epilogue ({QConv-pool-BN-HardTanh} / {QConv-BN-HardTanh}, Sec. III-E)
// runs in registers before the only store.
#include <type_traits>

#include <stdio.h>
#include <string.h>

#include "qconv_internal.h"

namespace qc {

namespace {

template <int PA, int PW>
struct Pairing {
  static constexpr int NA = (PA == 1) ? 1 : PA - 1;  // magnitude planes of a
  static constexpr int NW = (PW == 1) ? 1 : PW - 1;
  static constexpr int MAXE_A = (PA == 4) ? 2 : 0;
  static constexpr int MAXE_W = (PW == 4) ? 2 : 0;
  static constexpr int NCLS = MAXE_A + MAXE_W + 1;  // shift classes when both have masks
};

template <int PA, int PW>
constexpr int default_tn() {
  return (PA == 4 && PW == 4) ? 8 : ((PA == 4 || PW == 4) ? 16 : 32);
}

__device__ __forceinline__ uint32_t quant_planes_rt(float z, int bits, Thr t) {
  if (bits == 1) return quant_planes<1>(z, t);
  if (bits == 2) return quant_planes<2>(z, t);
  return quant_planes<3>(z, t);
}

// Accumulator of one output pixel over the whole receptive field, for TN
// channels starting at co0.  Returns acc in code units in acc[].
template <int PA, int PW, int TN>
__device__ __forceinline__ void dot_pixel(const ConvArgs& a, const uint32_t* __restrict__ actb,
                                          const uint32_t* __restrict__ wbase, int oh, int ow,
                                          int32_t (&acc)[TN]) {
  using PP = Pairing<PA, PW>;
  constexpr bool BOTH_MASK = (PA > 1 && PW > 1);
  // counters
  uint32_t cx[TN][BOTH_MASK ? PP::NCLS : (PA > 1 ? PP::NA : PP::NW)];
  uint32_t cm[BOTH_MASK ? TN : 1][BOTH_MASK ? PP::NCLS : 1];
  uint32_t cma[PP::NA];        // activation-only mask counts (PW == 1)
  uint32_t cmw[TN][PP::NW];    // weight-only mask counts (PA == 1)
  constexpr int NCX = BOTH_MASK ? PP::NCLS : (PA > 1 ? PP::NA : PP::NW);
#pragma unroll
  for (int n = 0; n < TN; ++n) {
#pragma unroll
    for (int q = 0; q < NCX; ++q) cx[n][q] = 0u;
#pragma unroll
    for (int q = 0; q < PP::NW; ++q) cmw[n][q] = 0u;
  }
#pragma unroll
  for (int n = 0; n < (BOTH_MASK ? TN : 1); ++n)
#pragma unroll
    for (int q = 0; q < (BOTH_MASK ? PP::NCLS : 1); ++q) cm[n][q] = 0u;
#pragma unroll
  for (int j = 0; j < PP::NA; ++j) cma[j] = 0u;

  const int apix = a.cw * PA;
  const int wstep = a.cop * PW;
  for (int ky = 0; ky < a.kh; ++ky) {
    const int ih = oh * a.stride - a.pad + ky;
    const bool rok = (ih >= 0) && (ih < a.h);
    for (int kx = 0; kx < a.kw; ++kx) {
      const int iw = ow * a.stride - a.pad + kx;
      const bool ok = rok && (iw >= 0) && (iw < a.w);
      // Out-of-range taps read word 0 of the image (always valid memory) and
      // are replaced by 0, which is the padding level Q(0) in every encoding.
      const uint32_t* ap = actb + (ok ? ((int64_t)ih * a.w + iw) * apix : 0);
      const uint32_t* wk = wbase + (int64_t)((ky * a.kw + kx) * a.cw) * wstep;
      for (int c = 0; c < a.cw; ++c) {
        uint32_t av[PA];
#pragma unroll
        for (int p = 0; p < PA; ++p) {
          const uint32_t v = ap[c * PA + p];
          av[p] = ok ? v : 0u;
        }
        if constexpr (PA > 1 && PW == 1) {
#pragma unroll
          for (int j = 0; j < PP::NA; ++j) cma[j] += __builtin_popcount(av[1 + j]);
        }
        const uint32_t* wc = wk + (int64_t)c * wstep;
#pragma unroll
        for (int n = 0; n < TN; ++n) {
          uint32_t wv[PW];
#pragma unroll
          for (int q = 0; q < PW; ++q) wv[q] = wc[n * PW + q];
          const uint32_t x = av[0] ^ wv[0];
          if constexpr (PA == 1 && PW == 1) {
            cx[n][0] += __builtin_popcount(x);
          } else if constexpr (PW == 1) {
#pragma unroll
            for (int j = 0; j < PP::NA; ++j) cx[n][j] += __builtin_popcount(x & av[1 + j]);
          } else if constexpr (PA == 1) {
#pragma unroll
            for (int r = 0; r < PP::NW; ++r) {
              cx[n][r] += __builtin_popcount(x & wv[1 + r]);
              cmw[n][r] += __builtin_popcount(wv[1 + r]);
            }
          } else {
#pragma unroll
            for (int cls = 0; cls < PP::NCLS; ++cls) {
              uint32_t m = 0u;
#pragma unroll
              for (int j = 0; j < PP::NA; ++j)
#pragma unroll
                for (int r = 0; r < PP::NW; ++r)
                  if (plane_exp(PA, 1 + j) + plane_exp(PW, 1 + r) == cls) m |= av[1 + j] & wv[1 + r];
              cm[n][cls] += __builtin_popcount(m);
              cx[n][cls] += __builtin_popcount(m & x);
            }
          }
        }
      }
    }
  }
  // shift-combine
#pragma unroll
  for (int n = 0; n < TN; ++n) {
    int32_t v = 0;
    if constexpr (PA == 1 && PW == 1) {
      v = a.kreal - 2 * (int32_t)cx[n][0];
    } else if constexpr (PW == 1) {
#pragma unroll
      for (int j = 0; j < PP::NA; ++j)
        v += ((int32_t)cma[j] - 2 * (int32_t)cx[n][j]) << plane_exp(PA, 1 + j);
    } else if constexpr (PA == 1) {
#pragma unroll
      for (int r = 0; r < PP::NW; ++r)
        v += ((int32_t)cmw[n][r] - 2 * (int32_t)cx[n][r]) << plane_exp(PW, 1 + r);
    } else {
#pragma unroll
      for (int cls = 0; cls < PP::NCLS; ++cls)
        v += ((int32_t)cm[n][cls] - 2 * (int32_t)cx[n][cls]) << cls;
    }
    acc[n] = v;
  }
}

template <int PA, int PW, int TN, bool POOL>
__global__ __launch_bounds__(256) void conv_bitplane_kernel(const ConvArgs a) {
  const int64_t g = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const int64_t groups = (int64_t)a.n * a.oh_out * a.ow_out;
  if (g >= groups) return;
  const int co0 = blockIdx.y * TN;
  const int px = (int)(g % a.ow_out);
  const int64_t r = g / a.ow_out;
  const int py = (int)(r % a.oh_out);
  const int b = (int)(r / a.oh_out);

  const uint32_t* actb = a.act + (int64_t)b * a.h * a.w * a.cw * PA;
  const uint32_t* wbase = a.wt + (int64_t)co0 * PW;

  int32_t best[TN];
  constexpr int TP = POOL ? 4 : 1;
#pragma unroll 1
  for (int t = 0; t < TP; ++t) {
    const int oh = POOL ? 2 * py + (t >> 1) : py;
    const int ow = POOL ? 2 * px + (t & 1) : px;
    int32_t acc[TN];
    dot_pixel<PA, PW, TN>(a, actb, wbase, oh, ow, acc);
#pragma unroll
    for (int n = 0; n < TN; ++n) best[n] = (t == 0) ? acc[n] : max(best[n], acc[n]);
  }

  // ---- epilogue ----
  const float inv = 1.0f / (float)(1 << a.shift);  // exact power of two
  const int64_t plane = (int64_t)a.oh_out * a.ow_out;
  const int64_t obase = (int64_t)b * a.cout * plane + (int64_t)py * a.ow_out + px;
  const int pout = planes_of(a.out_bits);
  uint32_t ow_words[4] = {0u, 0u, 0u, 0u};
  const bool want_pack = (a.mode == QCONV_EPI_BN_PACK) || (a.out_packed != nullptr);
#pragma unroll
  for (int n = 0; n < TN; ++n) {
    const int co = co0 + n;
    if (co >= a.cout) break;
    const int64_t oi = obase + (int64_t)co * plane;
    if (a.mode == QCONV_EPI_INT32) {
      static_cast<int32_t*>(a.out)[oi] = best[n];
      continue;
    }
    const float ar = (float)best[n] * inv;
    if (a.mode == QCONV_EPI_SCALE_F32) {
      static_cast<float*>(a.out)[oi] = a.scale[co] * ar;
      continue;
    }
    float z = fmaf(a.bn_k[co], ar, a.bn_b[co]);
    if (a.mode == QCONV_EPI_BN_F32) {
      if (a.residual_on) z = z + a.residual[oi];
      static_cast<float*>(a.out)[oi] = z;
    }
    if (want_pack) {
      const uint32_t pl = quant_planes_rt(hardtanh(z), a.out_bits, a.othr);
#pragma unroll
      for (int p = 0; p < 4; ++p) ow_words[p] |= ((pl >> p) & 1u) << n;
    }
  }
  if (want_pack) {
    const int64_t wbase_o = (((int64_t)b * a.oh_out + py) * a.ow_out + px) * a.out_cw + (co0 >> 5);
    if constexpr (TN == 32) {
      uint32_t* dst = a.out_packed + wbase_o * pout;
      for (int p = 0; p < pout; ++p) dst[p] = ow_words[p];
    } else {
      // Sub-word store of this tile's TN channels.  The tile holding the last
      // channel also clears the rest of that word (no tile covers those
      // channels, and bits past the last channel must read 0).
      constexpr int SUBS = 32 / TN;
      const int sub = (co0 & 31) / TN;
      const int last_sub = (co0 + TN >= a.cout) ? SUBS - 1 : sub;
      using sub_t = typename std::conditional<TN == 16, uint16_t, uint8_t>::type;
      sub_t* dst = reinterpret_cast<sub_t*>(a.out_packed + wbase_o * pout);
      for (int p = 0; p < pout; ++p) {
        dst[SUBS * p + sub] = (sub_t)ow_words[p];
        for (int s2 = sub + 1; s2 <= last_sub; ++s2) dst[SUBS * p + s2] = (sub_t)0;
      }
    }
  }
}

template <int PA, int PW>
int launch_pp(const ConvArgs& a, hipStream_t s) {
  constexpr int TN = default_tn<PA, PW>();
  const int64_t groups = (int64_t)a.n * a.oh_out * a.ow_out;
  if (groups == 0) return QCONV_OK;
  const dim3 grid((unsigned)((groups + 255) / 256), (unsigned)ceil_div(a.cout, TN));
  if (a.pool)
    conv_bitplane_kernel<PA, PW, TN, true><<<grid, 256, 0, s>>>(a);
  else
    conv_bitplane_kernel<PA, PW, TN, false><<<grid, 256, 0, s>>>(a);
  return hip_status();
}

}  // namespace

int bitplane_kernel_name(const ConvArgs& a, char* buf, int len) {
  if (xnor_supports(a)) return xnor_kernel_name(a, buf, len);
  const int pa = planes_of(a.a_bits), pw = planes_of(a.w_bits);
  int tn = 0;
#define QC_CASE(A, W) \
  if (pa == A && pw == W) tn = default_tn<A, W>();
  QC_CASE(1, 1)
  QC_CASE(2, 1)
  QC_CASE(1, 2)
  QC_CASE(2, 2)
  QC_CASE(4, 4)
  QC_CASE(4, 1)
  QC_CASE(1, 4)
  QC_CASE(4, 2)
  QC_CASE(2, 4)
#undef QC_CASE
  if (!tn) return QCONV_EUNSUPPORTED;
  char name[96];
  snprintf(name, sizeof(name), "conv_bitplane_kernel<%d, %d, %d, %s>", pa, pw, tn, a.pool ? "true" : "false");
  if (buf && len > 0) snprintf(buf, (size_t)len, "%s", name);
  return (int)strlen(name);
}

int launch_conv_bitplane(const ConvArgs& a, hipStream_t s) {
  if (xnor_supports(a)) return launch_conv_xnor(a, s);
  const int pa = planes_of(a.a_bits), pw = planes_of(a.w_bits);
#define QC_CASE(A, W) \
  if (pa == A && pw == W) return launch_pp<A, W>(a, s);
  QC_CASE(1, 1)
  QC_CASE(2, 1)
  QC_CASE(1, 2)
  QC_CASE(2, 2)
  QC_CASE(4, 4)
  QC_CASE(4, 1)
  QC_CASE(1, 4)
  QC_CASE(4, 2)
  QC_CASE(2, 4)
#undef QC_CASE
  return QCONV_EUNSUPPORTED;
}

}  // namespace qc
