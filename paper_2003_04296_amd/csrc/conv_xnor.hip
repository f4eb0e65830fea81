// conv_xnor.hip -- the layer product of Algorithm 1 (inference branch) as
// XNOR/AND + popcount over channel-packed bitplanes on the VALU, for 1- and
// 2-bit operands (Sec. III-C: XNOR replaces the multiply; Sec. IV-C and
// Tables I-II: XNOR is the operation whenever the smaller width is <= 2).
//
// Per 32-channel word pair (sign planes S, nonzero masks M; a 1-bit operand
// has M = all ones):
//   sum_c a_c w_c = pc(M_a & M_w) - 2 pc(M_a & M_w & (S_a xor S_w)),
// which gfx950 evaluates with v_bitop3_b32 (any 3-input bit function in one
// instruction) and v_bcnt_u32_b32 (popcount plus an accumulator):
//   1W1A  xor, bcnt                        (pc(M) = K is a constant)
//   2W1A  bitop3((Sa^Sw)&Ma), bcnt         (pc(Ma) counted once per pixel)
//   1W2A  bitop3((Sa^Sw)&Mw), bcnt         (pc(Mw) counted once per channel)
//   2W2A  and, bitop3, bcnt, bcnt
//
// Block: an 8 x 8 tile of output pixels of one image x CO_B = 128 / KS output
// channels, 256 threads.  The packed halo tile and the block's weights are
// staged in LDS chunk by chunk of input words (both read from HBM once per
// block, coalesced).  A thread owns 4 consecutive pixels of a row x 8
// channels (32 accumulators per counter), reading 4 activation words and 8
// weight words per plane from LDS per (tap, word) step (weight reads are
// broadcasts within a channel group).  KS adjacent lanes split the (tap,
// word) steps of the same outputs and their counters are summed with DPP
// quad permutations (xor 1, xor 2), so small layers still give every CU
// several waves; each of the KS lanes then runs the epilogue for 8 / KS of
// the channels.  Blocks are renumbered so that the channel tiles of one
// pixel tile run on the same XCD (its L2 holds the halo).
//
// Epilogues: int32 accumulators, s_c * acc, BN fmaf (+ fp32 residual); the
// packed and pooled epilogues stay with conv_bitplane_kernel.
#include <stdio.h>
#include <string.h>

#include <type_traits>

#include "qconv_internal.h"

namespace qc {

namespace {

constexpr int XT = 8;         // output tile side of 3x3 layers (th = tw = 8)
constexpr int XNC = 8;        // channels per thread
constexpr int XMP = 4;        // pixels per thread (one row segment)
constexpr int XCHUNK_LDS = 48 * 1024;  // LDS budget of one block's staged chunk

struct XArgs {
  ConvArgs c;
  int tiles_x, tiles_y, co_tiles;
  int th, tw, gshift;  // output tile rows x columns (th * tw = 64); log2 of the 4-pixel groups per row
  int cwc, nchunks;  // input words staged per chunk
  int hr, hc, hcs;   // halo rows, columns, LDS words per (word, plane) row segment
  int half;          // stride 2: columns stored by parity, odd ones from `half`
  int k1;            // 1x1 kernel: only the sampled pixels are staged (halo = the tile)
  int act_words;     // LDS words of the staged activations (per chunk)
  int nblocks;
  int xcd_remap;     // renumber blocks so consecutive logical ids share an XCD
};

// LDS column of halo column hcol (stride 2: even columns first, then odd).
__device__ __forceinline__ int halo_col(int hcol, int stride, int half) {
  return stride == 2 ? (hcol & 1) * half + (hcol >> 1) : hcol;
}

template <int PA, int PW, int KS>
__global__ __launch_bounds__(256) void conv_xnor_kernel(const XArgs x) {
  constexpr int CO_B = 128 / KS;
  constexpr bool MA = PA > 1, MW = PW > 1;  // operands with a nonzero mask
  extern __shared__ __attribute__((aligned(16))) uint32_t xlds[];
  const ConvArgs& a = x.c;
  // block -> (image, pixel tile, channel tile); the channel tile varies fastest
  int bid = blockIdx.x;
  if (x.xcd_remap) {
    const int per = x.nblocks / 8;
    bid = (bid & 7) * per + (bid >> 3);
  }
  const int ct = bid % x.co_tiles;
  int rest = bid / x.co_tiles;
  const int tx = rest % x.tiles_x;
  rest /= x.tiles_x;
  const int ty = rest % x.tiles_y;
  const int img = rest / x.tiles_y;
  const int co_blk = ct * CO_B;
  const int oy0 = ty * x.th, ox0 = tx * x.tw;
  const int iy0 = oy0 * a.stride - a.pad, ix0 = ox0 * a.stride - a.pad;

  const int tid = threadIdx.x;
  const int ks = tid % KS;
  const int pg = (tid / KS) % 16;  // pixel group: row pg / (tw / 4), columns 4 (pg % (tw / 4)) ..
  const int cg = tid / (16 * KS);  // channel group: channels 8 cg .. 8 cg + 7 of the block
  const int prow = pg >> x.gshift, pcol = (pg & ((1 << x.gshift) - 1)) * XMP;

  uint32_t* act_l = xlds;                   // [cwc][PA][hr][hcs]
  uint32_t* wt_l = xlds + x.act_words;      // [tap][cwc][CO_B][PW]
  // the epilogue's per-channel parameters: [0, CO_B) k or s_c, [CO_B, 2 CO_B) b
  float* ep_l = reinterpret_cast<float*>(xlds + x.act_words + a.kh * a.kw * x.cwc * CO_B * PW);
  const int taps = a.kh * a.kw;
  const int plane_words = x.hr * x.hcs;

  uint32_t cx[XMP][XNC], cm[MA && MW ? XMP : 1][MA && MW ? XNC : 1];
  uint32_t cma[MA && !MW ? XMP : 1], cmw[MW && !MA ? XNC : 1];
#pragma unroll
  for (int i = 0; i < XMP; ++i)
#pragma unroll
    for (int n = 0; n < XNC; ++n) cx[i][n] = 0u;
  if constexpr (MA && MW) {
#pragma unroll
    for (int i = 0; i < XMP; ++i)
#pragma unroll
      for (int n = 0; n < XNC; ++n) cm[i][n] = 0u;
  }
  cma[0] = 0u;
#pragma unroll
  for (int i = 0; i < (MA && !MW ? XMP : 1); ++i) cma[i] = 0u;
#pragma unroll
  for (int n = 0; n < (MW && !MA ? XNC : 1); ++n) cmw[n] = 0u;

  const int64_t apix = (int64_t)a.cw * PA;
  const uint32_t* actb = a.act + (int64_t)img * a.h * a.w * apix;
  for (int chunk = 0; chunk < x.nchunks; ++chunk) {
    const int cw0 = chunk * x.cwc;
    const int ncw = min(x.cwc, a.cw - cw0);
    const int hpix = x.hr * x.hc;
    const int wrows = taps * ncw;
    // halo word `it` of this chunk (0 outside the image = Q(0)): its LDS
    // slot and, inside the image, its source
    auto halo_item = [&](int it, const uint32_t** src) __attribute__((always_inline)) {
      const int c = it % ncw;  // consecutive threads: consecutive words of one pixel
      const int hp = it / ncw;
      const int hrow = hp / x.hc, hcol = hp - (hp / x.hc) * x.hc;
      const int step = x.k1 ? a.stride : 1;
      const int iy = iy0 + hrow * step, ix = ix0 + hcol * step;
      *src = (iy >= 0 && iy < a.h && ix >= 0 && ix < a.w)
                 ? actb + ((int64_t)iy * a.w + ix) * apix + (int64_t)(cw0 + c) * PA
                 : nullptr;
      const int col = x.k1 ? hcol : halo_col(hcol, a.stride, x.half);
      return c * PA * plane_words + hrow * x.hcs + col;
    };
    // weight word `it` of this chunk, [tap][word][channel][plane] (rows past
    // cout are 0 in the packed layout: cop >= co_blk + CO_B)
    auto wt_item = [&](int it, const uint32_t** src) __attribute__((always_inline)) {
      const int col = it % CO_B;
      const int r = it / CO_B;
      const int tap = r / ncw, c = r - (r / ncw) * ncw;
      *src = a.wt + ((int64_t)(tap * a.cw + cw0 + c) * a.cop + co_blk + col) * PW;
      return ((tap * x.cwc + c) * CO_B + col) * PW;
    };
    auto ld = [](const uint32_t* src, uint32_t* v, auto np) __attribute__((always_inline)) {
      constexpr int NP = decltype(np)::value;
      if constexpr (NP == 1) {
        v[0] = src ? src[0] : 0u;
      } else {
        const uint2 u = src ? *reinterpret_cast<const uint2*>(src) : make_uint2(0u, 0u);
        v[0] = u.x;
        v[1] = u.y;
      }
    };
    // ---- stage the chunk: the first halo word and weight word of every
    // thread are both in flight before either is stored ----
    {
      uint32_t va[PA], vw[PW];
      const uint32_t *sa = nullptr, *sw = nullptr;
      int da = 0, dw = 0;
      if (tid < hpix * ncw) da = halo_item(tid, &sa);
      if (tid < wrows * CO_B) dw = wt_item(tid, &sw);
      ld(sa, va, std::integral_constant<int, PA>());
      if (tid < wrows * CO_B) ld(sw, vw, std::integral_constant<int, PW>());
      // with the first chunk, the epilogue parameters of the block's channels
      const bool pt = chunk == 0 && tid < 2 * CO_B && a.mode != QCONV_EPI_INT32;
      float pv = 0.0f;
      if (pt) {
        const int col = tid % CO_B, co = co_blk + col;
        const float* src = a.mode == QCONV_EPI_SCALE_F32 ? a.scale : (tid < CO_B ? a.bn_k : a.bn_b);
        if (co < a.cout && (tid < CO_B || a.mode != QCONV_EPI_SCALE_F32)) pv = src[co];
      }
      if (pt) ep_l[tid] = pv;
      if (tid < hpix * ncw) {
#pragma unroll
        for (int p = 0; p < PA; ++p) act_l[da + p * plane_words] = va[p];
      }
      if (tid < wrows * CO_B) {
#pragma unroll
        for (int p = 0; p < PW; ++p) wt_l[dw + p] = vw[p];
      }
    }
    for (int it = tid + 256; it < hpix * ncw; it += 256) {
      const uint32_t* sa;
      const int da = halo_item(it, &sa);
      uint32_t va[PA];
      ld(sa, va, std::integral_constant<int, PA>());
#pragma unroll
      for (int p = 0; p < PA; ++p) act_l[da + p * plane_words] = va[p];
    }
    for (int it = tid + 256; it < wrows * CO_B; it += 256) {
      const uint32_t* sw;
      const int dw = wt_item(it, &sw);
      uint32_t vw[PW];
      ld(sw, vw, std::integral_constant<int, PW>());
#pragma unroll
      for (int p = 0; p < PW; ++p) wt_l[dw + p] = vw[p];
    }
    __syncthreads();

    // ---- this lane's (tap, word) steps: s = ks, ks + KS, ... ----
    const int nsteps = taps * ncw;
    int tap = 0, c = ks;
    while (c >= ncw) {  // ncw may be smaller than KS
      c -= ncw;
      ++tap;
    }
    for (int s = ks; s < nsteps; s += KS) {
      const int ky = tap / a.kw, kx = tap - (tap / a.kw) * a.kw;
      // activation words of the 4 pixels: halo row prow*stride + ky, columns (pcol + i)*stride + kx
      int hrow, col0;
      if (x.k1) {
        hrow = prow;
        col0 = pcol;
      } else {
        hrow = prow * a.stride + ky;
        col0 = halo_col(pcol * a.stride + kx, a.stride, x.half);
      }
      uint32_t av[PA][XMP];
#pragma unroll
      for (int p = 0; p < PA; ++p) {
        const uint32_t* ap = act_l + (c * PA + p) * plane_words + hrow * x.hcs + col0;
#pragma unroll
        for (int i = 0; i < XMP; ++i) av[p][i] = ap[i];
      }
      uint32_t wv[PW][XNC];
      const uint4* wp = reinterpret_cast<const uint4*>(wt_l + ((tap * x.cwc + c) * CO_B + cg * XNC) * PW);
#pragma unroll
      for (int q = 0; q < XNC * PW / 4; ++q) {
        const uint4 u = wp[q];
        const uint32_t e[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const int flat = 4 * q + r;  // channel flat / PW, plane flat % PW
          wv[flat % PW][flat / PW] = e[r];
        }
      }
      if constexpr (MA && !MW) {
#pragma unroll
        for (int i = 0; i < XMP; ++i) cma[i] += __builtin_popcount(av[1][i]);
      }
      if constexpr (MW && !MA) {
#pragma unroll
        for (int n = 0; n < XNC; ++n) cmw[n] += __builtin_popcount(wv[1][n]);
      }
#pragma unroll
      for (int i = 0; i < XMP; ++i)
#pragma unroll
        for (int n = 0; n < XNC; ++n) {
          const uint32_t xs = av[0][i] ^ wv[0][n];
          if constexpr (!MA && !MW) {
            cx[i][n] += __builtin_popcount(xs);
          } else if constexpr (MA && !MW) {
            cx[i][n] += __builtin_popcount(xs & av[1][i]);
          } else if constexpr (!MA && MW) {
            cx[i][n] += __builtin_popcount(xs & wv[1][n]);
          } else {
            const uint32_t m = av[1][i] & wv[1][n];
            cm[i][n] += __builtin_popcount(m);
            cx[i][n] += __builtin_popcount(xs & m);
          }
        }
      c += KS;
      while (c >= ncw) {
        c -= ncw;
        ++tap;
      }
    }
    __syncthreads();
  }

  // ---- sum the KS lanes' counters (DPP quad permutations: xor 1, xor 2) ----
  auto red = [&](uint32_t& v) __attribute__((always_inline)) {
    if constexpr (KS >= 2) v += (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0xB1, 0xF, 0xF, false);
    if constexpr (KS >= 4) v += (uint32_t)__builtin_amdgcn_mov_dpp((int)v, 0x4E, 0xF, 0xF, false);
  };
#pragma unroll
  for (int i = 0; i < XMP; ++i)
#pragma unroll
    for (int n = 0; n < XNC; ++n) {
      red(cx[i][n]);
      if constexpr (MA && MW) red(cm[i][n]);
    }
  if constexpr (MA && !MW) {
#pragma unroll
    for (int i = 0; i < XMP; ++i) red(cma[i]);
  }
  if constexpr (MW && !MA) {
#pragma unroll
    for (int n = 0; n < XNC; ++n) red(cmw[n]);
  }

  // ---- epilogue: lane ks handles channels n = ks, ks + KS, ... of its 8 ----
  const int oy = oy0 + prow, oxs = ox0 + pcol;
  if (oy >= a.ho) return;
  const float inv = 1.0f / (float)(1 << a.shift);
  const int64_t plane = (int64_t)a.ho * a.wo;
  const bool vec = (a.wo % 4 == 0) && (oxs + XMP <= a.wo);
#pragma unroll
  for (int n = 0; n < XNC; ++n) {
    if (n % KS != ks) continue;
    const int co = co_blk + cg * XNC + n;
    if (co >= a.cout) continue;
    int32_t acc[XMP];
#pragma unroll
    for (int i = 0; i < XMP; ++i) {
      if constexpr (!MA && !MW)
        acc[i] = a.kreal - 2 * (int32_t)cx[i][n];
      else if constexpr (MA && !MW)
        acc[i] = (int32_t)cma[i] - 2 * (int32_t)cx[i][n];
      else if constexpr (!MA && MW)
        acc[i] = (int32_t)cmw[n] - 2 * (int32_t)cx[i][n];
      else
        acc[i] = (int32_t)cm[i][n] - 2 * (int32_t)cx[i][n];
    }
    const int64_t oi = ((int64_t)img * a.cout + co) * plane + (int64_t)oy * a.wo + oxs;
    if (a.mode == QCONV_EPI_INT32) {
      int32_t* o = static_cast<int32_t*>(a.out) + oi;
      if (vec) {
        *reinterpret_cast<int4*>(o) = make_int4(acc[0], acc[1], acc[2], acc[3]);
      } else {
#pragma unroll
        for (int i = 0; i < XMP; ++i)
          if (oxs + i < a.wo) o[i] = acc[i];
      }
      continue;
    }
    float z[XMP];
    const int cl = cg * XNC + n;
    if (a.mode == QCONV_EPI_SCALE_F32) {
      const float sc = ep_l[cl];
#pragma unroll
      for (int i = 0; i < XMP; ++i) z[i] = sc * ((float)acc[i] * inv);
    } else {
      const float kk = ep_l[cl], bb = ep_l[CO_B + cl];
#pragma unroll
      for (int i = 0; i < XMP; ++i) z[i] = fmaf(kk, (float)acc[i] * inv, bb);
      if (a.residual_on) {
        const float* r = a.residual + oi;
        if (vec) {
          const float4 rv = *reinterpret_cast<const float4*>(r);
          z[0] = z[0] + rv.x;
          z[1] = z[1] + rv.y;
          z[2] = z[2] + rv.z;
          z[3] = z[3] + rv.w;
        } else {
#pragma unroll
          for (int i = 0; i < XMP; ++i)
            if (oxs + i < a.wo) z[i] = z[i] + r[i];
        }
      }
    }
    float* o = static_cast<float*>(a.out) + oi;
    if (vec) {
      *reinterpret_cast<float4*>(o) = make_float4(z[0], z[1], z[2], z[3]);
    } else {
#pragma unroll
      for (int i = 0; i < XMP; ++i)
        if (oxs + i < a.wo) o[i] = z[i];
    }
  }
}

// Block plan for a layer; false if the kernel does not serve it.
bool xnor_plan(const ConvArgs& a, int ks, XArgs* x) {
  memset(x, 0, sizeof(*x));
  x->c = a;
  if (a.a_bits > 2 || a.w_bits > 2) return false;  // the SHIFT pairs stay with the generic kernel
  if (a.pool || a.out_packed || a.mode == QCONV_EPI_BN_PACK) return false;
  if (!((a.kh == 1 && a.kw == 1) || (a.kh == 3 && a.kw == 3)) || a.stride > 2 || a.n == 0) return false;
  const int co_b = 128 / ks;
  x->k1 = a.kh == 1 ? 1 : 0;
  // 1x1 layers stage only the sampled pixels, so their tile may be wider than
  // tall at no staging cost: of 2 x 32, 4 x 16 and 8 x 8 the shape with the
  // fewest pixel slots over the output, the widest on ties (longer runs of
  // each output row in one store: ResNet-18's 28 x 28 shortcut output in
  // rows of 28 instead of 8); 3x3 layers keep 8 x 8 (the least halo)
  x->tw = XT;
  if (x->k1) {
    int64_t best = -1;
    for (int tw : {32, 16, 8}) {
      const int64_t slots = (int64_t)ceil_div(a.wo, tw) * ceil_div(a.ho, 64 / tw);
      if (best < 0 || slots < best) {
        best = slots;
        x->tw = tw;
      }
    }
  }
  x->th = 64 / x->tw;
  x->gshift = x->tw == 32 ? 3 : (x->tw == 16 ? 2 : 1);
  x->tiles_x = ceil_div(a.wo, x->tw);
  x->tiles_y = ceil_div(a.ho, x->th);
  x->co_tiles = ceil_div(a.cout, co_b);
  if (x->k1) {
    x->hr = x->th;
    x->hc = x->hcs = x->tw;
  } else {
    x->hr = (x->th - 1) * a.stride + a.kh;
    x->hc = (x->tw - 1) * a.stride + a.kw;
    x->half = (x->hc + 1) / 2;
    x->hcs = a.stride == 2 ? 2 * x->half : x->hc;
  }
  const int pa = planes_of(a.a_bits), pw = planes_of(a.w_bits);
  const int taps = a.kh * a.kw;
  // words per chunk: as many as fit the LDS budget, at most all of them
  const size_t per_word = (size_t)pa * x->hr * x->hcs * 4 + (size_t)taps * co_b * pw * 4;
  int cwc = (int)(XCHUNK_LDS / per_word);
  if (cwc < 1) return false;
  if (cwc > a.cw) cwc = a.cw;
  x->cwc = cwc;
  x->nchunks = ceil_div(a.cw, cwc);
  x->act_words = ((cwc * pa * x->hr * x->hcs) + 3) & ~3;  // the weight tile starts 16-byte aligned
  const int64_t nb = (int64_t)a.n * x->tiles_y * x->tiles_x * x->co_tiles;
  if (nb >= ((int64_t)1 << 31) || a.cop < x->co_tiles * co_b) return false;
  x->nblocks = (int)nb;
  x->xcd_remap = (nb % 8 == 0) ? 1 : 0;
  return true;
}

size_t xnor_lds(const XArgs& x, int ks) {
  const int co_b = 128 / ks;
  return ((size_t)x.act_words + (size_t)x.c.kh * x.c.kw * x.cwc * co_b * planes_of(x.c.w_bits) + 2 * co_b) * 4;
}

int device_cus_x() {
  int dev = 0, v = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) return 256;
  return v;
}

// The K split: the smallest KS (1, 2, 4) that gives every CU at least two
// blocks, else 4.
int pick_ks(const ConvArgs& a) {
  const int cus = device_cus_x();
  for (int ks : {1, 2, 4}) {
    XArgs x;
    if (!xnor_plan(a, ks, &x)) return 0;
    if (x.nblocks >= 2 * cus) return ks;
  }
  return 4;
}

template <int PA, int PW>
int launch_ks(const XArgs& x, int ks, hipStream_t s) {
  const size_t lds = xnor_lds(x, ks);
  if (ks == 1) conv_xnor_kernel<PA, PW, 1><<<dim3((unsigned)x.nblocks), 256, lds, s>>>(x);
  else if (ks == 2) conv_xnor_kernel<PA, PW, 2><<<dim3((unsigned)x.nblocks), 256, lds, s>>>(x);
  else conv_xnor_kernel<PA, PW, 4><<<dim3((unsigned)x.nblocks), 256, lds, s>>>(x);
  return hip_status();
}

}  // namespace

bool xnor_supports(const ConvArgs& a) {
  XArgs x;
  return xnor_plan(a, 1, &x);
}

int xnor_kernel_name(const ConvArgs& a, char* buf, int len) {
  const int ks = pick_ks(a);
  if (!ks) return QCONV_EUNSUPPORTED;
  char name[96];
  snprintf(name, sizeof(name), "conv_xnor_kernel<%d, %d, %d>", planes_of(a.a_bits), planes_of(a.w_bits), ks);
  if (buf && len > 0) snprintf(buf, (size_t)len, "%s", name);
  return (int)strlen(name);
}

int launch_conv_xnor(const ConvArgs& a, hipStream_t s) {
  const int ks = pick_ks(a);
  XArgs x;
  if (!ks || !xnor_plan(a, ks, &x)) return QCONV_EUNSUPPORTED;
  const int pa = planes_of(a.a_bits), pw = planes_of(a.w_bits);
  if (pa == 1 && pw == 1) return launch_ks<1, 1>(x, ks, s);
  if (pa == 2 && pw == 1) return launch_ks<2, 1>(x, ks, s);
  if (pa == 1 && pw == 2) return launch_ks<1, 2>(x, ks, s);
  return launch_ks<2, 2>(x, ks, s);
}

}  // namespace qc
