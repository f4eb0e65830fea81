// conv_mfma.hip -- the same layer product (Algorithm 1, inference branch) on
// the gfx950 matrix cores.  The level codes of both operands ({-1,+1},
// {-1,0,+1}, {0,+-1,+-2,+-4}) are exact as int8 and as E2M1 (fp4), and every
// partial sum is an integer below 2^24, so both
//   v_mfma_i32_32x32x32_i8            (int32 accumulate) and
//   v_mfma_scale_f32_32x32x64_f8f6f4  (fp4 operands, unit scales, fp32 accumulate)
// give the exact integer accumulator of the bitplane kernel.
//
// Tiling: a block (4 waves, 2 x 2) owns 2 * MTW M-tiles of 32 output pixels
// and 64 * NTW output channels (2 * NTW N-tiles of 32); a wave owns MTW
// M-tiles x NTW N-tiles of 32 x 32 accumulators (MTW = 2: 128-pixel blocks,
// three waves per SIMD, so one block's stores overlap other blocks' MFMAs).  The block's input rows plus halo
// are expanded once per channel chunk from the packed bitplanes into LDS
// (int8: 4 words = 128 bytes per pixel, fp4: 8 words = 128 bytes, + 16 bytes
// of padding so that 16-byte fragment reads of neighbouring pixels fall in
// different banks).  Each expanded value then feeds every tap and every
// output channel of the block.  The weights were expanded once at packing
// time into the same operand format; a lane reads its 16-byte B fragment
// straight from global memory (L2-resident, shared by all blocks).
// The epilogue reads the accumulator layout (register v of lane l holds row
// 8(v/4) + 4(l/32) + v%4, column l%32) and packs requantized outputs with one
// wave ballot per plane: 32 channels of a pixel become one word.
#include <string.h>

#include <type_traits>

#include "qconv_internal.h"

namespace qc {

namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));

#ifndef QC_MFMA_MTW
#define QC_MFMA_MTW 2
#endif
constexpr int MTW = QC_MFMA_MTW;       // M-tiles (of 32 pixels) per wave
constexpr int BLOCK_PIX = 2 * MTW * 32;  // 2 waves along M
#ifndef QC_MFMA_WPE
#define QC_MFMA_WPE 3
#endif
constexpr int MAX_LDS = 64 * 1024;


template <int FP4>
struct OpT;
template <>
struct OpT<0> {
  static constexpr int CHUNK_WORDS = 4;  // words of 32 channels staged per chunk
  static constexpr int WORD_BYTES = 32;  // LDS bytes per word per pixel
  static constexpr int WORDS_PER_STEP = 1;
  using acc_t = v16i;
};
template <>
struct OpT<1> {
  static constexpr int CHUNK_WORDS = 8;
  static constexpr int WORD_BYTES = 16;
  static constexpr int WORDS_PER_STEP = 2;
  using acc_t = v16f;
};

struct MfmaArgs {
  ConvArgs c;
  const uint8_t* wx;    // expanded weights in the chosen operand format
  int wx_bytes;         // size of that operand copy (bounds of the B buffer reads)
  int ipb;              // whole images per block (1: the block is a pixel range of one image)
  int blocks_per_img;   // ipb == 1: blocks per image
  int hr, hc;           // halo rows / cols per image slot
  int pix_bytes;        // LDS bytes per halo pixel (chunk words * WORD_BYTES + 16)
  int chunk_words;      // words staged per chunk
  int ksteps;           // k-steps per tap over all words (int8: cw, fp4: ceil(cw/2))
  int nchunks;
  int vec_store;        // ho*wo % 4 == 0: 4 consecutive pixels are one aligned 16-byte run
  int tiles_px;         // pixel tiles (blocks of BLOCK_PIX pixels or ipb images)
  int tiles_co;         // output-channel tiles (64 * NTW channels)
  int halo_bytes;       // LDS bytes of the halo tile (reused as the output stage)
  int pool_wo;          // 2x2 max pooling: the conv output width (8, 16, 32 or 64), else 0
  int mt_interleave;    // wave wm owns M-tiles wm, wm + 2, ... instead of a contiguous run
};

__device__ __forceinline__ v16i mfma(v4i a, v4i b, v16i c) {
  return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ v16f mfma(v4i a, v4i b, v16f c) {
  v8i a8 = {a[0], a[1], a[2], a[3], 0, 0, 0, 0};
  v8i b8 = {b[0], b[1], b[2], b[3], 0, 0, 0, 0};
  // operand format 4 = E2M1 for both; scales 127 = 2^0
  return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, c, 4, 4, 0, 127, 0, 127);
}
__device__ __forceinline__ int acc_value(const v16i& a, int v) { return a[v]; }
__device__ __forceinline__ int acc_value(const v16f& a, int v) { return (int)a[v]; }

template <int FP4, int PA>
__device__ __forceinline__ void expand_to_lds(const uint32_t* pl, uint8_t* dst) {
  if constexpr (FP4) {
    uint32_t o[4];
    expand_fp4_word<PA>(pl, 0xFFFFFFFFu, o);
    *reinterpret_cast<uint4*>(dst) = make_uint4(o[0], o[1], o[2], o[3]);
  } else {
    uint32_t o[8];
    expand_i8_word<PA>(pl, 0xFFFFFFFFu, o);
    reinterpret_cast<uint4*>(dst)[0] = make_uint4(o[0], o[1], o[2], o[3]);
    reinterpret_cast<uint4*>(dst)[1] = make_uint4(o[4], o[5], o[6], o[7]);
  }
}

__device__ __forceinline__ uint32_t quant_rt(float z, int bits, Thr t) {
  if (bits == 1) return quant_planes<1>(z, t);
  if (bits == 2) return quant_planes<2>(z, t);
  return quant_planes<3>(z, t);
}

// Compile-time loop: f(integral_constant<I>) for I in [B, E), so that the
// accumulator tiles are only ever indexed with constants (no scratch copy).
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

struct EpiCtx {
  int img0, p0, co_blk, hwo, lane;
};

constexpr int STAGE_LD = 36;                      // floats per staged channel row (32 + 4 pad)
constexpr int STAGE_BYTES = 32 * STAGE_LD * 4;    // one 32 x 32 tile per wave

// Image and pixel of block pixel t; false past the end of the block's work.
__device__ __forceinline__ bool block_pixel(const MfmaArgs& m, const EpiCtx& x, int t, int* img,
                                            int* pp) {
  int slot;
  if (m.ipb == 1) {
    slot = 0;
    *pp = x.p0 + t;
    if (*pp >= x.hwo) return false;
  } else {
    slot = t / x.hwo;
    *pp = t - slot * x.hwo;
    if (slot >= m.ipb || x.img0 + slot >= m.c.n) return false;
  }
  *img = x.img0 + slot;
  return true;
}

// Flat NCHW index of block pixel t for channel co, or -1 past the end.
__device__ __forceinline__ int64_t out_index(const MfmaArgs& m, const EpiCtx& x, int t, int co) {
  int img, pp;
  if (!block_pixel(m, x, t, &img, &pp)) return -1;
  return ((int64_t)img * m.c.cout + co) * x.hwo + pp;
}

// Epilogue of one 32 x 32 accumulator tile: block pixels [32 mt, 32 mt + 32)
// x output channels [c32, c32 + 32).  Unpacked outputs go through the wave's
// LDS stage so that every store instruction writes whole 128-byte runs of
// one channel's pixels; packed outputs are assembled with ballots.
template <class AccT>
__device__ __forceinline__ void store_tile(const MfmaArgs& m, const EpiCtx& x, const AccT& acc,
                                           int mt, int c32, float* stage) {
  const ConvArgs& a = m.c;
  const int g = x.lane >> 5, r32 = x.lane & 31;
  const float inv = 1.0f / (float)(1 << a.shift);
  const bool pack = a.out_packed != nullptr && c32 < a.cout;  // uniform
  const int co = c32 + r32;
  const bool co_ok = co < a.cout;
  const int cs = min(co, a.cout - 1);
  float kk = 0.0f, bb = 0.0f, ss = 0.0f;
  if (a.mode == QCONV_EPI_BN_F32 || a.mode == QCONV_EPI_BN_PACK) {
    kk = a.bn_k[cs];
    bb = a.bn_b[cs];
  } else if (a.mode == QCONV_EPI_SCALE_F32) {
    ss = a.scale[cs];
  }
  // value of register v before any residual: int32 accumulator (INT32 mode)
  // or the fp32 scale / BN result, bit-cast into the stage
  auto value_bits = [&](int v) -> uint32_t {
    const int av = acc_value(acc, v);
    if (a.mode == QCONV_EPI_INT32) return (uint32_t)av;
    const float ar = (float)av * inv;
    const float z = (a.mode == QCONV_EPI_SCALE_F32) ? ss * ar : fmaf(kk, ar, bb);
    return __float_as_uint(z);
  };

  if (a.mode != QCONV_EPI_BN_PACK && c32 < a.cout) {
    // stage: lane (column r32, half g) holds rows 8q + 4g + i, i = 0..3
#pragma unroll
    for (int q = 0; q < 4; ++q) {
      const uint4 w4 = make_uint4(value_bits(4 * q), value_bits(4 * q + 1), value_bits(4 * q + 2),
                                  value_bits(4 * q + 3));
      *reinterpret_cast<uint4*>(stage + r32 * STAGE_LD + 8 * q + 4 * g) = w4;
    }
    // read back: lane l takes channel 8k + l/8, pixels 4(l%8) .. 4(l%8)+3
#pragma unroll
    for (int k = 0; k < 4; ++k) {
      const int cl = 8 * k + (x.lane >> 3);
      const int px = 4 * (x.lane & 7);
      const uint4 w4 = *reinterpret_cast<const uint4*>(stage + cl * STAGE_LD + px);
      const int c = c32 + cl;
      if (c >= a.cout) continue;
      const int t = 32 * mt + px;
      const int64_t i0 = out_index(m, x, t, c);
      uint32_t w[4] = {w4.x, w4.y, w4.z, w4.w};
      if (m.vec_store && i0 >= 0) {
        // ho*wo % 4 == 0: the four pixels are one aligned 16-byte run of one image
        if (a.residual_on) {
          const float4 rv = *reinterpret_cast<const float4*>(a.residual + i0);
          w[0] = __float_as_uint(__uint_as_float(w[0]) + rv.x);
          w[1] = __float_as_uint(__uint_as_float(w[1]) + rv.y);
          w[2] = __float_as_uint(__uint_as_float(w[2]) + rv.z);
          w[3] = __float_as_uint(__uint_as_float(w[3]) + rv.w);
        }
        *reinterpret_cast<uint4*>(static_cast<uint32_t*>(a.out) + i0) = make_uint4(w[0], w[1], w[2], w[3]);
      } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          const int64_t ie = out_index(m, x, t + e, c);
          if (ie < 0) continue;
          uint32_t we = w[e];
          if (a.residual_on) we = __float_as_uint(__uint_as_float(we) + a.residual[ie]);
          static_cast<uint32_t*>(a.out)[ie] = we;
        }
      }
    }
  }

  if (pack) {
    // one ballot per (pixel row, plane): lanes 0-31 hold the 32 channels of
    // row t + e (g = 0), lanes 32-63 those of row t + 4 + e (g = 1)
    const int pout = planes_of(a.out_bits);
    const int cword = c32 >> 5;
#pragma unroll
    for (int v4 = 0; v4 < 16; v4 += 4) {
      const int t = 32 * mt + 8 * (v4 >> 2) + 4 * g;
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        const int64_t ie = out_index(m, x, t + e, cs);
        float z = __uint_as_float(value_bits(v4 + e));
        if (a.residual_on && ie >= 0) z = z + a.residual[ie];
        const uint32_t pl = (co_ok && ie >= 0) ? quant_rt(hardtanh(z), a.out_bits, a.othr) : 0u;
        int img, pp;
        const bool pix_ok = block_pixel(m, x, t + e, &img, &pp);
        for (int p = 0; p < pout; ++p) {
          const uint64_t bal = __ballot((pl >> p) & 1u);
          if (r32 == 0 && pix_ok) {
            const uint32_t word = g ? (uint32_t)(bal >> 32) : (uint32_t)bal;
            a.out_packed[(((int64_t)img * x.hwo + pp) * a.out_cw + cword) * pout + p] = word;
          }
        }
      }
    }
  }
}

// Pooled epilogue (2x2 max over the integer accumulator, before BN) of one
// wave's two M-tiles for output channels [c32, c32 + 32).  The block starts
// at an even conv row and the M-tiles are assigned so that all four pixels of
// every window sit in the same lane:
//   wo = 32: the two tiles are rows 2r and 2r+1 (same register);
//   wo = 64: the tiles are the same half of rows 2r and 2r+1 (interleaved tiles);
//   wo = 16: one tile is two rows, the lower pixel is register v + 8;
//   wo =  8: one tile is four rows, the lower pixel is register v + 4;
// and the horizontal neighbour of an even pixel (even v) is register v + 1.
// Lane (g, r32) ends with 8 pooled pixels of channel c32 + r32.
template <int WO, class AccT>
__device__ __forceinline__ void store_pool_tiles(const MfmaArgs& m, const EpiCtx& x, const AccT& a0,
                                                 const AccT& a1, int mt0, int mt1, int c32) {
  const ConvArgs& a = m.c;
  const int g = x.lane >> 5, r32 = x.lane & 31;
  const float inv = 1.0f / (float)(1 << a.shift);
  const bool pack = a.out_packed != nullptr && c32 < a.cout;  // uniform
  const int co = c32 + r32;
  const bool co_ok = co < a.cout;
  const int cs = min(co, a.cout - 1);
  float kk = 0.0f, bb = 0.0f, ss = 0.0f;
  if (a.mode == QCONV_EPI_BN_F32 || a.mode == QCONV_EPI_BN_PACK) {
    kk = a.bn_k[cs];
    bb = a.bn_b[cs];
  } else if (a.mode == QCONV_EPI_SCALE_F32) {
    ss = a.scale[cs];
  }
  const int64_t plane = (int64_t)a.oh_out * a.ow_out;
  const int pout = pack ? planes_of(a.out_bits) : 0;
  const int cword = c32 >> 5;
  Unroll<0, 8>::run([&](auto S) {
    constexpr int s = decltype(S)::value;
    constexpr bool pair_tiles = WO >= 32;
    constexpr int ti = pair_tiles ? 0 : s / 4;  // tile holding the window's upper row
    constexpr int u = pair_tiles ? s : s % 4;
    constexpr int v = (WO == 8) ? (u & 1) * 2 + (u >> 1) * 8 : 2 * u;
    constexpr int dv = pair_tiles ? 0 : (WO == 16 ? 8 : 4);
    const AccT& top = (ti == 0) ? a0 : a1;
    const AccT& bot = pair_tiles ? a1 : top;
    const int best = max(max(acc_value(top, v), acc_value(top, v + 1)),
                         max(acc_value(bot, v + dv), acc_value(bot, v + dv + 1)));
    const int t = 32 * ((ti == 0) ? mt0 : mt1) + 8 * (v / 4) + 4 * g + (v % 4);
    int img = 0, pp = 0;
    bool ok = block_pixel(m, x, t, &img, &pp);
    const int oy = pp / a.wo, ox = pp - (pp / a.wo) * a.wo;
    const int py = oy >> 1, px = ox >> 1;
    ok = ok && py < a.oh_out;  // an odd last conv row has no pooled row
    const float ar = (float)best * inv;
    float z = (a.mode == QCONV_EPI_SCALE_F32) ? ss * ar : fmaf(kk, ar, bb);
    const int64_t oi = ((int64_t)img * a.cout + cs) * plane + (int64_t)py * a.ow_out + px;
    if (a.mode != QCONV_EPI_BN_PACK && co_ok && ok) {
      if (a.mode == QCONV_EPI_INT32) {
        static_cast<int32_t*>(a.out)[oi] = best;
      } else {
        if (a.residual_on) z = z + a.residual[oi];
        static_cast<float*>(a.out)[oi] = z;
      }
    }
    if (pack) {
      const uint32_t pl = (co_ok && ok) ? quant_rt(hardtanh(z), a.out_bits, a.othr) : 0u;
      for (int p = 0; p < pout; ++p) {
        const uint64_t bal = __ballot((pl >> p) & 1u);
        if (r32 == 0 && ok) {
          const uint32_t word = g ? (uint32_t)(bal >> 32) : (uint32_t)bal;
          a.out_packed[((((int64_t)img * a.oh_out + py) * a.ow_out + px) * a.out_cw + cword) * pout + p] =
              word;
        }
      }
    }
  });
}

template <int FP4, int PA, int NTW>
__global__ __launch_bounds__(256, QC_MFMA_WPE) void conv_mfma_kernel(const MfmaArgs m) {
  using O = OpT<FP4>;
  using acc_t = typename O::acc_t;
  extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
  const ConvArgs& a = m.c;
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;
  const int g = lane >> 5, r32 = lane & 31;
  const int hwo = a.ho * a.wo;

  const int slot_pix = m.hr * m.hc;
  const int apix = a.cw * PA;
  const int n_slots = (m.ipb == 1) ? 1 : m.ipb;
  const int items_per_chunk = n_slots * slot_pix * m.chunk_words;
  const int taps = a.kh * a.kw;
  const int steps_per_chunk = m.chunk_words / O::WORDS_PER_STEP;
  // B fragments are read through a buffer resource: the per-lane part of
  // the address is a vector offset, the per-step part a scalar offset, and
  // reads past the operand copy return 0.
  const __amdgpu_buffer_rsrc_t brsrc =
      __builtin_amdgcn_make_buffer_rsrc((void*)m.wx, (short)0, m.wx_bytes, 0x00020000);
  const int bstride = a.cop * 32;  // bytes between consecutive k-steps
  // one (pixel tile, channel tile) per block
  {
    const int pb = blockIdx.x;
    const int co_blk = blockIdx.y * (64 * NTW);
    int img0, p0;
    if (m.ipb == 1) {
      img0 = pb / m.blocks_per_img;
      p0 = (pb % m.blocks_per_img) * BLOCK_PIX;
    } else {
      img0 = pb * m.ipb;
      p0 = 0;
    }
    const int oy0 = p0 / a.wo;
    const int iy0 = oy0 * a.stride - a.pad;

    // LDS byte offset of each of the wave's M-tile rows at tap (0, 0), plus
    // this lane's 16-byte half of the k-step.
    int abase[MTW];
#pragma unroll
    for (int i = 0; i < MTW; ++i) {
      const int t = 32 * (m.mt_interleave ? wm + 2 * i : wm * MTW + i) + r32;
      int slot, pp;
      if (m.ipb == 1) {
        slot = 0;
        pp = p0 + t;
      } else {
        slot = t / hwo;
        pp = t - slot * hwo;
      }
      bool ok = (m.ipb == 1) ? (pp < hwo) : (slot < m.ipb);
      if (!ok) {  // a row past the end: read any valid LDS pixel, its result is dropped
        slot = 0;
        pp = p0;
      }
      const int oy = pp / a.wo, ox = pp - (pp / a.wo) * a.wo;
      const int hp = slot * slot_pix + (oy - oy0) * a.stride * m.hc + ox * a.stride;
      abase[i] = hp * m.pix_bytes + g * 16;
    }

    acc_t acc[MTW][NTW];
#pragma unroll
    for (int i = 0; i < MTW; ++i)
#pragma unroll
      for (int j = 0; j < NTW; ++j)
#pragma unroll
        for (int v = 0; v < 16; ++v) acc[i][j][v] = 0;

    int bvoff[NTW];
#pragma unroll
    for (int j = 0; j < NTW; ++j) bvoff[j] = (co_blk + 32 * (wn * NTW + j) + r32) * 32 + g * 16;

    for (int chunk = 0; chunk < m.nchunks; ++chunk) {
      __syncthreads();
      // ---- expand the halo tile of this channel chunk into LDS ----
      // loads of up to 4 items are issued together before any is expanded
      for (int it0 = 0; it0 < items_per_chunk; it0 += 4 * 256) {
        uint32_t pl[4][PA];
        int dst[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int it = it0 + u * 256 + tid;
          dst[u] = -1;
#pragma unroll
          for (int p = 0; p < PA; ++p) pl[u][p] = 0u;
          if (it < items_per_chunk) {
            const int cwl = it % m.chunk_words;
            const int hp = it / m.chunk_words;
            const int slot = hp / slot_pix;
            const int rem = hp - slot * slot_pix;
            const int hrow = rem / m.hc, hcol = rem - (rem / m.hc) * m.hc;
            const int img = img0 + slot;
            const int iy = iy0 + hrow, ix = hcol - a.pad;
            const int cw = chunk * m.chunk_words + cwl;
            dst[u] = hp * m.pix_bytes + cwl * O::WORD_BYTES;
            if (img < a.n && iy >= 0 && iy < a.h && ix >= 0 && ix < a.w && cw < a.cw) {
              const uint32_t* src = a.act + (((int64_t)img * a.h + iy) * a.w + ix) * apix + cw * PA;
#pragma unroll
              for (int p = 0; p < PA; ++p) pl[u][p] = src[p];
            }
          }
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (dst[u] >= 0) expand_to_lds<FP4, PA>(pl[u], lds + dst[u]);
      }
      __syncthreads();

      // ---- MFMA over (tap, k-step) of this chunk ----
      // B fragments come from a ring of three register sets, each loaded two
      // k-steps before its MFMAs (buffer loads, so the compiler keeps them
      // where they are issued).  A fragments are read from LDS in the step
      // that uses them.  Steps advance (tap, k-step) incrementally.
      const int ks0 = chunk * steps_per_chunk;
      const int spc = min(m.ksteps, ks0 + steps_per_chunk) - ks0;  // k-steps per tap in this chunk
      const int nsteps = taps * spc;
      // load stream (runs two steps ahead of the compute stream)
      int l_tap = 0, l_ksl = 0, l_count = 0;
      auto bload = [&](v4i (&dst)[NTW]) {
        const int so = (l_tap * m.ksteps + ks0 + l_ksl) * bstride;
#pragma unroll
        for (int j = 0; j < NTW; ++j)
          dst[j] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(brsrc, bvoff[j], so, 0));
        if (l_count + 1 < nsteps) {  // the last step is reloaded past the end (never used)
          ++l_count;
          if (++l_ksl == spc) {
            l_ksl = 0;
            ++l_tap;
          }
        }
      };
      // compute stream
      int c_ksl = 0, c_ky = 0, c_kx = 0;
      auto step = [&](const v4i (&bf)[NTW]) {
        const int lo = (c_ky * m.hc + c_kx) * m.pix_bytes + c_ksl * 32;
        v4i af[MTW];
#pragma unroll
        for (int i = 0; i < MTW; ++i) af[i] = *reinterpret_cast<const v4i*>(lds + abase[i] + lo);
#pragma unroll
        for (int i = 0; i < MTW; ++i)
#pragma unroll
          for (int j = 0; j < NTW; ++j) acc[i][j] = mfma(af[i], bf[j], acc[i][j]);
        if (++c_ksl == spc) {
          c_ksl = 0;
          if (++c_kx == a.kw) {
            c_kx = 0;
            ++c_ky;
          }
        }
      };
      v4i B0[NTW], B1[NTW], B2[NTW];
      bload(B0);
      bload(B1);
      for (int st = 0; st < nsteps; st += 3) {
        bload(B2);
        step(B0);
        if (st + 1 >= nsteps) break;
        bload(B0);
        step(B1);
        if (st + 2 >= nsteps) break;
        bload(B1);
        step(B2);
      }
    }

    // ---- epilogue ----
    __syncthreads();  // every wave is done with the halo tile; LDS becomes the output stage
    float* stage = reinterpret_cast<float*>(lds + wave * STAGE_BYTES);
    const EpiCtx x = {img0, p0, co_blk, hwo, lane};
    if constexpr (MTW == 2) {
      if (m.pool_wo) {
        const int mt0 = m.mt_interleave ? wm : 2 * wm;
        const int mt1 = m.mt_interleave ? wm + 2 : 2 * wm + 1;
        Unroll<0, NTW>::run([&](auto J) {
          const int c32 = co_blk + 32 * (wn * NTW + J);
          switch (m.pool_wo) {
            case 8: store_pool_tiles<8>(m, x, acc[0][J], acc[1][J], mt0, mt1, c32); break;
            case 16: store_pool_tiles<16>(m, x, acc[0][J], acc[1][J], mt0, mt1, c32); break;
            case 32: store_pool_tiles<32>(m, x, acc[0][J], acc[1][J], mt0, mt1, c32); break;
            default: store_pool_tiles<64>(m, x, acc[0][J], acc[1][J], mt0, mt1, c32); break;
          }
        });
        return;
      }
    }
    Unroll<0, MTW>::run([&](auto I) {
      Unroll<0, NTW>::run([&](auto J) {
        store_tile(m, x, acc[I][J], wm * MTW + I, co_blk + 32 * (wn * NTW + J), stage);
      });
    });
  }
}

bool plan(const ConvArgs& a, MfmaArgs* m) {
  memset(m, 0, sizeof(*m));
  m->c = a;
  const int fp4 = a.mfma_fp4;
  const int chunk_max = fp4 ? OpT<1>::CHUNK_WORDS : OpT<0>::CHUNK_WORDS;
  const int wpstep = fp4 ? 2 : 1;
  const int word_bytes = fp4 ? 16 : 32;
  const int cw_round = ceil_div(a.cw, wpstep) * wpstep;
  m->ksteps = ceil_div(a.cw, wpstep);
  m->wx = fp4 ? a.w_fp4 : a.w_i8;
  m->wx_bytes = (int)(a.kh * a.kw * m->ksteps * a.cop * 32);
  const int hwo = a.ho * a.wo;
  m->hc = (a.wo - 1) * a.stride + a.kw;
  m->vec_store = (hwo % 4 == 0) ? 1 : 0;
  // Candidate channel chunks, largest first; smaller chunks shrink the LDS
  // tile so that more small images fit in one block.
  int best_pix = -1;
  MfmaArgs best = *m;
  for (int cwc = min(chunk_max, cw_round); cwc >= wpstep; cwc /= 2) {
    if (cwc % wpstep) break;
    MfmaArgs t = *m;
    t.chunk_words = cwc;
    t.pix_bytes = cwc * word_bytes + 16;
    t.nchunks = ceil_div(cw_round, cwc);
    int pix;
    if (hwo * 2 <= BLOCK_PIX) {
      t.hr = (a.ho - 1) * a.stride + a.kh;
      const size_t slot = (size_t)t.hr * t.hc * t.pix_bytes;
      const int fit = (int)(MAX_LDS / slot);
      t.ipb = min(BLOCK_PIX / hwo, fit);
      t.blocks_per_img = 0;
      if (t.ipb < 1) continue;
      pix = t.ipb * hwo;
    } else {
      t.ipb = 1;
      t.blocks_per_img = ceil_div(hwo, BLOCK_PIX);
      const int rows = min(a.ho, ceil_div(BLOCK_PIX, a.wo) + 1);
      t.hr = (rows - 1) * a.stride + a.kh;
      if ((size_t)t.hr * t.hc * t.pix_bytes > (size_t)MAX_LDS) continue;
      pix = BLOCK_PIX;
    }
    if (pix > best_pix) {
      best_pix = pix;
      best = t;
    }
    if (pix == BLOCK_PIX || (hwo * 2 <= BLOCK_PIX && t.ipb == BLOCK_PIX / hwo)) break;
  }
  if (best_pix < 0) return false;
  *m = best;
  if (a.pool) {
    // every 2x2 window must fall in one lane of one wave (see store_pool_tiles)
    if (MTW != 2 || !(a.wo == 8 || a.wo == 16 || a.wo == 32 || a.wo == 64)) return false;
    if (m->ipb > 1 && a.ho % 2 != 0) return false;
    m->pool_wo = a.wo;
    m->mt_interleave = (a.wo == 64) ? 1 : 0;
  }
  if (m->ipb == 1 && m->blocks_per_img == 0) m->blocks_per_img = 1;
  m->tiles_px = (m->ipb == 1) ? a.n * m->blocks_per_img : ceil_div(a.n, m->ipb);
  m->tiles_co = (a.cout > 64) ? ceil_div(a.cout, 128) : 1;
  m->halo_bytes = m->hr * m->hc * m->pix_bytes * (m->ipb == 1 ? 1 : m->ipb);
  return true;
}

template <int FP4, int PA>
int launch_fp(const MfmaArgs& m, hipStream_t s) {
  const ConvArgs& a = m.c;
  const size_t lds = max((size_t)m.halo_bytes, (size_t)(4 * STAGE_BYTES));
  const dim3 grid((unsigned)m.tiles_px, (unsigned)m.tiles_co);
  if (a.cout > 64)
    conv_mfma_kernel<FP4, PA, 2><<<grid, 256, lds, s>>>(m);
  else
    conv_mfma_kernel<FP4, PA, 1><<<grid, 256, lds, s>>>(m);
  return hip_status();
}

}  // namespace

bool mfma_supports(const ConvArgs& a) {
  if (a.stride > 2 || a.n == 0) return false;
  MfmaArgs m;
  return plan(a, &m);
}

int launch_conv_mfma(const ConvArgs& a, hipStream_t s) {
  MfmaArgs m;
  if (!plan(a, &m)) return QCONV_EUNSUPPORTED;
  const int pa = planes_of(a.a_bits);
  if (a.mfma_fp4) {
    if (pa == 1) return launch_fp<1, 1>(m, s);
    if (pa == 2) return launch_fp<1, 2>(m, s);
    return launch_fp<1, 4>(m, s);
  }
  if (pa == 1) return launch_fp<0, 1>(m, s);
  if (pa == 2) return launch_fp<0, 2>(m, s);
  return launch_fp<0, 4>(m, s);
}

}  // namespace qc
