#pragma once
// conv_mfma.h -- the layer product of Algorithm 1 (inference branch) on the
// gfx950 matrix cores.  The level codes of both operands ({-1,+1},
// {-1,0,+1}, {0,+-1,+-2,+-4}) are exact as int8 and as E2M1 (fp4), and every
// partial sum is an integer below 2^24, so both
//   v_mfma_i32_32x32x32_i8            (int32 accumulate) and
//   v_mfma_scale_f32_32x32x64_f8f6f4  (fp4 operands, unit scales, fp32 accumulate)
// give the exact integer accumulator of the bitplane kernel.
//
// 16-bit inputs (Table I, rows with 16-bit inputs and 1..3-bit weights: the
// "XNOR ADDER" / "SHIFT ADDER" operation at 16-bit floating precision): the
// activations stay fp16 and the weight codes are exact in fp16, so
//   v_mfma_f32_32x32x16_f16           (fp32 accumulate)
// sums exact products; only the fp32 accumulation rounds.  The halo is
// staged in LDS as it is stored (64 bytes per 32 channels), with the same
// fragment addressing (32 bytes per k-step, 16 per lane half).  The rows
// with 1..3-bit inputs and 16-bit weights use the same kernel with the roles
// of the formats swapped: the activation bitplanes are expanded into the
// fp16 codes of their levels in LDS and the weights are fp16.
//
// Work unit.  The block's M dimension is a list of "units": output pixels, or
// with 2x2 pooling whole pooling windows (the pooled output pixels), each of
// which occupies four consecutive M rows.  A block owns a run of units of one
// image, or several whole images, and 32 * NT * WN output channels.
//
// Tiling.  4 waves in a WM x WN grid; a wave owns MT x NT tiles of 32 x 32
// accumulators.  The block's input rows plus halo are expanded once per
// channel chunk from the packed bitplanes into LDS (int8: 32 bytes per 32
// channels, fp4: 16 bytes; + 16 bytes of padding per pixel, so that 16-byte
// fragment reads of neighbouring pixels fall in different banks).  Each
// expanded value then feeds every tap and every output channel of the block.
// The weights were expanded at packing time into the same operand format; a
// lane reads its 16-byte B fragment from global memory (L2-resident) through
// a buffer resource, two k-steps ahead of its use.
//
// Epilogue.  Register v of lane l holds M row 8(v/4) + 4(l/32) + v%4 and
// output channel l%32.  Row r of an M-tile is unit r for plain convolutions,
// so a lane's registers 4q..4q+3 are four consecutive pixels of one channel
// (one 16-byte NCHW store).  With pooling, row r is element r%4 of window
// 4((r/4)%2) + r/8, so registers 4q..4q+3 are the four pixels of one window
// and a lane ends with four consecutive pooled pixels.  Packed outputs are
// built with one wave ballot per (register, plane): lanes 0-31 give the 32
// channels of one pixel, lanes 32-63 those of another, and the words are
// moved into lanes with writelane so that each lane stores one pixel's word.
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <type_traits>

#include "qconv_internal.h"

namespace qc {
namespace mfma {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v8i __attribute__((ext_vector_type(8)));
typedef int v16i __attribute__((ext_vector_type(16)));
typedef float v16f __attribute__((ext_vector_type(16)));
typedef _Float16 v8h __attribute__((ext_vector_type(8)));

constexpr int MAX_LDS = 38 * 1024;  // one halo buffer (two per block, two blocks per CU)
// fp16 operands have no bitplane fallback: input tiles up to twice that size
// are staged with one block per CU instead
constexpr int MAX_LDS_WIDE = 76 * 1024;
constexpr int BRING = 2;  // weight-fragment register sets in flight (deeper rings measured slower)
// Packed words of the next stage held per thread in registers (bounded by
// the registers left next to the accumulators); items past 256 times this
// are loaded when the stage is expanded, each pair then waiting a full
// global-memory latency.  The 128-channel block shape holds up to 2048
// items of 1- and 2-bit inputs (its 3x3 halo tiles of 128 channels); the
// smaller shapes, whose tiles are narrower and which run three blocks per
// CU within 168 registers, hold 1024.
// fp16 halo words (64 bytes each) are not held across the MFMAs: they are
// loaded at the end of the stage instead (two per thread in flight), so
// that no weight-fragment load of the MFMA loop waits behind them (loads of
// a wave complete in order) and the registers stay free.
__host__ __device__ constexpr int halo_items_per_thread(int words, int cfg) {
  return words == 16 ? 0 : (cfg == 0 && words <= 2 ? 8 : (words == 1 ? 4 : 8 / words));
}

// Blocks of conv_mfma_kernel per CU that its register budget is compiled
// for (512 registers per SIMD lane shared by the resident waves): three for
// the fp4 shapes of up to 64 output channels per block (168 registers), two
// otherwise (the 128-channel shape holds twice the accumulators; the int8
// and fp16 shapes spill within 168).
__host__ __device__ constexpr int blocks_per_cu(int opk, int cfg) { return opk == OP_FP4 && cfg != 0 ? 3 : 2; }


// Operand formats (MfmaOp): what one 32-channel word of a pixel becomes in
// LDS and how many channels one k-step of the MFMA consumes.
template <int OPK>
struct OpT;
template <>
struct OpT<OP_I8> {
  static constexpr int CHUNK_WORDS = 4;  // 32-channel words staged per chunk
  static constexpr int WORD_BYTES = 32;  // LDS bytes per word per pixel
  static constexpr int K_PER_STEP = 32;  // channels per k-step
  using acc_t = v16i;
};
template <>
struct OpT<OP_FP4> {
  static constexpr int CHUNK_WORDS = 8;
  static constexpr int WORD_BYTES = 16;
  static constexpr int K_PER_STEP = 64;
  using acc_t = v16f;
};
template <>
struct OpT<OP_F16> {
  static constexpr int CHUNK_WORDS = 2;
  static constexpr int WORD_BYTES = 64;
  static constexpr int K_PER_STEP = 16;
  using acc_t = v16f;
};

// Block shapes: WM x WN x SK waves (SK: waves splitting the K range of the
// same output tile, their partial tiles summed through LDS), each owning
// MT x NT tiles of 32 x 32 accumulators.
template <int CFG>
struct Cfg;
template <>
struct Cfg<0> {  // 256 rows x 128 channels
  static constexpr int WM = 2, WN = 2, SK = 1, MT = 4, NT = 2;
};
template <>
struct Cfg<1> {  // 256 rows x 64 channels (layers with <= 64 output channels)
  static constexpr int WM = 4, WN = 1, SK = 1, MT = 2, NT = 2;
};
template <>
struct Cfg<2> {  // 64 rows x 64 channels, K split over the four waves (small layers)
  static constexpr int WM = 1, WN = 1, SK = 4, MT = 2, NT = 2;
};
inline int cfg_rows(int cfg) { return cfg == 2 ? 64 : 256; }
inline int cfg_block_co(int cfg) { return cfg == 0 ? 128 : 64; }
constexpr int PARAM_BYTES = 2 * 128 * 4;  // per-channel epilogue parameters of the block, in LDS
constexpr int RED_BYTES = 4 * 4 * 16 * 64 * 4;  // split-K partial tiles: 4 waves x 4 tiles

struct MfmaArgs {
  ConvArgs c;
  const uint8_t* wx;  // expanded weights in the chosen operand format
  int wx_bytes;       // size of that operand copy (bounds of the B buffer reads)
  int pool;           // units are 2x2 windows
  int upi;            // units per image
  int uw;             // units per output row
  FastDiv fd_upi, fd_uw;
  int ipb;            // whole images per block (1: the block is a run of units of one image)
  int bpi;            // ipb == 1: blocks per image
  int units_pb;       // units per block
  int hr, hc;         // halo rows / cols per image slot
  int slot_pix;       // hr * hc
  FastDiv fd_slot, fd_hc, fd_cwc;
  int pix_bytes;      // LDS bytes per halo pixel
  int chunk_words;    // words staged per chunk
  int ksteps;         // k-steps per tap over all words (int8: cw, fp4: ceil(cw/2), fp16: 2 cw)
  int nchunks;
  int vec;            // upi % 4 == 0: four consecutive units are one aligned 16-byte run
  int tiles_px, tiles_co;
  int halo_bytes;
  int ht_needed;      // requantization thresholds reach 1: apply HardTanh before comparing
  int out_bytes;      // byte size of the unpacked output (buffer-resource bound, < 2^31)
  int buf_bytes;      // LDS bytes of one halo buffer
  int grid;           // blocks launched (each loops over the work items)
  int act_bytes;      // byte size of the packed activations (buffer-resource bound; 0 if >= 2^31)
};

// One 32 x 32 MFMA of operand format OPK on 16-byte fragments.
template <int OPK, class AccT>
__device__ __forceinline__ AccT mfma(v4i a, v4i b, AccT c) {
  if constexpr (OPK == OP_I8) {
    return __builtin_amdgcn_mfma_i32_32x32x32_i8(a, b, c, 0, 0, 0);
  } else if constexpr (OPK == OP_FP4) {
    v8i a8 = {a[0], a[1], a[2], a[3], 0, 0, 0, 0};
    v8i b8 = {b[0], b[1], b[2], b[3], 0, 0, 0, 0};
    // operand format 4 = E2M1 for both; scales 127 = 2^0
    return __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, c, 4, 4, 0, 127, 0, 127);
  } else {
    return __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(v8h, a), __builtin_bit_cast(v8h, b), c, 0,
                                                  0, 0);
  }
}
// Accumulator register as an exact float / int.
__device__ __forceinline__ float acc_f(const v16i& a, int v) { return (float)a[v]; }
__device__ __forceinline__ float acc_f(const v16f& a, int v) { return a[v]; }
__device__ __forceinline__ int acc_i(const v16i& a, int v) { return a[v]; }
__device__ __forceinline__ int acc_i(const v16f& a, int v) { return (int)a[v]; }

// One word of a halo pixel into LDS in operand format OPK.  fp16: a word of
// 16-bit inputs is already an operand (64 bytes copied as they are); the
// bitplanes of 1..3-bit inputs (against 16-bit weights) become the fp16
// codes of their levels.
template <int OPK, int PA>
__device__ __forceinline__ void expand_to_lds(const uint32_t* pl, uint8_t* dst) {
  if constexpr (OPK == OP_F16 && PA == 16) {
#pragma unroll
    for (int q = 0; q < 4; ++q)
      reinterpret_cast<uint4*>(dst)[q] = make_uint4(pl[4 * q], pl[4 * q + 1], pl[4 * q + 2], pl[4 * q + 3]);
  } else if constexpr (OPK == OP_F16) {
    uint32_t o[8], h[16];
    expand_i8_word<PA>(pl, 0xFFFFFFFFu, o);
#pragma unroll
    for (int q = 0; q < 8; ++q) i8_word_to_f16(o[q], &h[2 * q], &h[2 * q + 1]);
#pragma unroll
    for (int q = 0; q < 4; ++q)
      reinterpret_cast<uint4*>(dst)[q] = make_uint4(h[4 * q], h[4 * q + 1], h[4 * q + 2], h[4 * q + 3]);
  } else if constexpr (OPK == OP_FP4) {
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

template <int P>
__device__ __forceinline__ void store_words(uint32_t* dst, const uint32_t* w) {
  if constexpr (P == 1)
    *dst = w[0];
  else if constexpr (P == 2)
    *reinterpret_cast<uint2*>(dst) = make_uint2(w[0], w[1]);
  else
    *reinterpret_cast<uint4*>(dst) = make_uint4(w[0], w[1], w[2], w[3]);
}

// Image and in-image unit of block unit t; false past the end of the block's work.
__device__ __forceinline__ bool unit_of(const MfmaArgs& m, int img0, int u0, int t, int* img, int* uu) {
  if (m.ipb == 1) {
    *img = img0;
    *uu = u0 + t;
    return *uu < m.upi;
  }
  const int slot = (int)fdiv((uint32_t)t, m.fd_upi);
  *img = img0 + slot;
  *uu = t - slot * m.upi;
  return (slot < m.ipb) & (*img < m.c.n);
}

enum EpiKind { K_INT32 = 0, K_SCALE = 1, K_BNF32 = 2, K_PACK = 3 };

// Epilogue of one 32 x 32 accumulator tile: M-tile T of the block (units
// 32T.. or, pooled, windows 8T..) x output channels co32 .. co32 + 31.
// KIND: what the unpacked output holds; OB: bits of the packed output
// (0 = none); POOL: units are 2x2 windows.
template <int KIND, int OB, int POOL, class AccT>
__device__ __forceinline__ void tile_epilogue(const MfmaArgs& m, const AccT& acc, int img0, int u0,
                                              int T, int co32, float kk, float bb, int lane) {
  const ConvArgs& a = m.c;
  constexpr int POUT = OB ? planes_of(OB) : 1;
  const int g = lane >> 5, r32 = lane & 31;
  const float inv = 1.0f / (float)(1 << a.shift);
  const int co = co32 + r32;
  const bool cok = co < a.cout;
  const int64_t oplane = (int64_t)m.upi;  // NCHW channel-plane stride of the output
  uint32_t pw[POUT];  // packed words of this tile, gathered into lanes
#pragma unroll
  for (int p = 0; p < POUT; ++p) pw[p] = 0u;

  constexpr int NQ = POOL ? 1 : 4;  // 16-byte groups per lane: 4 plain, 1 pooled
  Unroll<0, NQ>::run([&](auto QI) {
    constexpr int QQ = decltype(QI)::value;
    // the lane's four consecutive units
    const int t0 = POOL ? 8 * T + 4 * g : 32 * T + 8 * QQ + 4 * g;
    int img, uu;
    const bool ok0 = unit_of(m, img0, u0, t0, &img, &uu);
    float z[4];
    int zi[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      if constexpr (POOL) {
        // window i: registers 4i .. 4i + 3; an int32 accumulator takes its
        // maximum as an integer (exact at any magnitude), an fp32 one (exact
        // integers below 2^24) as a float
        if constexpr (std::is_same<AccT, v16i>::value) {
          zi[i] = max(max(acc[4 * i], acc[4 * i + 1]), max(acc[4 * i + 2], acc[4 * i + 3]));
          z[i] = (float)zi[i] * inv;
        } else {
          const float m4 = fmaxf(fmaxf(acc_f(acc, 4 * i), acc_f(acc, 4 * i + 1)),
                                 fmaxf(acc_f(acc, 4 * i + 2), acc_f(acc, 4 * i + 3)));
          zi[i] = (int)m4;
          z[i] = m4 * inv;
        }
      } else {
        zi[i] = acc_i(acc, 4 * QQ + i);
        z[i] = acc_f(acc, 4 * QQ + i) * inv;
      }
      if constexpr (KIND == K_SCALE) z[i] = kk * z[i];
      if constexpr (KIND == K_BNF32 || KIND == K_PACK) z[i] = fmaf(kk, z[i], bb);
    }
    // unpacked output (+ residual)
    if constexpr (KIND != K_PACK) {
      if (m.vec) {
        if (ok0 && cok) {
          const int64_t oi = ((int64_t)img * a.cout + co) * oplane + uu;
          if constexpr (KIND == K_BNF32) {
            if (a.residual_on) {
              const float4 rv = *reinterpret_cast<const float4*>(a.residual + oi);
              z[0] = z[0] + rv.x;
              z[1] = z[1] + rv.y;
              z[2] = z[2] + rv.z;
              z[3] = z[3] + rv.w;
            }
          }
          if constexpr (KIND == K_INT32)
            *reinterpret_cast<int4*>(static_cast<int32_t*>(a.out) + oi) = make_int4(zi[0], zi[1], zi[2], zi[3]);
          else
            *reinterpret_cast<float4*>(static_cast<float*>(a.out) + oi) = make_float4(z[0], z[1], z[2], z[3]);
        }
      } else {
        for (int i = 0; i < 4; ++i) {
          int im, ui;
          if (!unit_of(m, img0, u0, t0 + i, &im, &ui) || !cok) continue;
          const int64_t oi = ((int64_t)im * a.cout + co) * oplane + ui;
          float zv = z[0];
          int ziv = zi[0];
          if (i == 1) { zv = z[1]; ziv = zi[1]; }
          if (i == 2) { zv = z[2]; ziv = zi[2]; }
          if (i == 3) { zv = z[3]; ziv = zi[3]; }
          if constexpr (KIND == K_BNF32) {
            if (a.residual_on) zv = zv + a.residual[oi];
          }
          if constexpr (KIND == K_INT32)
            static_cast<int32_t*>(a.out)[oi] = ziv;
          else
            static_cast<float*>(a.out)[oi] = zv;
          if constexpr (OB > 0) {
            if (i == 0) z[0] = zv;
            if (i == 1) z[1] = zv;
            if (i == 2) z[2] = zv;
            if (i == 3) z[3] = zv;
          }
        }
      }
    }
    // packed output: one ballot per (unit, plane); lanes 0-31 hold unit
    // t0 + i of half g = 0, lanes 32-63 that of half g = 1
    if constexpr (OB > 0) {
      uint64_t bl[4][POUT];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        float zz = z[i];
        if (m.ht_needed) zz = hardtanh(zz);
        int im, ui;
        const bool uok = unit_of(m, img0, u0, t0 + i, &im, &ui);
        plane_ballots<OB>(zz, uok & cok, a.othr, bl[i]);
      }
      constexpr int B = POOL ? 0 : 8 * QQ;
#pragma unroll
      for (int p = 0; p < POUT; ++p)
        pw[p] = writelanes8<B, B + 1, B + 2, B + 3, B + 4, B + 5, B + 6, B + 7>(
            pw[p], (uint32_t)bl[0][p], (uint32_t)bl[1][p], (uint32_t)bl[2][p], (uint32_t)bl[3][p],
            (uint32_t)(bl[0][p] >> 32), (uint32_t)(bl[1][p] >> 32), (uint32_t)(bl[2][p] >> 32),
            (uint32_t)(bl[3][p] >> 32));
    }
  });
  if constexpr (OB > 0) {
    // lane L < (POOL ? 8 : 32) stores the words of tile unit L
    const int nl = POOL ? 8 : 32;
    int img, uu;
    if (lane < nl && unit_of(m, img0, u0, nl * T + lane, &img, &uu)) {
      uint32_t* dst = a.out_packed + (((int64_t)img * m.upi + uu) * a.out_cw + (co32 >> 5)) * POUT;
      store_words<POUT>(dst, pw);
    }
  }
}

// Plane bits of Q(HardTanh(z)) for the 16 values a lane holds in the
// swapped orientation (Eqs. 4, 21, 22; the quantizer's compares): value
// v = 4q + i goes to bit 8q + i; the caller shifts the words by 4g, masks
// missing channels and merges the other half of the word.  HT: apply
// HardTanh first (only when a threshold reaches 1 does it change a result).
template <int OB, bool HT>
__device__ __forceinline__ void swap_plane_bits(const float (&zs)[16], const Thr& t, uint32_t* pw) {
#pragma unroll
  for (int v = 0; v < 16; ++v) {
    const int pos = 8 * (v / 4) + (v % 4);
    const float zz = HT ? hardtanh(zs[v]) : zs[v];
    const uint32_t s = zz > 0.0f ? 1u : 0u;
    if constexpr (OB == 1) {
      pw[0] |= s << pos;
    } else if constexpr (OB == 2) {
      const uint32_t nz = !(fabsf(zz) <= t.t0) ? 1u : 0u;
      pw[0] |= (s & nz) << pos;
      pw[1] |= nz << pos;
    } else {
      const float az = fabsf(zz);
      const uint32_t a1 = !(az <= t.t0) ? 1u : 0u;
      const uint32_t a2 = !(az <= t.t1) ? 1u : 0u;
      const uint32_t a3 = !(az <= t.t2) ? 1u : 0u;
      pw[0] |= (s & a1) << pos;
      pw[1] |= a3 << pos;
      pw[2] |= (a2 & ~a3) << pos;
      pw[3] |= (a1 & ~a2) << pos;
    }
  }
}

// Residual values of one tile of the swapped orientation (register
// v = 4q + i of lane l: channel co32 + 8q + 4(l/32) + i, unit 32T + l%32),
// loaded in one batch: on gfx9 loads and stores share one in-order counter,
// so a residual load issued after a store also waits for that store.
__device__ __forceinline__ void swap_res_load(const MfmaArgs& m, int img0, int u0, int T, int co32, int lane,
                                              float (&r)[16]) {
  const ConvArgs& a = m.c;
  const int g = lane >> 5, r32 = lane & 31;
  int img, uu;
  const bool uok = unit_of(m, img0, u0, 32 * T + r32, &img, &uu);
  const int voff = uok ? (int)((((int64_t)img * a.cout + co32 + 4 * g) * m.upi + uu) * 4) : 0x7FFFFFF0;
  const __amdgpu_buffer_rsrc_t rrsrc =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.residual, (short)0, m.out_bytes, 0x00020000);
  const int pstride = m.upi * 4;
#pragma unroll
  for (int v = 0; v < 16; ++v)
    r[v] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rrsrc, voff, (8 * (v / 4) + v % 4) * pstride, 0));
}

// Epilogue of one tile in the swapped orientation (weights as the A
// operand; RES: 0 no residual, 1 residual, 2 as the arguments say; the
// residual values come from `pre` when given, else from one batch of loads
// before the tile's stores): register v = 4q + i of lane l holds output channel
// co32 + 8q + 4(l/32) + i of unit 32T + l%32.  Each register is one store
// instruction writing two 128-byte runs (32 consecutive units of two
// channels) through a buffer resource; the per-register part of the offset
// is a scalar.  Lanes whose unit does not exist get an offset past the end
// of the buffer, so their stores and residual loads are dropped.  The
// block's per-channel parameters come from LDS.
// OB > 0: the packed planes of Q(HardTanh(z)) (Eqs. 4, 21, 22) as well (KIND
// K_PACK: only those).  A lane holds 16 of the 32 channels of its unit, so
// it sets its 16 bits of each plane word with the quantizer's compares, and
// one exchange with lane l ^ 32 completes the word, which lanes 0-31 store
// (PERM: through v_permlane32_swap, else a shuffle through LDS, which takes
// no extra register).
template <int KIND, int RES = 2, int OB = 0, bool PERM = false, class AccT>
__device__ __forceinline__ void tile_epilogue_swap(const MfmaArgs& m, const AccT& acc, int img0, int u0,
                                                   int T, int co32, int co_blk, const float* prm,
                                                   int lane, const float (*pre)[16] = nullptr) {
  constexpr int POUT = OB ? planes_of(OB) : 1;
  uint32_t pw[POUT];
#pragma unroll
  for (int p = 0; p < POUT; ++p) pw[p] = 0u;
  float zs[16];  // z of the 16 values, for the packed planes
  const ConvArgs& a = m.c;
  const int g = lane >> 5, r32 = lane & 31;
  const float inv = 1.0f / (float)(1 << a.shift);
  int img, uu;
  const bool uok = unit_of(m, img0, u0, 32 * T + r32, &img, &uu);
  const int cbase = co32 + 4 * g;
  const int voff = uok ? (int)((((int64_t)img * a.cout + cbase) * m.upi + uu) * 4) : 0x7FFFFFF0;
  const __amdgpu_buffer_rsrc_t orsrc =
      __builtin_amdgcn_make_buffer_rsrc(a.out, (short)0, m.out_bytes, 0x00020000);
  const bool res = KIND == K_BNF32 && (RES == 1 || (RES == 2 && a.residual_on));
  float rv[16];
  if (res) {
    if (pre) {
#pragma unroll
      for (int v = 0; v < 16; ++v) rv[v] = (*pre)[v];
    } else {
      swap_res_load(m, img0, u0, T, co32, lane, rv);
    }
  }
  const bool full = co32 + 32 <= a.cout;  // uniform: no channel of the tile is missing
  const int pstride = m.upi * 4;
#pragma unroll
  for (int q = 0; q < 4; ++q) {
    float4 k4 = make_float4(0.f, 0.f, 0.f, 0.f), b4 = k4;
    if constexpr (KIND != K_INT32) {
      const int pc = co32 - co_blk + 8 * q + 4 * g;
      k4 = *reinterpret_cast<const float4*>(prm + pc);
      b4 = *reinterpret_cast<const float4*>(prm + 128 + pc);
    }
    const float kv[4] = {k4.x, k4.y, k4.z, k4.w};
    const float bv[4] = {b4.x, b4.y, b4.z, b4.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int so = (8 * q + i) * pstride;
      uint32_t bits;
      float z = 0.0f;
      if constexpr (KIND == K_INT32) {
        bits = (uint32_t)acc_i(acc, 4 * q + i);
      } else {
        z = acc_f(acc, 4 * q + i) * inv;
        if constexpr (KIND == K_SCALE) z = kv[i] * z;
        if constexpr (KIND == K_BNF32 || KIND == K_PACK) z = fmaf(kv[i], z, bv[i]);
        if constexpr (KIND == K_BNF32) {
          if (res) z = z + rv[4 * q + i];
        }
        bits = __float_as_uint(z);
      }
      if constexpr (KIND != K_PACK) {
        if (full || cbase + 8 * q + i < a.cout) __builtin_amdgcn_raw_buffer_store_b32(bits, orsrc, voff, so, 0);
      }
      zs[4 * q + i] = z;
    }
  }
  if constexpr (OB > 0) {
    if (m.ht_needed)
      swap_plane_bits<OB, true>(zs, a.othr, pw);
    else
      swap_plane_bits<OB, false>(zs, a.othr, pw);
    if (!full) {
      // channels past the last one are 0 in every plane: bit 8q + i holds
      // channel cbase + 8q + i
      const int lim = a.cout - cbase;
      uint32_t vm = 0u;
#pragma unroll
      for (int q = 0; q < 4; ++q) {
        const int nb = min(max(lim - 8 * q, 0), 4);
        vm |= ((1u << nb) - 1u) << (8 * q);
      }
#pragma unroll
      for (int p = 0; p < POUT; ++p) pw[p] &= vm;
    }
#pragma unroll
    for (int p = 0; p < POUT; ++p) {
      pw[p] <<= 4 * g;  // this lane's channels are cbase + ...: nibbles of half g
      if constexpr (PERM) {
        // lanes 0-31 take the word of lane l + 32 (one VALU op, no LDS round
        // trip); OR-ing both results is the same whichever of the two
        // carries the swapped half
        const auto sw = __builtin_amdgcn_permlane32_swap(pw[p], pw[p], false, false);
        pw[p] |= sw[0] | sw[1];
      } else {
        pw[p] |= (uint32_t)__shfl_xor((int)pw[p], 32);
      }
    }
    if (g == 0 && uok) {
      uint32_t* dst = a.out_packed + (((int64_t)img * m.upi + uu) * a.out_cw + (co32 >> 5)) * POUT;
      store_words<POUT>(dst, pw);
    }
  }
}

// The swapped tile epilogue for the layer's output mode.
template <class AccT>
__device__ __forceinline__ void tile_epilogue_swap_mode(const MfmaArgs& m, const AccT& acc, int img0, int u0,
                                                        int T, int co32, int co_blk, const float* prm,
                                                        int lane) {
  const ConvArgs& a = m.c;
  const int ob = a.out_packed ? a.out_bits : 0;
  if (a.mode == QCONV_EPI_INT32) {
    tile_epilogue_swap<K_INT32>(m, acc, img0, u0, T, co32, co_blk, prm, lane);
  } else if (a.mode == QCONV_EPI_SCALE_F32) {
    tile_epilogue_swap<K_SCALE>(m, acc, img0, u0, T, co32, co_blk, prm, lane);
  } else if (a.mode == QCONV_EPI_BN_F32) {
    if (ob == 0) tile_epilogue_swap<K_BNF32, 2, 0>(m, acc, img0, u0, T, co32, co_blk, prm, lane);
    else if (ob == 1) tile_epilogue_swap<K_BNF32, 2, 1>(m, acc, img0, u0, T, co32, co_blk, prm, lane);
    else if (ob == 2) tile_epilogue_swap<K_BNF32, 2, 2>(m, acc, img0, u0, T, co32, co_blk, prm, lane);
    else tile_epilogue_swap<K_BNF32, 2, 3>(m, acc, img0, u0, T, co32, co_blk, prm, lane);
  } else {
    if (ob == 1) tile_epilogue_swap<K_PACK, 0, 1>(m, acc, img0, u0, T, co32, co_blk, prm, lane);
    else if (ob == 2) tile_epilogue_swap<K_PACK, 0, 2>(m, acc, img0, u0, T, co32, co_blk, prm, lane);
    else tile_epilogue_swap<K_PACK, 0, 3>(m, acc, img0, u0, T, co32, co_blk, prm, lane);
  }
}

// The epilogue over the wave's MT x NT tiles.  The per-channel parameters
// come from the block's LDS copy (kk at prm[c], bb at prm[128 + c] for
// channel co_blk + c).  UNROLL: the tiles as a compile-time sequence, so that
// independent tiles' loads, arithmetic and stores interleave; otherwise a
// loop at run time that copies one tile at a time out of the (statically
// indexed) accumulator array, which keeps the code of the rarely used output
// modes small.
template <int KIND, int OB, int POOL, bool UNROLL, int MT, int NT, class AccT>
__device__ __forceinline__ void epilogue(const MfmaArgs& m, const AccT (&acc)[MT][NT], int img0,
                                         int u0, int tile_m0, int co_w, int co_blk, const float* prm, int lane) {
  const ConvArgs& a = m.c;
  const int r32 = lane & 31;
  auto one = [&](const AccT& t, int i, int j) __attribute__((always_inline)) {
    const int co32 = co_w + 32 * j;
    const int c = co32 - co_blk + r32;
    const float kj = KIND == K_INT32 ? 0.0f : prm[c];
    const float bj = (KIND == K_BNF32 || KIND == K_PACK) ? prm[128 + c] : 0.0f;
    tile_epilogue<KIND, OB, POOL>(m, t, img0, u0, tile_m0 + i, co32, kj, bj, lane);
  };
  if constexpr (UNROLL) {
    Unroll<0, MT * NT>::run([&](auto TT) {
      constexpr int tt = decltype(TT)::value;
      if (co_w + 32 * (tt % NT) < a.cout) one(acc[tt / NT][tt % NT], tt / NT, tt % NT);  // uniform
    });
  } else {
#pragma nounroll
    for (int tt = 0; tt < MT * NT; ++tt) {
      const int i = tt / NT, j = tt - (tt / NT) * NT;
      if (co_w + 32 * j >= a.cout) continue;  // uniform: tile past the last channel
      AccT cur;
      switch (tt) {
#define QC_PICK(K)                   \
  case K:                            \
    if constexpr (K < MT * NT) cur = acc[K / NT][K % NT]; \
    break;
        QC_PICK(0) QC_PICK(1) QC_PICK(2) QC_PICK(3) QC_PICK(4) QC_PICK(5) QC_PICK(6) QC_PICK(7)
#undef QC_PICK
        default: break;
      }
      one(cur, i, j);
    }
  }
}

// The packed and BN outputs of pooled layers (the case of this orientation
// in networks) run the unrolled tile sequence; other outputs the loop.
template <int KIND, int POOL, int MT, int NT, class AccT>
__device__ __forceinline__ void epilogue_ob(const MfmaArgs& m, const AccT (&acc)[MT][NT], int img0,
                                            int u0, int tile_m0, int co_w, int co_blk, const float* prm, int lane) {
  const int ob = m.c.out_packed ? m.c.out_bits : 0;
  constexpr bool U = POOL == 1;  // unpooled layers take the swapped orientation
  if (ob == 0) epilogue<KIND, 0, POOL, U && KIND == K_BNF32>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane);
  else if (ob == 1) epilogue<KIND, 1, POOL, U>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane);
  else if (ob == 2) epilogue<KIND, 2, POOL, U>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane);
  else epilogue<KIND, 3, POOL, U>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane);
}

template <int POOL, int MT, int NT, class AccT>
__device__ __forceinline__ void epilogue_mode(const MfmaArgs& m, const AccT (&acc)[MT][NT], int img0,
                                              int u0, int tile_m0, int co_w, int co_blk, const float* prm,
                                              int lane) {
  switch (m.c.mode) {
    case QCONV_EPI_INT32:
      epilogue<K_INT32, 0, POOL, false>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane);
      break;
    case QCONV_EPI_SCALE_F32:
      epilogue<K_SCALE, 0, POOL, false>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane);
      break;
    case QCONV_EPI_BN_F32: epilogue_ob<K_BNF32, POOL>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane); break;
    default: epilogue_ob<K_PACK, POOL>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane); break;
  }
}

// The swapped epilogue over the wave's MT x NT tiles: packed and BN outputs
// as an unrolled tile sequence (mode fixed at compile time), int32 and scaled
// outputs one tile at a time.
template <int KIND, int RES, int OB, int MT, int NT, class AccT>
__device__ __forceinline__ void epilogue_swap_tiles(const MfmaArgs& m, const AccT (&acc)[MT][NT], int img0,
                                                    int u0, int tile_m0, int co_w, int co_blk, const float* prm,
                                                    int lane) {
  Unroll<0, MT * NT>::run([&](auto TT) {
    constexpr int tt = decltype(TT)::value;
    const int co32 = co_w + 32 * (tt % NT);
    if (co32 < m.c.cout)  // uniform
      tile_epilogue_swap<KIND, RES, OB, true>(m, acc[tt / NT][tt % NT], img0, u0, tile_m0 + tt / NT, co32, co_blk,
                                              prm, lane);
  });
}

template <int MT, int NT, class AccT>
__device__ __forceinline__ void epilogue_swap_all(const MfmaArgs& m, const AccT (&acc)[MT][NT], int img0, int u0,
                                                  int tile_m0, int co_w, int co_blk, const float* prm, int lane) {
  const ConvArgs& a = m.c;
  const int ob = a.out_packed ? a.out_bits : 0;
  if (a.mode == QCONV_EPI_BN_PACK) {
    if (ob == 1) epilogue_swap_tiles<K_PACK, 0, 1>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane);
    else if (ob == 2) epilogue_swap_tiles<K_PACK, 0, 2>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane);
    else epilogue_swap_tiles<K_PACK, 0, 3>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane);
  } else if (a.mode == QCONV_EPI_BN_F32) {
    if (ob == 0) epilogue_swap_tiles<K_BNF32, 2, 0>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane);
    else if (ob == 1) epilogue_swap_tiles<K_BNF32, 2, 1>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane);
    else if (ob == 2) epilogue_swap_tiles<K_BNF32, 2, 2>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane);
    else epilogue_swap_tiles<K_BNF32, 2, 3>(m, acc, img0, u0, tile_m0, co_w, co_blk, prm, lane);
  } else {
    const int r32 = lane & 31;
    (void)r32;
#pragma nounroll
    for (int tt = 0; tt < MT * NT; ++tt) {
      const int i = tt / NT, j = tt - (tt / NT) * NT;
      const int co32 = co_w + 32 * j;
      if (co32 >= a.cout) continue;
      AccT tcur;
      switch (tt) {
#define QC_PICK(K)                                         \
  case K:                                                  \
    if constexpr (K < MT * NT) tcur = acc[K / NT][K % NT]; \
    break;
        QC_PICK(0) QC_PICK(1) QC_PICK(2) QC_PICK(3) QC_PICK(4) QC_PICK(5) QC_PICK(6) QC_PICK(7)
#undef QC_PICK
        default: break;
      }
      tile_epilogue_swap_mode(m, tcur, img0, u0, tile_m0 + i, co32, co_blk, prm, lane);
    }
  }
}

// Geometry of one work item (a pixel tile x a channel tile) as seen by one lane.
template <int MT>
struct Item {
  int img0, u0, co_blk, iy0;
  int abase[MT];  // LDS byte offset (tap (0, 0), this lane's k-half) of the pixel fed into row r32 of each M-tile
};

// First image and first unit of work item w.
__device__ __forceinline__ void item_units(const MfmaArgs& m, int w, int* img0, int* u0) {
  const int pt = w / m.tiles_co;
  if (m.ipb == 1) {
    *img0 = pt / m.bpi;
    *u0 = (pt - *img0 * m.bpi) * m.units_pb;
  } else {
    *img0 = pt * m.ipb;
    *u0 = 0;
  }
}

// Image and first input row of the halo tile of work item w.
__device__ __forceinline__ void item_origin(const MfmaArgs& m, int w, int* img0, int* iy0) {
  const int pt = w / m.tiles_co;
  int u0;
  if (m.ipb == 1) {
    *img0 = pt / m.bpi;
    u0 = (pt - *img0 * m.bpi) * m.units_pb;
  } else {
    *img0 = pt * m.ipb;
    u0 = 0;
  }
  const int uy0 = (int)fdiv((uint32_t)u0, m.fd_uw);
  *iy0 = (m.pool ? 2 * uy0 : uy0) * m.c.stride - m.c.pad;
}

template <int MT, int NT, int WN>
__device__ __forceinline__ void decode_item(const MfmaArgs& m, int w, int wm, int r32, int g, Item<MT>* it) {
  const ConvArgs& a = m.c;
  const int pt = w / m.tiles_co;
  const int ct = w - pt * m.tiles_co;
  it->co_blk = ct * (32 * NT * WN);
  if (m.ipb == 1) {
    it->img0 = pt / m.bpi;
    it->u0 = (pt - it->img0 * m.bpi) * m.units_pb;
  } else {
    it->img0 = pt * m.ipb;
    it->u0 = 0;
  }
  // first conv row held in the halo tile (ipb > 1: every slot starts at row 0)
  const int uy0 = (int)fdiv((uint32_t)it->u0, m.fd_uw);
  const int oy0 = m.pool ? 2 * uy0 : uy0;
  it->iy0 = oy0 * a.stride - a.pad;
#pragma unroll
  for (int i = 0; i < MT; ++i) {
    const int T = wm * MT + i;
    int unit, e = 0;
    if (m.pool) {
      unit = 8 * T + 4 * ((r32 >> 2) & 1) + (r32 >> 3);
      e = r32 & 3;
    } else {
      unit = 32 * T + r32;
    }
    int img, uu;
    if (!unit_of(m, it->img0, it->u0, unit, &img, &uu)) {
      uu = it->u0;  // a row past the end: read any valid pixel, its result is dropped
      img = it->img0;
    }
    const int slot = img - it->img0;
    const int uy = (int)fdiv((uint32_t)uu, m.fd_uw);
    const int ux = uu - uy * m.uw;
    const int oy = m.pool ? 2 * uy + (e >> 1) : uy;
    const int ox = m.pool ? 2 * ux + (e & 1) : ux;
    const int hp = slot * m.slot_pix + (oy - oy0) * a.stride * m.hc + ox * a.stride;
    it->abase[i] = hp * m.pix_bytes + g * 16;
  }
}

// Packed words of this thread's share of a halo tile: item it = tid + 256 u
// is (halo pixel it / chunk_words, word it % chunk_words).  Pixels outside
// the image and words past the last channel read as 0 (= Q(0)).
template <int PA, int NI, int NR>
__device__ __forceinline__ void load_halo(const MfmaArgs& m, int img0, int iy0, int chunk, int tid,
                                          uint32_t (&raw)[NR][PA]) {
  static_assert(NI <= NR, "items past the register array");
  const ConvArgs& a = m.c;
  const int items = m.ipb * m.slot_pix * m.chunk_words;
  const int apix = a.cw * PA;
#pragma unroll
  for (int u = 0; u < NI; ++u) {
    const int it = tid + 256 * u;
#pragma unroll
    for (int p = 0; p < PA; ++p) raw[u][p] = 0u;
    if (it < items) {
      const int hp = (int)fdiv((uint32_t)it, m.fd_cwc);
      const int cwl = it - hp * m.chunk_words;
      const int slot = (int)fdiv((uint32_t)hp, m.fd_slot);
      const int rem = hp - slot * m.slot_pix;
      const int hrow = (int)fdiv((uint32_t)rem, m.fd_hc);
      const int hcol = rem - hrow * m.hc;
      const int img = img0 + slot;
      const int iy = iy0 + hrow, ix = hcol - a.pad;
      const int cw = chunk * m.chunk_words + cwl;
      if (img < a.n && iy >= 0 && iy < a.h && ix >= 0 && ix < a.w && cw < a.cw) {
        const uint32_t* src = a.act + (((int64_t)img * a.h + iy) * a.w + ix) * apix + cw * PA;
        if constexpr (PA == 1) {
          raw[u][0] = src[0];
        } else if constexpr (PA == 2) {
          const uint2 v = *reinterpret_cast<const uint2*>(src);
          raw[u][0] = v.x;
          raw[u][1] = v.y;
        } else {
#pragma unroll
          for (int q = 0; q < PA / 4; ++q) {
            const uint4 v = reinterpret_cast<const uint4*>(src)[q];
            raw[u][4 * q] = v.x;
            raw[u][4 * q + 1] = v.y;
            raw[u][4 * q + 2] = v.z;
            raw[u][4 * q + 3] = v.w;
          }
        }
      }
    }
  }
}

// Expands this thread's share of a halo tile into an LDS buffer: the items
// already held in raw, then any items past NI * 256 loaded here directly.
template <int OPK, int PA, int NI, int NR>
__device__ __forceinline__ void store_halo(const MfmaArgs& m, int img0, int iy0, int chunk, int tid,
                                           const uint32_t (&raw)[NR][PA], uint8_t* buf) {
  const int items = m.ipb * m.slot_pix * m.chunk_words;
#pragma unroll
  for (int u = 0; u < NI; ++u) {
    const int it = tid + 256 * u;
    if (it < items) {
      const int hp = (int)fdiv((uint32_t)it, m.fd_cwc);
      const int cwl = it - hp * m.chunk_words;
      expand_to_lds<OPK, PA>(raw[u], buf + hp * m.pix_bytes + cwl * OpT<OPK>::WORD_BYTES);
    }
  }
  // the rest two at a time: both loads in flight before the first store
  for (int it = NI * 256 + tid; it < items; it += 512) {
    uint32_t two[2][PA];
    load_halo<PA, 2>(m, img0, iy0, chunk, it, two);
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int iu = it + 256 * u;
      if (iu < items) {
        const int hp = (int)fdiv((uint32_t)iu, m.fd_cwc);
        const int cwl = iu - hp * m.chunk_words;
        expand_to_lds<OPK, PA>(two[u], buf + hp * m.pix_bytes + cwl * OpT<OPK>::WORD_BYTES);
      }
    }
  }
}

// Per-channel parameters of the swapped epilogue for channels co_blk.. of the item.
template <int BCO>
__device__ __forceinline__ void load_params(const ConvArgs& a, int co_blk, int tid, float* prm) {
  if (tid < 2 * BCO) {
    const int half = tid / BCO, c = tid - half * BCO;
    const int cs = min(co_blk + c, a.cout - 1);
    float v = 0.0f;
    if (a.mode == QCONV_EPI_SCALE_F32) v = half ? 0.0f : a.scale[cs];
    else if (a.mode == QCONV_EPI_BN_F32 || a.mode == QCONV_EPI_BN_PACK) v = half ? a.bn_b[cs] : a.bn_k[cs];
    prm[half * 128 + c] = v;
  }
}

// The convolution kernel.  Blocks loop over work items (pixel tile x channel
// tile) with a stride of the grid size.  Each (item, channel chunk) is a
// stage; the packed words of stage s + 1 are loaded into registers before
// the MFMAs of stage s and expanded into the other of two LDS halo buffers
// after them, so that global latency, the expansion and the epilogue's
// stores overlap the matrix work.  Split-K shapes run one item per block.
template <int OPK, int PA, int CFG, int SWAP>
__global__ __launch_bounds__(256, blocks_per_cu(OPK, CFG)) void conv_mfma_kernel(const MfmaArgs m) {
  using O = OpT<OPK>;
  using acc_t = typename O::acc_t;
  using C = Cfg<CFG>;
  constexpr int MT = C::MT, NT = C::NT, WN = C::WN, SK = C::SK;
  constexpr int BCO = 32 * NT * WN;
  constexpr int NI = halo_items_per_thread(PA, CFG);  // halo items per thread and stage
  static_assert(SK == 1 || SK == MT * NT, "a split-K block has one tile per wave");
  extern __shared__ __attribute__((aligned(16))) uint8_t lds_raw[];
  const ConvArgs& a = m.c;
  // wave-uniform indices in scalar registers; per-lane indices are derived
  // afresh from fresh_tid() wherever a loop iteration needs them, so that
  // nothing computed from them stays live across the item loop (held there,
  // such values were spilled to scratch, and every reload waited for all
  // stores in flight: loads and stores share one in-order counter)
  const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  auto fresh_tid = [&]() __attribute__((always_inline)) {
    int t = tid;
    asm volatile("" : "+v"(t));
    return t;
  };
  const int wk = wave % SK;  // K-split index
  const int wmn = wave / SK;
  const int wm = wmn / WN, wn = wmn - (wmn / WN) * WN;
  const int g = lane >> 5, r32 = lane & 31;
  const int total = m.tiles_px * m.tiles_co;
  // LDS: two parameter sets, then two halo buffers
  float* prm_base = reinterpret_cast<float*>(lds_raw);
  uint8_t* halo_base = lds_raw + 2 * PARAM_BYTES;
  const int buf_bytes = m.buf_bytes;

  int w = blockIdx.x;
  if (w >= total) return;
  Item<MT> cur;
  decode_item<MT, NT, WN>(m, w, wm, r32, g, &cur);
  uint32_t raw[NI > 0 ? NI : 1][PA];
  load_halo<PA, NI>(m, cur.img0, cur.iy0, 0, tid, raw);
  load_params<BCO>(a, cur.co_blk, tid, prm_base);
  store_halo<OPK, PA, NI>(m, cur.img0, cur.iy0, 0, tid, raw, halo_base);
  lds_barrier();

  acc_t acc[MT][NT];
#pragma unroll
  for (int i = 0; i < MT; ++i)
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) acc[i][j][v] = 0;

  // B fragments are read through a buffer resource: the per-lane part of the
  // address is a vector offset, the per-step part a scalar offset, and reads
  // past the operand copy return 0.
  const __amdgpu_buffer_rsrc_t brsrc =
      __builtin_amdgcn_make_buffer_rsrc((void*)m.wx, (short)0, m.wx_bytes, 0x00020000);
  const int bstride = a.cop * 32;  // bytes between consecutive k-steps
  const int taps = a.kh * a.kw;
  const int steps_per_chunk = m.chunk_words * 32 / O::K_PER_STEP;
  int chunk = 0, sbuf = 0, ipar = 0;

  for (;;) {
    // ---- the next stage: its packed words go into registers now ----
    int nw = w, nchunk = chunk + 1;
    if (nchunk == m.nchunks) {
      nchunk = 0;
      nw = w + gridDim.x;
    }
    const bool has_next = nw < total;
    int nimg0 = cur.img0, niy0 = cur.iy0;
    if (has_next) {
      if (nchunk == 0) item_origin(m, nw, &nimg0, &niy0);
      load_halo<PA, NI>(m, nimg0, niy0, nchunk, fresh_tid(), raw);
    }

    // ---- MFMA over this wave's share of the (tap, k-step) steps of the stage ----
    // B fragments come from a ring of BRING register sets, each loaded
    // BRING - 1 steps before its MFMAs; A fragments are read from LDS one
    // step ahead.
    {
      const uint8_t* lds = halo_base + sbuf * buf_bytes;
      const int co_w = cur.co_blk + 32 * NT * wn;
      const int bt = fresh_tid();
      int bvoff[NT];
#pragma unroll
      for (int j = 0; j < NT; ++j) bvoff[j] = (co_w + 32 * j + (bt & 31)) * 32 + ((bt >> 5) & 1) * 16;
      const int ks0 = chunk * steps_per_chunk;
      const int spc = min(m.ksteps, ks0 + steps_per_chunk) - ks0;  // k-steps per tap in this chunk
      const int nsteps_all = taps * spc;
      const int sbeg = (nsteps_all * wk) / SK, send = (nsteps_all * (wk + 1)) / SK;
      const int nsteps = send - sbeg;
      if (nsteps > 0) {
        const int tap0 = sbeg / spc;
        int l_tap = tap0, l_ksl = sbeg - tap0 * spc, l_count = 0;
        auto bload = [&](v4i (&dstb)[NT]) {
          const int so = (l_tap * m.ksteps + ks0 + l_ksl) * bstride;
#pragma unroll
          for (int j = 0; j < NT; ++j)
            dstb[j] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(brsrc, bvoff[j], so, 0));
          if (l_count + 1 < nsteps) {  // the last step is reloaded past the end (never used)
            ++l_count;
            if (++l_ksl == spc) {
              l_ksl = 0;
              ++l_tap;
            }
          }
        };
        int r_ksl = sbeg - tap0 * spc, r_ky = tap0 / a.kw, r_kx = tap0 - (tap0 / a.kw) * a.kw, r_count = 0;
        auto aload = [&](v4i (&dsta)[MT]) {
          const int lo = (r_ky * m.hc + r_kx) * m.pix_bytes + r_ksl * 32;
#pragma unroll
          for (int i = 0; i < MT; ++i) dsta[i] = *reinterpret_cast<const v4i*>(lds + cur.abase[i] + lo);
          ++r_count;
          if (++r_ksl == spc) {
            r_ksl = 0;
            if (++r_kx == a.kw) {
              r_kx = 0;
              ++r_ky;
            }
          }
        };
        v4i Acur[MT], Anext[MT];
        auto step = [&](const v4i (&bf)[NT]) {
#pragma unroll
          for (int i = 0; i < MT; ++i) Acur[i] = Anext[i];
          if (r_count < nsteps) aload(Anext);
#pragma unroll
          for (int i = 0; i < MT; ++i)
#pragma unroll
            for (int j = 0; j < NT; ++j) {
              if constexpr (SWAP)
                acc[i][j] = mfma<OPK>(bf[j], Acur[i], acc[i][j]);
              else
                acc[i][j] = mfma<OPK>(Acur[i], bf[j], acc[i][j]);
            }
        };
        // ring of BRING register sets: the set of step st + BRING - 1 is
        // loaded just before the MFMAs of step st
        v4i Bq[BRING][NT];
        Unroll<0, BRING - 1>::run([&](auto D) { bload(Bq[decltype(D)::value]); });
        aload(Anext);
        for (int st = 0; st < nsteps; st += BRING) {
          Unroll<0, BRING>::run([&](auto D) {
            constexpr int d = decltype(D)::value;
            if (st + d < nsteps) {
              bload(Bq[(d + BRING - 1) % BRING]);
              step(Bq[d]);
            }
          });
        }
      }
    }

    // ---- the next stage's halo into the other buffer (the epilogue below
    // reads no halo buffer; a split-K block never has a next stage) ----
    if (has_next)
      store_halo<OPK, PA, NI>(m, nimg0, niy0, nchunk, fresh_tid(), raw, halo_base + (sbuf ^ 1) * buf_bytes);

    // ---- epilogue of a finished item ----
    if (chunk == m.nchunks - 1) {
      const int elane = fresh_tid() & 63;
      const float* prm = prm_base + ipar * (PARAM_BYTES / 4);
      const int co_w = cur.co_blk + 32 * NT * wn;
      if constexpr (SK > 1) {
        // split-K: sum the partial tiles through LDS (both halo buffers:
        // a split-K block has no next stage), one tile per wave
        // (the raw accumulator bits: int32 partials are summed as integers,
        // exact at any magnitude; fp32 ones hold exact integers below 2^24)
        lds_barrier();
        using elem_t = typename std::conditional<std::is_same<acc_t, v16i>::value, int, float>::type;
        typedef elem_t e4 __attribute__((ext_vector_type(4)));
        e4* red = reinterpret_cast<e4*>(halo_base);
#pragma unroll
        for (int i = 0; i < MT; ++i)
#pragma unroll
          for (int j = 0; j < NT; ++j)
#pragma unroll
            for (int v4 = 0; v4 < 4; ++v4) {
              e4 t;
              t.x = acc[i][j][4 * v4];
              t.y = acc[i][j][4 * v4 + 1];
              t.z = acc[i][j][4 * v4 + 2];
              t.w = acc[i][j][4 * v4 + 3];
              red[((wave * (MT * NT) + i * NT + j) * 4 + v4) * 64 + elane] = t;
            }
        lds_barrier();
        const int tile = wave;  // this wave's tile after the reduction
        acc_t sum;
#pragma unroll
        for (int v4 = 0; v4 < 4; ++v4) {
          e4 s4 = {0, 0, 0, 0};
#pragma unroll
          for (int ww = 0; ww < SK; ++ww) s4 += red[((ww * (MT * NT) + tile) * 4 + v4) * 64 + elane];
          sum[4 * v4] = s4.x;
          sum[4 * v4 + 1] = s4.y;
          sum[4 * v4 + 2] = s4.z;
          sum[4 * v4 + 3] = s4.w;
        }
        const int ti = tile / NT, tj = tile - (tile / NT) * NT;
        const int co32 = co_w + 32 * tj;
        if (co32 < a.cout) {
          if constexpr (SWAP) {
            tile_epilogue_swap_mode(m, sum, cur.img0, cur.u0, ti, co32, cur.co_blk, prm, elane);
          } else {
            acc_t one[1][1] = {{sum}};
            if (m.pool)
              epilogue_mode<1>(m, one, cur.img0, cur.u0, ti, co32, cur.co_blk, prm, elane);
            else
              epilogue_mode<0>(m, one, cur.img0, cur.u0, ti, co32, cur.co_blk, prm, elane);
          }
        }
      } else if (co_w < a.cout) {
        if constexpr (SWAP) {
          epilogue_swap_all(m, acc, cur.img0, cur.u0, wm * MT, co_w, cur.co_blk, prm, elane);
        } else {
          if (m.pool)
            epilogue_mode<1>(m, acc, cur.img0, cur.u0, wm * MT, co_w, cur.co_blk, prm, elane);
          else
            epilogue_mode<0>(m, acc, cur.img0, cur.u0, wm * MT, co_w, cur.co_blk, prm, elane);
        }
      }
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j)
#pragma unroll
          for (int v = 0; v < 16; ++v) acc[i][j][v] = 0;
    }

    if (!has_next) break;
    if (nchunk == 0) {
      ipar ^= 1;
      w = nw;
      const int dt = fresh_tid();
      decode_item<MT, NT, WN>(m, w, wm, dt & 31, (dt >> 5) & 1, &cur);
      load_params<BCO>(a, cur.co_blk, fresh_tid(), prm_base + ipar * (PARAM_BYTES / 4));
    }
    chunk = nchunk;
    sbuf ^= 1;
    lds_barrier();
  }
}

// s_waitcnt vmcnt(0): every vector memory access of the wave has completed.
__device__ __forceinline__ void vm_wait_all() { __builtin_amdgcn_s_waitcnt(0x0F70); }


// Packed words of this thread's share of a halo tile (items it = tid +
// STRIDE u, as in load_halo), read through a buffer resource over the packed
// activations: every lane issues every load, and words outside the image or
// past the last channel use an offset past the end of the buffer, which
// reads as 0 (= Q(0)).  The destination registers are written by the loads
// alone.
template <int PA, int NI, int STRIDE>
__device__ __forceinline__ void load_halo_rsrc(const MfmaArgs& m, __amdgpu_buffer_rsrc_t rsrc, int img0,
                                               int iy0, int tid, uint32_t (&raw)[NI][PA]) {
  const ConvArgs& a = m.c;
  const int items = m.ipb * m.slot_pix * m.chunk_words;
  const int apix = a.cw * PA;
#pragma unroll
  for (int u = 0; u < NI; ++u) {
    const int it = tid + STRIDE * u;
    const int hp = (int)fdiv((uint32_t)it, m.fd_cwc);
    const int cw = it - hp * m.chunk_words;
    const int slot = (int)fdiv((uint32_t)hp, m.fd_slot);
    const int rem = hp - slot * m.slot_pix;
    const int hrow = (int)fdiv((uint32_t)rem, m.fd_hc);
    const int hcol = rem - hrow * m.hc;
    const int img = img0 + slot;
    const int iy = iy0 + hrow, ix = hcol - a.pad;
    const bool ok = it < items && img < a.n && iy >= 0 && iy < a.h && ix >= 0 && ix < a.w && cw < a.cw;
    const int off = ok ? (((img * a.h + iy) * a.w + ix) * apix + cw * PA) * 4 : 0x7FFFFFF0;
    if constexpr (PA == 1) {
      raw[u][0] = __builtin_amdgcn_raw_buffer_load_b32(rsrc, off, 0, 0);
    } else if constexpr (PA == 2) {
      const auto v = __builtin_amdgcn_raw_buffer_load_b64(rsrc, off, 0, 0);
      raw[u][0] = v[0];
      raw[u][1] = v[1];
    } else {
      const auto v = __builtin_amdgcn_raw_buffer_load_b128(rsrc, off, 0, 0);
      raw[u][0] = v[0];
      raw[u][1] = v[1];
      raw[u][2] = v[2];
      raw[u][3] = v[3];
    }
  }
}

// Expands a thread's share of a halo tile into LDS: the NI items held in raw,
// then the items past NI * STRIDE, loaded here one at a time.
template <int OPK, int PA, int NI, int STRIDE>
__device__ __forceinline__ void expand_halo(const MfmaArgs& m, __amdgpu_buffer_rsrc_t rsrc, int img0, int iy0,
                                            int tid, const uint32_t (&raw)[NI][PA], uint8_t* buf) {
  const int items = m.ipb * m.slot_pix * m.chunk_words;
#pragma unroll
  for (int u = 0; u < NI; ++u) {
    const int it = tid + STRIDE * u;
    if (it < items) {
      const int hp = (int)fdiv((uint32_t)it, m.fd_cwc);
      expand_to_lds<OPK, PA>(raw[u], buf + hp * m.pix_bytes + (it - hp * m.chunk_words) * OpT<OPK>::WORD_BYTES);
    }
  }
  for (int it0 = NI * STRIDE; it0 < items; it0 += STRIDE) {
    uint32_t one[1][PA];
    load_halo_rsrc<PA, 1, STRIDE>(m, rsrc, img0, iy0, it0 + tid, one);
    const int it = it0 + tid;
    if (it < items) {
      const int hp = (int)fdiv((uint32_t)it, m.fd_cwc);
      expand_to_lds<OPK, PA>(one[0], buf + hp * m.pix_bytes + (it - hp * m.chunk_words) * OpT<OPK>::WORD_BYTES);
    }
  }
}

// Block shapes of the store-overlapped kernel: a group of 8 waves covers 256
// units x BCO channels, WM x WN waves of MT x NT tiles of 32 x 32.
template <int CFG>
struct PCfg;
template <>
struct PCfg<0> {  // 256 x 128
  static constexpr int WM = 4, WN = 2, MT = 2, NT = 2;
};
template <>
struct PCfg<1> {  // 256 x 64
  static constexpr int WM = 4, WN = 2, MT = 2, NT = 1;
};
constexpr int PP_GROUP = 512;  // threads per wave group

// Layers whose output is written unpacked in fp32/int32 are bound by those
// stores, and the store rate of a CU grows with the number of waves that
// store at once.  This variant runs 16 waves in one block per CU, in two
// groups of eight: while one group runs the MFMAs of an item, the other
// expands the halo tile of its next item and stores the item it finished
// before, and the roles swap at every LDS barrier.  The block's weights stay
// in LDS for the whole launch (every item of a block has the same output
// channels); the only global accesses of a computing group are the loads of
// its next halo tile, issued first so that they arrive under the MFMAs.  The
// stores are issued last in a phase and the barrier does not wait for them,
// so they drain while the same group computes its next item.
// The block's items are w = blockIdx.x + k * gridDim.x; group k % 2 owns
// item k, computes it in phase k and stores it in phase k + 1; its halo
// words are loaded in phase k - 2 (the prologue for k < 2) and expanded in
// phase k - 1.  Each group runs its own loop over pairs of phases, so that
// every path from one phase to the next is the program order (the loads of
// a compute phase are always consumed by the following store phase).
// LDS: parameters, weights [tap][k-step][k-half][channel][16 B], one halo
// buffer per group.  Serves unpacked, unpooled outputs (pixels as the A
// operand, so that a lane holds one channel); needs a single channel chunk
// and packed activations below 2 GiB.
template <int OPK, int PA, int CFG, int OB>
__global__ __launch_bounds__(1024, 1) void conv_mfma_pp_kernel(const MfmaArgs m) {
  using O = OpT<OPK>;
  using acc_t = typename O::acc_t;
  using C = PCfg<CFG>;
  constexpr int MT = C::MT, NT = C::NT, WN = C::WN;
  constexpr int BCO = 32 * NT * WN;
  constexpr int NI = PA == 4 ? 2 : 3;  // halo items per thread held in registers
  extern __shared__ __attribute__((aligned(16))) uint8_t lds_raw[];
  const ConvArgs& a = m.c;
  // wave-uniform indices in scalar registers
  const int tid = threadIdx.x, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int grp = wave >> 3, wq = wave & 7;
  const int wm = wq / WN, wn = wq - (wq / WN) * WN;
  const int total = m.tiles_px * m.tiles_co;
  if ((int)blockIdx.x >= total) return;
  const int n_my = (total - (int)blockIdx.x + (int)gridDim.x - 1) / (int)gridDim.x;
  const int taps = a.kh * a.kw;
  const int ksteps = m.ksteps;
  float* prm = reinterpret_cast<float*>(lds_raw);
  uint8_t* bw = lds_raw + PARAM_BYTES;
  const int bw_bytes = taps * ksteps * BCO * 32;
  uint8_t* halo = bw + bw_bytes + grp * m.buf_bytes;
  const int co_blk = ((int)blockIdx.x % m.tiles_co) * BCO;  // gridDim.x is a multiple of tiles_co
  const int co_w = co_blk + 32 * NT * wn;
  const __amdgpu_buffer_rsrc_t arsrc =
      __builtin_amdgcn_make_buffer_rsrc((void*)a.act, (short)0, m.act_bytes, 0x00020000);
  auto item_w = [&](int k) __attribute__((always_inline)) { return (int)blockIdx.x + k * (int)gridDim.x; };

  // ---- prologue: each group loads the halo words of its first item, then
  // all 16 waves copy the weights into LDS (up to eight 16-byte loads in
  // flight per thread, all issued before the first is used: one round for
  // up to 128 KB); group 1 then loads the parameters while group 0 expands
  // item 0 ----
  uint32_t raw[NI][PA];
  const int gtid0 = tid & (PP_GROUP - 1);
  int img0, iy0;
  item_origin(m, item_w(grp < n_my ? grp : 0), &img0, &iy0);
  load_halo_rsrc<PA, NI, PP_GROUP>(m, arsrc, img0, iy0, gtid0, raw);
  {
    const __amdgpu_buffer_rsrc_t brsrc =
        __builtin_amdgcn_make_buffer_rsrc((void*)m.wx, (short)0, m.wx_bytes, 0x00020000);
    const int chunks = taps * ksteps * BCO * 2;  // 16-byte pieces
    for (int c0 = 0; c0 < chunks; c0 += 8 * 2 * PP_GROUP) {
      // a thread past the last piece copies the last piece again (same
      // value, same place), so that every load is consumed
      v4i v[8];
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int c = min(c0 + u * 2 * PP_GROUP + tid, chunks - 1);
        const int tk = c / (2 * BCO);
        const int rem = c - tk * (2 * BCO);
        v[u] = __builtin_bit_cast(v4i, __builtin_amdgcn_raw_buffer_load_b128(
                                           brsrc, (tk * a.cop + co_blk + (rem >> 1)) * 32 + (rem & 1) * 16, 0, 0));
      }
#pragma unroll
      for (int u = 0; u < 8; ++u) {
        const int c = min(c0 + u * 2 * PP_GROUP + tid, chunks - 1);
        const int tk = c / (2 * BCO);
        const int rem = c - tk * (2 * BCO);
        *reinterpret_cast<v4i*>(bw + ((tk * 2 + (rem & 1)) * BCO + (rem >> 1)) * 16) = v[u];
      }
    }
  }
  if (grp == 1)
    load_params<BCO>(a, co_blk, gtid0, prm);
  else
    expand_halo<OPK, PA, NI, PP_GROUP>(m, arsrc, img0, iy0, gtid0, raw, halo);
  // Explicit waits for every outstanding global access where that costs
  // nothing (here, and at the start of each store phase, where the only ones
  // are the halo loads of a phase ago): no load issued before them is then
  // taken as pending anywhere in the loops below, so the compute phases
  // never wait for the stores still draining from the phase before.
  vm_wait_all();
  lds_barrier();

  // Accumulators and the loaded halo words are the only per-lane state
  // carried from one phase to the next; the first (tap, k-step) of an item
  // starts from a zero C operand, and the item geometry is recomputed in
  // every phase.
  acc_t acc[MT][NT];

  // The thread index passes through an empty asm in every phase, so that the
  // index arithmetic derived from it is recomputed there rather than hoisted
  // out of the loops (where it would be held in scratch memory).
  auto fresh_tid = [&]() __attribute__((always_inline)) {
    int t = tid;
    asm volatile("" : "+v"(t));
    return t;
  };

  // compute item k; first the halo words of item k + 2
  auto compute = [&](int k) __attribute__((always_inline)) {
    const int ptid = fresh_tid();
    const int plane = ptid & 63, pg = plane >> 5, pr32 = plane & 31;
    if (k + 2 < n_my) {
      int nimg0, niy0;
      item_origin(m, item_w(k + 2), &nimg0, &niy0);
      load_halo_rsrc<PA, NI, PP_GROUP>(m, arsrc, nimg0, niy0, ptid & (PP_GROUP - 1), raw);
    }
    Item<MT> cur;
    decode_item<MT, NT, WN>(m, item_w(k), wm, pr32, pg, &cur);
    int boff[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) boff[j] = (32 * NT * wn + 32 * j + pr32) * 16 + pg * (BCO * 16);
    // A (pixels) and B (weights) fragments from LDS in two register sets,
    // each read one (tap, k-step) before its MFMAs
    const int nsteps = taps * ksteps;
    int t_ky = 0, t_kx = 0, t_ks = 0, t_tk = 0;
    auto fetch = [&](v4i (&A)[MT], v4i (&B)[NT]) {
      const int lo = (t_ky * m.hc + t_kx) * m.pix_bytes + t_ks * 32;
#pragma unroll
      for (int i = 0; i < MT; ++i) A[i] = *reinterpret_cast<const v4i*>(halo + cur.abase[i] + lo);
      const uint8_t* bs = bw + t_tk * (2 * BCO * 16);
#pragma unroll
      for (int j = 0; j < NT; ++j) B[j] = *reinterpret_cast<const v4i*>(bs + boff[j]);
      ++t_tk;
      if (++t_ks == ksteps) {
        t_ks = 0;
        if (++t_kx == a.kw) {
          t_kx = 0;
          ++t_ky;
        }
      }
    };
    auto mm = [&](const v4i (&A)[MT], const v4i (&B)[NT]) {
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = mfma<OPK>(B[j], A[i], acc[i][j]);
    };
    v4i AX[MT], BX[NT], AY[MT], BY[NT];
    fetch(AX, BX);                  // step 0
    if (nsteps > 1) fetch(AY, BY);  // step 1
    {
      const acc_t zero = {};
#pragma unroll
      for (int i = 0; i < MT; ++i)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[i][j] = mfma<OPK>(BX[j], AX[i], zero);
    }
    // steps 1 .. nsteps - 1 in pairs (Y, X); reads run one step ahead
    int st = 1;
    for (; st + 2 < nsteps; st += 2) {
      fetch(AX, BX);  // step st + 1
      mm(AY, BY);     // step st
      fetch(AY, BY);  // step st + 2
      mm(AX, BX);     // step st + 1
    }
    if (st < nsteps) {
      if (st + 1 < nsteps) fetch(AX, BX);
      mm(AY, BY);
      if (st + 1 < nsteps) mm(AX, BX);
    }
  };

  // store item k - 1 and expand the halo words of item k + 1 (loaded a
  // phase ago), one halo item after each tile's stores: the stores' issue is
  // limited by the memory system, and the expansion fills those stalls
  auto store = [&](int k) __attribute__((always_inline)) {
    vm_wait_all();
    const int ptid = fresh_tid();
    const int plane = ptid & 63, gt = ptid & (PP_GROUP - 1);
    const bool stage = k + 1 < n_my;
    int nimg0 = 0, niy0 = 0;
    if (stage) item_origin(m, item_w(k + 1), &nimg0, &niy0);
    const int items = m.ipb * m.slot_pix * m.chunk_words;
    auto expand_one = [&](auto UI) __attribute__((always_inline)) {
      constexpr int U = decltype(UI)::value;
      const int it = gt + PP_GROUP * U;
      if (stage && it < items) {
        const int hp = (int)fdiv((uint32_t)it, m.fd_cwc);
        expand_to_lds<OPK, PA>(raw[U], halo + hp * m.pix_bytes + (it - hp * m.chunk_words) * O::WORD_BYTES);
      }
    };
    const bool st = k >= 1 && co_w < a.cout;
    int pimg0 = 0, pu0 = 0;
    if (st) item_units(m, item_w(k - 1), &pimg0, &pu0);
    // BN tiles (OB > 0: with the packed Q(HardTanh(z)) of the next layer)
    auto bn_tile = [&](auto RESC, const acc_t& A, int T, int co32, const float(*pre)[16])
                       __attribute__((always_inline)) {
      tile_epilogue_swap<K_BNF32, decltype(RESC)::value, OB>(m, A, pimg0, pu0, T, co32, co_blk, prm, plane, pre);
    };
    if (a.mode == QCONV_EPI_BN_F32 && a.residual_on) {
      // residual layers: the residual values of tile t + 1 are loaded before
      // the stores of tile t, so no load waits for the stores of its own tile
      float rcur[16], rnext[16];
      if (st && co_w < a.cout) swap_res_load(m, pimg0, pu0, wm * MT, co_w, plane, rcur);
      Unroll<0, MT * NT>::run([&](auto TI) __attribute__((always_inline)) {
        constexpr int TT = decltype(TI)::value;
        constexpr int i = TT / NT, j = TT % NT;
        const int co32 = co_w + 32 * j;
        if constexpr (TT + 1 < MT * NT) {
          constexpr int i1 = (TT + 1) / NT, j1 = (TT + 1) % NT;
          if (st && co_w + 32 * j1 < a.cout) swap_res_load(m, pimg0, pu0, wm * MT + i1, co_w + 32 * j1, plane, rnext);
        }
        if (st && co32 < a.cout) bn_tile(std::integral_constant<int, 1>{}, acc[i][j], wm * MT + i, co32, &rcur);
        if constexpr (TT + 1 < MT * NT) {
#pragma unroll
          for (int v = 0; v < 16; ++v) rcur[v] = rnext[v];
        }
        if constexpr (TT < NI) expand_one(std::integral_constant<int, TT>{});
      });
    } else {
      Unroll<0, MT * NT>::run([&](auto TI) __attribute__((always_inline)) {
        constexpr int TT = decltype(TI)::value;
        constexpr int i = TT / NT, j = TT % NT;
        const int co32 = co_w + 32 * j;
        if (st && co32 < a.cout) {
          const int T = wm * MT + i;
          if (a.mode == QCONV_EPI_INT32) {
            tile_epilogue_swap<K_INT32, 0>(m, acc[i][j], pimg0, pu0, T, co32, co_blk, prm, plane);
          } else if (a.mode == QCONV_EPI_SCALE_F32) {
            tile_epilogue_swap<K_SCALE, 0>(m, acc[i][j], pimg0, pu0, T, co32, co_blk, prm, plane);
          } else if (a.mode == QCONV_EPI_BN_PACK) {
            // the packed output alone (its width is the input's: OB)
            if constexpr (OB > 0) tile_epilogue_swap<K_PACK, 0, OB>(m, acc[i][j], pimg0, pu0, T, co32, co_blk, prm, plane);
          } else {
            bn_tile(std::integral_constant<int, 0>{}, acc[i][j], T, co32, nullptr);
          }
        }
        if constexpr (TT < NI) expand_one(std::integral_constant<int, TT>{});
      });
    }
    Unroll<(MT * NT < NI ? MT * NT : NI), NI>::run([&](auto UI) __attribute__((always_inline)) { expand_one(UI); });
    // halo items past NI per thread (large tiles): loaded here, one at a time
    if (stage) {
      for (int it0 = NI * PP_GROUP; it0 < items; it0 += PP_GROUP) {
        uint32_t one[1][PA];
        load_halo_rsrc<PA, 1, PP_GROUP>(m, arsrc, nimg0, niy0, it0 + gt, one);
        const int it = it0 + gt;
        if (it < items) {
          const int hp = (int)fdiv((uint32_t)it, m.fd_cwc);
          expand_to_lds<OPK, PA>(one[0], halo + hp * m.pix_bytes + (it - hp * m.chunk_words) * O::WORD_BYTES);
        }
      }
    }
  };

  // phases 0 .. n_my: group 0 computes in the even ones, group 1 in the odd
  // ones; both groups pass n_my + 1 barriers
  if (grp == 0) {
    for (int p = 0; p <= n_my; p += 2) {
      if (p < n_my) compute(p);
      lds_barrier();
      if (p + 1 <= n_my) {
        store(p + 1);
        lds_barrier();
      }
    }
  } else {
    for (int p = 0; p <= n_my; p += 2) {
      store(p);
      lds_barrier();
      if (p + 1 <= n_my) {
        if (p + 1 < n_my) compute(p + 1);
        lds_barrier();
      }
    }
  }
}

// Host-side planning (conv_mfma.hip).
int device_cus();
bool use_swap(const MfmaArgs& m);
bool use_pp(const MfmaArgs& m, int cfg, int cus);
size_t pp_lds(const MfmaArgs& m, int cfg);
size_t block_lds(const MfmaArgs& m);
constexpr int LDS_PER_CU = 160 * 1024;
constexpr int MAX_DEVICES = 64;

// Raises the dynamic-LDS limit of one kernel instantiation to `bytes`, once
// per device and size (the pointer identifies the instantiation).
template <void (*K)(const MfmaArgs)>
bool raise_lds_limit_of(size_t bytes) {
  static std::atomic<int> done[MAX_DEVICES];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return false;
  std::atomic<int>* d = (dev >= 0 && dev < MAX_DEVICES) ? &done[dev] : nullptr;
  if (d && d->load(std::memory_order_relaxed) >= (int)bytes) return true;
  if (hipFuncSetAttribute(reinterpret_cast<const void*>(K), hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) !=
      hipSuccess)
    return false;
  if (d) d->store((int)bytes, std::memory_order_relaxed);
  return true;
}

template <int OPK, int PA, int CFG>
int launch_cfg(MfmaArgs m, hipStream_t s) {
  const size_t lds = block_lds(m);
  const int total = m.tiles_px * m.tiles_co;
  const int cus = device_cus();
  if constexpr (CFG != 2 && OPK != OP_F16) {
    if (use_pp(m, CFG, cus)) {
      const size_t plds = pp_lds(m, CFG);
      // every block keeps one output-channel tile: a multiple of tiles_co blocks
      m.grid = max(m.tiles_co, (min(total, cus) / m.tiles_co) * m.tiles_co);
      // OB: the bits of a packed copy of a BN output; one width per input
      // width (the one a network of that width asks for), others are refused
      // by use_pp
      constexpr int OB_NET = PA == 1 ? 1 : (PA == 2 ? 2 : 3);
      auto kern = conv_mfma_pp_kernel<OPK, PA, CFG, 0>;
      if (m.c.out_packed) kern = conv_mfma_pp_kernel<OPK, PA, CFG, OB_NET>;
      // the dynamic-LDS limit of this instantiation, raised once per device
      static std::atomic<int> lds_set[MAX_DEVICES];
      int dev = 0;
      if (hipGetDevice(&dev) != hipSuccess) return QCONV_EHIP;
      std::atomic<int>* done = (dev >= 0 && dev < MAX_DEVICES) ? &lds_set[dev] : nullptr;
      if (!done || done->load(std::memory_order_relaxed) < (int)plds) {
        if (hipFuncSetAttribute(reinterpret_cast<const void*>(kern), hipFuncAttributeMaxDynamicSharedMemorySize,
                                (int)plds) != hipSuccess)
          return QCONV_EHIP;
        if (done) done->store((int)plds, std::memory_order_relaxed);
      }
      kern<<<dim3((unsigned)m.grid), 2 * PP_GROUP, plds, s>>>(m);
      return hip_status();
    }
  }
  if (CFG == 2) {
    m.grid = total;  // split-K: one item per block
  } else {
    // resident blocks per CU: the register bound of the kernel, then LDS
    const int per_cu = max(1, min(blocks_per_cu(OPK, CFG), (int)(LDS_PER_CU / lds)));
    m.grid = min(total, per_cu * cus);
  }
  if (use_swap(m)) {
    if (lds > 64 * 1024 && !raise_lds_limit_of<conv_mfma_kernel<OPK, PA, CFG, 1>>(lds)) return QCONV_EHIP;
    conv_mfma_kernel<OPK, PA, CFG, 1><<<dim3((unsigned)m.grid), 256, lds, s>>>(m);
  } else {
    if (lds > 64 * 1024 && !raise_lds_limit_of<conv_mfma_kernel<OPK, PA, CFG, 0>>(lds)) return QCONV_EHIP;
    conv_mfma_kernel<OPK, PA, CFG, 0><<<dim3((unsigned)m.grid), 256, lds, s>>>(m);
  }
  return hip_status();
}

template <int OPK, int PA>
int launch_fp(const MfmaArgs& m, int cfg, hipStream_t s) {
  if (cfg == 0) return launch_cfg<OPK, PA, 0>(m, s);
  if (cfg == 1) return launch_cfg<OPK, PA, 1>(m, s);
  return launch_cfg<OPK, PA, 2>(m, s);
}

// One launcher per (operand format, activation words) pair, each compiled in
// a translation unit of its own (conv_mfma_<format>_p<words>.hip).
#define QC_MFMA_LAUNCHERS(X) \
  X(i8_p1, OP_I8, 1) X(i8_p2, OP_I8, 2) X(i8_p4, OP_I8, 4) \
  X(fp4_p1, OP_FP4, 1) X(fp4_p2, OP_FP4, 2) X(fp4_p4, OP_FP4, 4) \
  X(f16_p1, OP_F16, 1) X(f16_p2, OP_F16, 2) X(f16_p4, OP_F16, 4) X(f16_p16, OP_F16, 16)
#define QC_MFMA_DECLARE(NAME, OPK, PA) int launch_mfma_##NAME(const MfmaArgs& m, int cfg, hipStream_t s);
QC_MFMA_LAUNCHERS(QC_MFMA_DECLARE)
#undef QC_MFMA_DECLARE
#define QC_MFMA_DEFINE(NAME, OPK, PA) \
  int launch_mfma_##NAME(const MfmaArgs& m, int cfg, hipStream_t s) { return launch_fp<OPK, PA>(m, cfg, s); }

}  // namespace mfma
}  // namespace qc
