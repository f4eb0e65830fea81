// conv_f32_mfma.hip -- the full-precision first convolution on the fp32
// matrix cores (v_mfma_f32_32x32x2_f32) or, for the pooled 7 x 7 / 2
// geometry, on the bf16 matrix cores through exact three-way splits (the
// bf16x6 kernel below), with its batch norm, ReLU, an optional 3x3 / 2 max
// pooling (pad 1) and the packed Q(HardTanh(.)) of the next layer's input
// fused into the epilogue.  The first layer's input is
// the image, which stays unquantized (Sec. III-E; the workloads fix fp32
// first layers); its sums are taken in the matrix cores' order, so results
// match the fixed fmaf-chain kernels (fp32_layers.hip) within fp32 rounding,
// not bit for bit.
//
// Implicit GEMM: M = conv pixels of a tile, N = 32 output channels per
// block, K = cin * k * k (per input channel the k * k taps in OIHW order,
// padded to even).  A block (4 waves, 2 M-tiles of 32 pixels each) stages
// the tile's input window in LDS, zero outside the image; its 32 channels'
// weights stay in LDS for the whole launch.  The tile geometry, kernel size
// and stride are compile-time, so every operand read is one LDS access at a
// per-lane base plus an immediate offset.  Blocks loop over (image, tile)
// items; the next item's window is loaded into registers under the current
// item's matrix work.
//
// Tiles.  With pooling, a tile is 7 x 8 pooled outputs, which need the
// 15 x 17 = 255 conv pixels of their windows (8 M-tiles of 32, one row
// unused): BN + ReLU go into an LDS tile and the 3x3 maxima come out of it
// (pixels outside the conv output never win; a NaN never replaces the
// running maximum).  Without pooling a tile is 8 conv rows x 32 columns,
// one M-tile per row.  Tiles and windows wholly inside the image skip the
// bounds checks.
//
// LDS banks (64 on gfx950).  An operand read is one ds_read_b32 of 64
// lanes: lanes 0-31 read 32 consecutive tile pixels at one tap, lanes 32-63
// the same pixels at the k-step's other tap.  With stride 2 the window is
// stored split by row and column parity (odd columns 32 floats after the
// even ones, rows 81 floats apart, odd rows at an offset of 32 mod 64), so
// that the 32 pixels of a half fall in 32 consecutive banks and the taps are
// paired so that the other half reads exactly 32 banks away: (ky, 2a) with
// (ky, 2a + 1), then (2b, k - 1) with (2b + 1, k - 1), the last tap with a
// zero-weight padding tap.  The conv tile of the pooling epilogue is stored
// pixel-major (40 floats per pixel: the two halves of an accumulator
// register land 32 banks apart) and read with lanes on channels and the two
// halves on pooled columns two apart (again 32 banks apart).
#include <stdio.h>
#include <algorithm>
#include <string.h>

#include "qconv_internal.h"

namespace qc {

namespace {

typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int PT_H = 7, PT_W = 8;    // pooled outputs per tile
constexpr int PT_H0 = 8, PT_W0 = 32;  // conv tile without pooling
constexpr int CT_PITCH = 40;          // LDS floats per pixel of the pooling conv tile (pixel-major)
constexpr int CT_PIX = 256;           // pixel slots of the pooling conv tile
constexpr int PO_PITCH = PT_H * PT_W + 1;  // LDS floats per channel of the staged pooled tile
constexpr int F32M_NJ = 16;           // input window elements per thread (windows up to 4096 floats)
constexpr int NCT_MAX = 4;            // 32-channel tiles per block over one staged window (plain tiles)
constexpr size_t F32M_LDS_MAX = 80 * 1024;  // two blocks per CU
constexpr int S2_HW = 32;             // stride 2: offset of the odd-column phase within a row
constexpr int S2_WP = 81;             // stride 2: row pitch (17 mod 64)

// smallest v >= x with v = 32 (mod 64)
__host__ __device__ constexpr int up_32mod64(int x) { return x <= 32 ? 32 : ((x - 32 + 63) / 64) * 64 + 32; }

// bf16x6 (the 7 x 7 / 2 pooled geometry): the window is held as three bf16
// planes of the exact split x = x0 + x1 + x2, rows of X6_RPW words (two
// bf16 each) and channels of X6_CIPW words; 21 words per row keep the 32
// pixels of each half of a wave's read in 32 distinct banks.
constexpr int X6_RPW = 21;
constexpr int X6_CIPW = 35 * X6_RPW;  // 35 window rows of the pooled 7 x 7 / 2 tile
constexpr int X6_PLW = 3 * X6_CIPW + 1;  // words per plane: up to 3 input channels and a spare word

// Exact split of an fp32 value into three bf16 parts, x = p0 + p1 + p2:
// p0 is x cut to its top 16 bits (the leading 8 significand bits), the
// remainder x - p0 is exact in fp32 (same sign and exponent range), and so
// is the second cut; what is left has at most 8 significant bits, so it is
// itself a bf16.  Cutting rather than rounding keeps every part no larger
// than what it splits, and no part overflows.  A non-finite x makes the
// remainder NaN (inf - inf, or NaN), so its products spread NaN.
__device__ __forceinline__ void split_bf16x3(float x, uint32_t& h0, uint32_t& h1, uint32_t& h2) {
  const uint32_t u = __float_as_uint(x);
  const float r1 = x - __uint_as_float(u & 0xFFFF0000u);
  const uint32_t v = __float_as_uint(r1);
  const float r2 = r1 - __uint_as_float(v & 0xFFFF0000u);
  h0 = u >> 16;
  h1 = v >> 16;
  h2 = __float_as_uint(r2) >> 16;
}

template <int KSZ, int S, int POOL>
struct Geo {
  static constexpr int CT_H = POOL ? 2 * PT_H + 1 : PT_H0;  // conv pixels of a tile
  static constexpr int CT_W = POOL ? 2 * PT_W + 1 : PT_W0;
  static constexpr int IH = (CT_H - 1) * S + KSZ;           // staged input window
  static constexpr int IW = (CT_W - 1) * S + KSZ;
  static constexpr int WIN = IH * IW;                       // window elements per input channel
  static constexpr int KK = KSZ * KSZ, KS2 = (KK + 1) / 2;  // taps, k-steps of two taps
  // LDS floats per input channel of the staged window, and the offset of
  // the odd-row phase (stride 2)
  static constexpr int HRP = S == 2 ? up_32mod64(((IH + 1) / 2) * S2_WP) : 0;
  static constexpr int CIP = S == 2 ? HRP + (IH / 2) * S2_WP : WIN;
  static_assert(S == 1 || ((IW + 1) / 2 <= S2_HW && S2_HW + IW / 2 <= S2_WP), "stride-2 row layout");
};

// Taps of k-step st: t0 (lanes 0-31) and t1 (lanes 32-63; -1 = padding).
// Stride 1: taps 2 st and 2 st + 1 in OIHW order.  Stride 2: the pairing
// that puts the two taps 32 banks apart in the phase-split window.
template <int KSZ, int S>
__host__ __device__ constexpr int step_tap(int st, int half) {
  constexpr int KK = KSZ * KSZ;
  if (S == 1) {
    const int t = 2 * st + half;
    return t < KK ? t : -1;
  }
  constexpr int HP = (KSZ - 1) / 2;  // column pairs per row
  constexpr int NCOL = KSZ * HP;
  if (st < NCOL) return (st / HP) * KSZ + 2 * (st % HP) + half;
  if (st < NCOL + HP) return (2 * (st - NCOL) + half) * KSZ + KSZ - 1;
  return half ? -1 : KK - 1;
}

// Whether the lanes 32-63 of k-step st read through the second base (the
// odd-row phase with stride 2, the next window row with stride 1).
template <int KSZ, int S>
__host__ __device__ constexpr bool step_row(int st) {
  if (S == 1) return (2 * st) % KSZ == KSZ - 1;
  constexpr int HP = (KSZ - 1) / 2;
  return st >= KSZ * HP && st < KSZ * HP + HP;
}

// Offset of tap t inside one channel's staged window.
template <int KSZ, int S, int POOL>
__host__ __device__ constexpr int tap_off(int t) {
  using G = Geo<KSZ, S, POOL>;
  const int ky = t / KSZ, kx = t % KSZ;
  if (S == 1) return ky * G::IW + kx;
  return (ky & 1) * G::HRP + (ky >> 1) * S2_WP + (kx & 1) * S2_HW + (kx >> 1);
}

struct F32M {
  const float* x;
  const float* wt;  // OIHW
  const float* bn_k;
  const float* bn_b;
  int n, cin, h, w, cout;
  int pad;
  int ho, wo;  // conv output
  int relu;
  int oh, ow;  // layer output (pooled when pooling)
  int tiles_y, tiles_x, co_tiles, items;
  FastDiv fd_tx, fd_ty;  // item -> (image, tile row, tile column) without a division
  int nct, co_groups;  // 32-channel tiles per block (plain tiles: up to 4 over one staged window), blocks per item
  float* out;
  uint32_t* out_packed;
  int out_cw;
  Thr othr;  // requantization thresholds for |z| (HardTanh folded in)
  int l_w, l_pk;  // LDS float offsets: weights, packed staging (window / conv tile region at 0)
};

// ALG 0: the fp32 matrix cores.  ALG 1 (bf16x6; the pooled 7 x 7 / 2
// geometry only): each window element and weight is split exactly into
// three bf16 parts, x = x0 + x1 + x2 and w = w0 + w1 + w2, and the six
// partial products with i + j <= 2 are summed on the bf16 matrix cores
// (v_mfma_f32_32x32x16_bf16), x0 w0 in one accumulator and the five
// smaller ones in a second, added at the end.  The three dropped products
// are below 2^-20 |x w| together, and the small products' own sum rounds
// below 2^-20.4 sum |x w| for K <= 147, so each output is within
// (gamma_K + 2^-19 + 2^-24) sum |x w| of the exact sum.  A
// k-step of 16 is two (ci, ky) tap rows: lanes 0-31 take row 2 j, lanes
// 32-63 row 2 j + 1, each as 4 words of two bf16 (taps kx, kx + 1; the
// eighth slot reads the next window column against a zero weight).
// Inputs and weights must be finite: a non-finite value makes NaN in the
// outputs it meets (including, through the eighth slot, the output one
// column to its left).
template <int ALG, int KSZ, int S, int POOL, int OB>
__device__ __forceinline__ void f32m_body(const F32M& m) {
  static_assert(ALG == 0 || (KSZ == 7 && S == 2 && POOL == 1), "bf16x6 geometry");
  using G = Geo<KSZ, S, POOL>;
  constexpr int KS2 = G::KS2, IW = G::IW, WIN = G::WIN, CIP = G::CIP, CT_W = G::CT_W;
  extern __shared__ __attribute__((aligned(16))) float fl[];
  float* xin = fl;
  float* wB = fl + m.l_w;
  uint16_t* xh = reinterpret_cast<uint16_t*>(fl);             // bf16x6: the window's three planes
  const uint32_t* xw = reinterpret_cast<const uint32_t*>(fl);
  uint16_t* wh = reinterpret_cast<uint16_t*>(fl + m.l_w);     // bf16x6: the weights' parts
  float* ctile = fl;                       // pooling: conv tile over the consumed window
  float* ptile = fl + CT_PIX * CT_PITCH;   // pooling: staged fp32 pooled tile
  uint32_t* pk = reinterpret_cast<uint32_t*>(fl + m.l_pk);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  // the block's channel tiles ct0 .. ct0 + nct - 1 (pooled tiles: one; the
  // last group of a layer whose tile count is not a multiple of m.nct has
  // fewer)
  const int ct0 = (blockIdx.x % m.co_groups) * (POOL ? 1 : m.nct);
  const int nct = POOL ? 1 : min(m.nct, m.co_tiles - ct0);

  // bf16x6: tap rows (ci, ky) of the contraction and its k-steps of two rows
  const int x6_rows = m.cin * KSZ, x6_steps = (x6_rows + 1) / 2;
  if constexpr (ALG == 0) {
    // weights of the block's channels, [tile][ci][k-step][half][32] (padding
    // taps and channels past cout 0)
    for (int i = tid; i < nct * m.cin * KS2 * 64; i += 256) {
      const int c = i & 31, h = (i >> 5) & 1, r = i >> 6, cq = r / (m.cin * KS2), r2 = r - cq * (m.cin * KS2);
      const int ci = r2 / KS2, st = r2 - ci * KS2, co = (ct0 + cq) * 32 + c;
      const int tap = step_tap<KSZ, S>(st, h);
      wB[i] = (tap >= 0 && co < m.cout) ? m.wt[((int64_t)co * m.cin + ci) * G::KK + tap] : 0.0f;
    }
  } else {
    // the three parts of the weights as B operands: k-step j holds, per
    // part, 64 lanes x 8 bf16 (lane = row half x channel; slot e = tap kx,
    // slot 7 zero), 1536 bf16 per k-step; with an odd row count the last
    // k-step holds only its first row's 32 lanes per part
    const int last_lanes = (x6_rows & 1) ? 32 : 64;
    for (int i = tid; i < 64 * x6_steps; i += 256) {
      const int j = i >> 6, ln = i & 63, ll = j == x6_steps - 1 ? last_lanes : 64;
      if (ln >= ll) continue;
      const int g = 2 * j + (ln >> 5), ci = g / KSZ, ky = g - ci * KSZ, co = ct0 * 32 + (ln & 31);
      uint32_t pw[3][4];
#pragma unroll
      for (int e = 0; e < 8; e += 2) {
        uint32_t a[3], b[3];
        const float* wr = m.wt + (((int64_t)co * m.cin + ci) * KSZ + ky) * KSZ;
        const bool ok = co < m.cout;
        split_bf16x3(ok ? wr[e] : 0.0f, a[0], a[1], a[2]);
        split_bf16x3(ok && e + 1 < KSZ ? wr[e + 1] : 0.0f, b[0], b[1], b[2]);
#pragma unroll
        for (int q = 0; q < 3; ++q) pw[q][e / 2] = a[q] | (b[q] << 16);
      }
#pragma unroll
      for (int q = 0; q < 3; ++q)
        *reinterpret_cast<uint4*>(wh + j * 1536 + (q * ll + ln) * 8) = make_uint4(pw[q][0], pw[q][1], pw[q][2], pw[q][3]);
    }
  }
  // per-channel epilogue parameters of this lane's channel in each tile
  float bkv[NCT_MAX], bbv[NCT_MAX];
#pragma unroll
  for (int cq = 0; cq < NCT_MAX; ++cq) {
    const int co = (ct0 + cq) * 32 + l32;
    const bool ok = cq < nct && co < m.cout;
    bkv[cq] = ok ? m.bn_k[co] : 0.0f;
    bbv[cq] = ok ? m.bn_b[co] : 0.0f;
  }
  // Wait for these loads here: used inside the item loop's conditional
  // blocks, a value still counted as in flight makes the compiler wait
  // for every load in flight there, the next window's prefetch included.
  __builtin_amdgcn_s_waitcnt(0x0F70);  // vmcnt(0)

  // The input window is cin * WIN elements; thread t owns elements t + 256 j.
  // Their offset inside one image, their window row / column and their LDS
  // slot are the same for every item, so they are computed once.
  const int welems = m.cin * WIN;
  const int64_t img_elems = (int64_t)m.cin * m.h * m.w;
  int eoff[F32M_NJ];      // ci * h * w + yy * w + xx (window origin at 0, 0)
  uint32_t eyx[F32M_NJ];  // yy << 16 | xx, or all ones past the window
  int edst[F32M_NJ];      // LDS slot (past the window: the spare slot after it)
#pragma unroll
  for (int j = 0; j < F32M_NJ; ++j) {
    const int e = tid + 256 * j;
    eoff[j] = 0;
    eyx[j] = 0xFFFFFFFFu;
    edst[j] = ALG ? m.cin * X6_CIPW * 2 : m.cin * CIP;
    if (e < welems) {
      const int ci = e / WIN, r = e - ci * WIN, yy = r / IW, xx = r - (r / IW) * IW;
      eoff[j] = (ci * m.h + yy) * m.w + xx;
      eyx[j] = ((uint32_t)yy << 16) | (uint32_t)xx;
      if constexpr (ALG == 1)
        edst[j] = (ci * X6_CIPW + yy * X6_RPW) * 2 + xx;  // bf16 slot in each plane
      else
        edst[j] = S == 2 ? ci * CIP + (yy & 1) * G::HRP + (yy >> 1) * S2_WP + (xx & 1) * S2_HW + (xx >> 1) : e;
    }
  }
  float wval[F32M_NJ];
  auto origin = [&](int item, int* img, int* ty, int* tx, int* cy0, int* cx0) __attribute__((always_inline)) {
    const int r0 = (int)fdiv((uint32_t)item, m.fd_tx);
    *tx = item - r0 * m.tiles_x;
    *img = (int)fdiv((uint32_t)r0, m.fd_ty);
    *ty = r0 - *img * m.tiles_y;
    *cy0 = POOL ? 2 * *ty * PT_H - 1 : *ty * PT_H0;
    *cx0 = POOL ? 2 * *tx * PT_W - 1 : *tx * PT_W0;
  };
  // One buffer load per element through a resource over the tile's image:
  // elements outside the image or past the window get an offset past the
  // buffer's end and read 0 without a memory access, so the loads go out
  // back to back with no mask applied after them.
  auto load_window = [&](int item) __attribute__((always_inline)) {
    int img, ty, tx, cy0, cx0;
    origin(item, &img, &ty, &tx, &cy0, &cx0);
    const int iy0 = cy0 * S - m.pad, ix0 = cx0 * S - m.pad;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(m.x + (int64_t)img * img_elems), (short)0, (int)(img_elems * 4), 0x00020000);
    const int org = iy0 * m.w + ix0;  // may be negative: added only to in-image elements
    const bool inside = iy0 >= 0 && iy0 + G::IH <= m.h && ix0 >= 0 && ix0 + IW <= m.w;
    // two straight runs of loads (a window inside the image needs no
    // bounds test) rather than a branch around each element's test
    if (inside) {
#pragma unroll
      for (int j = 0; j < F32M_NJ; ++j) {
        const int voff = eyx[j] != 0xFFFFFFFFu ? (org + eoff[j]) * 4 : 0x7FFFFFF0;
        wval[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, voff, 0, 0));
      }
    } else {
#pragma unroll
      for (int j = 0; j < F32M_NJ; ++j) {
        const int gy = iy0 + (int)(eyx[j] >> 16), gx = ix0 + (int)(eyx[j] & 0xFFFFu);
        const bool ok = eyx[j] != 0xFFFFFFFFu && (unsigned)gy < (unsigned)m.h && (unsigned)gx < (unsigned)m.w;
        const int voff = ok ? (org + eoff[j]) * 4 : 0x7FFFFFF0;
        wval[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rs, voff, 0, 0));
      }
    }
  };
  const int first = blockIdx.x / m.co_groups, step_items = gridDim.x / m.co_groups;
  if (first < m.items) load_window(first);

  // per-lane operand bases of the wave's two M-tiles (the unused pooled row
  // reads pixel 0; its result is dropped): lanes 32-63 read the k-step's
  // second tap through base A (next column phase / next column) or base B
  // (odd-row phase / next window row)
  int bA[2], bB[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int pi = (wave * 2 + t) * 32 + l32;
    const int pc = pi < G::CT_H * CT_W ? pi : 0;
    const int pr = pc / CT_W, pcol = pc - (pc / CT_W) * CT_W;
    const int pb = S == 2 ? pr * S2_WP + pcol : pr * IW + pcol;
    bA[t] = pb + half * (S == 2 ? S2_HW : 1);
    bB[t] = pb + half * (S == 2 ? G::HRP : IW - (KSZ - 1));
  }
  // bf16x6: word offset of each M-tile's pixel in a plane (window row 2 r,
  // word c: taps kx, kx + 1 of column 2 c + kx)
  int pbw[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int pi = (wave * 2 + t) * 32 + l32;
    const int pc = pi < G::CT_H * CT_W ? pi : 0;
    const int pr = pc / CT_W;
    pbw[t] = 2 * pr * X6_RPW + (pc - pr * CT_W);
  }

  for (int item = first; item < m.items; item += step_items) {
    int img, ty, tx, cy0, cx0;
    origin(item, &img, &ty, &tx, &cy0, &cx0);
    lds_barrier();  // the previous item's LDS tiles are consumed
    if constexpr (ALG == 1) {
      // the column after the window's last one, which the eighth slot of the
      // last pixel column reads, is 0 in every row and part (the pooled
      // epilogue's conv tile overlays these rows)
      if (tid < m.cin * G::IH) {  // at most 3 x 35 rows
        const int ci = tid / G::IH, yy = tid - ci * G::IH;
#pragma unroll
        for (int q = 0; q < 3; ++q) xh[2 * q * X6_PLW + (ci * X6_CIPW + yy * X6_RPW) * 2 + IW] = 0;
      }
    }
#pragma unroll
    for (int j = 0; j < F32M_NJ; ++j) {  // elements past the window land on the spare slot
      if constexpr (ALG == 1) {
        uint32_t p0, p1, p2;
        split_bf16x3(wval[j], p0, p1, p2);
        xh[edst[j]] = (uint16_t)p0;
        xh[2 * X6_PLW + edst[j]] = (uint16_t)p1;
        xh[4 * X6_PLW + edst[j]] = (uint16_t)p2;
      } else {
        xin[edst[j]] = wval[j];
      }
    }
    lds_barrier();
    if (item + step_items < m.items) load_window(item + step_items);

    for (int cq = 0; cq < nct; ++cq) {
    const int ct = ct0 + cq, co_blk = ct * 32, co_l = co_blk + l32;
    const bool cok = co_l < m.cout;
    float bk = bkv[0], bb = bbv[0];
#pragma unroll
    for (int j = 1; j < NCT_MAX; ++j)
      if (cq == j) {
        bk = bkv[j];
        bb = bbv[j];
      }
    // ---- MFMAs: this wave's 2 M-tiles x 32 channels ----
    v16f acc0 = {}, acc1 = {};
    if constexpr (ALG == 1) {
      typedef __bf16 v8bf __attribute__((ext_vector_type(8)));
      auto mm = [](uint4 a, uint4 b, v16f c) __attribute__((always_inline)) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(v8bf, a), __builtin_bit_cast(v8bf, b), c, 0,
                                                       0, 0);
      };
      v16f cor0 = {}, cor1 = {};
      // one k-step: B parts from wj (ll lanes per part, this lane's at lb),
      // A parts of both M-tiles from word offset rb (zero: all operands 0)
      auto kstep = [&](const uint16_t* wj, int ll, int lb, int rb, bool zero) __attribute__((always_inline)) {
        uint4 b[3], a0[3], a1[3];
#pragma unroll
        for (int q = 0; q < 3; ++q) b[q] = *reinterpret_cast<const uint4*>(wj + (q * ll + lb) * 8);
        const uint32_t* r0 = xw + rb + pbw[0];
        const uint32_t* r1 = xw + rb + pbw[1];
#pragma unroll
        for (int q = 0; q < 3; ++q) {
          const int o = q * X6_PLW;
          // slot 7 holds the window column after the row's taps, against a
          // zero weight (finite inputs: a zero product)
          a0[q] = make_uint4(r0[o], r0[o + 1], r0[o + 2], r0[o + 3]);
          a1[q] = make_uint4(r1[o], r1[o + 1], r1[o + 2], r1[o + 3]);
          if (zero) {
            a0[q] = make_uint4(0u, 0u, 0u, 0u);
            a1[q] = make_uint4(0u, 0u, 0u, 0u);
          }
        }
        // the five small products first, into their own accumulator
        cor0 = mm(a0[2], b[0], cor0);
        cor1 = mm(a1[2], b[0], cor1);
        cor0 = mm(a0[1], b[1], cor0);
        cor1 = mm(a1[1], b[1], cor1);
        cor0 = mm(a0[0], b[2], cor0);
        cor1 = mm(a1[0], b[2], cor1);
        cor0 = mm(a0[1], b[0], cor0);
        cor1 = mm(a1[1], b[0], cor1);
        cor0 = mm(a0[0], b[1], cor0);
        cor1 = mm(a1[0], b[1], cor1);
        acc0 = mm(a0[0], b[0], acc0);
        acc1 = mm(a1[0], b[0], acc1);
      };
      // this lane's tap row 2 j + half as (ci, ky) and its word offset
      int ky = half, rb = half * X6_RPW;
      const int nfull = x6_rows >> 1;
      for (int j = 0; j < nfull; ++j) {
        kstep(wh + j * 1536, 64, lane, rb, false);
        ky += 2;
        rb += 2 * X6_RPW;
        if (ky >= KSZ) {
          ky -= KSZ;
          rb += X6_CIPW - KSZ * X6_RPW;
        }
      }
      // an odd row count: the last row alone, lanes 32-63 with zero
      // activations (read at row 0) against the first half's weights
      if (x6_rows & 1) kstep(wh + nfull * 1536, 32, l32, half ? 0 : rb, half != 0);
      acc0 += cor0;
      acc1 += cor1;
    } else {
    for (int ci = 0; ci < m.cin; ++ci) {
      const float* xa0 = xin + ci * CIP + bA[0];
      const float* xa1 = xin + ci * CIP + bA[1];
      const float* xb0 = xin + ci * CIP + bB[0];
      const float* xb1 = xin + ci * CIP + bB[1];
      const float* wc = wB + (cq * m.cin + ci) * (KS2 * 64) + half * 32 + l32;
#pragma unroll
      for (int st = 0; st < KS2; ++st) {
        const int o = tap_off<KSZ, S, POOL>(step_tap<KSZ, S>(st, 0));
        const bool rowb = step_row<KSZ, S>(st);
        float a0 = rowb ? xb0[o] : xa0[o];
        float a1 = rowb ? xb1[o] : xa1[o];
        if (step_tap<KSZ, S>(st, 1) < 0 && half) {
          a0 = 0.0f;  // the padding tap: keep the operand of its zero weight finite
          a1 = 0.0f;
        }
        const float bv = wc[st * 64];
        acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, bv, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, bv, acc1, 0, 0, 0);
      }
    }
    }  // ALG

    // ---- epilogue ----
    // register v of lane l: channel co_blk + l % 32, tile pixel 32 T + 8 (v / 4) + 4 (l / 32) + v % 4
    if constexpr (POOL) {
      lds_barrier();  // every wave's operand reads are done: the conv tile overwrites the window
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int pi = (wave * 2 + t) * 32 + 8 * (v / 4) + 4 * half + (v % 4);
          float z = fmaf(bk, t == 0 ? acc0[v] : acc1[v], bb);
          z = (m.relu && !(z > 0.0f)) ? 0.0f : z;
          // the unused pixel 255 holds -inf: the pooling reads it for taps
          // outside the conv output
          if (t == 1 && v == 15) z = (wave == 3 && half) ? -INFINITY : z;
          ctile[pi * CT_PITCH + l32] = z;
        }
      }
      lds_barrier();
      // pooling: lane -> channel, wave / half -> one pooled column (the
      // halves two columns apart), all PT_H pooled rows of it, from the row
      // maxima of the 15 conv rows
      const int pxl = ((wave >> 1) << 2) + (wave & 1) + 2 * half;
      const int px = tx * PT_W + pxl;
      const bool interior = cy0 >= 0 && cy0 + G::CT_H <= m.ho && cx0 >= 0 && cx0 + CT_W <= m.wo;
      bool vx[3];
#pragma unroll
      for (int d = 0; d < 3; ++d) {
        const int gx = cx0 + 2 * pxl + d;
        vx[d] = interior || (gx >= 0 && gx < m.wo);
      }
      float rmax[G::CT_H];
      if (interior) {
#pragma unroll
        for (int r = 0; r < G::CT_H; ++r) {
          const float* cp = ctile + (r * CT_W + 2 * pxl) * CT_PITCH + l32;
          rmax[r] = fmaxf(fmaxf(cp[0], cp[CT_PITCH]), cp[2 * CT_PITCH]);  // a NaN never replaces the maximum
        }
      } else {
        // taps outside the conv output read the -inf of pixel 255
        const float* sent = ctile + 255 * CT_PITCH + l32;
#pragma unroll
        for (int r = 0; r < G::CT_H; ++r) {
          const int gy = cy0 + r;
          const bool vy = gy >= 0 && gy < m.ho;
          const float* cp = ctile + (r * CT_W + 2 * pxl) * CT_PITCH + l32;
          float mx = -INFINITY;
#pragma unroll
          for (int d = 0; d < 3; ++d) mx = fmaxf(mx, *((vy && vx[d]) ? cp + d * CT_PITCH : sent));
          rmax[r] = mx;
        }
      }
#pragma unroll
      for (int p = 0; p < PT_H; ++p) {
        const float z = fmaxf(fmaxf(rmax[2 * p], rmax[2 * p + 1]), rmax[2 * p + 2]);
        const int py = ty * PT_H + p;
        if (m.out) ptile[l32 * PO_PITCH + p * PT_W + pxl] = z;
        if constexpr (OB > 0) {
          // one ballot per plane: lanes 0-31 give the word of (py, px) of
          // the lower half, lanes 32-63 that of the upper half
          constexpr int P = planes_of(OB);
          uint64_t bl[P];
          plane_ballots<OB>(z, cok, m.othr, bl);
          if (l32 == 0 && py < m.oh && px < m.ow) {
#pragma unroll
            for (int q = 0; q < P; ++q)
              m.out_packed[((((int64_t)img * m.oh + py) * m.ow + px) * m.out_cw + ct) * P + q] =
                  half ? (uint32_t)(bl[q] >> 32) : (uint32_t)bl[q];
          }
        }
      }
      if (m.out) {
        lds_barrier();
        // the staged pooled tile out in rows of 8 pixels: thread -> (pooled
        // pixel of the tile, the wave's 8 channels)
        const int pp = tid & 63;
        const int pyl = pp / PT_W, pxo = pp - (pp / PT_W) * PT_W;
        const int py = ty * PT_H + pyl, pxg = tx * PT_W + pxo;
        if (pp < PT_H * PT_W && py < m.oh && pxg < m.ow) {
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int c = wave * 8 + j, co = co_blk + c;
            if (co < m.cout) m.out[(((int64_t)img * m.cout + co) * m.oh + py) * m.ow + pxg] = ptile[c * PO_PITCH + pp];
          }
        }
      }
    } else {
      // one M-tile = one conv row of 32 columns: lane l holds columns
      // 8 (v / 4) + 4 (l / 32) + v % 4 of its channel
#pragma unroll
      for (int v = 0; v < 16; ++v) {
        float z0 = fmaf(bk, acc0[v], bb), z1 = fmaf(bk, acc1[v], bb);
        if (m.relu) {
          z0 = (z0 > 0.0f) ? z0 : 0.0f;
          z1 = (z1 > 0.0f) ? z1 : 0.0f;
        }
        acc0[v] = z0;
        acc1[v] = z1;
      }
      if (m.out != nullptr) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
          const int oy = cy0 + wave * 2 + t;
          if (oy < m.oh && cok) {
            float* orow = m.out + (((int64_t)img * m.cout + co_l) * m.oh + oy) * m.ow;
#pragma unroll
            for (int g = 0; g < 4; ++g) {
              const int ox = cx0 + 8 * g + 4 * half;
              float z[4];
#pragma unroll
              for (int i = 0; i < 4; ++i) z[i] = t == 0 ? acc0[4 * g + i] : acc1[4 * g + i];
              if (m.ow % 4 == 0 && ox + 4 <= m.ow) {
                *reinterpret_cast<float4*>(orow + ox) = make_float4(z[0], z[1], z[2], z[3]);
              } else {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                  if (ox + i < m.ow) orow[ox + i] = z[i];
              }
            }
          }
        }
      }
      if constexpr (OB > 0) {
        // one ballot per (value, plane): lanes 0-31 give the word of column
        // 8 g + i, lanes 32-63 that of column 8 g + 4 + i; the words go to
        // lane 32 t + column of a register per plane, stored in one pass
        constexpr int P = planes_of(OB);
        uint32_t pw[P] = {};
        Unroll<0, 8>::run([&](auto tg) {
          constexpr int T = decltype(tg)::value / 4, GG = decltype(tg)::value % 4, B = 32 * T + 8 * GG;
          uint64_t bl[4][P];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float z = T == 0 ? acc0[4 * GG + i] : acc1[4 * GG + i];
            plane_ballots<OB>(z, cok, m.othr, bl[i]);
          }
#pragma unroll
          for (int p = 0; p < P; ++p)
            pw[p] = writelanes8<B, B + 1, B + 2, B + 3, B + 4, B + 5, B + 6, B + 7>(
                pw[p], (uint32_t)bl[0][p], (uint32_t)bl[1][p], (uint32_t)bl[2][p], (uint32_t)bl[3][p],
                (uint32_t)(bl[0][p] >> 32), (uint32_t)(bl[1][p] >> 32), (uint32_t)(bl[2][p] >> 32),
                (uint32_t)(bl[3][p] >> 32));
        });
        uint32_t* d = pk + (((wave * 2 + half) * PT_W0 + l32) * nct + cq) * P;
        if constexpr (P == 1) {
          d[0] = pw[0];
        } else if constexpr (P == 2) {
          *reinterpret_cast<uint2*>(d) = make_uint2(pw[0], pw[1]);
        } else {
          *reinterpret_cast<uint4*>(d) = make_uint4(pw[0], pw[1], pw[2], pw[3]);
        }
      }
    }
    }  // channel tiles
    if constexpr (!POOL && OB > 0) {
      // every channel tile's words of a pixel, stored together (one
      // contiguous run per pixel when the block holds all its channels)
      constexpr int P = planes_of(OB);
      lds_barrier();
      const int wpp = nct * P;  // staged words per pixel
      for (int i = tid; i < PT_H0 * PT_W0 * wpp; i += 256) {
        const int qq = i / wpp, r = i - qq * wpp;
        const int qy = cy0 + qq / PT_W0, qx = cx0 + qq % PT_W0;
        if (qy < m.oh && qx < m.ow)
          m.out_packed[(((int64_t)img * m.oh + qy) * m.ow + qx) * m.out_cw * P + ct0 * P + r] = pk[i];
      }
    }
  }
}

template <int KSZ, int S, int POOL, int OB>
__global__ __launch_bounds__(256, 2) void conv_f32_mfma_kernel(const F32M m) {
  f32m_body<0, KSZ, S, POOL, OB>(m);
}

template <int KSZ, int S, int POOL, int OB>
__global__ __launch_bounds__(256, 2) void conv_f32_bf16x6_kernel(const F32M m) {
  f32m_body<1, KSZ, S, POOL, OB>(m);
}

int device_cus_f() {
  int dev = 0, v = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) return 256;
  return v;
}

// Window of a tile for kernel size k and stride s, and its LDS floats per
// input channel (run-time mirror of Geo).
void geo_rt(int k, int s, int pool, int* ih, int* iw, int* cip) {
  const int ct_h = pool ? 2 * PT_H + 1 : PT_H0, ct_w = pool ? 2 * PT_W + 1 : PT_W0;
  *ih = (ct_h - 1) * s + k;
  *iw = (ct_w - 1) * s + k;
  *cip = s == 2 ? up_32mod64(((*ih + 1) / 2) * S2_WP) + (*ih / 2) * S2_WP : *ih * *iw;
}

size_t f32m_lds(const F32M& m, int pool);

bool f32m_plan(int n, int cin, int h, int w, int cout, int k, int stride, int pad, int pool, int alg, F32M* m) {
  memset(m, 0, sizeof(*m));
  if (n < 1 || cin < 1 || pad < 0 || cout < 1) return false;
  if (k != 3 && k != 5 && k != 7) return false;               // instantiated kernel sizes
  if (!(stride == 1 || (stride == 2 && pool))) return false;  // instantiated strides
  if (alg && !(k == 7 && stride == 2 && pool && cin <= 3)) return false;  // the bf16x6 geometry
  m->n = n;
  m->cin = cin;
  m->h = h;
  m->w = w;
  m->cout = cout;
  m->pad = pad;
  if (h + 2 * pad < k || w + 2 * pad < k) return false;
  m->ho = (h + 2 * pad - k) / stride + 1;
  m->wo = (w + 2 * pad - k) / stride + 1;
  int ih, iw, cip;
  geo_rt(k, stride, pool, &ih, &iw, &cip);
  if ((int64_t)cin * ih * iw > 256 * F32M_NJ) return false;  // the window's register share
  // one image's bytes fit a buffer resource, with the out-of-range offset
  // 0x7FFFFFF0 past its end
  if ((int64_t)cin * h * w * 4 >= 0x7FFFFFF0 || ih >= (1 << 16) || iw >= (1 << 16)) return false;
  if (pool) {
    m->oh = (m->ho - 1) / 2 + 1;
    m->ow = (m->wo - 1) / 2 + 1;
    m->tiles_y = ceil_div(m->oh, PT_H);
    m->tiles_x = ceil_div(m->ow, PT_W);
  } else {
    m->oh = m->ho;
    m->ow = m->wo;
    m->tiles_y = ceil_div(m->oh, PT_H0);
    m->tiles_x = ceil_div(m->ow, PT_W0);
  }
  m->co_tiles = ceil_div(cout, 32);
  const int64_t items = (int64_t)n * m->tiles_y * m->tiles_x;
  if (items * m->co_tiles >= ((int64_t)1 << 31)) return false;
  // the multiply-high divisions of an item index are exact
  if (items * m->tiles_x >= ((int64_t)1 << 32) || (items / m->tiles_x + 1) * m->tiles_y >= ((int64_t)1 << 32))
    return false;
  m->items = (int)items;
  m->fd_tx = make_fastdiv((uint32_t)m->tiles_x);
  m->fd_ty = make_fastdiv((uint32_t)m->tiles_y);
  // LDS: the staged window (with pooling also the conv tile and the staged
  // pooled tile over it), the weights, then (plain tiles) the packed
  // staging; plain tiles take as many channel tiles per block (up to 4) as
  // fit, so that a window staged once feeds all of them
  const int taps2 = 2 * ((k * k + 1) / 2);  // padded taps per input channel
  int64_t region = alg ? 3 * X6_PLW : (int64_t)cin * cip + 1;  // + the spare slot of the elements past the window
  if (pool) region = std::max<int64_t>(region, (int64_t)CT_PIX * CT_PITCH + 32 * PO_PITCH);
  m->l_w = (int)((region + 3) & ~(int64_t)3);
  for (int nct = pool ? 1 : std::min(m->co_tiles, NCT_MAX); nct >= 1; --nct) {
    m->nct = nct;
    m->co_groups = ceil_div(m->co_tiles, nct);
    const int x6_rows = cin * k;  // bf16x6: 1536 bf16 per k-step of two tap rows, 768 for a last single row
    m->l_pk = m->l_w + (alg ? ((x6_rows / 2) * 1536 + (x6_rows & 1) * 768) / 2 : nct * cin * taps2 * 32);
    if (f32m_lds(*m, pool) <= F32M_LDS_MAX) return true;
  }
  return false;
}

size_t f32m_lds(const F32M& m, int pool) {
  return (size_t)(m.l_pk + (pool ? 0 : PT_H0 * PT_W0 * 4 * m.nct)) * 4;
}

template <int KSZ, int S, int POOL>
int launch_geo(const F32M& m, int ob, int alg, int grid, size_t lds, hipStream_t s) {
  auto go = [&](auto kern) -> int {
    if (lds > 64 * 1024 && hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               (int)F32M_LDS_MAX) != hipSuccess)
      return QCONV_EHIP;
    kern<<<dim3((unsigned)grid), 256, lds, s>>>(m);
    return hip_status();
  };
  if constexpr (KSZ == 7 && S == 2 && POOL == 1) {
    if (alg) {
      switch (ob) {
        case 0: return go(conv_f32_bf16x6_kernel<KSZ, S, POOL, 0>);
        case 1: return go(conv_f32_bf16x6_kernel<KSZ, S, POOL, 1>);
        case 2: return go(conv_f32_bf16x6_kernel<KSZ, S, POOL, 2>);
        default: return go(conv_f32_bf16x6_kernel<KSZ, S, POOL, 3>);
      }
    }
  }
  switch (ob) {
    case 0: return go(conv_f32_mfma_kernel<KSZ, S, POOL, 0>);
    case 1: return go(conv_f32_mfma_kernel<KSZ, S, POOL, 1>);
    case 2: return go(conv_f32_mfma_kernel<KSZ, S, POOL, 2>);
    default: return go(conv_f32_mfma_kernel<KSZ, S, POOL, 3>);
  }
}

}  // namespace

bool conv_f32_mfma_supports(int n, int cin, int h, int w, int cout, int k, int stride, int pad, int pool, int alg) {
  F32M m;
  return f32m_plan(n > 0 ? n : 1, cin, h, w, cout, k, stride, pad, pool, alg, &m);
}

int launch_conv_f32_mfma(const float* x, const float* w, int n, int cin, int h, int wd, int cout, int k, int stride,
                         int pad, const float* bn_k, const float* bn_b, int relu, int pool, float* out,
                         uint32_t* out_packed, int out_bits, Thr othr, int alg, hipStream_t s) {
  F32M m;
  if (n == 0) return QCONV_OK;
  if (!f32m_plan(n, cin, h, wd, cout, k, stride, pad, pool, alg, &m)) return QCONV_EUNSUPPORTED;
  m.x = x;
  m.wt = w;
  m.bn_k = bn_k;
  m.bn_b = bn_b;
  m.relu = relu;
  m.out = out;
  m.out_packed = out_packed;
  m.out_cw = ceil_div(cout, 32);
  m.othr = thr_unclamped(othr);
  const int ob = out_packed ? out_bits : 0;
  const int blocks_per = (pool ? 2 : 3) * device_cus_f() / m.co_groups;
  const int64_t want = (int64_t)(blocks_per < 1 ? 1 : blocks_per);
  const int grid = (int)((want < m.items ? want : m.items) * m.co_groups);
  const size_t lds = f32m_lds(m, pool);
  if (pool) {
    if (stride == 1) {
      if (k == 3) return launch_geo<3, 1, 1>(m, ob, alg, grid, lds, s);
      if (k == 5) return launch_geo<5, 1, 1>(m, ob, alg, grid, lds, s);
      return launch_geo<7, 1, 1>(m, ob, alg, grid, lds, s);
    }
    if (k == 3) return launch_geo<3, 2, 1>(m, ob, alg, grid, lds, s);
    if (k == 5) return launch_geo<5, 2, 1>(m, ob, alg, grid, lds, s);
    return launch_geo<7, 2, 1>(m, ob, alg, grid, lds, s);
  }
  if (k == 3) return launch_geo<3, 1, 0>(m, ob, alg, grid, lds, s);
  if (k == 5) return launch_geo<5, 1, 0>(m, ob, alg, grid, lds, s);
  return launch_geo<7, 1, 0>(m, ob, alg, grid, lds, s);
}

}  // namespace qc
