// conv_f32_mfma.hip -- the full-precision first convolution on the fp32
// matrix cores (v_mfma_f32_32x32x2_f32), with its batch norm, ReLU, an
// optional 3x3 / 2 max pooling (pad 1) and the packed Q(HardTanh(.)) of the
// next layer's input fused into the epilogue.  The first layer's input is
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
#include <stdio.h>
#include <string.h>

#include "qconv_internal.h"

namespace qc {

namespace {

typedef float v16f __attribute__((ext_vector_type(16)));

constexpr int PT_H = 7, PT_W = 8;    // pooled outputs per tile
constexpr int PT_H0 = 8, PT_W0 = 32;  // conv tile without pooling
constexpr int CT_STRIDE = 257;        // LDS floats per channel of the conv tile (odd: no bank conflicts)
constexpr int F32M_NJ = 16;           // input window elements per thread (windows up to 4096 floats)
constexpr size_t F32M_LDS_MAX = 80 * 1024;  // two blocks per CU

template <int KSZ, int S, int POOL>
struct Geo {
  static constexpr int CT_H = POOL ? 2 * PT_H + 1 : PT_H0;  // conv pixels of a tile
  static constexpr int CT_W = POOL ? 2 * PT_W + 1 : PT_W0;
  static constexpr int IH = (CT_H - 1) * S + KSZ;           // staged input window
  static constexpr int IW = (CT_W - 1) * S + KSZ;
  static constexpr int WIN = IH * IW;
  static constexpr int KK = KSZ * KSZ, KS2 = (KK + 1) / 2;  // taps, k-steps of two taps
};

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
  float* out;
  uint32_t* out_packed;
  int out_cw;
  Thr othr;
  int l_w, l_ct, l_pk;  // LDS float offsets: weights, conv tile, packed staging (window at 0)
};

// Tap t (t < KK) as an offset inside the window.
template <int KSZ, int IW>
__host__ __device__ constexpr int tap_off(int t) {
  return (t / KSZ) * IW + (t % KSZ);
}

template <int KSZ, int S, int POOL, int OB>
__global__ __launch_bounds__(256, 2) void conv_f32_mfma_kernel(const F32M m) {
  using G = Geo<KSZ, S, POOL>;
  constexpr int KK = G::KK, KS2 = G::KS2, IW = G::IW, WIN = G::WIN, CT_W = G::CT_W;
  extern __shared__ __attribute__((aligned(16))) float fl[];
  float* xin = fl;
  float* wB = fl + m.l_w;
  float* ctile = fl + m.l_ct;
  uint32_t* pk = reinterpret_cast<uint32_t*>(fl + m.l_pk);
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int half = lane >> 5, l32 = lane & 31;
  const int ct = blockIdx.x % m.co_tiles;
  const int co_blk = ct * 32;

  // weights of the block's 32 channels, [ci][2 KS2 taps][32] (padding taps 0)
  for (int i = tid; i < m.cin * 2 * KS2 * 32; i += 256) {
    const int c = i & 31, r = i >> 5, ci = r / (2 * KS2), kq = r - ci * (2 * KS2), co = co_blk + c;
    wB[i] = (kq < KK && co < m.cout) ? m.wt[((int64_t)co * m.cin + ci) * KK + kq] : 0.0f;
  }
  // per-channel epilogue parameters of this lane's channel
  const int co_l = co_blk + l32;
  const bool cok = co_l < m.cout;
  const float bk = cok ? m.bn_k[co_l] : 0.0f, bb = cok ? m.bn_b[co_l] : 0.0f;

  // The input window is cin * WIN floats; thread t owns elements t + 256 j.
  // Their offset inside one image, and their window row / column, are the
  // same for every item, so they are computed once.
  const int welems = m.cin * WIN;
  const int64_t img_elems = (int64_t)m.cin * m.h * m.w;
  int eoff[F32M_NJ];      // ci * h * w + yy * w + xx (window origin at 0, 0)
  uint32_t eyx[F32M_NJ];  // yy << 16 | xx, or all ones past the window
#pragma unroll
  for (int j = 0; j < F32M_NJ; ++j) {
    const int e = tid + 256 * j;
    eoff[j] = 0;
    eyx[j] = 0xFFFFFFFFu;
    if (e < welems) {
      const int ci = e / WIN, r = e - ci * WIN, yy = r / IW, xx = r - (r / IW) * IW;
      eoff[j] = (ci * m.h + yy) * m.w + xx;
      eyx[j] = ((uint32_t)yy << 16) | (uint32_t)xx;
    }
  }
  float wval[F32M_NJ];
  auto origin = [&](int item, int* img, int* ty, int* tx, int* cy0, int* cx0) __attribute__((always_inline)) {
    *tx = item % m.tiles_x;
    const int r0 = item / m.tiles_x;
    *ty = r0 % m.tiles_y;
    *img = r0 / m.tiles_y;
    *cy0 = POOL ? 2 * *ty * PT_H - 1 : *ty * PT_H0;
    *cx0 = POOL ? 2 * *tx * PT_W - 1 : *tx * PT_W0;
  };
  auto load_window = [&](int item) __attribute__((always_inline)) {
    int img, ty, tx, cy0, cx0;
    origin(item, &img, &ty, &tx, &cy0, &cx0);
    const int iy0 = cy0 * S - m.pad, ix0 = cx0 * S - m.pad;
    const float* xb = m.x + (int64_t)img * img_elems;
    const int64_t org = (int64_t)iy0 * m.w + ix0;  // may be negative: added only to in-image elements
    if (iy0 >= 0 && iy0 + G::IH <= m.h && ix0 >= 0 && ix0 + IW <= m.w) {
#pragma unroll
      for (int j = 0; j < F32M_NJ; ++j) wval[j] = eyx[j] != 0xFFFFFFFFu ? xb[org + eoff[j]] : 0.0f;
    } else {
#pragma unroll
      for (int j = 0; j < F32M_NJ; ++j) {
        const int gy = iy0 + (int)(eyx[j] >> 16), gx = ix0 + (int)(eyx[j] & 0xFFFFu);
        const bool ok = eyx[j] != 0xFFFFFFFFu && gy >= 0 && gy < m.h && gx >= 0 && gx < m.w;
        wval[j] = ok ? xb[org + eoff[j]] : 0.0f;
      }
    }
  };
  const int first = blockIdx.x / m.co_tiles, step_items = gridDim.x / m.co_tiles;
  if (first < m.items) load_window(first);

  // per-lane pixel bases of the wave's two M-tiles (the unused pooled row
  // reads pixel 0; its result is dropped)
  int pb[2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const int pi = (wave * 2 + t) * 32 + l32;
    const int pc = pi < G::CT_H * CT_W ? pi : 0;
    pb[t] = (pc / CT_W) * S * IW + (pc % CT_W) * S;
  }
  // lanes of the upper half take the second tap of each k-step: one window
  // column further, or the first column of the next row
  const int dh_col = half, dh_row = half * (IW - (KSZ - 1));

  for (int item = first; item < m.items; item += step_items) {
    int img, ty, tx, cy0, cx0;
    origin(item, &img, &ty, &tx, &cy0, &cx0);
    lds_barrier();  // the previous item's LDS tiles are consumed
#pragma unroll
    for (int j = 0; j < F32M_NJ; ++j)
      if (eyx[j] != 0xFFFFFFFFu) xin[tid + 256 * j] = wval[j];
    lds_barrier();
    if (item + step_items < m.items) load_window(item + step_items);

    // ---- MFMAs: this wave's 2 M-tiles x 32 channels ----
    v16f acc0 = {}, acc1 = {};
    for (int ci = 0; ci < m.cin; ++ci) {
      const float* xc0 = xin + ci * WIN + pb[0];
      const float* xc1 = xin + ci * WIN + pb[1];
      const float* x0c = xc0 + dh_col;  // a k-step whose two taps share a row
      const float* x1c = xc1 + dh_col;
      const float* x0r = xc0 + dh_row;  // a k-step whose second tap starts the next row
      const float* x1r = xc1 + dh_row;
      const float* wc = wB + ci * (2 * KS2 * 32) + half * 32 + l32;
#pragma unroll
      for (int st = 0; st < KS2; ++st) {
        const int t0 = 2 * st;
        const bool wrap = (t0 % KSZ) == KSZ - 1;  // taps 2 st and 2 st + 1 on different rows
        const int o = tap_off<KSZ, IW>(t0);
        float a0 = wrap ? x0r[o] : x0c[o];
        float a1 = wrap ? x1r[o] : x1c[o];
        if (st == KS2 - 1 && (KK % 2 == 1) && half) {
          a0 = 0.0f;  // the padding tap of an odd KK: keep the operand of its zero weight finite
          a1 = 0.0f;
        }
        const float bv = wc[st * 64];
        acc0 = __builtin_amdgcn_mfma_f32_32x32x2f32(a0, bv, acc0, 0, 0, 0);
        acc1 = __builtin_amdgcn_mfma_f32_32x32x2f32(a1, bv, acc1, 0, 0, 0);
      }
    }

    // ---- epilogue ----
    // register v of lane l: channel co_blk + l % 32, tile pixel 32 T + 8 (v / 4) + 4 (l / 32) + v % 4
    if constexpr (POOL) {
#pragma unroll
      for (int t = 0; t < 2; ++t) {
#pragma unroll
        for (int v = 0; v < 16; ++v) {
          const int pi = (wave * 2 + t) * 32 + 8 * (v / 4) + 4 * half + (v % 4);
          float z = fmaf(bk, t == 0 ? acc0[v] : acc1[v], bb);
          if (m.relu) z = (z > 0.0f) ? z : 0.0f;
          if (pi < G::CT_H * CT_W) ctile[l32 * CT_STRIDE + pi] = z;
        }
      }
      if constexpr (OB > 0) {
        for (int i = tid; i < PT_H * PT_W * planes_of(OB); i += 256) pk[i] = 0u;
      }
      lds_barrier();
      // pooling: thread -> (pooled pixel of the tile, the wave's 8 channels)
      const int pp = tid & 63, cq = wave;
      const int pyl = pp / PT_W, pxl = pp - (pp / PT_W) * PT_W;
      const int py = ty * PT_H + pyl, px = tx * PT_W + pxl;
      const bool interior = cy0 >= 0 && cy0 + G::CT_H <= m.ho && cx0 >= 0 && cx0 + CT_W <= m.wo;
      if (pp < PT_H * PT_W && py < m.oh && px < m.ow) {
        constexpr int P = OB > 0 ? planes_of(OB) : 1;
        uint32_t bits[P];
#pragma unroll
        for (int p = 0; p < P; ++p) bits[p] = 0u;
        const float* cb = ctile + cq * 8 * CT_STRIDE + (2 * pyl) * CT_W + 2 * pxl;
        // window taps inside the conv output (all of them in an interior tile)
        bool vy[3], vx[3];
#pragma unroll
        for (int d = 0; d < 3; ++d) {
          const int gy = cy0 + 2 * pyl + d, gx = cx0 + 2 * pxl + d;
          vy[d] = interior || (gy >= 0 && gy < m.ho);
          vx[d] = interior || (gx >= 0 && gx < m.wo);
        }
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int co = co_blk + cq * 8 + j;
          float mx = -INFINITY;
#pragma unroll
          for (int dy = 0; dy < 3; ++dy)
#pragma unroll
            for (int dx = 0; dx < 3; ++dx) {
              const float v = cb[j * CT_STRIDE + dy * CT_W + dx];
              if (vy[dy] && vx[dx]) mx = fmaxf(mx, v);  // a NaN never replaces the maximum
            }
          if (co < m.cout) {
            if (m.out) m.out[(((int64_t)img * m.cout + co) * m.oh + py) * m.ow + px] = mx;
            if constexpr (OB > 0) {
              const uint32_t qv = quant_planes<OB>(hardtanh(mx), m.othr);
#pragma unroll
              for (int p = 0; p < P; ++p) bits[p] |= ((qv >> p) & 1u) << j;
            }
          }
        }
        if constexpr (OB > 0) {
#pragma unroll
          for (int p = 0; p < P; ++p) atomicOr(&pk[pp * P + p], bits[p] << (8 * cq));
        }
      }
      if constexpr (OB > 0) {
        constexpr int P = planes_of(OB);
        lds_barrier();
        for (int i = tid; i < PT_H * PT_W * P; i += 256) {
          const int qq = i / P, p = i - (i / P) * P;
          const int qy = ty * PT_H + qq / PT_W, qx = tx * PT_W + qq % PT_W;
          if (qy < m.oh && qx < m.ow)
            m.out_packed[((((int64_t)img * m.oh + qy) * m.ow + qx) * m.out_cw + ct) * P + p] = pk[i];
        }
      }
    } else {
      // one M-tile = one conv row of 32 columns: lane l holds columns
      // 8 (v / 4) + 4 (l / 32) + v % 4 of its channel
      if constexpr (OB > 0) {
        for (int i = tid; i < PT_H0 * PT_W0 * planes_of(OB); i += 256) pk[i] = 0u;
        lds_barrier();
      }
#pragma unroll
      for (int t = 0; t < 2; ++t) {
        const int row = wave * 2 + t;
        const int oy = cy0 + row;
#pragma unroll
        for (int g = 0; g < 4; ++g) {
          const int col = 8 * g + 4 * half;
          float z[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            z[i] = fmaf(bk, t == 0 ? acc0[4 * g + i] : acc1[4 * g + i], bb);
            if (m.relu) z[i] = (z[i] > 0.0f) ? z[i] : 0.0f;
          }
          const int ox = cx0 + col;
          if (oy < m.oh && cok && m.out) {
            float* o = m.out + (((int64_t)img * m.cout + co_l) * m.oh + oy) * m.ow + ox;
            if (m.ow % 4 == 0 && ox + 4 <= m.ow) {
              *reinterpret_cast<float4*>(o) = make_float4(z[0], z[1], z[2], z[3]);
            } else {
#pragma unroll
              for (int i = 0; i < 4; ++i)
                if (ox + i < m.ow) o[i] = z[i];
            }
          }
          if constexpr (OB > 0) {
            constexpr int P = planes_of(OB);
#pragma unroll
            for (int i = 0; i < 4; ++i) {
              const uint32_t qv = cok ? quant_planes<OB>(hardtanh(z[i]), m.othr) : 0u;
#pragma unroll
              for (int p = 0; p < P; ++p) {
                // lanes 0-31: the 32 channels of column col + i, lanes 32-63: of column col + 4 + i
                const uint64_t bl = __ballot((qv >> p) & 1u);
                if (lane == 0) {
                  pk[(row * PT_W0 + 8 * g + i) * P + p] = (uint32_t)bl;
                  pk[(row * PT_W0 + 8 * g + 4 + i) * P + p] = (uint32_t)(bl >> 32);
                }
              }
            }
          }
        }
      }
      if constexpr (OB > 0) {
        constexpr int P = planes_of(OB);
        lds_barrier();
        for (int i = tid; i < PT_H0 * PT_W0 * P; i += 256) {
          const int qq = i / P, p = i - (i / P) * P;
          const int qy = cy0 + qq / PT_W0, qx = cx0 + qq % PT_W0;
          if (qy < m.oh && qx < m.ow)
            m.out_packed[((((int64_t)img * m.oh + qy) * m.ow + qx) * m.out_cw + ct) * P + p] = pk[i];
        }
      }
    }
  }
}

int device_cus_f() {
  int dev = 0, v = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) return 256;
  return v;
}

// Window of a tile for kernel size k and stride s (run-time mirror of Geo).
void geo_rt(int k, int s, int pool, int* ih, int* iw) {
  const int ct_h = pool ? 2 * PT_H + 1 : PT_H0, ct_w = pool ? 2 * PT_W + 1 : PT_W0;
  *ih = (ct_h - 1) * s + k;
  *iw = (ct_w - 1) * s + k;
}

bool f32m_plan(int n, int cin, int h, int w, int cout, int k, int stride, int pad, int pool, F32M* m) {
  memset(m, 0, sizeof(*m));
  if (n < 1 || cin < 1 || pad < 0 || cout < 1) return false;
  if (k != 3 && k != 5 && k != 7) return false;               // instantiated kernel sizes
  if (!(stride == 1 || (stride == 2 && pool))) return false;  // instantiated strides
  m->n = n;
  m->cin = cin;
  m->h = h;
  m->w = w;
  m->cout = cout;
  m->pad = pad;
  if (h + 2 * pad < k || w + 2 * pad < k) return false;
  m->ho = (h + 2 * pad - k) / stride + 1;
  m->wo = (w + 2 * pad - k) / stride + 1;
  int ih, iw;
  geo_rt(k, stride, pool, &ih, &iw);
  if ((int64_t)cin * ih * iw > 256 * F32M_NJ) return false;  // the window's register share
  if ((int64_t)cin * h * w >= ((int64_t)1 << 31) || ih >= (1 << 16) || iw >= (1 << 16)) return false;
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
  m->items = (int)items;
  const int taps2 = 2 * ((k * k + 1) / 2);  // padded taps per input channel
  m->l_w = (cin * ih * iw + 3) & ~3;
  m->l_ct = m->l_w + cin * taps2 * 32;
  m->l_pk = m->l_ct + (pool ? 32 * CT_STRIDE : 0);
  const int pk_words = pool ? PT_H * PT_W * 4 : PT_H0 * PT_W0 * 4;
  return (size_t)(m->l_pk + pk_words) * 4 <= F32M_LDS_MAX;
}

size_t f32m_lds(const F32M& m, int pool) {
  return (size_t)(m.l_pk + (pool ? PT_H * PT_W * 4 : PT_H0 * PT_W0 * 4)) * 4;
}

template <int KSZ, int S, int POOL>
int launch_geo(const F32M& m, int ob, int grid, size_t lds, hipStream_t s) {
  auto go = [&](auto kern) -> int {
    if (lds > 64 * 1024 && hipFuncSetAttribute(reinterpret_cast<const void*>(kern),
                                               hipFuncAttributeMaxDynamicSharedMemorySize,
                                               (int)F32M_LDS_MAX) != hipSuccess)
      return QCONV_EHIP;
    kern<<<dim3((unsigned)grid), 256, lds, s>>>(m);
    return hip_status();
  };
  switch (ob) {
    case 0: return go(conv_f32_mfma_kernel<KSZ, S, POOL, 0>);
    case 1: return go(conv_f32_mfma_kernel<KSZ, S, POOL, 1>);
    case 2: return go(conv_f32_mfma_kernel<KSZ, S, POOL, 2>);
    default: return go(conv_f32_mfma_kernel<KSZ, S, POOL, 3>);
  }
}

}  // namespace

bool conv_f32_mfma_supports(int n, int cin, int h, int w, int cout, int k, int stride, int pad, int pool) {
  F32M m;
  return f32m_plan(n > 0 ? n : 1, cin, h, w, cout, k, stride, pad, pool, &m);
}

int launch_conv_f32_mfma(const float* x, const float* w, int n, int cin, int h, int wd, int cout, int k, int stride,
                         int pad, const float* bn_k, const float* bn_b, int relu, int pool, float* out,
                         uint32_t* out_packed, int out_bits, Thr othr, hipStream_t s) {
  F32M m;
  if (n == 0) return QCONV_OK;
  if (!f32m_plan(n, cin, h, wd, cout, k, stride, pad, pool, &m)) return QCONV_EUNSUPPORTED;
  m.x = x;
  m.wt = w;
  m.bn_k = bn_k;
  m.bn_b = bn_b;
  m.relu = relu;
  m.out = out;
  m.out_packed = out_packed;
  m.out_cw = ceil_div(cout, 32);
  m.othr = othr;
  const int ob = out_packed ? out_bits : 0;
  const int blocks_per = 2 * device_cus_f() / m.co_tiles;
  const int64_t want = (int64_t)(blocks_per < 1 ? 1 : blocks_per);
  const int grid = (int)((want < m.items ? want : m.items) * m.co_tiles);
  const size_t lds = f32m_lds(m, pool);
  if (pool) {
    if (stride == 1) {
      if (k == 3) return launch_geo<3, 1, 1>(m, ob, grid, lds, s);
      if (k == 5) return launch_geo<5, 1, 1>(m, ob, grid, lds, s);
      return launch_geo<7, 1, 1>(m, ob, grid, lds, s);
    }
    if (k == 3) return launch_geo<3, 2, 1>(m, ob, grid, lds, s);
    if (k == 5) return launch_geo<5, 2, 1>(m, ob, grid, lds, s);
    return launch_geo<7, 2, 1>(m, ob, grid, lds, s);
  }
  if (k == 3) return launch_geo<3, 1, 0>(m, ob, grid, lds, s);
  if (k == 5) return launch_geo<5, 1, 0>(m, ob, grid, lds, s);
  return launch_geo<7, 1, 0>(m, ob, grid, lds, s);
}

}  // namespace qc
