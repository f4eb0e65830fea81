// conv_mfma.hip -- planning of the matrix-core convolution (block shape,
// halo tiles, which kernel) and the dispatch to the launcher of the operand
// format; the kernels are in conv_mfma.h, instantiated one (format, planes)
// pair per translation unit.
#include <stdio.h>
#include <string.h>

#include <atomic>

#include "conv_mfma.h"

namespace qc {
namespace mfma {

bool plan(const ConvArgs& a, int cfg, MfmaArgs* m) {
  memset(m, 0, sizeof(*m));
  m->c = a;
  const int op = a.mfma_op;
  // fp16 operands exactly for 16-bit inputs or 16-bit weights
  if ((op == OP_F16) != (a.a_bits == 16 || a.w_bits == 16)) return false;
  // fp4 products accumulate in fp32: exact only while every partial sum
  // (at most K * max|a| * max|w| in magnitude) stays below 2^24
  if (op == OP_FP4 &&
      (int64_t)a.kreal * (a.a_bits == 3 ? 4 : 1) * (a.w_bits == 3 ? 4 : 1) >= ((int64_t)1 << 24))
    return false;
  // Split-K items (cfg 2: fully connected layers and small maps) have few
  // k-steps per wave per stage, so each stage is a serial round of halo
  // loads, expansion and barriers: their fp4 stages take up to four times
  // the channels when the tile fits (ConvNet's 1024 -> 1024 FC 9.1 -> 6.8
  // us, ResNet-18's 512-channel 7x7 layers 4-6 % faster).
  const int chunk_max = op == OP_FP4 ? (cfg == 2 ? 4 : 1) * OpT<OP_FP4>::CHUNK_WORDS
                                     : (op == OP_F16 ? OpT<OP_F16>::CHUNK_WORDS : OpT<OP_I8>::CHUNK_WORDS);
  const int wpstep = op == OP_FP4 ? 2 : 1;  // words per k-step, rounded up to whole words
  const int word_bytes = op == OP_FP4 ? OpT<OP_FP4>::WORD_BYTES
                                      : (op == OP_F16 ? OpT<OP_F16>::WORD_BYTES : OpT<OP_I8>::WORD_BYTES);
  const int k_per_step = op == OP_FP4 ? OpT<OP_FP4>::K_PER_STEP
                                      : (op == OP_F16 ? OpT<OP_F16>::K_PER_STEP : OpT<OP_I8>::K_PER_STEP);
  const int cw_round = ceil_div(a.cw, wpstep) * wpstep;
  m->ksteps = ceil_div(a.cw * 32, k_per_step);
  m->wx = op == OP_FP4 ? a.w_fp4 : (op == OP_F16 ? a.w_f16 : a.w_i8);
  const int64_t wxb = (int64_t)a.kh * a.kw * m->ksteps * a.cop * 32;
  if (wxb >= ((int64_t)1 << 31)) return false;
  m->wx_bytes = (int)wxb;
  m->pool = a.pool;
  m->uw = a.pool ? a.wo / 2 : a.wo;
  const int uh = a.pool ? a.ho / 2 : a.ho;
  m->upi = uh * m->uw;
  if (m->upi < 1) return false;
  const int rows = cfg_rows(cfg);
  const int rows_per_unit = a.pool ? 4 : 1;
  const int units_pb = rows / rows_per_unit;
  m->units_pb = units_pb;
  m->hc = (a.wo - 1) * a.stride + a.kw;
  m->vec = (m->upi % 4 == 0) ? 1 : 0;
  // Channel chunks, largest first; smaller chunks shrink the LDS tile so
  // that more small images fit in one block.
  int best_units = -1;
  MfmaArgs best = *m;
  for (int wide = 0; wide < 2 && best_units < 0; ++wide) {
  // the wide buffer (one block per CU) serves the fp16 tiles and the
  // 256-row tiles of stride-2 layers, whose input rows are twice as many
  // (ResNet-18's 64 -> 128 stride-2 layer at batch 64 took 26 us on 64-row
  // split-K items, 15 us on 256-row ones)
  if (wide && op != OP_F16 && (cfg == 2 || a.stride == 1)) break;
  const size_t lim = wide ? (size_t)MAX_LDS_WIDE : (size_t)MAX_LDS;
  for (int cwc = min(chunk_max, cw_round); cwc >= wpstep; cwc /= 2) {
    if (cwc % wpstep) break;
    MfmaArgs t = *m;
    t.chunk_words = cwc;
    t.pix_bytes = cwc * word_bytes + 16;
    t.nchunks = ceil_div(cw_round, cwc);
    int units;
    const int conv_rows_img = a.pool ? 2 * uh : a.ho;
    if (m->upi * 2 <= units_pb) {
      t.hr = (conv_rows_img - 1) * a.stride + a.kh;
      const size_t slot = (size_t)t.hr * t.hc * t.pix_bytes;
      const int fit = (int)(lim / slot);
      t.ipb = min(units_pb / m->upi, fit);
      if (cfg == 2) {
        // split-K items of whole images (fully connected layers): no more
        // images per item than leaves one item per CU, so that every CU
        // works and the largest channel chunk fits (fewer serial stages)
        const int64_t per_cu = (int64_t)a.n * ceil_div(a.cout, cfg_block_co(cfg)) / device_cus();
        if (per_cu < t.ipb) t.ipb = per_cu < 1 ? 1 : (int)per_cu;
      }
      if (t.ipb < 1) continue;
      // one image per item is the single-image mode: one block per image
      t.bpi = t.ipb == 1 ? 1 : 0;
      units = t.ipb * m->upi;
    } else {
      t.ipb = 1;
      t.bpi = ceil_div(m->upi, units_pb);
      // unit rows a run of units_pb units can touch, then conv rows
      const int urows = min(uh, ceil_div(units_pb, m->uw) + 1);
      const int crows = a.pool ? 2 * urows : urows;
      t.hr = (crows - 1) * a.stride + a.kh;
      if ((size_t)t.hr * t.hc * t.pix_bytes > lim) continue;
      units = units_pb;
    }
    if (units > best_units) {
      best_units = units;
      best = t;
    }
    if (units == units_pb || (m->upi * 2 <= units_pb && t.ipb == units_pb / m->upi)) break;
  }
  }
  if (best_units < 0) return false;
  *m = best;
  m->slot_pix = m->hr * m->hc;
  m->fd_upi = make_fastdiv((uint32_t)m->upi);
  m->fd_uw = make_fastdiv((uint32_t)m->uw);
  m->fd_slot = make_fastdiv((uint32_t)m->slot_pix);
  m->fd_hc = make_fastdiv((uint32_t)m->hc);
  m->fd_cwc = make_fastdiv((uint32_t)m->chunk_words);
  // every fast division stays exact: dividend * divisor < 2^32
  const uint64_t items = (uint64_t)m->ipb * m->slot_pix * m->chunk_words;
  const uint64_t max_unit = (uint64_t)m->upi + 256;
  if (items * m->chunk_words >= (1ull << 32) || items * m->slot_pix >= (1ull << 32) ||
      (uint64_t)m->slot_pix * m->hc >= (1ull << 32) || max_unit * m->upi >= (1ull << 32) ||
      max_unit * m->uw >= (1ull << 32))
    return false;
  m->tiles_px = (m->ipb == 1) ? a.n * m->bpi : ceil_div(a.n, m->ipb);
  m->tiles_co = ceil_div(a.cout, cfg_block_co(cfg));
  if (m->tiles_px < 1 || m->tiles_co < 1) return false;  // never an empty launch
  m->halo_bytes = m->slot_pix * m->pix_bytes * m->ipb;
  m->ht_needed = a.out_packed && hardtanh_needed(a.out_bits, a.othr);
  const int64_t ab = (int64_t)a.n * a.h * a.w * a.cw * act_words(a.a_bits) * 4;
  m->act_bytes = ab < ((int64_t)1 << 31) ? (int)ab : 0;
  const int64_t ob = (int64_t)a.n * a.cout * m->upi * 4;
  m->out_bytes = ob < ((int64_t)1 << 31) ? (int)ob : 0;
  m->buf_bytes = (m->halo_bytes + 15) & ~15;
  if (cfg == 2) m->buf_bytes = max(m->buf_bytes, RED_BYTES / 2);  // the two buffers hold the split-K partials
  return true;
}

// LDS bytes of one block: two parameter sets and two halo buffers.
size_t block_lds(const MfmaArgs& m) { return 2 * PARAM_BYTES + (size_t)m.buf_bytes * 2; }


// Block shape: 256 rows x 128 (or 64) output channels; when those leave
// compute units without a block, 256 x 64 if that gives every CU one, else
// 64-row split-K blocks (measured on the ConvNet and ResNet-18 layers: with
// one or more 256-row items per CU the unsplit shapes are faster, with fewer
// the split one); split-K too when the 256-row input tile does not fit the
// staging buffer.
bool use_pp(const MfmaArgs& m, int cfg, int cus);

int pick_cfg_base(const ConvArgs& a) {
  const int big = a.cout <= 64 ? 1 : 0;
  MfmaArgs m;
  if (!plan(a, big, &m)) {
    // the 256-row halo does not fit (wide rows, stride 2): 64-row items
    MfmaArgs s;
    return plan(a, 2, &s) ? 2 : big;
  }
  const int64_t blocks = (int64_t)m.tiles_px * m.tiles_co;
  const int steps = a.kh * a.kw * m.ksteps;
  // fewer 128-channel items than CUs, or (stride 1) than two per CU
  if ((blocks < device_cus() || (a.stride == 1 && blocks < 2 * device_cus())) && steps >= 8) {
    // 64-channel blocks double the block count; when that gives every CU a
    // block they beat the split-K shape (ResNet-18 3x3 layers: 512 ch at
    // 7x7, batch 256, 59 -> 43 us; 256 ch at 14x14, batch 64, 22 -> 18 us),
    // and at one 128-channel item per CU they beat it too, three blocks per
    // CU against two (ConvNet's 256 -> 512 layer at 8x8 23.7 -> 21.6 us,
    // its pooled 512 -> 512 layer 36.9 -> 34.0 us; ResNet-18's 128-channel
    // 28x28 layer 15.9 -> 14.8 us; its stride-2 layers measured slower)
    MfmaArgs h;
    if (big == 0 && plan(a, 1, &h) && (int64_t)h.tiles_px * h.tiles_co >= device_cus()) return 1;
    MfmaArgs s;
    if (plan(a, 2, &s)) return 2;
  }
  return big;
}

// The store-overlapped kernel needs two items per CU: a layer whose
// 128-channel items are too few for it takes 64-channel items when those
// are enough (its epilogue then runs beside the other group's MFMAs instead
// of after them).
int pick_cfg(const ConvArgs& a) {
  const int cfg = pick_cfg_base(a);
  if (cfg != 0) return cfg;
  MfmaArgs m0, m1;
  const int cus = device_cus();
  if (plan(a, 0, &m0) && !use_pp(m0, 0, cus) && plan(a, 1, &m1) && use_pp(m1, 1, cus)) return 1;
  return 0;
}

// The swapped orientation serves unpacked, unpooled outputs whose byte size
// fits a buffer resource.
bool use_swap(const MfmaArgs& m) {
  const ConvArgs& a = m.c;
  return !a.pool && m.out_bytes > 0;
}

// Compute units of the current device, queried once per device.
int device_cus() {
  static std::atomic<int> cache[MAX_DEVICES];
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  const bool cached = dev >= 0 && dev < MAX_DEVICES;
  if (cached) {
    const int c = cache[dev].load(std::memory_order_relaxed);
    if (c > 0) return c;
  }
  int v = 0;
  if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0) return 256;
  if (cached) cache[dev].store(v, std::memory_order_relaxed);
  return v;
}

// LDS bytes of one store-overlapped block: parameters, the block's weights,
// one halo buffer per group.
size_t pp_lds(const MfmaArgs& m, int cfg) {
  const int bco = cfg_block_co(cfg);
  return PARAM_BYTES + (size_t)m.c.kh * m.c.kw * m.ksteps * bco * 32 + (size_t)m.buf_bytes * 2;
}

// The ping-pong kernel serves 256-row shapes with unpooled outputs whose
// channels fit one stage and whose weights fit next to two halo buffers,
// when every block gets at least one item per group.
bool use_pp(const MfmaArgs& m, int cfg, int cus) {
  if (cfg == 2 || m.c.mfma_op == OP_F16 || !use_swap(m) || m.nchunks != 1 || m.act_bytes == 0) return false;
  // packed outputs (alone, or as the copy of a BN output) of the input's
  // width (the case of a network of one activation width)
  if (m.c.out_packed != nullptr &&
      ((m.c.mode != QCONV_EPI_BN_F32 && m.c.mode != QCONV_EPI_BN_PACK) || m.c.out_bits != m.c.a_bits))
    return false;
  if (pp_lds(m, cfg) > (size_t)LDS_PER_CU) return false;
  if ((int64_t)m.tiles_px * m.tiles_co < 2 * (int64_t)cus) return false;
  // a packed output alone: only where the base kernel's own shape leaves
  // fewer than two items per CU (measured on ResNet-18 and ConvNet layers:
  // with 2-3 items per CU of the base kernel its blocks overlap each other
  // better than the two groups do; with one item per CU the groups win)
  if (m.c.mode == QCONV_EPI_BN_PACK) {
    MfmaArgs b;
    if (plan(m.c, pick_cfg_base(m.c), &b) && (int64_t)b.tiles_px * b.tiles_co >= 2 * (int64_t)cus) return false;
  }
  return true;
}


}  // namespace mfma

using namespace mfma;

bool mfma_supports(const ConvArgs& a) {
  if (a.stride > 2 || a.n == 0) return false;
  MfmaArgs m;
  return plan(a, pick_cfg(a), &m);
}

int mfma_kernel_name(const ConvArgs& a, char* buf, int len) {
  MfmaArgs m;
  const int cfg = pick_cfg(a);
  if (!plan(a, cfg, &m)) return QCONV_EUNSUPPORTED;
  char name[96];
  if (use_pp(m, cfg, device_cus()))
    snprintf(name, sizeof(name), "conv_mfma_pp_kernel<%d, %d, %d, %d>", a.mfma_op, act_words(a.a_bits), cfg,
             a.out_packed ? a.out_bits : 0);
  else
    snprintf(name, sizeof(name), "conv_mfma_kernel<%d, %d, %d, %d>", a.mfma_op, act_words(a.a_bits), cfg,
             use_swap(m) ? 1 : 0);
  if (buf && len > 0) snprintf(buf, (size_t)len, "%s", name);
  return (int)strlen(name);
}

int launch_conv_mfma(const ConvArgs& a, hipStream_t s) {
  MfmaArgs m;
  const int cfg = pick_cfg(a);
  if (!plan(a, cfg, &m)) return QCONV_EUNSUPPORTED;
  const int pa = act_words(a.a_bits);
  if (a.mfma_op == OP_F16) {
    if (pa == 16) return launch_mfma_f16_p16(m, cfg, s);
    if (pa == 1) return launch_mfma_f16_p1(m, cfg, s);
    if (pa == 2) return launch_mfma_f16_p2(m, cfg, s);
    return launch_mfma_f16_p4(m, cfg, s);
  }
  if (a.mfma_op == OP_FP4) {
    if (pa == 1) return launch_mfma_fp4_p1(m, cfg, s);
    if (pa == 2) return launch_mfma_fp4_p2(m, cfg, s);
    return launch_mfma_fp4_p4(m, cfg, s);
  }
  if (pa == 1) return launch_mfma_i8_p1(m, cfg, s);
  if (pa == 2) return launch_mfma_i8_p2(m, cfg, s);
  return launch_mfma_i8_p4(m, cfg, s);
}

}  // namespace qc
