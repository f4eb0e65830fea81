// api.hip -- the C ABI declared in include/qconv.h: argument validation,
// kernel selection and the layer loop of whole networks.  Nothing here
// allocates device memory or synchronises; every launch goes to the
// caller's stream.
#include <math.h>
#include <stdio.h>
#include <string.h>

#include <atomic>
#include <mutex>
#include <new>
#include <vector>

#include "qconv_internal.h"

using namespace qc;

namespace {

constexpr int MAX_DEVICES_API = 64;

constexpr float kActThr2[1] = {0.5f};
constexpr float kActThr3[3] = {0.125f, 0.375f, 0.75f};
constexpr float kWgtThr2[1] = {0.7f};
constexpr float kWgtThr3[3] = {0.125f, 0.375f, 0.75f};

bool bits_ok(int b) { return b >= 1 && b <= 3; }
bool act_bits_ok(int b) { return bits_ok(b) || b == 16; }
int max_code(int bits) { return bits == 3 ? 4 : 1; }
int code_shift(int bits) { return bits == 3 ? 2 : 0; }

// Threshold set for `bits`, from a host array (validated) or the defaults.
int act_thresholds(int bits, const float* user, Thr* t) {
  *t = {0.0f, 0.0f, 0.0f};
  if (bits == 1) return QCONV_OK;
  if (bits == 2) {
    t->t0 = user ? user[0] : kActThr2[0];
    if (!(t->t0 >= 0.0f)) return QCONV_EINVAL;
    return QCONV_OK;
  }
  const float* s = user ? user : kActThr3;
  t->t0 = s[0];
  t->t1 = s[1];
  t->t2 = s[2];
  if (!(t->t0 >= 0.0f && t->t0 <= t->t1 && t->t1 <= t->t2)) return QCONV_EINVAL;
  return QCONV_OK;
}

size_t packed_bytes(int64_t n, int c, int64_t h, int64_t w, int bits) {
  return (size_t)(n * h * w * ceil_div(c, 32) * act_words(bits)) * sizeof(uint32_t);
}

}  // namespace

extern "C" {

const char* qconv_error_string(int status) {
  switch (status) {
    case QCONV_OK: return "ok";
    case QCONV_EINVAL: return "invalid argument";
    case QCONV_EUNSUPPORTED: return "unsupported configuration";
    case QCONV_EWORKSPACE: return "workspace too small";
    case QCONV_EOVERFLOW: return "int32 accumulator could overflow (K * max|a| * max|w| >= 2^31)";
    case QCONV_EHIP: return "HIP launch or runtime error";
    case QCONV_ESCRATCH: return "needs more than the library's fixed no-allocation scratch (qnet_noalloc_limit bytes)";
    default: return "unknown status";
  }
}

int qconv_version(void) { return 101; }

int qconv_inference_op(int m, int n, int* op, int* precision_bits) {
  auto valid = [](int b) { return b == 1 || b == 2 || b == 3 || b == 16 || b == 32; };
  if (!op || !precision_bits || !valid(m) || !valid(n)) return QCONV_EINVAL;
  const int lo = m < n ? m : n, hi = m < n ? n : m;
  if (lo == 32) {
    *op = QCONV_OP_MAC;
    *precision_bits = 32;
  } else if (hi >= 16) {
    if (hi == 32) return QCONV_EUNSUPPORTED;  // not a row of the tables
    *op = (lo == 3) ? QCONV_OP_SHIFT_ADDER : QCONV_OP_XNOR_ADDER;
    *precision_bits = 16;
  } else {
    *op = (lo == 3) ? QCONV_OP_SHIFT : QCONV_OP_XNOR;
    *precision_bits = (hi <= 2) ? 1 : 2;
  }
  return QCONV_OK;
}

size_t qconv_packed_act_bytes(int n, int c, int h, int w, int bits) {
  if (n < 0 || c < 1 || h < 1 || w < 1 || !act_bits_ok(bits)) return 0;
  return packed_bytes(n, c, h, w, bits);
}

int qconv_pack_act(const float* x, int n, int c, int h, int w, int bits, const float* thresholds,
                   uint32_t* out_packed, void* stream) {
  if (n < 0 || c < 1 || h < 1 || w < 1 || !act_bits_ok(bits)) return QCONV_EINVAL;
  if (n > 0 && (!x || !out_packed)) return QCONV_EINVAL;
  if (bits == 16) return launch_pack_act_f16(x, n, c, h, w, out_packed, (hipStream_t)stream);
  Thr t;
  const int rc = act_thresholds(bits, thresholds, &t);
  if (rc) return rc;
  return launch_pack_act(x, n, c, h, w, bits, t, out_packed, (hipStream_t)stream);
}

size_t qconv_packed_weight_bytes(int cout, int cin, int kh, int kw, int bits) {
  if (cout < 1 || cin < 1 || kh < 1 || kw < 1 || !act_bits_ok(bits)) return 0;
  if (bits == 16) return wbytes_f16(cout, cin, kh, kw);
  return wbytes_planes(cout, cin, kh, kw, bits) + wbytes_i8(cout, cin, kh, kw) +
         wbytes_fp4(cout, cin, kh, kw) + wbytes_f16(cout, cin, kh, kw);
}

int qconv_pack_weight(const float* w, int cout, int cin, int kh, int kw, int bits,
                      const float* base_thresholds, uint32_t* out_packed, float* out_scale,
                      void* stream) {
  if (!w || !out_packed || !out_scale || cout < 1 || cin < 1 || kh < 1 || kw < 1 || !act_bits_ok(bits))
    return QCONV_EINVAL;
  if (bits == 16) return launch_pack_weight_f16(w, cout, cin, kh, kw, out_packed, out_scale, (hipStream_t)stream);
  float base[3] = {0.0f, 0.0f, 0.0f};
  if (bits == 2) base[0] = base_thresholds ? base_thresholds[0] : kWgtThr2[0];
  if (bits == 3)
    for (int j = 0; j < 3; ++j) base[j] = base_thresholds ? base_thresholds[j] : kWgtThr3[j];
  if (bits == 2 && !(base[0] >= 0.0f)) return QCONV_EINVAL;
  if (bits == 3 && !(base[0] >= 0.0f && base[0] <= base[1] && base[1] <= base[2])) return QCONV_EINVAL;
  return launch_pack_weight(w, cout, cin, kh, kw, bits, base, out_packed, out_scale,
                            (hipStream_t)stream);
}

int qconv_fold_bn(const float* gamma, const float* beta, const float* mean, const float* var,
                  double eps, int c, float* k_out, float* b_out) {
  if (!gamma || !beta || !mean || !var || !k_out || !b_out || c < 1 || !(eps >= 0.0))
    return QCONV_EINVAL;
  for (int i = 0; i < c; ++i) {
    const double kd = (double)gamma[i] / sqrt((double)var[i] + eps);
    k_out[i] = (float)kd;
    b_out[i] = (float)((double)beta[i] - kd * (double)mean[i]);
  }
  return QCONV_OK;
}

int qconv_out_size(int in, int k, int stride, int pad) {
  if (in < 1 || k < 1 || stride < 1 || pad < 0) return QCONV_EINVAL;
  const int o = (in + 2 * pad - k) / stride + 1;
  return (in + 2 * pad - k) < 0 ? QCONV_EINVAL : o;
}

}  // extern "C"

namespace {

// Validates a qconv_forward call and fills the kernel arguments; returns the
// concrete algorithm to run (> 0) or a negative status.
int prepare_conv(const qconv_desc* d, const uint32_t* act_packed, const uint32_t* w_packed,
                 const qconv_epilogue* epi, void* out, uint32_t* out_packed, bool check_ptrs,
                 ConvArgs* args) {
  if (!d || !epi) return QCONV_EINVAL;
  if (d->n < 0 || d->cin < 1 || d->h < 1 || d->w < 1 || d->cout < 1 || d->kh < 1 || d->kw < 1 ||
      d->stride < 1 || d->pad < 0 || !act_bits_ok(d->a_bits) || !act_bits_ok(d->w_bits))
    return QCONV_EINVAL;
  if (d->algo < QCONV_ALGO_AUTO || d->algo > QCONV_ALGO_MFMA_F16) return QCONV_EINVAL;
  // one side 16-bit (Table I: 16-bit inputs with 1..3-bit weights, or
  // 1..3-bit inputs with 16-bit weights) runs on the fp16 matrix cores only,
  // and only such layers do; 16 x 16 is not a row of the tables
  const bool f16 = d->a_bits == 16 || d->w_bits == 16;
  if (d->a_bits == 16 && d->w_bits == 16) return QCONV_EUNSUPPORTED;
  if (f16 ? (d->algo != QCONV_ALGO_AUTO && d->algo != QCONV_ALGO_MFMA_F16) : d->algo == QCONV_ALGO_MFMA_F16)
    return QCONV_EUNSUPPORTED;
  const int ho = qconv_out_size(d->h, d->kh, d->stride, d->pad);
  const int wo = qconv_out_size(d->w, d->kw, d->stride, d->pad);
  if (ho < 1 || wo < 1) return QCONV_EINVAL;
  const int64_t K = (int64_t)d->cin * d->kh * d->kw;
  if (!f16 && K * max_code(d->a_bits) * max_code(d->w_bits) >= (int64_t)1 << 31) return QCONV_EOVERFLOW;
  if (epi->mode < QCONV_EPI_INT32 || epi->mode > QCONV_EPI_BN_PACK) return QCONV_EINVAL;
  if (f16 && epi->mode == QCONV_EPI_INT32) return QCONV_EUNSUPPORTED;  // the accumulator is fp32
  if (epi->flags & ~(QCONV_EPI_POOL2 | QCONV_EPI_RESIDUAL)) return QCONV_EINVAL;
  const bool pool = (epi->flags & QCONV_EPI_POOL2) != 0;
  const bool resid = (epi->flags & QCONV_EPI_RESIDUAL) != 0;
  if (pool && (ho < 2 || wo < 2)) return QCONV_EINVAL;
  if (resid && epi->mode != QCONV_EPI_BN_F32) return QCONV_EINVAL;
  if (check_ptrs) {
    if (resid && !epi->residual) return QCONV_EINVAL;
    if (epi->mode == QCONV_EPI_SCALE_F32 && !epi->scale) return QCONV_EINVAL;
    if ((epi->mode == QCONV_EPI_BN_F32 || epi->mode == QCONV_EPI_BN_PACK) && (!epi->bn_k || !epi->bn_b))
      return QCONV_EINVAL;
  }
  const bool pack = epi->mode == QCONV_EPI_BN_PACK || (epi->mode == QCONV_EPI_BN_F32 && out_packed);
  if (check_ptrs && epi->mode == QCONV_EPI_BN_PACK && !out_packed) return QCONV_EINVAL;
  if (check_ptrs && epi->mode != QCONV_EPI_BN_PACK && !out && d->n > 0) return QCONV_EINVAL;
  if (pack && !bits_ok(epi->out_bits)) return QCONV_EINVAL;
  if (check_ptrs && d->n > 0 && (!act_packed || !w_packed)) return QCONV_EINVAL;

  ConvArgs& a = *args;
  memset(&a, 0, sizeof(a));
  a.act = act_packed;
  a.wt = w_packed;
  a.n = d->n;
  a.h = d->h;
  a.w = d->w;
  a.cw = ceil_div(d->cin, 32);
  a.cout = d->cout;
  a.cop = cout_pad(d->cout);
  a.kh = d->kh;
  a.kw = d->kw;
  a.stride = d->stride;
  a.pad = d->pad;
  a.ho = ho;
  a.wo = wo;
  a.oh_out = pool ? ho / 2 : ho;
  a.ow_out = pool ? wo / 2 : wo;
  a.kreal = (int)K;
  a.shift = code_shift(d->a_bits) + code_shift(d->w_bits);
  a.a_bits = d->a_bits;
  a.w_bits = d->w_bits;
  a.mode = epi->mode;
  a.pool = pool ? 1 : 0;
  a.residual_on = resid ? 1 : 0;
  a.scale = epi->scale;
  a.bn_k = epi->bn_k;
  a.bn_b = epi->bn_b;
  a.residual = epi->residual;
  a.out = out;
  a.out_packed = pack ? out_packed : nullptr;
  a.out_bits = pack ? epi->out_bits : 0;
  a.out_cw = ceil_div(d->cout, 32);
  if (pack) {
    const int rc = act_thresholds(epi->out_bits, epi->out_thresholds, &a.othr);
    if (rc) return rc;
  }
  a.cin = d->cin;
  if (d->w_bits == 16) {
    // the whole buffer is the fp16 operand copy
    a.w_f16 = reinterpret_cast<const uint8_t*>(w_packed);
  } else {
    const uint8_t* wb = reinterpret_cast<const uint8_t*>(w_packed);
    a.w_i8 = wb ? wb + wbytes_planes(d->cout, d->cin, d->kh, d->kw, d->w_bits) : nullptr;
    a.w_fp4 = wb ? a.w_i8 + wbytes_i8(d->cout, d->cin, d->kh, d->kw) : nullptr;
    a.w_f16 = wb ? a.w_fp4 + wbytes_fp4(d->cout, d->cin, d->kh, d->kw) : nullptr;
  }
  if (f16) {
    a.mfma_op = OP_F16;
    if (d->n > 0 && !mfma_supports(a)) return QCONV_EUNSUPPORTED;
    return QCONV_ALGO_MFMA_F16;
  }
  // the fp4 matrix cores accumulate in fp32: every partial sum is an integer
  // of magnitude at most K * max|a| * max|w|, exact only below 2^24
  const bool fp4_exact = K * max_code(d->a_bits) * max_code(d->w_bits) < ((int64_t)1 << 24);
  if (d->algo == QCONV_ALGO_MFMA_FP4 && !fp4_exact) return QCONV_EUNSUPPORTED;
  if (d->algo == QCONV_ALGO_MFMA_I8 || d->algo == QCONV_ALGO_MFMA_FP4) {
    a.mfma_op = d->algo == QCONV_ALGO_MFMA_FP4 ? OP_FP4 : OP_I8;
    if (d->n > 0 && !mfma_supports(a)) return QCONV_EUNSUPPORTED;
    return d->algo;
  }
  // AUTO: the fp4 matrix cores (int8 ones, whose int32 accumulator is exact
  // at any size, past the fp4 bound), except for tiny contractions (K <= 256,
  // the 1x1 shortcut convolutions of ResNet-18) that the LDS-tiled XNOR
  // kernel serves, where staging a matrix-core input tile costs more than
  // the whole bitplane product (measured 18-19 us on the bitplane kernels
  // against 21-29 us on the matrix cores for those layers).  Small
  // contractions the XNOR kernel does not serve (packed or pooled outputs,
  // 3-bit operands) would fall to the one-lane-per-pixel kernel, which the
  // matrix cores beat (1x1, K = 64 and 128, packed 2-bit outputs: 11-12 us
  // against 22-30 us).
  if (d->algo == QCONV_ALGO_AUTO && d->n > 0 && (K > 256 || !xnor_supports(a))) {
    a.mfma_op = fp4_exact ? OP_FP4 : OP_I8;
    if (mfma_supports(a)) return fp4_exact ? QCONV_ALGO_MFMA_FP4 : QCONV_ALGO_MFMA_I8;
  }
  return QCONV_ALGO_BITPLANE;
}

}  // namespace

extern "C" {

int qconv_resolve_algo(const qconv_desc* d, const qconv_epilogue* epi) {
  ConvArgs a;
  return prepare_conv(d, nullptr, nullptr, epi, nullptr, nullptr, false, &a);
}

int aqe_forward(const float* x, int64_t n, int bits, float alpha, const float* thresholds, const float* scale,
                int64_t group_size, float* y, void* stream) {
  if (n < 0 || !bits_ok(bits) || !(alpha >= 0.0f && alpha <= 1.0f) || group_size < 0) return QCONV_EINVAL;
  if (n > 0 && (!x || !y)) return QCONV_EINVAL;
  Thr t = {0.0f, 0.0f, 0.0f};
  if (group_size == 0) {
    if (scale) return QCONV_EINVAL;
    const int rc = act_thresholds(bits, thresholds, &t);
    if (rc) return rc;
  } else {
    if (n % group_size != 0 || (n > 0 && !scale)) return QCONV_EINVAL;
    if (bits == 2) t.t0 = thresholds ? thresholds[0] : kWgtThr2[0];
    if (bits == 3) {
      t.t0 = thresholds ? thresholds[0] : kWgtThr3[0];
      t.t1 = thresholds ? thresholds[1] : kWgtThr3[1];
      t.t2 = thresholds ? thresholds[2] : kWgtThr3[2];
    }
    if (bits == 2 && !(t.t0 >= 0.0f)) return QCONV_EINVAL;
    if (bits == 3 && !(t.t0 >= 0.0f && t.t0 <= t.t1 && t.t1 <= t.t2)) return QCONV_EINVAL;
  }
  return launch_aqe_forward(x, n, bits, alpha, t, group_size ? scale : nullptr, group_size ? group_size : 1, y,
                            (hipStream_t)stream);
}

int aqe_backward(const float* x, const float* gy, int64_t n, float alpha, float* gx, void* stream) {
  if (n < 0 || !(alpha >= 0.0f && alpha <= 1.0f)) return QCONV_EINVAL;
  if (n > 0 && (!x || !gy || !gx)) return QCONV_EINVAL;
  return launch_aqe_backward(x, gy, n, alpha, gx, (hipStream_t)stream);
}

int aqe_sgd_clip(float* w, const float* g, int64_t n, float lr, void* stream) {
  if (n < 0 || !(lr == lr)) return QCONV_EINVAL;
  if (n > 0 && (!w || !g)) return QCONV_EINVAL;
  return launch_aqe_sgd_clip(w, g, n, lr, (hipStream_t)stream);
}

int qconv_kernel_name(const qconv_desc* d, const qconv_epilogue* epi, int packed_out, char* buf, int len) {
  ConvArgs a;
  static uint32_t marker;  // stands for a packed output buffer; never accessed
  const int algo = prepare_conv(d, nullptr, nullptr, epi, nullptr, packed_out ? &marker : nullptr, false, &a);
  if (algo < 0) return algo;
  if (algo == QCONV_ALGO_BITPLANE) return bitplane_kernel_name(a, buf, len);
  return mfma_kernel_name(a, buf, len);
}

int qconv_forward(const qconv_desc* d, const uint32_t* act_packed, const uint32_t* w_packed,
                  const qconv_epilogue* epi, void* out, uint32_t* out_packed, void* stream) {
  ConvArgs a;
  const int algo = prepare_conv(d, act_packed, w_packed, epi, out, out_packed, true, &a);
  if (algo < 0) return algo;
  if (d->n == 0) return QCONV_OK;
  hipStream_t s = (hipStream_t)stream;
  if (algo == QCONV_ALGO_BITPLANE) return launch_conv_bitplane(a, s);
  return launch_conv_mfma(a, s);
}

// ---------------------------------------------------------------------------
// Networks
// ---------------------------------------------------------------------------

}  // extern "C"

namespace {

enum LayerKind { L_CONV_F32, L_MAXPOOL_F32, L_QUANTIZE, L_QCONV, L_AVGPOOL, L_FC_F32 };

struct QTensor {
  int c, h, w, bits;  // bits 0 = fp32 NCHW, else packed bitplanes
};

struct QLayer {
  int kind = 0, src = 0, src2 = -1;
  const float* wf = nullptr;
  const uint32_t* wq = nullptr;
  const float* bn_k = nullptr;
  const float* bn_b = nullptr;
  const float* bias = nullptr;
  int cout = 0, k = 0, stride = 1, pad = 0, w_bits = 0, pool2 = 0, relu = 0, out_bits = 0;
  // a quantized conv with an fp32 output also writes tensor pack_dst, the
  // packed Q(HardTanh(z)) of its output, from the same epilogue; the
  // quantize layer that made that tensor is then `fused` and launches nothing
  int pack_dst = -1, fused = 0;
  // fp32 conv on the matrix cores (the network's fp32 algorithm when the
  // layer fits it); pool_dst: the tensor of a 3x3 / 2 max pooling fused into
  // its epilogue (the conv's own output is then never written)
  int f32_mfma = 0, pool_dst = -1;
};

size_t tensor_bytes(const QTensor& t, int batch) {
  if (t.bits == 0) return (size_t)batch * t.c * t.h * t.w * sizeof(float);
  return packed_bytes(batch, t.c, t.h, t.w, t.bits);
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

}  // namespace

struct qnet {
  std::vector<QTensor> t;
  std::vector<QLayer> L;
  int f32_algo = QNET_F32_MFMA;
};

namespace {
int run_layers(const qnet* net, const float* x, int batch, float* logits, char* ws, const size_t* toff,
               const size_t* woff, int first, int count, hipStream_t s);

// Whether fp32 conv layer l runs on the matrix cores: the kernel must fit it
// as it will run (with its fused pooling or without); otherwise the chain.
bool conv_uses_mfma(const qnet* net, const QLayer& l) {
  if (l.kind != L_CONV_F32 || !l.f32_mfma) return false;
  const QTensor& s = net->t[l.src];
  return conv_f32_mfma_supports(1, s.c, s.h, s.w, l.cout, l.k, l.stride, l.pad, l.pool_dst > 0 ? 1 : 0, 0);
}

// The matrix-core arithmetic of such a layer: 1 (exact bf16 splits, six
// partial products) when the network asks for it and the layer is a pooled
// geometry that kernel takes, else 0 (fp32 matrix cores).
int conv_mfma_alg(const qnet* net, const QLayer& l) {
  if (net->f32_algo != QNET_F32_BF16X6 || l.pool_dst <= 0) return 0;
  const QTensor& s = net->t[l.src];
  return conv_f32_mfma_supports(1, s.c, s.h, s.w, l.cout, l.k, l.stride, l.pad, 1, 1) ? 1 : 0;
}
}  // namespace

namespace {

// Workspace plan: every tensor except the input (0) and the last one gets
// its own 256-byte aligned region, then one region per fp32 conv for its
// re-laid-out weights.  Returns the total; offsets[id] = (size_t)-1 if none.
size_t plan(const qnet* net, int batch, std::vector<size_t>* toff, std::vector<size_t>* woff) {
  size_t off = 0;
  const int last = (int)net->t.size() - 1;
  if (toff) toff->assign(net->t.size(), (size_t)-1);
  for (int id = 1; id < last; ++id) {
    if (toff) (*toff)[id] = off;
    off = align256(off + tensor_bytes(net->t[id], batch));
  }
  if (woff) woff->assign(net->L.size(), (size_t)-1);
  for (size_t i = 0; i < net->L.size(); ++i) {
    const QLayer& l = net->L[i];
    if (l.kind != L_CONV_F32) continue;
    if (woff) (*woff)[i] = off;
    const int cin = net->t[l.src].c;
    off = align256(off + (size_t)cin * l.k * l.k * ceil_div(l.cout, 64) * 64 * sizeof(float));
  }
  return off;
}

int add_tensor(qnet* net, QLayer l, QTensor out) {
  if (out.c < 1 || out.h < 1 || out.w < 1) return QCONV_EINVAL;
  net->L.push_back(l);
  net->t.push_back(out);
  return (int)net->t.size() - 1;
}

bool valid_src(const qnet* net, int id) { return net && id >= 0 && id < (int)net->t.size(); }

}  // namespace

extern "C" {

qnet* qnet_create(int in_c, int in_h, int in_w) {
  if (in_c < 1 || in_h < 1 || in_w < 1) return nullptr;
  qnet* net = new (std::nothrow) qnet();
  if (!net) return nullptr;
  net->t.push_back({in_c, in_h, in_w, 0});
  return net;
}

void qnet_destroy(qnet* net) { delete net; }

int qnet_add_conv_f32(qnet* net, int src, const float* w, int cout, int k, int stride, int pad,
                      const float* bn_k, const float* bn_b, int relu, int out_bits) {
  if (!valid_src(net, src) || !w || !bn_k || !bn_b || cout < 1 || k < 1 || stride < 1 || pad < 0 ||
      out_bits < 0 || out_bits > 3)
    return QCONV_EINVAL;
  const QTensor& s = net->t[src];
  if (s.bits != 0) return QCONV_EINVAL;
  QLayer l;
  l.kind = L_CONV_F32;
  l.src = src;
  l.wf = w;
  l.bn_k = bn_k;
  l.bn_b = bn_b;
  l.cout = cout;
  l.k = k;
  l.stride = stride;
  l.pad = pad;
  l.relu = relu ? 1 : 0;
  l.out_bits = out_bits;
  const int ho = qconv_out_size(s.h, k, stride, pad), wo = qconv_out_size(s.w, k, stride, pad);
  if (ho < 1 || wo < 1) return QCONV_EINVAL;
  // matrix cores when the network asks for them and the kernel fits the layer
  // unpooled or pooled (a fused pooling decides which, see conv_uses_mfma)
  l.f32_mfma = net->f32_algo != QNET_F32_FMAF_CHAIN && (conv_f32_mfma_supports(1, s.c, s.h, s.w, cout, k, stride, pad, 0, 0) ||
                                                  conv_f32_mfma_supports(1, s.c, s.h, s.w, cout, k, stride, pad, 1, 0));
  return add_tensor(net, l, {cout, ho, wo, out_bits});
}

int qnet_set_f32_algo(qnet* net, int algo) {
  if (!net || (algo != QNET_F32_FMAF_CHAIN && algo != QNET_F32_MFMA && algo != QNET_F32_BF16X6) || !net->L.empty())
    return QCONV_EINVAL;
  net->f32_algo = algo;
  return QCONV_OK;
}

int qnet_add_maxpool_f32(qnet* net, int src, int k, int stride, int pad) {
  if (!valid_src(net, src) || k < 1 || stride < 1 || pad < 0 || pad >= k) return QCONV_EINVAL;
  const QTensor& s = net->t[src];
  if (s.bits != 0) return QCONV_EINVAL;
  QLayer l;
  l.kind = L_MAXPOOL_F32;
  l.src = src;
  l.k = k;
  l.stride = stride;
  l.pad = pad;
  const int ho = qconv_out_size(s.h, k, stride, pad), wo = qconv_out_size(s.w, k, stride, pad);
  if (ho < 1 || wo < 1) return QCONV_EINVAL;
  // 3x3 / 2 pooling (pad 1) of a matrix-core fp32 conv's own output runs in
  // that conv's epilogue
  if (src > 0 && k == 3 && stride == 2 && pad == 1) {
    QLayer& prod = net->L[src - 1];
    const QTensor& ps = net->t[prod.src];
    if (prod.kind == L_CONV_F32 && prod.f32_mfma && prod.out_bits == 0 && prod.pool_dst < 0 && prod.pack_dst < 0 &&
        conv_f32_mfma_supports(1, ps.c, ps.h, ps.w, prod.cout, prod.k, prod.stride, prod.pad, 1, 0)) {
      prod.pool_dst = (int)net->t.size();
      l.fused = 1;
    }
  }
  return add_tensor(net, l, {s.c, ho, wo, 0});
}

int qnet_add_quantize(qnet* net, int src, int bits) {
  if (!valid_src(net, src) || !bits_ok(bits)) return QCONV_EINVAL;
  const QTensor s = net->t[src];
  if (s.bits != 0) return QCONV_EINVAL;
  QLayer l;
  l.kind = L_QUANTIZE;
  l.src = src;
  l.out_bits = bits;
  // Q(x) of a quantized conv's fp32 output comes out of that conv's own
  // epilogue (Algorithm 1: a_l^q = h(a_l) right after the layer), as the
  // packed Q(HardTanh(z)); with the default thresholds (all below 1)
  // HardTanh changes no level, so the bits are those of Q(x)
  QLayer& prod = net->L[src - 1 >= 0 ? src - 1 : 0];
  const int id = (int)net->t.size();
  if (src > 0 && prod.kind == L_QCONV && prod.out_bits == 0 && prod.pack_dst < 0) {
    prod.pack_dst = id;
    l.fused = 1;
  } else if (src > 0 && prod.kind == L_MAXPOOL_F32 && prod.fused) {
    // a pooling fused into a matrix-core fp32 conv: that conv packs its pooled output
    QLayer& conv = net->L[prod.src - 1];
    if (conv.pack_dst < 0) {
      conv.pack_dst = id;
      l.fused = 1;
    }
  } else if (src > 0 && prod.kind == L_CONV_F32 && prod.f32_mfma && prod.out_bits == 0 && prod.pool_dst < 0 &&
             prod.pack_dst < 0) {
    const QTensor& ps = net->t[prod.src];
    if (conv_f32_mfma_supports(1, ps.c, ps.h, ps.w, prod.cout, prod.k, prod.stride, prod.pad, 0, 0)) {
      prod.pack_dst = id;
      l.fused = 1;
    }
  }
  return add_tensor(net, l, {s.c, s.h, s.w, bits});
}

int qnet_add_qconv(qnet* net, int src, const uint32_t* w_packed, int cout, int k, int stride,
                   int pad, int w_bits, int pool2, const float* bn_k, const float* bn_b,
                   int residual_src, int out_bits) {
  if (!valid_src(net, src) || !w_packed || !bn_k || !bn_b || cout < 1 || k < 1 || stride < 1 ||
      pad < 0 || !(bits_ok(w_bits) || w_bits == 16) || out_bits < 0 || out_bits > 3)
    return QCONV_EINVAL;
  const QTensor s = net->t[src];
  if (s.bits == 0) return QCONV_EINVAL;
  int ho = qconv_out_size(s.h, k, stride, pad), wo = qconv_out_size(s.w, k, stride, pad);
  if (ho < 1 || wo < 1) return QCONV_EINVAL;
  if (pool2) {
    if (ho < 2 || wo < 2) return QCONV_EINVAL;
    ho /= 2;
    wo /= 2;
  }
  // 16-bit weights accumulate in fp32: no int32 bound
  if (w_bits != 16 && (int64_t)s.c * k * k * max_code(s.bits) * max_code(w_bits) >= (int64_t)1 << 31)
    return QCONV_EOVERFLOW;
  if (residual_src > 0) {
    if (!valid_src(net, residual_src) || out_bits != 0) return QCONV_EINVAL;
    const QTensor& r = net->t[residual_src];
    if (r.bits != 0 || r.c != cout || r.h != ho || r.w != wo) return QCONV_EINVAL;
  }
  QLayer l;
  l.kind = L_QCONV;
  l.src = src;
  l.src2 = residual_src > 0 ? residual_src : -1;
  l.wq = w_packed;
  l.bn_k = bn_k;
  l.bn_b = bn_b;
  l.cout = cout;
  l.k = k;
  l.stride = stride;
  l.pad = pad;
  l.w_bits = w_bits;
  l.pool2 = pool2 ? 1 : 0;
  l.out_bits = out_bits;
  return add_tensor(net, l, {cout, ho, wo, out_bits});
}

int qnet_add_avgpool(qnet* net, int src) {
  if (!valid_src(net, src)) return QCONV_EINVAL;
  const QTensor s = net->t[src];
  if (s.bits != 0) return QCONV_EINVAL;
  QLayer l;
  l.kind = L_AVGPOOL;
  l.src = src;
  return add_tensor(net, l, {s.c, 1, 1, 0});
}

int qnet_add_fc_f32(qnet* net, int src, const float* w, const float* bias, int out_features) {
  if (!valid_src(net, src) || !w || out_features < 1) return QCONV_EINVAL;
  const QTensor s = net->t[src];
  if (s.bits != 0 && !(s.bits == 1 && s.h == 1 && s.w == 1)) return QCONV_EUNSUPPORTED;
  QLayer l;
  l.kind = L_FC_F32;
  l.src = src;
  l.wf = w;
  l.bias = bias;
  l.cout = out_features;
  return add_tensor(net, l, {out_features, 1, 1, 0});
}

size_t qnet_workspace_bytes(const qnet* net, int batch) {
  if (!net || batch < 0) return 0;
  return plan(net, batch, nullptr, nullptr);
}

int qnet_tensor_info(const qnet* net, int id, int batch, int* c, int* h, int* w, int* bits,
                     size_t* ws_offset) {
  if (!valid_src(net, id) || batch < 0) return QCONV_EINVAL;
  const QTensor& t = net->t[id];
  if (c) *c = t.c;
  if (h) *h = t.h;
  if (w) *w = t.w;
  if (bits) *bits = t.bits;
  if (ws_offset) {
    std::vector<size_t> toff;
    plan(net, batch, &toff, nullptr);
    *ws_offset = toff[id];
  }
  return QCONV_OK;
}

int qnet_forward_range(const qnet* net, const float* x, int batch, float* logits, void* workspace,
                       size_t workspace_bytes, int first, int count, void* stream) {
  if (!net || batch < 0 || net->L.empty()) return QCONV_EINVAL;
  if (first < 0 || count < 0 || first + count > (int)net->L.size()) return QCONV_EINVAL;
  if (batch == 0 || count == 0) return QCONV_OK;
  if (!x || !logits) return QCONV_EINVAL;
  const QTensor& last = net->t.back();
  if (last.bits != 0) return QCONV_EUNSUPPORTED;
  std::vector<size_t> toff, woff;
  const size_t need = plan(net, batch, &toff, &woff);
  if (workspace_bytes < need) return QCONV_EWORKSPACE;
  if (need > 0 && !workspace) return QCONV_EINVAL;
  return run_layers(net, x, batch, logits, static_cast<char*>(workspace), toff.data(), woff.data(), first, count,
                    (hipStream_t)stream);
}

}  // extern "C"

namespace {

// The layer loop of qnet_forward over layers [first, first + count), with
// tensor `id` at ws + toff[id] and the re-laid-out weights of fp32 conv
// layer i at ws + woff[i] (inputs already validated).
int run_layers(const qnet* net, const float* x, int batch, float* logits, char* ws, const size_t* toff,
               const size_t* woff, int first, int count, hipStream_t s) {
  const int last_id = (int)net->t.size() - 1;
  auto ptr = [&](int id) -> void* {
    if (id == 0) return const_cast<float*>(x);
    if (id == last_id) return logits;
    return ws + toff[id];
  };
  Thr dflt[4];
  for (int b = 1; b <= 3; ++b) act_thresholds(b, nullptr, &dflt[b]);
  for (size_t i = (size_t)first; i < (size_t)(first + count); ++i) {
    const QLayer& l = net->L[i];
    const int dst = (int)i + 1;
    const QTensor& si = net->t[l.src];
    const QTensor& so = net->t[dst];
    int rc = QCONV_OK;
    switch (l.kind) {
      case L_CONV_F32: {
        if (conv_uses_mfma(net, l)) {
          const bool pool = l.pool_dst > 0;
          const int ob = l.out_bits ? l.out_bits : (l.pack_dst > 0 ? net->t[l.pack_dst].bits : 0);
          float* outf = pool ? static_cast<float*>(ptr(l.pool_dst)) : (l.out_bits ? nullptr : static_cast<float*>(ptr(dst)));
          uint32_t* outp = l.out_bits ? static_cast<uint32_t*>(ptr(dst))
                                      : (l.pack_dst > 0 ? static_cast<uint32_t*>(ptr(l.pack_dst)) : nullptr);
          rc = launch_conv_f32_mfma(static_cast<const float*>(ptr(l.src)), l.wf, batch, si.c, si.h, si.w, l.cout, l.k,
                                    l.stride, l.pad, l.bn_k, l.bn_b, l.relu, pool ? 1 : 0, outf, outp, ob,
                                    dflt[ob ? ob : 1], conv_mfma_alg(net, l), s);
          break;
        }
        float* wt = reinterpret_cast<float*>(ws + woff[i]);
        rc = launch_transpose_conv_weight(l.wf, l.cout, si.c, l.k, wt, s);
        if (rc) return rc;
        rc = launch_conv_f32(static_cast<const float*>(ptr(l.src)), wt, batch, si.c, si.h, si.w,
                             l.cout, l.k, l.stride, l.pad, l.bn_k, l.bn_b, l.relu, l.out_bits,
                             dflt[l.out_bits ? l.out_bits : 1],
                             l.out_bits ? nullptr : static_cast<float*>(ptr(dst)),
                             l.out_bits ? static_cast<uint32_t*>(ptr(dst)) : nullptr, s);
        break;
      }
      case L_MAXPOOL_F32:
        if (l.fused) break;  // in the epilogue of the fp32 conv that made its source
        rc = launch_maxpool_f32(static_cast<const float*>(ptr(l.src)), batch, si.c, si.h, si.w,
                                l.k, l.stride, l.pad, static_cast<float*>(ptr(dst)), s);
        break;
      case L_QUANTIZE:
        if (l.fused) break;  // written by the epilogue of the conv that made its source
        rc = launch_pack_act(static_cast<const float*>(ptr(l.src)), batch, si.c, si.h, si.w,
                             l.out_bits, dflt[l.out_bits], static_cast<uint32_t*>(ptr(dst)), s);
        break;
      case L_QCONV: {
        qconv_desc d = {batch, si.c, si.h, si.w, l.cout, l.k, l.k, l.stride, l.pad,
                        si.bits, l.w_bits, QCONV_ALGO_AUTO};
        qconv_epilogue e;
        memset(&e, 0, sizeof(e));
        e.mode = l.out_bits ? QCONV_EPI_BN_PACK : QCONV_EPI_BN_F32;
        e.flags = (l.pool2 ? QCONV_EPI_POOL2 : 0) | (l.src2 > 0 ? QCONV_EPI_RESIDUAL : 0);
        e.bn_k = l.bn_k;
        e.bn_b = l.bn_b;
        e.residual = l.src2 > 0 ? static_cast<const float*>(ptr(l.src2)) : nullptr;
        e.out_bits = l.out_bits;
        uint32_t* packed = l.out_bits ? static_cast<uint32_t*>(ptr(dst)) : nullptr;
        if (l.pack_dst > 0) {
          packed = static_cast<uint32_t*>(ptr(l.pack_dst));
          e.out_bits = net->t[l.pack_dst].bits;
        }
        rc = qconv_forward(&d, static_cast<const uint32_t*>(ptr(l.src)), l.wq, &e,
                           l.out_bits ? nullptr : ptr(dst), packed, s);
        break;
      }
      case L_AVGPOOL:
        rc = launch_avgpool_f32(static_cast<const float*>(ptr(l.src)), batch, si.c, si.h, si.w,
                                static_cast<float*>(ptr(dst)), s);
        break;
      case L_FC_F32:
        rc = launch_fc_f32(ptr(l.src), si.bits, batch, si.c * si.h * si.w, l.wf, l.bias, l.cout,
                           static_cast<float*>(ptr(dst)), s);
        break;
      default:
        return QCONV_EINVAL;
    }
    (void)so;
    if (rc) return rc;
  }
  return QCONV_OK;
}

}  // namespace

extern "C" {

int qnet_forward(const qnet* net, const float* x, int batch, float* logits, void* workspace,
                 size_t workspace_bytes, void* stream) {
  return qnet_forward_range(net, x, batch, logits, workspace, workspace_bytes, 0, net ? (int)net->L.size() : 0,
                            stream);
}

int qnet_num_layers(const qnet* net) { return net ? (int)net->L.size() : QCONV_EINVAL; }

int qnet_layer_kernel(const qnet* net, int layer, int batch, char* buf, int len) {
  if (!net || layer < 0 || layer >= (int)net->L.size() || batch < 1) return QCONV_EINVAL;
  const QLayer& l = net->L[layer];
  const QTensor& si = net->t[l.src];
  char name[128];
  name[0] = 0;
  if (l.fused) {
    // written by an earlier layer's epilogue: no launch of its own
  } else if (l.kind == L_CONV_F32) {
    if (conv_uses_mfma(net, l)) {
      const int ob = l.out_bits ? l.out_bits : (l.pack_dst > 0 ? net->t[l.pack_dst].bits : 0);
      snprintf(name, sizeof(name), "conv_f32_%s_kernel<%d, %d, %d, %d>", conv_mfma_alg(net, l) ? "bf16x6" : "mfma", l.k,
               l.stride, l.pool_dst > 0 ? 1 : 0, ob);
    } else {
      snprintf(name, sizeof(name), "conv_f32_kernel<%d, %d>", l.out_bits, (l.out_bits == 0 && l.cout > 32) ? 64 : 32);
    }
  } else if (l.kind == L_QCONV) {
    qconv_desc d = {batch, si.c, si.h, si.w, l.cout, l.k, l.k, l.stride, l.pad, si.bits, l.w_bits, QCONV_ALGO_AUTO};
    qconv_epilogue e;
    memset(&e, 0, sizeof(e));
    e.mode = l.out_bits ? QCONV_EPI_BN_PACK : QCONV_EPI_BN_F32;
    e.flags = (l.pool2 ? QCONV_EPI_POOL2 : 0) | (l.src2 > 0 ? QCONV_EPI_RESIDUAL : 0);
    e.out_bits = l.out_bits ? l.out_bits : (l.pack_dst > 0 ? net->t[l.pack_dst].bits : 0);
    const int rc = qconv_kernel_name(&d, &e, (l.out_bits || l.pack_dst > 0) ? 1 : 0, name, (int)sizeof(name));
    if (rc < 0) return rc;
  } else if (l.kind == L_MAXPOOL_F32) {
    snprintf(name, sizeof(name), "%s", (l.k == 3 && l.stride == 2 && l.pad == 1 && si.w % 2 == 0)
                                           ? "maxpool3s2_f32_kernel" : "maxpool_f32_kernel");
  } else if (l.kind == L_QUANTIZE) {
    snprintf(name, sizeof(name), "pack_act_lds_kernel<%d>", l.out_bits);
  } else if (l.kind == L_AVGPOOL) {
    snprintf(name, sizeof(name), "%s", si.h * si.w <= 60 ? "avgpool_lds_kernel" : "avgpool_f32_kernel");
  } else {
    snprintf(name, sizeof(name), "fc_f32_kernel<%d>", si.bits);
  }
  if (buf && len > 0) snprintf(buf, (size_t)len, "%s", name);
  return (int)strlen(name);
}

int qnet_layer_fused_into(const qnet* net, int layer) {
  if (!net || layer < 0 || layer >= (int)net->L.size()) return QCONV_EINVAL;
  const int id = layer + 1;
  for (int i = 0; i < layer; ++i) {
    const QLayer& l = net->L[i];
    if (l.pack_dst == id || l.pool_dst == id) return i;
  }
  return layer;
}

}  // extern "C"

// ---------------------------------------------------------------------------
// Networks without a caller workspace: every intermediate tensor lives in one
// fixed device array of the library, reused as soon as the layers that read
// a tensor have run.
// ---------------------------------------------------------------------------

namespace {

constexpr size_t kScratchBytes = (size_t)QNET_NOALLOC_SCRATCH_MIB << 20;
constexpr int kScratchTensors = 1024;  // tensors (plus fp32 conv weight regions) a plan can place

// The array itself.  In host code its name is only a stand-in for the
// symbol: kernels get the device address hipGetSymbolAddress returns.
__device__ __align__(256) uint8_t scratch[kScratchBytes];

// Device address of `scratch` on each device, looked up once per device.
std::atomic<uint8_t*> g_scratch_ptr[MAX_DEVICES_API];
std::mutex g_scratch_mu;

int scratch_ptr(uint8_t** out) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= MAX_DEVICES_API) return QCONV_EHIP;
  uint8_t* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      void* sym = nullptr;
      if (hipGetSymbolAddress(&sym, HIP_SYMBOL(scratch)) != hipSuccess || !sym) return QCONV_EHIP;
      p = static_cast<uint8_t*>(sym);
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return QCONV_OK;
}

// Liveness plan: tensor id (made by layer id - 1) stays placed until the last
// layer that reads it has run; the re-laid-out weights of fp32 conv layer i
// live during layer i only.  Each region takes the lowest 256-byte aligned
// offset that overlaps no region still live (first fit over the ends of
// the live regions).  Writes toff[id] / woff[i] (fixed arrays, no heap) and
// returns the bytes used, or 0 with *rc set when the network has more
// regions than the arrays hold.
size_t liveness_plan(const qnet* net, int batch, size_t* toff, size_t* woff, int* rc) {
  const int nt = (int)net->t.size(), nl = (int)net->L.size();
  *rc = QCONV_OK;
  if (nt + nl > kScratchTensors) {
    *rc = QCONV_EUNSUPPORTED;
    return 0;
  }
  int last_use[kScratchTensors];
  for (int id = 0; id < nt; ++id) last_use[id] = id - 1;
  for (int i = 0; i < nl; ++i) {
    const QLayer& l = net->L[i];
    if (last_use[l.src] < i) last_use[l.src] = i;
    if (l.src2 > 0 && last_use[l.src2] < i) last_use[l.src2] = i;
  }
  struct Region {
    size_t off, end;
    int until;  // last layer that uses it
  };
  Region live[kScratchTensors];
  int nlive = 0;
  size_t top = 0;
  auto place = [&](size_t bytes, int layer, int until) -> size_t {
    // drop regions whose last use came before this layer
    int k = 0;
    for (int j = 0; j < nlive; ++j)
      if (live[j].until >= layer) live[k++] = live[j];
    nlive = k;
    size_t best = (size_t)-1;
    for (int c = -1; c < nlive; ++c) {
      const size_t cand = c < 0 ? 0 : align256(live[c].end);
      bool ok = true;
      for (int j = 0; j < nlive && ok; ++j) ok = cand + bytes <= live[j].off || cand >= live[j].end;
      if (ok && cand < best) best = cand;
    }
    live[nlive++] = {best, best + bytes, until};
    if (align256(best + bytes) > top) top = align256(best + bytes);
    return best;
  };
  for (int i = 0; i < nl; ++i) {
    const QLayer& l = net->L[i];
    woff[i] = (size_t)-1;
    if (l.kind == L_CONV_F32 && !conv_uses_mfma(net, l)) {
      const int cin = net->t[l.src].c;
      woff[i] = place((size_t)cin * l.k * l.k * ceil_div(l.cout, 64) * 64 * sizeof(float), i, i);
    }
    const int id = i + 1;
    if ((l.kind == L_QUANTIZE || l.kind == L_MAXPOOL_F32) && l.fused) continue;  // placed with the conv that writes it
    toff[id] = (size_t)-1;
    // a conv whose pooling is fused never writes its own output
    if (id != nt - 1 && !(l.kind == L_CONV_F32 && l.pool_dst > 0))
      toff[id] = place(tensor_bytes(net->t[id], batch), i, last_use[id]);
    if (l.pool_dst > 0) toff[l.pool_dst] = place(tensor_bytes(net->t[l.pool_dst], batch), i, last_use[l.pool_dst]);
    if (l.pack_dst > 0) toff[l.pack_dst] = place(tensor_bytes(net->t[l.pack_dst], batch), i, last_use[l.pack_dst]);
  }
  toff[0] = (size_t)-1;
  return top;
}

}  // namespace

extern "C" {

size_t qnet_noalloc_bytes(const qnet* net, int batch) {
  if (!net || batch < 0 || net->L.empty()) return 0;
  size_t toff[kScratchTensors], woff[kScratchTensors];
  int rc = 0;
  return liveness_plan(net, batch, toff, woff, &rc);
}

size_t qnet_noalloc_limit(void) { return kScratchBytes; }

int qnet_forward_noalloc(const qnet* net, const float* x, int batch, float* logits, void* stream) {
  if (!net || batch < 0 || net->L.empty()) return QCONV_EINVAL;
  if (batch == 0) return QCONV_OK;
  if (!x || !logits) return QCONV_EINVAL;
  if (net->t.back().bits != 0) return QCONV_EUNSUPPORTED;
  size_t toff[kScratchTensors], woff[kScratchTensors];
  int rc = 0;
  const size_t need = liveness_plan(net, batch, toff, woff, &rc);
  if (rc) return rc;
  if (need > kScratchBytes) return QCONV_ESCRATCH;
  uint8_t* base = nullptr;
  rc = scratch_ptr(&base);
  if (rc) return rc;
  return run_layers(net, x, batch, logits, reinterpret_cast<char*>(base), toff, woff, 0, (int)net->L.size(),
                    (hipStream_t)stream);
}

}  // extern "C"
