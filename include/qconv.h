/*
 * qconv.h -- C ABI of the MI355X (gfx950) quantized-convolution library.
 *
 * The library computes the inference forward pass of MINW-Net ("M-bit
 * Inputs and N-bit Weights Network"; Chen et al., "Propagating
 * Asymptotic-Estimated Gradients for Low Bitwidth Quantized Neural
 * Networks"): weights and activations quantized by the inference quantizers
 * of Sec. III-C (Eq. 20 applying Eq. 4 sign, Eq. 21 ternary, Eq. 22
 * power-of-two), the layer product of Algorithm 1's inference branch
 * evaluated as XNOR/AND-popcount over channel-packed bitplanes with a
 * shift-weighted sum over plane pairs (Sec. III-C: bitwise and shift
 * operations replace multiplies), and the layer constructs of Sec. III-E
 * ({QConv-pooling-BN-HardTanh}, {QConv-BN-HardTanh}) fused into the
 * convolution's epilogue.
 *
 * Conventions shared by every entry point:
 *  - Pointers named x, w, act, out, scale, bn_*, residual, logits, workspace
 *    are DEVICE pointers owned by the caller; "host" marks host pointers.
 *    The library never allocates device memory, never synchronises, keeps no
 *    mutable global state, and enqueues all work on `stream` (a hipStream_t
 *    passed as void*; NULL = the null stream).
 *  - Every call validates its arguments synchronously and returns a negative
 *    qconv_status WITHOUT launching anything when they are invalid.  A launch
 *    failure returns QCONV_EHIP.  Faults inside kernels surface at the
 *    caller's next synchronisation.
 *  - Overlapping input and output buffers are not supported.
 *
 * Integer level codes (what a packed value means):
 *   1 bit : {-1, +1}                         (Eq. 4)
 *   2 bits: {-1, 0, +1}                      (Eq. 21)
 *   3 bits: {0, +-1, +-2, +-4} = 4 x {0, +-1/4, +-1/2, +-1}   (Eq. 22)
 *   Integer accumulators are in code units: the real product is
 *   acc * 2^-(2[a_bits==3] + 2[w_bits==3]).
 *
 * Quantizer thresholds (the paper leaves them open; these are the defaults):
 *   activations: 2 bits |x| <= 0.5 -> 0;  3 bits |x| <= 1/8 -> 0,
 *                <= 3/8 -> 1/4, <= 3/4 -> 1/2, else 1 (nearest level);
 *   weights:     the same rules with thresholds multiplied by s_c = mean|W_c|
 *                (2 bits: 0.7 s_c; 3 bits: {1/8, 3/8, 3/4} s_c), each
 *                threshold computed in double and rounded once to float.
 *   sign(x) = +1 only for x > 0 (0, -0 and NaN give -1; Sec. II-A).
 *
 * Packed bitplane layouts (uint32 words, bit (c % 32) of word (c / 32) holds
 * channel c; bits past the last channel are 0 in every plane):
 *   planes P = 1 / 2 / 4 for 1 / 2 / 3 bits;
 *   plane 0: sign, 1 <=> level > 0;
 *   2 bits : plane 1 = level != 0;
 *   3 bits : plane 1 = |level| == 1, plane 2 = |level| == 1/2,
 *            plane 3 = |level| == 1/4.
 *   activations: [n][h][w][cw][P],              cw = ceil(c / 32)
 *   weights    : [kh][kw][cw][cout_pad][P],     cout_pad = ceil(cout / 128) * 128
 *                (rows of padding channels are 0), followed in the same
 *                buffer by three matrix-core operand copies of the same
 *                levels, expanded from those bitplanes (channels past cin
 *                and padding output channels are 0): int8 codes [kh][kw][cw][cout_pad][32 B], E2M1 (fp4)
 *                codes [kh][kw][ceil(cw/2)][cout_pad][32 B] (64 channels:
 *                16 B per 32-channel word, whose u32 q holds channels q,
 *                q + 4, ..., q + 28 in nibbles 0..7) and IEEE fp16 codes
 *                [kh][kw][2 cw][cout_pad][16 x 2 B] (16 channels per
 *                record); the codes 0, +-1, +-2, +-4 are exact in all three.
 *   An all-zero activation word reads as level -1 for 1 bit and 0 for 2/3
 *   bits, i.e. Q(0): the value padding taps take in the product.
 *
 * 16-bit inputs (Table I / Table IV: 16-bit floating inputs with 1..3-bit
 * weights, the "XNOR ADDER" / "SHIFT ADDER" rows): bits = 16 stands for an
 * unquantized IEEE fp16 activation tensor [n][h][w][cw * 32] (channel-last,
 * channels past c hold +0; viewed as uint32 words, channel 2i in the low
 * half of word i).  The product sums fp16 activation x weight code exactly
 * and accumulates in fp32 (padding taps hold 0); its real value is
 * acc * 2^-(2[w_bits==3]).  Only the fp32 accumulation rounds, so results
 * match the exact product within K * 2^-24 * sum|x * code| (in code units),
 * and exactly when every partial sum is an integer below 2^24.
 *
 * 16-bit weights (Table I rows with 1..3-bit inputs and 16-bit weights):
 * w_bits = 16 packs fp32 OIHW weights into IEEE fp16 (round to nearest even)
 * laid out as the fp16 operand copy above, [kh][kw][2 cw][cout_pad][16 x 2 B],
 * and that is the whole packed buffer; out_scale still receives mean|W_c|.
 * The product of the inputs' level codes (padding taps at Q(0)) with the
 * fp16 weights is summed as for 16-bit inputs; its real value is
 * acc * 2^-(2[a_bits==3]).
 */
#ifndef QCONV_H
#define QCONV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  QCONV_OK = 0,
  QCONV_EINVAL = -1,       /* null pointer, bad size, bad enum value          */
  QCONV_EUNSUPPORTED = -2, /* valid but not implemented (shape, bits, algo)   */
  QCONV_EWORKSPACE = -3,   /* workspace too small                             */
  QCONV_EOVERFLOW = -4,    /* K * max|a| * max|w| >= 2^31 (int32 accumulator) */
  QCONV_EHIP = -5,         /* a HIP launch or runtime call failed             */
  QCONV_ESCRATCH = -6      /* qnet_forward_noalloc: the network needs more
                              than the fixed scratch array holds             */
} qconv_status;

/* Human-readable text for a status code (never NULL). */
const char* qconv_error_string(int status);

/* Library ABI version (major * 100 + minor). */
int qconv_version(void);

/* ------------------------------------------------------------------------ */
/* Inference-operation rule (Sec. IV-C; Tables I and II, columns 3-4)        */
/* ------------------------------------------------------------------------ */
typedef enum {
  QCONV_OP_XNOR = 1,        /* min(M, N) <= 2                               */
  QCONV_OP_SHIFT = 2,       /* min(M, N) == 3                               */
  QCONV_OP_XNOR_ADDER = 3,  /* one side 16-bit float, other side <= 2 bits  */
  QCONV_OP_SHIFT_ADDER = 4, /* one side 16-bit float, other side 3 bits     */
  QCONV_OP_MAC = 5          /* both 32-bit float                            */
} qconv_op;

/* For M-bit inputs and N-bit weights (M, N in {1, 2, 3, 16, 32}) report the
 * inference operation (by the smaller width) and the computational precision
 * in bits (by the larger width: 1 -> "1-bit fixed", 2 -> "2-bit fixed",
 * 16/32 -> floating).  *op and *precision_bits are host pointers. */
int qconv_inference_op(int m_bits, int n_bits, int* op, int* precision_bits);

/* ------------------------------------------------------------------------ */
/* Quantize + pack (Sec. III-C, Eq. 20)                                      */
/* ------------------------------------------------------------------------ */

/* Bytes of the packed activation tensor [n][h][w][ceil(c/32)][P]
 * (bits = 16: the fp16 tensor [n][h][w][ceil(c/32) * 32]). */
size_t qconv_packed_act_bytes(int n, int c, int h, int w, int bits);

/* Quantize fp32 NCHW activations x[n][c][h][w] with h(.) of `bits` and pack
 * them into out_packed.  thresholds (host, may be NULL for the defaults):
 * 2 bits {delta}; 3 bits {t1, t2, t3} increasing; ignored for 1 bit.
 * bits = 16: convert to the fp16 channel-last layout above instead (round to
 * nearest, ties to even; beyond the fp16 range -> +-inf; NaN stays NaN;
 * thresholds ignored). */
int qconv_pack_act(const float* x, int n, int c, int h, int w, int bits,
                   const float* thresholds, uint32_t* out_packed, void* stream);

/* Bytes of the packed weight buffer: the bitplanes [kh][kw][ceil(cin/32)][cout_pad][P]
 * plus the int8, fp4 and fp16 operand copies described above (bits = 16: the
 * fp16 weights alone). */
size_t qconv_packed_weight_bytes(int cout, int cin, int kh, int kw, int bits);

/* Quantize fp32 OIHW weights w[cout][cin][kh][kw] (Eq. 20) and pack them.
 * out_scale[cout] (device) receives s_c = mean |W_c| (double sum over
 * (cin, kh, kw) in storage order, rounded once to float).  base_thresholds
 * (host, NULL = defaults) are multiplied by s_c per channel.  bits = 16:
 * round to fp16 instead (16-bit weights, see above; thresholds ignored). */
int qconv_pack_weight(const float* w, int cout, int cin, int kh, int kw, int bits,
                      const float* base_thresholds, uint32_t* out_packed, float* out_scale,
                      void* stream);

/* Host helper: fold batch norm (all host arrays of length c) in double,
 * k = gamma / sqrt(var + eps), b = beta - k * mean, each rounded once. */
int qconv_fold_bn(const float* gamma, const float* beta, const float* mean, const float* var,
                  double eps, int c, float* k_out, float* b_out);

/* ------------------------------------------------------------------------ */
/* Quantized convolution with fused epilogue (Algorithm 1 + Sec. III-E)      */
/* ------------------------------------------------------------------------ */
typedef enum {
  QCONV_ALGO_AUTO = 0,     /* library choice: fp4 matrix cores where supported
                              (int8 ones where fp4 would not be exact, see
                              QCONV_ALGO_MFMA_FP4), the bitplane kernel for
                              K = cin*kh*kw <= 256 where its LDS-tiled XNOR
                              form applies (1-2 bit operands, 1x1 or 3x3,
                              stride <= 2, unpacked unpooled outputs)       */
  QCONV_ALGO_BITPLANE = 1, /* VALU XNOR/AND + popcount over bitplanes         */
  QCONV_ALGO_MFMA_I8 = 2,  /* int8 matrix cores on the expanded level codes   */
  QCONV_ALGO_MFMA_FP4 = 3, /* fp4 (E2M1) matrix cores on the same codes; they
                              accumulate in fp32, exact only while
                              K * max|a| * max|w| < 2^24: past that this
                              algorithm returns QCONV_EUNSUPPORTED             */
  QCONV_ALGO_MFMA_F16 = 4  /* fp16 matrix cores: the only one with a 16-bit side */
} qconv_algo;

typedef struct {
  int n, cin, h, w;     /* input activations (packed with a_bits)         */
  int cout, kh, kw;     /* weights (packed with w_bits)                   */
  int stride, pad;      /* same stride / padding on both axes             */
  int a_bits, w_bits;   /* 1..3 each, or one of them 16 (fp16 side)       */
  int algo;             /* qconv_algo                                     */
} qconv_desc;

typedef enum {
  QCONV_EPI_INT32 = 0,     /* out: int32 [n][cout][ho][wo] accumulators (code units)    */
  QCONV_EPI_SCALE_F32 = 1, /* out: fp32 s_c * acc_real (one rounding)                   */
  QCONV_EPI_BN_F32 = 2,    /* out: fp32 z = fmaf(k_c, acc_real, b_c) [+ residual]       */
  QCONV_EPI_BN_PACK = 3    /* out_packed only: Q(HardTanh(z)) packed with out_bits     */
} qconv_epi_mode;

enum {
  QCONV_EPI_POOL2 = 1,    /* 2x2/2 max pool of the accumulators before anything else  */
  QCONV_EPI_RESIDUAL = 2  /* BN_F32: add residual[n][cout][ho][wo] after BN (fp32 add) */
};

typedef struct {
  int mode;                   /* qconv_epi_mode                                       */
  int flags;                  /* QCONV_EPI_POOL2 | QCONV_EPI_RESIDUAL                  */
  const float* scale;         /* [cout] s_c                      (SCALE_F32)          */
  const float* bn_k;          /* [cout] folded k_c               (BN_F32, BN_PACK)    */
  const float* bn_b;          /* [cout] folded b_c                                    */
  const float* residual;      /* fp32 NCHW, output shape          (RESIDUAL)          */
  int out_bits;               /* bits of out_packed (BN_PACK; BN_F32 when out_packed)  */
  const float* out_thresholds;/* host, NULL = default activation thresholds           */
} qconv_epilogue;

/* Output spatial size of the convolution (before pooling). */
int qconv_out_size(int in, int k, int stride, int pad);

/* One quantized layer: acc = (act * W) in code units over all taps (padding
 * taps take Q(0)), then the epilogue.  out is int32 or fp32 NCHW (may be
 * NULL in BN_PACK mode); out_packed ([n][ho'][wo'][ceil(cout/32)][P_out],
 * ho'/wo' after pooling) is written in BN_PACK mode and, when non-NULL, in
 * BN_F32 mode (quantizing the fp32 result).  Requires ceil(cout/32)*32
 * channels of room in out_packed's last word, K = cin*kh*kw with
 * K * max|a| * max|w| < 2^31.  The matrix-core algorithms support stride 1
 * or 2 (with or without pooling) and an input tile that fits their LDS
 * staging buffer (at least one input row of 64 output pixels' receptive
 * field); asked for explicitly otherwise they return QCONV_EUNSUPPORTED,
 * and AUTO falls back to the bitplane kernels.  Every algorithm returns the
 * same bits.  a_bits = 16 or w_bits = 16 (not both): act_packed is the
 * fp16 tensor above, resp. w_packed the fp16 weights; the algorithm is
 * QCONV_ALGO_MFMA_F16 (AUTO picks it; any other returns QCONV_EUNSUPPORTED,
 * as does QCONV_ALGO_MFMA_F16 for layers with no 16-bit side), the
 * epilogue runs on the fp32 accumulator (QCONV_EPI_INT32 returns
 * QCONV_EUNSUPPORTED) and the overflow check does not apply.  There is no
 * bitplane fallback for 16-bit inputs: input tiles that do not fit the
 * usual staging buffer are staged in one of up to 76 KB (one block per
 * compute unit), and a layer whose tile exceeds even that (80 bytes per
 * pixel per 32 channels; rows of several hundred pixels) returns
 * QCONV_EUNSUPPORTED. */
int qconv_forward(const qconv_desc* d, const uint32_t* act_packed, const uint32_t* w_packed,
                  const qconv_epilogue* epi, void* out, uint32_t* out_packed, void* stream);

/* The concrete algorithm (QCONV_ALGO_BITPLANE / _MFMA_I8 / _MFMA_FP4) that
 * qconv_forward would run for d and epi (d->algo may be AUTO), or a negative
 * status if the call would be rejected.  For QCONV_EPI_BN_F32 the answer is
 * that of a call without a packed copy (out_packed NULL; with one, AUTO may
 * choose differently for K <= 256: qconv_kernel_name takes it as an
 * argument).  Launches nothing. */
int qconv_resolve_algo(const qconv_desc* d, const qconv_epilogue* epi);

/* Name of the GPU kernel instantiation qconv_forward would launch for d and
 * epi on the current device (packed_out != 0: an out_packed buffer would be
 * passed; BN_PACK implies one), written NUL-terminated into buf (truncated
 * to len bytes; buf may be NULL).  The name and template arguments are those
 * a profiler shows, e.g. "conv_mfma_pp_kernel<1, 2, 0>".  Returns the length
 * of the full name, or a negative status if the call would be rejected.
 * Launches nothing; the choice depends on the device's compute-unit count. */
int qconv_kernel_name(const qconv_desc* d, const qconv_epilogue* epi, int packed_out, char* buf, int len);

/* ------------------------------------------------------------------------ */
/* Training with the asymptotic-quantized estimator (AQE): the elementwise   */
/* steps of Algorithm 1's training branch (Sec. III-B, III-D; Eqs.           */
/* activation and weight).  Device pointers, n values each, no allocation,   */
/* enqueued on `stream`; n == 0 launches nothing.                            */
/* ------------------------------------------------------------------------ */

/* Forward: y = fl(fl(alpha * h(x)) + fl(fl(1 - alpha) * x)) elementwise,
 * 0 <= alpha <= 1, where h(x) is the level (+-1, 0, +-1/2, +-1/4) that the
 * packing quantizers give for `bits` (same compares, ties and readings).
 *   group_size == 0: activation thresholds (host `thresholds`, NULL =
 *     defaults); scale must be NULL.
 *   group_size  > 0: weight thresholds: the base set (host `thresholds`,
 *     NULL = defaults) times scale[i / group_size] (device, e.g. the s_c that
 *     qconv_pack_weight writes; one group = one output channel's weights in
 *     OIHW order), rounded as the weight packing rounds them; n must be a
 *     multiple of group_size.
 * alpha = 1 gives h(x) for finite x (0 * inf is NaN), alpha = 0 gives x.
 * x and y may be the same buffer. */
int aqe_forward(const float* x, int64_t n, int bits, float alpha, const float* thresholds, const float* scale,
                int64_t group_size, float* y, void* stream);

/* Backward: gx = fl(2 alpha * gy) where |x| <= 1, else 0 (a NaN x gives 0).
 * alpha = 1/2 gives the straight-through estimator gy 1{|x| <= 1} (Eq. ste,
 * Theorem 1).  gx may alias gy. */
int aqe_backward(const float* x, const float* gy, int64_t n, float alpha, float* gx, void* stream);

/* Weight update of Algorithm 1 with plain SGD, then the clip to [-1, 1]:
 * w = fl(w - fl(lr * g)), then 1 if above 1, -1 if below -1 (a NaN stays).
 * In place. */
int aqe_sgd_clip(float* w, const float* g, int64_t n, float lr, void* stream);

/* ------------------------------------------------------------------------ */
/* Whole networks (Algorithm 1, inference branch, layer by layer)            */
/* ------------------------------------------------------------------------ */

/* A network is a list of layers over numbered tensors.  Tensor 0 is the fp32
 * NCHW network input [batch][in_c][in_h][in_w]; every qnet_add_* call
 * appends one layer producing one new tensor and returns its id (> 0), or a
 * negative qconv_status.  Device pointers handed to qnet_add_* (weights,
 * folded BN parameters) must stay valid while the network is used. */
typedef struct qnet qnet;

qnet* qnet_create(int in_c, int in_h, int in_w);
void qnet_destroy(qnet* net);

/* Arithmetic of the network's fp32 convolutions (call before adding
 * layers; returns QCONV_EINVAL afterwards):
 *   QNET_F32_MFMA (default): the fp32 matrix cores sum each output in their
 *     own order (results within fp32 rounding of the chain below); a 3x3 / 2
 *     max pooling (pad 1) of such a conv's output, and the quantize of
 *     either, run in the conv's epilogue.  Layers the matrix-core kernel
 *     does not fit (its LDS holds the input window, cin * k * k weights of
 *     32 channels and a pooled tile) fall back to the chain.
 *   QNET_F32_FMAF_CHAIN: each output one fmaf chain over (ci, kh, kw) from
 *     +0, a fixed order that makes networks reproducible bit for bit.
 *   QNET_F32_BF16X6: as QNET_F32_MFMA, except that a 7 x 7 / 2 conv with its
 *     3 x 3 / 2 pooling fused and cin <= 3 (the ResNet stem) runs on the bf16
 *     matrix cores: every input and weight is split exactly into three bf16
 *     parts (x = x0 + x1 + x2, each part the leading 8 significant bits of
 *     what is left) and the six partial products xi wj with i + j <= 2 are
 *     summed in fp32 (x0 w0 apart from the five smaller ones).  The three
 *     dropped products are below 2^-20 |x w|, so results stay within fp32
 *     rounding of the exact sum: |err| <= (gamma_K + 2^-19) sum |x w|.
 *     Inputs and weights must be finite: an inf or NaN makes NaN in the
 *     outputs whose windows hold it (and, for an input, in the output one
 *     column to its left, whose operand slot past its 7 taps reads it
 *     against a zero weight). */
enum { QNET_F32_FMAF_CHAIN = 0, QNET_F32_MFMA = 1, QNET_F32_BF16X6 = 2 };
int qnet_set_f32_algo(qnet* net, int algo);

/* fp32 conv (zero padding; the sum over (ci, kh, kw) as qnet_set_f32_algo
 * says), then z = fmaf(k, conv, b), then ReLU if relu != 0; out_bits == 0
 * keeps z as fp32 NCHW, out_bits 1..3 quantizes HardTanh(z) and packs it.
 * w: fp32 [cout][cin][k][k], read directly by the matrix-core kernel. */
int qnet_add_conv_f32(qnet* net, int src, const float* w, int cout, int k, int stride, int pad,
                      const float* bn_k, const float* bn_b, int relu, int out_bits);

/* fp32 k x k / stride max pooling with padding (padding never wins; the
 * window is scanned row by row and only a strictly greater value replaces
 * the running maximum).  3 x 3 / 2 with pad 1 right after a matrix-core fp32
 * conv with an fp32 output runs in that conv's epilogue (the conv's own
 * unpooled tensor is then never written). */
int qnet_add_maxpool_f32(qnet* net, int src, int k, int stride, int pad);

/* Quantize + pack an fp32 tensor with the default activation thresholds.
 * When src is the fp32 output of a qnet_add_qconv layer (out_bits 0, with or
 * without a residual) and no other quantize layer was folded into it yet,
 * that conv's epilogue writes this tensor as well (Algorithm 1: a_l^q =
 * h(a_l) right after the layer) and this layer launches nothing. */
int qnet_add_quantize(qnet* net, int src, int bits);

/* Quantized conv on a packed tensor with a BN epilogue (w_bits 1..3, or 16
 * for fp16 weights packed by qconv_pack_weight with bits = 16):
 * pool2 != 0 -> 2x2 max pool of the accumulators first;
 * out_bits 1..3 -> packed Q(HardTanh(BN)) output; out_bits 0 -> fp32 BN
 * output, plus the fp32 tensor residual_src when residual_src > 0. */
int qnet_add_qconv(qnet* net, int src, const uint32_t* w_packed, int cout, int k, int stride,
                   int pad, int w_bits, int pool2, const float* bn_k, const float* bn_b,
                   int residual_src, int out_bits);

/* Global average pooling of an fp32 tensor: sum over (h, w) from +0 in
 * storage order, one division by h*w. */
int qnet_add_avgpool(qnet* net, int src);

/* fp32 fully connected layer over the flattened (c, h, w) source, which is
 * fp32 or a 1-bit packed tensor read as +-1.0: each output one fmaf chain in
 * input order from +0, then + bias.  w: fp32 [out][in]; bias may be NULL. */
int qnet_add_fc_f32(qnet* net, int src, const float* w, const float* bias, int out_features);

/* Bytes of workspace qnet_forward needs for `batch` images. */
size_t qnet_workspace_bytes(const qnet* net, int batch);

/* Run the layers in order on x (device fp32 [batch][in_c][in_h][in_w]) and
 * write the last tensor (fp32 [batch][features]) to logits. */
int qnet_forward(const qnet* net, const float* x, int batch, float* logits, void* workspace,
                 size_t workspace_bytes, void* stream);

/* Layers [first, first + count) of qnet_forward only (layer i produces
 * tensor i + 1), on a workspace laid out for `batch` images exactly as
 * qnet_forward lays it out: the tensors those layers read must already hold
 * what earlier layers (of this or a previous call) wrote there.  Running
 * every range in order is the same as qnet_forward; used to time or
 * overlap parts of a network.  count == 0 launches nothing. */
int qnet_forward_range(const qnet* net, const float* x, int batch, float* logits, void* workspace,
                       size_t workspace_bytes, int first, int count, void* stream);

/* Number of layers added so far (negative status for a NULL network). */
int qnet_num_layers(const qnet* net);

/* The layer whose launch writes the tensor of layer `layer`: an earlier
 * layer when its epilogue takes over a folded quantize or max pooling (which
 * then launches nothing), else `layer` itself.  Negative status for a NULL
 * network or a layer index out of range. */
int qnet_layer_fused_into(const qnet* net, int layer);

/* Name of the main GPU kernel layer `layer` launches for `batch` images, as
 * a profiler shows it (an empty string for a layer written by an earlier
 * layer's epilogue); returns the name's length or a negative status.
 * Launches nothing. */
int qnet_layer_kernel(const qnet* net, int layer, int batch, char* buf, int len);

/* ------------------------------------------------------------------------ */
/* Networks without a workspace, for callers that cannot allocate device     */
/* memory (code under HIP graph capture, tight serving loops, harnesses that */
/* forbid allocation).                                                       */
/* ------------------------------------------------------------------------ */

/* Size of the library's fixed scratch array, in MiB: one array per device
 * the library runs on, allocated when the library's code is loaded on that
 * device and held until the process ends. */
#define QNET_NOALLOC_SCRATCH_MIB 128

/* qnet_forward without a workspace argument: the intermediate tensors live
 * in the library's scratch array of that device (qnet_noalloc_limit() bytes),
 * placed by a liveness plan (a tensor's bytes are reused once every layer
 * that reads it has run), so a network needs qnet_noalloc_bytes(net, batch)
 * of it, far less than qnet_workspace_bytes.  Returns QCONV_ESCRATCH, with
 * no launch, when that exceeds the array.  Allocates nothing, on the device
 * or the host (the plan is computed in fixed stack arrays; networks of more
 * than about 500 layers return QCONV_EUNSUPPORTED).  The array's device
 * address is looked up once per device, on the first call made with that
 * device current.  Every call on one device shares its array and leaves the
 * last call's tensors in it (no layer reads a region it has not written in
 * the same call, so nothing needs clearing): calls that overlap in time on
 * one device, from several streams or threads, race and give undefined
 * results.  The logits are bit-identical to qnet_forward's. */
int qnet_forward_noalloc(const qnet* net, const float* x, int batch, float* logits, void* stream);

/* Scratch bytes qnet_forward_noalloc needs for `batch` images (0 on bad
 * input), and the array's size. */
size_t qnet_noalloc_bytes(const qnet* net, int batch);
size_t qnet_noalloc_limit(void);

/* Shape of tensor `id` for `batch` images (host out-params; bits 0 = fp32),
 * and its byte offset inside the workspace after qnet_forward (the last
 * tensor lives in logits, offset reported as (size_t)-1). */
int qnet_tensor_info(const qnet* net, int id, int batch, int* c, int* h, int* w, int* bits,
                     size_t* ws_offset);

#ifdef __cplusplus
}
#endif

#endif /* QCONV_H */
