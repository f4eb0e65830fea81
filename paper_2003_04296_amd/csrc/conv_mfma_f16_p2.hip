// conv_mfma_f16_p2.hip -- the matrix-core convolution kernels for operand
// format OP_F16 with 2 activation word(s) per 32 channels (conv_mfma.h).
#include "conv_mfma.h"

namespace qc {
namespace mfma {
QC_MFMA_DEFINE(f16_p2, OP_F16, 2)
}  // namespace mfma
}  // namespace qc
