// conv_mfma_f16_p1.hip -- the matrix-core convolution kernels for operand
// format OP_F16 with 1 activation word(s) per 32 channels (conv_mfma.h).
#include "conv_mfma.h"

namespace qc {
namespace mfma {
QC_MFMA_DEFINE(f16_p1, OP_F16, 1)
}  // namespace mfma
}  // namespace qc
