// conv_mfma_i8_p1.hip -- the matrix-core convolution kernels for operand
// format OP_I8 with 1 activation word(s) per 32 channels (conv_mfma.h).
#include "conv_mfma.h"

namespace qc {
namespace mfma {
QC_MFMA_DEFINE(i8_p1, OP_I8, 1)
}  // namespace mfma
}  // namespace qc
