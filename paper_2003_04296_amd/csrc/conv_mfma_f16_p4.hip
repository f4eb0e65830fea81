// conv_mfma_f16_p4.hip -- the matrix-core convolution kernels for operand
// format OP_F16 with 4 activation word(s) per 32 channels (conv_mfma.h).
#include "conv_mfma.h"

namespace qc {
namespace mfma {
QC_MFMA_DEFINE(f16_p4, OP_F16, 4)
}  // namespace mfma
}  // namespace qc
