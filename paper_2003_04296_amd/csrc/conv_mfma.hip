// conv_mfma.hip -- int8 matrix-core path for the same layer product.
// Not enabled yet: every configuration reports unsupported, so the library
// dispatches to the bitplane kernels.
#include "qconv_internal.h"

namespace qc {

bool mfma_supports(const ConvArgs&) { return false; }

int launch_conv_mfma(const ConvArgs&, hipStream_t) { return QCONV_EUNSUPPORTED; }

}  // namespace qc
