// The matrix-core multi-channel kernels for K = 10, 11 (one translation unit
// per few filter sizes, so that they compile in parallel).
#include "multi_kernels.h"

namespace dconv {

DCONV_MFMA_LAUNCHER(10) { return launch_mfma_k<10>(p, I, F, O, a, st); }
DCONV_MFMA_LAUNCHER(11) { return launch_mfma_k<11>(p, I, F, O, a, st); }

}  // namespace dconv
