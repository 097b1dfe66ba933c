// The matrix-core multi-channel kernels for K = 1, 2, 3 (one translation unit
// per few filter sizes, so that they compile in parallel).
#include "multi_kernels.h"

namespace dconv {

DCONV_MFMA_LAUNCHER(1) { return launch_mfma_k<1>(p, I, F, O, a, st); }
DCONV_MFMA_LAUNCHER(2) { return launch_mfma_k<2>(p, I, F, O, a, st); }
DCONV_MFMA_LAUNCHER(3) { return launch_mfma_k<3>(p, I, F, O, a, st); }

}  // namespace dconv
