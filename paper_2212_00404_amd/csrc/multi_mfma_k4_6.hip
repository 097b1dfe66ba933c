// The matrix-core multi-channel kernels for K = 4, 5, 6 (one translation unit
// per few filter sizes, so that they compile in parallel).
#include "multi_kernels.h"

namespace dconv {

DCONV_MFMA_LAUNCHER(4) { return launch_mfma_k<4>(p, I, F, O, a, st); }
DCONV_MFMA_LAUNCHER(5) { return launch_mfma_k<5>(p, I, F, O, a, st); }
DCONV_MFMA_LAUNCHER(6) { return launch_mfma_k<6>(p, I, F, O, a, st); }

}  // namespace dconv
