// The matrix-core multi-channel kernels for K = 7, 8, 9 (one translation unit
// per few filter sizes, so that they compile in parallel).
#include "multi_kernels.h"

namespace dconv {

DCONV_MFMA_LAUNCHER(7) { return launch_mfma_k<7>(p, I, F, O, a, st); }
DCONV_MFMA_LAUNCHER(8) { return launch_mfma_k<8>(p, I, F, O, a, st); }
DCONV_MFMA_LAUNCHER(9) { return launch_mfma_k<9>(p, I, F, O, a, st); }

}  // namespace dconv
