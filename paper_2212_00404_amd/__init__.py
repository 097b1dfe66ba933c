"""libdconv for AMD Instinct MI355X: direct valid-mode stride-1 2-D convolution
in fp32 with hand-written gfx950 HIP kernels behind a C ABI.

``single(I, F)`` computes Eq. 2 and ``multi(I, F)`` Eq. 1 of Chang, Onishi,
Maruyama, "Fast convolution kernels on Pascal GPU with high memory
efficiency" (Section 2.1).  See ``dconv.py`` for the argument conventions and
``include/dconv.h`` for the C interface.
"""
from .dconv import (EXPORTED, GTX_1080TI, MI355X, Plan, load, model_latency,  # noqa: F401
                    model_multi, model_single, multi, plan_multi, plan_multi_candidates,
                    plan_multi_paper, plan_single, plan_single_candidates, plan_single_paper,
                    probe_latency, single, strerror)
