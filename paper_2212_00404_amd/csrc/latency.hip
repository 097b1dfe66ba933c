// Dependent-load latency probe: the measured latency that parameterises the
// paper's latency-hiding model (Section 2.2 takes the global-memory latency
// from a pointer-chasing measurement).
#include "internal.h"

#define DCONV_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

// One lane follows the chain j <- chain[j] from j = 0.  Every load's address
// depends on the previous load's value, so the elapsed time over `steps`
// loads divided by `steps` is the latency of one load from wherever the
// chain's footprint lives (caches or HBM).  The index is kept in a vector
// register so the loads are vector-memory loads like the kernels' own.
__global__ __launch_bounds__(64) void chase(const int *__restrict__ chain, int steps,
                                            long long *__restrict__ out) {
  if (threadIdx.x != 0) return;
  int j;
  asm volatile("v_mov_b32 %0, 0" : "=v"(j));
  const long long c0 = (long long)__builtin_amdgcn_s_memtime();
  const long long r0 = (long long)__builtin_amdgcn_s_memrealtime();
  for (int k = 0; k < steps; ++k) j = chain[j];
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  const long long c1 = (long long)__builtin_amdgcn_s_memtime();
  const long long r1 = (long long)__builtin_amdgcn_s_memrealtime();
  out[0] = c1 - c0;
  out[1] = r1 - r0;
  out[2] = j;
}

}  // namespace

DCONV_EXPORT int dconv_probe_latency(const int *chain, int steps, long long *out, void *stream) {
  if (!chain || !out) return DCONV_ENULL;
  if (steps < 1) return DCONV_EINVAL;
  (void)hipGetLastError();  // report this launch only
  hipLaunchKernelGGL(chase, dim3(1), dim3(64), 0, (hipStream_t)stream, chain, steps, out);
  return hipGetLastError() == hipSuccess ? DCONV_OK : DCONV_EHIP;
}
