// Internal declarations shared by the host planner (api.hip) and the kernel
// translation units.  Not part of the public interface (include/dconv.h).
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>
#include <vector>

#include "dconv.h"
#include "xcd.h"

namespace dconv {

// Debug builds (-DDCONV_POISON_LDS, libdconv_poison.so): every LDS buffer of
// a kernel starts filled with NaN, so an output computed from LDS that the
// kernel did not write first (a missing copy, wait or barrier before the
// first use of a buffer) comes out non-finite.  Ordinary builds: nothing.
#ifdef DCONV_POISON_LDS
template <class T>
__device__ __forceinline__ void poison_lds(T *p, int n) {
  float *f = reinterpret_cast<float *>(p);
  const int nf = n * (int)(sizeof(T) / sizeof(float));
  for (int i = threadIdx.x; i < nf; i += blockDim.x) f[i] = __builtin_nanf("");
}
#define DCONV_POISON(...) \
  do {                    \
    __VA_ARGS__;          \
    __syncthreads();      \
  } while (0)
#else
#define DCONV_POISON(...) \
  do {                    \
  } while (0)
#endif

// Stage-trace debug builds (-DDCONV_STAGE_TRACE, libdconv_trace.so): the
// multi-channel matrix-core kernel records clock counters around the phases
// of its stage loop into a buffer the caller registers with
// dconv_debug_stage_trace() (kStageTraceWords long longs per record, two
// records per workgroup: wave 0 and the last wave).  Record layout: [0] start
// (wall clock, 100 MHz), [1] start (shader clock), [2] before the first
// stage's copies, [3] after them, [4] after the stage loop (and channel-group
// sum), [5] end (wall clock), then for stage s < kStageTraceStages the shader
// clock at [6 + 5s + i]: i = 0 stage start, 1 after the copy wait, 2 after
// the barrier, 3 after issuing the next stage's copies, 4 after the MFMAs
// (shapes whose waves stage their own channels pass no barrier and issue
// the next stage's copies halfway through the MFMAs, between marks 3 and 4).
// Ordinary builds: none of this.
constexpr int kStageTraceStages = 64;
constexpr int kStageTraceWords = 6 + 5 * kStageTraceStages;
#ifdef DCONV_STAGE_TRACE
extern long long *g_stage_trace;
#endif

// ---------------------------------------------------------------------------
// Single-map kernels (Eq. 2)
// ---------------------------------------------------------------------------
struct SinglePlan {
  int kernel;     // 0: tiled (float4 rows), 1: generic, 2: tiled (unaligned rows), 3: matrix cores
  int K;
  int rows;       // output rows per lane (R)
  int lanes;      // lanes across a tile row (64, or fewer for narrow maps; vector kernels)
  int tile_h, tile_w;
  int tiles_x, tiles_y;
  int m_per_block;
  int grid;       // tiles_x * tiles_y
  int grid_z;     // ceil(M / m_per_block)
  int block;
  int lds_bytes;
};

constexpr int kMaxTiledK = 11;

// aligned: the input map pointer is 16-byte aligned (with Wx % 4 == 0 the
// tiled kernel then stages whole float4).
// variant: DCONV_VARIANT_AUTO / _VALU / _MFMA; DCONV_EUNSUPPORTED if the
// matrix-core kernel is forced where it has no instance (K < 5 or K > 11,
// or rows not 16-byte aligned).
int plan_single(int Wx, int Wy, int K, int M, int num_cu, bool aligned, int variant,
                SinglePlan *p);
// Every single-map plan for these sizes (each tile shape of the family the
// input's alignment allows, and the matrix-core kernel where it exists,
// crossed with the division of the filters over workgroups), in a fixed
// order; plan_single picks one of them.
int single_candidates(int Wx, int Wy, int K, int M, int num_cu, bool aligned, int variant,
                      std::vector<SinglePlan> &out);
hipError_t launch_single(const SinglePlan &p, const float *I, const float *F, float *O,
                         int Wx, int Wy, int M, hipStream_t s);
// The public description of a plan.
void export_single_plan(const SinglePlan &p, dconv_plan *out);

// ---------------------------------------------------------------------------
// Multi-channel kernels (Eq. 1)
// ---------------------------------------------------------------------------
struct MultiPlan {
  int variant;    // DCONV_VARIANT_VALU or DCONV_VARIANT_MFMA
  int kernel;     // instance id within the family
  int K;
  int tile_m;     // filters per workgroup
  int tpy, tpx;   // output tile rows x cols per workgroup
  int tiles_x, tiles_y;
  int chunk_c;    // channels per LDS stage
  int waves_c;    // wave groups splitting the channel sum inside a workgroup
  int grid_x, grid_y, grid_z;
  int block;
  int lds_bytes;
};

int plan_multi(int C, int M, int Wx, int Wy, int K, int variant, int num_cu, MultiPlan *p);
// Every plan of the family (or both families for DCONV_VARIANT_AUTO) that
// fits the device, in a fixed order; plan_multi picks one of them.
int multi_candidates(int C, int M, int Wx, int Wy, int K, int variant, int num_cu,
                     std::vector<MultiPlan> &out);
// The public description of a plan.
void export_multi_plan(const MultiPlan &p, dconv_plan *out);
hipError_t launch_multi(const MultiPlan &p, const float *I, const float *F, float *O, int C,
                        int M, int Wx, int Wy, hipStream_t s);

}  // namespace dconv
