// Microbenchmarks for the peaks the roofline fractions are quoted against
// (HBM streams, fp32 vector FMA, fp32 matrix instructions) and for the
// global->LDS copy path the convolution kernels stage their operands with.
// Built into libdconv_peaks.so, separate from libdconv; bench.py --peaks
// times each launch with HIP events and turns it into a rate.
//
// Every kernel stays inside the buffers it is given: the streams walk
// [0, n) with a grid-stride loop, the copy probe wraps its source offsets
// with a power-of-two mask and its LDS slots modulo a fixed count.
#include <hip/hip_runtime.h>
#include <cstdint>

#define PEAKS_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

// Sum of every float4 of src (non-temporal loads, four in flight per
// thread); one partial per thread to sink so the loads are not dead.
__global__ __launch_bounds__(256) void hbm_read(const f4 *__restrict__ src, int64_t n,
                                                float *__restrict__ sink) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  f4 acc = {0.f, 0.f, 0.f, 0.f};
  for (; i + 3 * stride < n; i += 4 * stride) {
    const f4 a = __builtin_nontemporal_load(src + i);
    const f4 b = __builtin_nontemporal_load(src + i + stride);
    const f4 c = __builtin_nontemporal_load(src + i + 2 * stride);
    const f4 d = __builtin_nontemporal_load(src + i + 3 * stride);
    acc += a + b + c + d;
  }
  for (; i < n; i += stride) acc += __builtin_nontemporal_load(src + i);
  sink[(int64_t)blockIdx.x * 256 + threadIdx.x] = acc.x + acc.y + acc.z + acc.w;
}

__global__ __launch_bounds__(256) void hbm_write(f4 *__restrict__ dst, int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  const f4 v = {1.f, 2.f, 3.f, 4.f};
  for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride)
    __builtin_nontemporal_store(v, dst + i);
}

__global__ __launch_bounds__(256) void hbm_copy(const f4 *__restrict__ src, f4 *__restrict__ dst,
                                                int64_t n) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  for (; i + stride < n; i += 2 * stride) {
    const f4 a = __builtin_nontemporal_load(src + i);
    const f4 b = __builtin_nontemporal_load(src + i + stride);
    __builtin_nontemporal_store(a, dst + i);
    __builtin_nontemporal_store(b, dst + i + stride);
  }
  for (; i < n; i += stride) __builtin_nontemporal_store(__builtin_nontemporal_load(src + i), dst + i);
}

// Eight independent fp32 FMA chains per lane (one FMA per lane per clock is
// the unpacked rate; packed fp32 instructions are disabled in this build).
__global__ __launch_bounds__(256) void fma_stream(float *__restrict__ out, int iters, float m,
                                                  float a) {
  float x[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = (float)(threadIdx.x + j);
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < 8; ++j) x[j] = __builtin_fmaf(x[j], m, a);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < 8; ++j) s += x[j];
  out[(int64_t)blockIdx.x * 256 + threadIdx.x] = s;
}

typedef float f16v __attribute__((ext_vector_type(16)));

// Four independent accumulators per wave of v_mfma_f32_32x32x2_f32
// (4096 flops each), v_mfma_f32_16x16x4_f32 (2048 flops each) or
// v_mfma_f32_4x4x1f32 (16 blocks of 4 x 4 x 1, 512 flops each).
template <int MF>
__global__ __launch_bounds__(256) void mfma_stream(float *__restrict__ out, int iters) {
  const float av = 1.0f + threadIdx.x * 1e-7f, bv = 1.0f - threadIdx.x * 1e-7f;
  if constexpr (MF == 32) {
    f16v c[4];
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) c[j][v] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < 4; ++j) c[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(av, bv, c[j], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j)
#pragma unroll
      for (int v = 0; v < 16; ++v) s += c[j][v];
    out[(int64_t)blockIdx.x * 256 + threadIdx.x] = s;
  } else {
    f4 c[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) c[j] = f4{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
      for (int j = 0; j < 4; ++j) {
        if constexpr (MF == 16)
          c[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av, bv, c[j], 0, 0, 0);
        else
          c[j] = __builtin_amdgcn_mfma_f32_4x4x1f32(av, bv, c[j], 0, 0, 0);
      }
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 4; ++j) s += c[j].x + c[j].y + c[j].z + c[j].w;
    out[(int64_t)blockIdx.x * 256 + threadIdx.x] = s;
  }
}

// NA independent accumulation chains of v_mfma_f32_4x4x1f32 per wave: with
// one wave per SIMD (grid = compute units, 256 threads) the time per
// instruction shows how far apart dependent instructions must be.
template <int NA>
__global__ __launch_bounds__(256) void mfma_chains(float *__restrict__ out, int iters) {
  const float av = 1.0f + threadIdx.x * 1e-7f, bv = 1.0f - threadIdx.x * 1e-7f;
  f4 c[NA];
#pragma unroll
  for (int j = 0; j < NA; ++j) c[j] = f4{0.f, 0.f, 0.f, 0.f};
  for (int it = 0; it < iters; ++it) {
#pragma unroll
    for (int j = 0; j < NA; ++j) c[j] = __builtin_amdgcn_mfma_f32_4x4x1f32(av, bv, c[j], 0, 0, 0);
  }
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < NA; ++j) s += c[j].x + c[j].y + c[j].z + c[j].w;
  out[(int64_t)blockIdx.x * 256 + threadIdx.x] = s;
}

typedef __attribute__((address_space(3))) void *lds_void_ptr;

// Direct global->LDS copies of W bytes per lane (4 or 16), 64 * W bytes per
// instruction, from a source region of mask + 1 floats (a power of two;
// small enough to stay in L2) into 16 LDS slots per wave, in bursts of 16
// copies followed by a wait.  Measures the rate the copy path delivers to
// LDS, per compute unit and in total.
// `shift` (0 to 3 floats) moves every source address off its W-byte
// alignment, so the unaligned case is measured too; the region then needs
// shift more floats after it.
template <int W>
__global__ __launch_bounds__(256) void lds_dma_stream(const float *__restrict__ src,
                                                      int64_t mask, int shift, int bursts,
                                                      float *__restrict__ out) {
  constexpr int SLOT = 64 * W / 4;       // floats per copy instruction
  __shared__ float buf[4 * 16 * SLOT];
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  float *mine = buf + wave * 16 * SLOT;
  int64_t base = ((int64_t)blockIdx.x * 4 + wave) * 16 * SLOT;
  for (int b = 0; b < bursts; ++b) {
#pragma unroll
    for (int s = 0; s < 16; ++s) {
      const int64_t off = ((base + (int64_t)s * SLOT + lane * (W / 4)) & mask) + shift;
      if constexpr (W == 4)
        __builtin_amdgcn_global_load_lds(src + off, (lds_void_ptr)(mine + s * SLOT), 4, 0, 0);
      else
        __builtin_amdgcn_global_load_lds(src + off, (lds_void_ptr)(mine + s * SLOT), 16, 0, 0);
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    base += 16 * SLOT * 7;  // move on through the region
  }
  __syncthreads();
  out[(int64_t)blockIdx.x * 256 + threadIdx.x] = buf[threadIdx.x];
}

// The same source walk as lds_dma_stream<16>, loaded into registers instead
// (16 float4 loads in flight per lane, then a wait and a sum): the rate the
// L2 -> vector L1 path delivers to ordinary loads, for comparison with the
// direct copies above.
__global__ __launch_bounds__(256) void vgpr_load_stream(const float *__restrict__ src,
                                                        int64_t mask, int bursts,
                                                        float *__restrict__ out) {
  constexpr int SLOT = 256;
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  int64_t base = ((int64_t)blockIdx.x * 4 + wave) * 16 * SLOT;
  f4 acc = f4{0.f, 0.f, 0.f, 0.f};
  for (int b = 0; b < bursts; ++b) {
    f4 x[16];
#pragma unroll
    for (int s = 0; s < 16; ++s)
      x[s] = *reinterpret_cast<const f4 *>(src + ((base + (int64_t)s * SLOT + lane * 4) & mask));
#pragma unroll
    for (int s = 0; s < 16; ++s) acc += x[s];
    base += 16 * SLOT * 7;
  }
  out[(int64_t)blockIdx.x * 256 + threadIdx.x] = acc.x + acc.y + acc.z + acc.w;
}

// Where a 16-byte-per-lane direct copy lands when its LDS destination is
// `shift` floats (0 to 3) past a 16-byte boundary: one wave copies 256
// floats of src into a zeroed LDS array at float offset shift, then writes
// the whole array (264 floats) to out.  Lane l's four floats are expected at
// shift + 4l .. shift + 4l + 3.
// With active < 64 only lanes 0 .. active-1 issue the copy (the others are
// masked off by a branch), which shows what masked-off lanes write.
__global__ __launch_bounds__(64) void lds_dma_layout(const float *__restrict__ src, int shift,
                                                     int active, float *__restrict__ out) {
  __shared__ __attribute__((aligned(16))) float buf[264];
  const int lane = threadIdx.x;
  for (int i = lane; i < 264; i += 64) buf[i] = 0.f;
  __syncthreads();
  if (lane < active)
    __builtin_amdgcn_global_load_lds(src + 4 * lane, (lds_void_ptr)(buf + shift), 16, 0, 0);
  asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
  __syncthreads();
  for (int i = lane; i < 264; i += 64) out[i] = buf[i];
}

}  // namespace

PEAKS_EXPORT int peaks_lds_dma_layout(const float *src, int shift, int active, float *out,
                                      void *stream) {
  if (!src || !out || shift < 0 || shift > 3 || active < 1 || active > 64) return -1;
  (void)hipGetLastError();
  hipLaunchKernelGGL(lds_dma_layout, dim3(1), dim3(64), 0, (hipStream_t)stream, src, shift, active,
                     out);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

PEAKS_EXPORT int peaks_vgpr_load(const float *src, long long region_floats, int bursts,
                                  float *out, int grid, void *stream) {
  if (!src || !out || bursts < 1 || grid < 1 || region_floats < 4096 ||
      (region_floats & (region_floats - 1)) != 0)
    return -1;
  (void)hipGetLastError();
  hipLaunchKernelGGL(vgpr_load_stream, dim3(grid), dim3(256), 0, (hipStream_t)stream, src,
                     (int64_t)(region_floats - 1), bursts, out);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// All calls: enqueue on `stream` and return 0, or -1 for a bad argument, or
// -4 if the launch failed.  `sink` / `out` hold grid x 256 floats.
PEAKS_EXPORT int peaks_hbm_read(const void *src, long long bytes, float *sink, int grid,
                                void *stream) {
  if (!src || !sink || bytes < 16 || grid < 1) return -1;
  (void)hipGetLastError();
  hipLaunchKernelGGL(hbm_read, dim3(grid), dim3(256), 0, (hipStream_t)stream,
                     (const f4 *)src, (int64_t)(bytes / 16), sink);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

PEAKS_EXPORT int peaks_hbm_write(void *dst, long long bytes, int grid, void *stream) {
  if (!dst || bytes < 16 || grid < 1) return -1;
  (void)hipGetLastError();
  hipLaunchKernelGGL(hbm_write, dim3(grid), dim3(256), 0, (hipStream_t)stream, (f4 *)dst,
                     (int64_t)(bytes / 16));
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

PEAKS_EXPORT int peaks_hbm_copy(const void *src, void *dst, long long bytes, int grid,
                                void *stream) {
  if (!src || !dst || bytes < 16 || grid < 1) return -1;
  (void)hipGetLastError();
  hipLaunchKernelGGL(hbm_copy, dim3(grid), dim3(256), 0, (hipStream_t)stream, (const f4 *)src,
                     (f4 *)dst, (int64_t)(bytes / 16));
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

PEAKS_EXPORT int peaks_fma(float *out, int iters, int grid, void *stream) {
  if (!out || iters < 1 || grid < 1) return -1;
  (void)hipGetLastError();
  hipLaunchKernelGGL(fma_stream, dim3(grid), dim3(256), 0, (hipStream_t)stream, out, iters,
                     0.999999f, 1e-6f);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

PEAKS_EXPORT int peaks_mfma(float *out, int iters, int grid, int shape, void *stream) {
  if (!out || iters < 1 || grid < 1 || (shape != 32 && shape != 16 && shape != 4)) return -1;
  (void)hipGetLastError();
  if (shape == 32)
    hipLaunchKernelGGL(mfma_stream<32>, dim3(grid), dim3(256), 0, (hipStream_t)stream, out, iters);
  else if (shape == 16)
    hipLaunchKernelGGL(mfma_stream<16>, dim3(grid), dim3(256), 0, (hipStream_t)stream, out, iters);
  else
    hipLaunchKernelGGL(mfma_stream<4>, dim3(grid), dim3(256), 0, (hipStream_t)stream, out, iters);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

PEAKS_EXPORT int peaks_mfma_chains(float *out, int chains, int iters, int grid, void *stream) {
  if (!out || iters < 1 || grid < 1) return -1;
  (void)hipGetLastError();
  switch (chains) {
    case 1: hipLaunchKernelGGL(mfma_chains<1>, dim3(grid), dim3(256), 0, (hipStream_t)stream, out, iters); break;
    case 2: hipLaunchKernelGGL(mfma_chains<2>, dim3(grid), dim3(256), 0, (hipStream_t)stream, out, iters); break;
    case 4: hipLaunchKernelGGL(mfma_chains<4>, dim3(grid), dim3(256), 0, (hipStream_t)stream, out, iters); break;
    case 8: hipLaunchKernelGGL(mfma_chains<8>, dim3(grid), dim3(256), 0, (hipStream_t)stream, out, iters); break;
    default: return -1;
  }
  return hipGetLastError() == hipSuccess ? 0 : -4;
}

// src: at least region_floats + shift floats, region_floats a power of two
// >= 4096, 0 <= shift <= 3.
PEAKS_EXPORT int peaks_lds_dma(const float *src, long long region_floats, int shift, int width,
                               int bursts, float *out, int grid, void *stream) {
  if (!src || !out || bursts < 1 || grid < 1 || region_floats < 4096 ||
      (region_floats & (region_floats - 1)) != 0 || (width != 4 && width != 16) || shift < 0 ||
      shift > 3)
    return -1;
  (void)hipGetLastError();
  if (width == 4)
    hipLaunchKernelGGL(lds_dma_stream<4>, dim3(grid), dim3(256), 0, (hipStream_t)stream, src,
                       (int64_t)(region_floats - 1), shift, bursts, out);
  else
    hipLaunchKernelGGL(lds_dma_stream<16>, dim3(grid), dim3(256), 0, (hipStream_t)stream, src,
                       (int64_t)(region_floats - 1), shift, bursts, out);
  return hipGetLastError() == hipSuccess ? 0 : -4;
}
