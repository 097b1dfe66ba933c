// Single-map direct convolution (paper, Section 2.1, Eq. 2; Section 3.1).
//
// One input map I[Wy][Wx], M filters F[M][K][K], output O[M][Hout][Wout].
//
// Design for gfx950 (the paper's SM partitioning for Pascal is prior art):
//  * A 256-thread workgroup owns a TH x 256 output tile (TH = 4 waves x R
//    rows).  It stages the input tile plus its K-1 halo rows and columns
//    (Section 3.1 adds the same K-1 extra lines to each map piece) in LDS
//    with coalesced float4 loads, then applies its share of the M filters to
//    the staged tile one after another, so the map is fetched from HBM once
//    per filter group (the map-split method of Section 3.1).
//  * Each lane owns 4 adjacent output columns x R output rows and streams the
//    R+K-1 input rows of its strip through registers: every row it reads from
//    LDS (W+K-1 values, 16-byte reads) feeds up to K filter rows x K taps x 4
//    columns of FMAs, so LDS traffic stays far below the FMA rate.
//  * The filter is wave-uniform; the compiler keeps it in scalar registers
//    (or VGPRs when K*K exceeds the scalar budget) and every FMA takes it as
//    an operand directly.
//  * Blocks are remapped so that each XCD walks a contiguous band of tiles
//    and halo rows shared by vertically adjacent tiles stay in one L2.
#include "internal.h"

namespace dconv {
namespace {

constexpr int kW = 4;           // output columns per lane
constexpr int kLanes = 64;
constexpr int kWaves = 4;
constexpr int kBlock = kLanes * kWaves;
constexpr int kTileW = kLanes * kW;  // 256 output columns per tile

// Output rows per lane, per filter size: enough rows that halo re-reads stay
// small, few enough that accumulators + filter + one input row fit in VGPRs.
template <int K> struct Rows { static constexpr int value = 8; };
// Output rows accumulated at once (a divisor of Rows).
template <int K> struct Group { static constexpr int value = 4; };

// Up to 7x7 the filter fits the scalar register file next to the addressing
// state.  Larger filters would spill scalar registers into VGPR lanes inside
// the FMA loop, so they are held in VGPRs instead (one copy per lane).
template <int K> struct FilterInVgpr { static constexpr bool value = K * K > 49; };

template <int K, int R>
struct TileShape {
  static constexpr int TH = kWaves * R;            // output rows per tile
  static constexpr int IH = TH + K - 1;            // staged input rows
  static constexpr int NQ = (kW + K - 1 + 3) / 4;  // float4 reads per lane per row
  static constexpr int IW4 = kLanes + NQ - 1;      // float4 per staged row
  static constexpr int LDS = IH * IW4 * 16;
};

template <int NQ>
__device__ __forceinline__ void load_row(const float4 *p, float *v) {
#pragma unroll
  for (int q = 0; q < NQ; ++q) {
    const float4 t = p[q];
    v[4 * q + 0] = t.x;
    v[4 * q + 1] = t.y;
    v[4 * q + 2] = t.z;
    v[4 * q + 3] = t.w;
  }
}

template <int K, int R>
__global__ __launch_bounds__(kBlock, 2) void single_tiled(
    const float *__restrict__ I, const float *__restrict__ F, float *__restrict__ O,
    int Wx, int Wy, int M, int tiles_x, int ntiles, int m_per_block, int vec4, int ostore) {
  using S = TileShape<K, R>;
  constexpr int IH = S::IH, IW4 = S::IW4, NQ = S::NQ;
  constexpr int G = Group<K>::value;
  static_assert(R % G == 0, "group must divide the strip");
  __shared__ float4 tile[IH * IW4];

  const int Hout = Wy - K + 1;
  const int Wout = Wx - K + 1;
  const int t = xcd_remap(blockIdx.x, ntiles);
  const int y0 = (t / tiles_x) * S::TH;
  const int x0 = (t % tiles_x) * kTileW;

  // Stage input rows [y0, y0+IH) x columns [x0, x0+4*IW4); zero outside the map.
  // All of a thread's loads are issued before the first LDS write so that
  // they are in flight together.  vec4: rows are 16-byte aligned (Wx % 4 == 0
  // and I 16-byte aligned).
  if (vec4) {
    constexpr int N = IH * IW4;
    constexpr int NL = (N + kBlock - 1) / kBlock;
    float4 v[NL];
#pragma unroll
    for (int j = 0; j < NL; ++j) {
      const int idx = threadIdx.x + j * kBlock;
      const int iy = idx / IW4;
      const int gy = y0 + iy;
      const int gx = x0 + 4 * (idx - iy * IW4);
      v[j] = make_float4(0.f, 0.f, 0.f, 0.f);
      if ((NL * kBlock == N || idx < N) && gy < Wy && gx < Wx)
        v[j] = *reinterpret_cast<const float4 *>(I + (size_t)gy * Wx + gx);
    }
#pragma unroll
    for (int j = 0; j < NL; ++j) {
      const int idx = threadIdx.x + j * kBlock;
      if (NL * kBlock == N || idx < N) tile[idx] = v[j];
    }
  } else {
    float *tf = reinterpret_cast<float *>(tile);
    constexpr int IWf = IW4 * 4;
    constexpr int N = IH * IWf;
    constexpr int NL = (N + kBlock - 1) / kBlock;
    constexpr int kBatch = 16;
#pragma unroll
    for (int b = 0; b < NL; b += kBatch) {
      float v[kBatch];
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int idx = threadIdx.x + (b + j) * kBlock;
        const int iy = idx / IWf;
        const int gy = y0 + iy;
        const int gx = x0 + (idx - iy * IWf);
        v[j] = 0.f;
        if (b + j < NL && idx < N && gy < Wy && gx < Wx) v[j] = I[(size_t)gy * Wx + gx];
      }
#pragma unroll
      for (int j = 0; j < kBatch; ++j) {
        const int idx = threadIdx.x + (b + j) * kBlock;
        if (b + j < NL && idx < N) tf[idx] = v[j];
      }
    }
  }
  __syncthreads();

  const int lane = threadIdx.x & (kLanes - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kLanes);
  const float4 *rowp = tile + wave * R * IW4 + lane;
  const int oy0 = y0 + wave * R;
  const int ox0 = x0 + lane * kW;

  const int m_begin = blockIdx.y * m_per_block;
  const int m_end = min(M, m_begin + m_per_block);
  for (int m = m_begin; m < m_end; ++m) {
    const float *Fm = F + (size_t)m * K * K;
    float f[K][K];
#pragma unroll
    for (int r = 0; r < K; ++r)
#pragma unroll
      for (int s = 0; s < K; ++s) {
        f[r][s] = Fm[r * K + s];
        if constexpr (FilterInVgpr<K>::value) asm volatile("" : "+v"(f[r][s]));
      }

    // Rows of the strip are processed G at a time; each group streams its
    // G+K-1 input rows once and keeps G x 4 accumulators.
#pragma unroll 1
    for (int g = 0; g < R / G; ++g) {
      const float4 *gp = rowp + g * G * IW4;
      float acc[G][kW];
#pragma unroll
      for (int j = 0; j < G; ++j)
#pragma unroll
        for (int w = 0; w < kW; ++w) acc[j][w] = 0.f;

      // One row of look-ahead: the next input row is requested from LDS
      // before the current one is consumed; the scheduling barrier keeps the
      // compiler from hoisting every row (which would exhaust the VGPRs).
      float cur[NQ * 4], nxt[NQ * 4];
      load_row<NQ>(gp, cur);
#pragma unroll
      for (int yy = 0; yy < G + K - 1; ++yy) {
        if (yy + 1 < G + K - 1) load_row<NQ>(gp + (yy + 1) * IW4, nxt);
#pragma unroll
        for (int r = 0; r < K; ++r) {
          const int j = yy - r;  // output row fed by filter row r
          if (j < 0 || j >= G) continue;
#pragma unroll
          for (int s = 0; s < K; ++s)
#pragma unroll
            for (int w = 0; w < kW; ++w)
              acc[j][w] = __builtin_fmaf(cur[w + s], f[r][s], acc[j][w]);
        }
        // Pin this row's FMAs before the barrier (the accumulators pass
        // through an empty asm statement, which is ordered like the barrier).
#pragma unroll
        for (int j = 0; j < G; ++j)
#pragma unroll
          for (int w = 0; w < kW; ++w) asm volatile("" : "+v"(acc[j][w]));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < NQ * 4; ++q) cur[q] = nxt[q];
      }

      float *Om = O + (size_t)m * Hout * Wout;
#pragma unroll
      for (int j = 0; j < G; ++j) {
        const int y = oy0 + g * G + j;
        if (y >= Hout) continue;
        float *orow = Om + (size_t)y * Wout + ox0;
        if (ox0 + kW <= Wout && ostore == 4) {
          *reinterpret_cast<float4 *>(orow) = make_float4(acc[j][0], acc[j][1], acc[j][2], acc[j][3]);
        } else if (ox0 + kW <= Wout && ostore == 2) {
          reinterpret_cast<float2 *>(orow)[0] = make_float2(acc[j][0], acc[j][1]);
          reinterpret_cast<float2 *>(orow)[1] = make_float2(acc[j][2], acc[j][3]);
        } else {
#pragma unroll
          for (int w = 0; w < kW; ++w)
            if (ox0 + w < Wout) orow[w] = acc[j][w];
        }
      }
    }
  }
}

// Any K: one output per thread, operands read through the caches.  Used for
// filters larger than the tiled kernels are instantiated for.
__global__ __launch_bounds__(256) void single_generic(
    const float *__restrict__ I, const float *__restrict__ F, float *__restrict__ O,
    int Wx, int Wy, int K, int M) {
  const int Hout = Wy - K + 1;
  const int Wout = Wx - K + 1;
  const int64_t total = (int64_t)M * Hout * Wout;
  const int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= total) return;
  const int x = (int)(idx % Wout);
  const int64_t my = idx / Wout;
  const int y = (int)(my % Hout);
  const int m = (int)(my / Hout);
  const float *Fm = F + (int64_t)m * K * K;
  float acc = 0.f;
  for (int r = 0; r < K; ++r) {
    const float *irow = I + (int64_t)(y + r) * Wx + x;
    const float *frow = Fm + r * K;
    for (int s = 0; s < K; ++s) acc = __builtin_fmaf(irow[s], frow[s], acc);
  }
  O[idx] = acc;
}

template <int K>
void plan_tiled(int Wx, int Wy, int M, int num_cu, SinglePlan *p) {
  constexpr int R = Rows<K>::value;
  using S = TileShape<K, R>;
  const int Hout = Wy - K + 1, Wout = Wx - K + 1;
  p->kernel = 0;
  p->rows = R;
  p->tile_h = S::TH;
  p->tile_w = kTileW;
  p->tiles_x = (Wout + kTileW - 1) / kTileW;
  p->tiles_y = (Hout + S::TH - 1) / S::TH;
  p->grid = p->tiles_x * p->tiles_y;
  // Filters reuse the staged tile; split them over workgroups only as far as
  // needed to give every compute unit several workgroups.
  const int want = 4 * num_cu;
  int splits = (want + p->grid - 1) / p->grid;
  if (splits > M) splits = M;
  if (splits < 1) splits = 1;
  p->m_per_block = (M + splits - 1) / splits;
  p->grid_z = (M + p->m_per_block - 1) / p->m_per_block;
  p->block = kBlock;
  p->lds_bytes = S::LDS;
}

// Widest output store every row of O allows: 4 floats if rows start on 16-byte
// boundaries, 2 if on 8-byte boundaries, else 1.  Lanes own 4 columns at
// multiples of 4, so aligned rows keep every lane's store aligned.
int store_width(const float *O, int Wout, int Hout) {
  const uintptr_t a = reinterpret_cast<uintptr_t>(O);
  (void)Hout;
  if (Wout % 4 == 0 && (a & 15) == 0) return 4;
  if (Wout % 2 == 0 && (a & 7) == 0) return 2;
  return 1;
}

template <int K>
hipError_t launch_tiled(const SinglePlan &p, const float *I, const float *F, float *O,
                        int Wx, int Wy, int M, hipStream_t s) {
  constexpr int R = Rows<K>::value;
  hipLaunchKernelGGL((single_tiled<K, R>), dim3(p.grid, p.grid_z), dim3(kBlock), 0, s,
                     I, F, O, Wx, Wy, M, p.tiles_x, p.grid, p.m_per_block,
                     (int)((Wx % 4 == 0) && ((reinterpret_cast<uintptr_t>(I) & 15) == 0)),
                     store_width(O, Wx - K + 1, Wy - K + 1));
  return hipGetLastError();
}

}  // namespace

void plan_single(int Wx, int Wy, int K, int M, int num_cu, SinglePlan *p) {
  *p = SinglePlan{};
  p->K = K;
  switch (K) {
#define DCONV_PLAN_K(k) \
  case k:               \
    plan_tiled<k>(Wx, Wy, M, num_cu, p); \
    return;
    DCONV_PLAN_K(1) DCONV_PLAN_K(2) DCONV_PLAN_K(3) DCONV_PLAN_K(4) DCONV_PLAN_K(5)
    DCONV_PLAN_K(6) DCONV_PLAN_K(7) DCONV_PLAN_K(8) DCONV_PLAN_K(9) DCONV_PLAN_K(10)
    DCONV_PLAN_K(11)
#undef DCONV_PLAN_K
    default:
      break;
  }
  const int64_t total = (int64_t)M * (Wy - K + 1) * (Wx - K + 1);
  p->kernel = 1;
  p->rows = 1;
  p->tile_h = 1;
  p->tile_w = 256;
  p->grid = (int)((total + 255) / 256);
  p->grid_z = 1;
  p->tiles_x = p->grid;
  p->tiles_y = 1;
  p->m_per_block = M;
  p->block = 256;
  p->lds_bytes = 0;
}

hipError_t launch_single(const SinglePlan &p, const float *I, const float *F, float *O,
                         int Wx, int Wy, int M, hipStream_t s) {
  if (p.kernel == 1) {
    hipLaunchKernelGGL(single_generic, dim3(p.grid), dim3(256), 0, s, I, F, O, Wx, Wy, p.K, M);
    return hipGetLastError();
  }
  switch (p.K) {
#define DCONV_LAUNCH_K(k) \
  case k:                 \
    return launch_tiled<k>(p, I, F, O, Wx, Wy, M, s);
    DCONV_LAUNCH_K(1) DCONV_LAUNCH_K(2) DCONV_LAUNCH_K(3) DCONV_LAUNCH_K(4) DCONV_LAUNCH_K(5)
    DCONV_LAUNCH_K(6) DCONV_LAUNCH_K(7) DCONV_LAUNCH_K(8) DCONV_LAUNCH_K(9) DCONV_LAUNCH_K(10)
    DCONV_LAUNCH_K(11)
#undef DCONV_LAUNCH_K
    default:
      return hipErrorInvalidValue;
  }
}

}  // namespace dconv
