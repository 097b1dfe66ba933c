// Single-map direct convolution (paper, Section 2.1, Eq. 2; Section 3.1).
//
// One input map I[Wy][Wx], M filters F[M][K][K], output O[M][Hout][Wout].
//
// Design for gfx950 (the paper's SM partitioning for Pascal is prior art):
//  * The output is cut into TH x 256 tiles (TH = 4 waves x R rows; R = 4 or 8,
//    4 where tall tiles would leave compute units idle), or for outputs up to
//    128 columns wide into 64-column tiles whose waves split into four row
//    groups.  A tile needs its input rows plus K-1 halo rows and columns
//    (Section 3.1 adds the same K-1 extra lines to each map piece).
//  * Workgroups are persistent: each walks every nwg-th tile and, while it
//    computes one tile from LDS, the global loads of its next tile are
//    already in flight into registers (the prefetching of Section 2.2,
//    method 1, done per workgroup).  After the compute the prefetched tile is
//    written to LDS.  Blocks are remapped per XCD so that neighbouring tiles,
//    which share halo rows, run on the same L2.
//  * Each lane owns 4 adjacent output columns x R output rows and streams the
//    input rows of its strip through registers G output rows at a time: one
//    16-byte LDS read per 4 input columns feeds up to K filter rows x K taps x
//    4 columns of FMAs, so LDS traffic stays far below the FMA rate.
//  * The filter is wave-uniform: up to 7x7 it stays in scalar registers and
//    every FMA takes it as an operand; larger filters are held in VGPRs.
//  * The filters of a workgroup (its share of the M filters) are applied to
//    each staged tile in turn, so the map is read from HBM once per filter
//    group (the map-split method of Section 3.1).
//  * Each lane writes its 4 columns of a row with one 16-byte store at any
//    row alignment, non-temporal except in one case chosen on the host.
#include <type_traits>

#include "internal.h"

namespace dconv {
namespace {

constexpr int kW = 4;           // output columns per lane
constexpr int kLanes = 64;
constexpr int kWaves = 4;
constexpr int kBlock = kLanes * kWaves;
constexpr int kTileW = kLanes * kW;  // 256 output columns per tile

// A lane's 4 output columns, stored as one 16-byte write.  Rows of O start
// wherever Wout puts them, so the type asks for 4-byte alignment only: the
// chip's global stores need dword alignment, and one 16-byte store per lane
// keeps every write a whole run of the row.  (Two 8-byte or four 4-byte
// non-temporal stores per lane, as an odd or 2 (mod 4) width would otherwise
// need, leave partly written lines: measured 1.05x slower at Wout = 4090 and
// 1.8-2.6x slower at Wout = 4089 and 4091.)
typedef float vf4u __attribute__((ext_vector_type(4), aligned(4)));

// Output rows per lane: enough that halo re-reads stay small, few enough that
// accumulators, filter, input rows and the prefetched tile fit in VGPRs (a
// tile prefetched as single floats takes four times the registers of one
// prefetched as float4, so unaligned maps get shorter tiles for large K).
// Small filters are bound by memory traffic: shorter tiles give each
// persistent workgroup more of them, so its first (unhidden) tile load is
// shorter and the loads of later tiles overlap more compute (measured 4-8%
// faster at K = 3 and 5 on a 4096 x 4096 map; no gain at K = 7).
template <int K, bool VEC4> struct Rows {
  static constexpr int value = (K <= 5 || (!VEC4 && K >= 8)) ? 4 : 8;
};
// Rows per lane of the short tiles used where tall ones would not give every
// compute unit a tile.
constexpr int kShortRows = 4;
// Output rows accumulated at once (a divisor of Rows).
template <int K> struct Group { static constexpr int value = 4; };
// Workgroups per compute unit the kernel is compiled for (register budget; a
// tile prefetched as single floats needs four times the registers).
template <int K, bool VEC4> struct Occupancy { static constexpr int value = (VEC4 && K <= 7) ? 4 : 2; };

// Up to 7x7 the filter fits the scalar register file next to the addressing
// state.  Larger filters would spill scalar registers into VGPR lanes inside
// the FMA loop, so they are held in VGPRs instead (one copy per lane).
template <int K> struct FilterInVgpr { static constexpr bool value = K * K > 49; };

// L: lanes across a row.  With L = 64 a wave covers R rows x 256 columns;
// with L < 64 its lanes form 64 / L row groups, each R rows x 4L columns
// (narrow maps, where most of a 256-column tile would hold no outputs).
template <int K, int R, int L = kLanes>
struct TileShape {
  static constexpr int RG = kLanes / L;            // row groups per wave
  static constexpr int TW = kW * L;                // output columns per tile
  static constexpr int TH = kWaves * RG * R;       // output rows per tile
  static constexpr int IH = TH + K - 1;            // staged input rows
  static constexpr int NQ = (kW + K - 1 + 3) / 4;  // float4 reads per lane per row
  static constexpr int IW4 = L + NQ - 1;           // float4 per staged row
  static constexpr int LW4 = IW4;                  // LDS stride of a staged row (float4)
  static constexpr int LDS = IH * LW4 * 16;
};
// Lanes across a row of the narrow tiles, and the widest output they serve.
constexpr int kNarrowLanes = 16;
constexpr int kNarrowMaxWout = 128;
constexpr int kNarrowMaxK = 5;

// s_waitcnt immediate for "vmcnt(0)" alone on gfx9-family chips: vmcnt in
// bits 3:0 and 15:14 (0), expcnt in bits 6:4 and lgkmcnt in bits 11:8 at their
// maxima (no wait).
constexpr int kWaitVmcnt0 = 0x0F70;

// Barrier for LDS hand-over inside a workgroup.  Unlike __syncthreads() it
// does not wait for outstanding global loads (the next tile's prefetch stays
// in flight across it) or global stores.
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Loads of one staged tile held in registers between fetch() and commit().
// VEC4: every map row starts on a 16-byte boundary, so whole float4 are
// loaded; otherwise single floats.  Values outside the map are zero.
// S: the tile shape (IH staged rows of IW4 float4, stored LW4 float4 apart).
template <class S, bool VEC4>
struct Stager {
  using T = typename std::conditional<VEC4, float4, float>::type;
  static constexpr int PER_ROW = VEC4 ? S::IW4 : S::IW4 * 4;
  static constexpr int LDS_ROW = VEC4 ? S::LW4 : S::LW4 * 4;
  static constexpr int N = S::IH * PER_ROW;
  static constexpr int NL = (N + kBlock - 1) / kBlock;
  T v[NL];

  __device__ __forceinline__ void fetch(const float *__restrict__ I, int Wx, int Wy, int y0, int x0) {
#pragma unroll
    for (int j = 0; j < NL; ++j) {
      const int idx = threadIdx.x + j * kBlock;
      const int iy = idx / PER_ROW;
      const int ix = idx - iy * PER_ROW;
      const int gy = y0 + iy;
      const bool ok = (NL * kBlock == N || idx < N) && gy < Wy;
      if constexpr (VEC4) {
        const int gx = x0 + 4 * ix;
        v[j] = make_float4(0.f, 0.f, 0.f, 0.f);
        if (ok && gx < Wx) v[j] = *reinterpret_cast<const float4 *>(I + (size_t)gy * Wx + gx);
      } else {
        const int gx = x0 + ix;
        v[j] = 0.f;
        if (ok && gx < Wx) v[j] = I[(size_t)gy * Wx + gx];
      }
    }
  }

  __device__ __forceinline__ void commit(float4 *tile) const {
    T *dst = reinterpret_cast<T *>(tile);
#pragma unroll
    for (int j = 0; j < NL; ++j) {
      const int idx = threadIdx.x + j * kBlock;
      if (NL * kBlock == N || idx < N) {
        if constexpr (LDS_ROW == PER_ROW) {
          dst[idx] = v[j];
        } else {
          const int iy = idx / PER_ROW;
          dst[iy * LDS_ROW + (idx - iy * PER_ROW)] = v[j];
        }
      }
    }
  }
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

template <int K>
__device__ __forceinline__ void load_filter(const float *__restrict__ F, int m, float (&f)[K][K]) {
  const float *Fm = F + (size_t)m * K * K;
  if constexpr (FilterInVgpr<K>::value) {
    // Vector loads through a pointer the compiler cannot prove uniform: all
    // K*K loads are in flight together (scalar loads of this many values
    // would be issued and waited for one at a time).
    int zero;
    asm volatile("v_mov_b32 %0, 0" : "=v"(zero));
    const float *p = Fm + zero;
#pragma unroll
    for (int r = 0; r < K; ++r)
#pragma unroll
      for (int s = 0; s < K; ++s) f[r][s] = p[r * K + s];
    // Wait for them here, with an instruction the compiler sees.  Otherwise
    // the first use of the filter, at a point the load may or may not have
    // been issued on every path, gets a wait for all loads in flight, which
    // includes the next tile's prefetch: prefetch and compute would then not
    // overlap even where no filter is reloaded.
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
  } else {
#pragma unroll
    for (int r = 0; r < K; ++r)
#pragma unroll
      for (int s = 0; s < K; ++s) f[r][s] = Fm[r * K + s];
  }
}

// One filter over the staged tile: this lane's R x 4 outputs at (oy0, ox0).
// NT: non-temporal output stores.  L: lanes across a row (TileShape).
template <int K, int R, bool NT, int L>
__device__ __forceinline__ void apply_filter(const float4 *rowp, const float (&f)[K][K],
                                             float *__restrict__ Om, int oy0, int ox0, int Hout,
                                             int Wout) {
  using S = TileShape<K, R, L>;
  constexpr int IW4 = S::IW4, NQ = S::NQ;
  constexpr int G = Group<K>::value;
  static_assert(R % G == 0, "group must divide the strip");
#pragma unroll 1
  for (int g = 0; g < R / G; ++g) {
    const float4 *gp = rowp + g * G * IW4;
    float acc[G][kW];
#pragma unroll
    for (int j = 0; j < G; ++j)
#pragma unroll
      for (int w = 0; w < kW; ++w) acc[j][w] = 0.f;

    // One row of look-ahead: the next input row is requested from LDS
    // before the current one is consumed.  The accumulators pass through an
    // empty asm statement and a scheduling barrier ends each row, which
    // keeps the compiler from hoisting every row's reads (and exhausting the
    // VGPRs).
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
#pragma unroll
      for (int j = 0; j < G; ++j)
#pragma unroll
        for (int w = 0; w < kW; ++w) asm volatile("" : "+v"(acc[j][w]));
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int q = 0; q < NQ * 4; ++q) cur[q] = nxt[q];
    }

#pragma unroll
    for (int j = 0; j < G; ++j) {
      const int y = oy0 + g * G + j;
      if (y >= Hout) continue;
      // The output is written once and never read back by this kernel:
      // non-temporal stores keep it from displacing the input tiles and
      // halos in the caches (measured: 15-20% faster across K).  The
      // exception (NT false) is chosen by the host.
      float *orow = Om + (size_t)y * Wout + ox0;
      const vf4u v = {acc[j][0], acc[j][1], acc[j][2], acc[j][3]};
      if (ox0 + kW <= Wout) {
        if constexpr (NT)
          __builtin_nontemporal_store(v, reinterpret_cast<vf4u *>(orow));
        else
          *reinterpret_cast<vf4u *>(orow) = v;
      } else {
#pragma unroll
        for (int w = 0; w < kW; ++w)
          if (ox0 + w < Wout) orow[w] = v[w];
      }
    }
  }
}

template <int K, int R, bool VEC4, bool NT, int L>
__global__ __launch_bounds__(kBlock, (Occupancy<K, VEC4>::value)) void single_tiled(
    const float *__restrict__ I, const float *__restrict__ F, float *__restrict__ O,
    int Wx, int Wy, int M, int tiles_x, int ntiles, int m_per_block) {
  using S = TileShape<K, R, L>;
  __shared__ float4 tile[S::IH * S::IW4];
  DCONV_POISON(poison_lds(tile, S::IH * S::IW4));

  const int Hout = Wy - K + 1;
  const int Wout = Wx - K + 1;
  // Persistent workgroup: tiles wg, wg + nwg, wg + 2 nwg, ...  At any moment
  // the workgroups in flight cover one contiguous band of tiles (rows of the
  // map), which measured faster than giving each workgroup its own run.
  const int nwg = gridDim.x;
  const int wg = xcd_remap(blockIdx.x, nwg);
  if (wg >= ntiles) return;
  const int m_begin = blockIdx.y * m_per_block;
  const int m_end = min(M, m_begin + m_per_block);

  const int lane = threadIdx.x & (kLanes - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kLanes);
  // This lane's row group (first output row within the tile) and column
  // quad.
  const int row0 = (wave * S::RG + lane / L) * R;
  const int cq = lane % L;
  const float4 *rowp = tile + row0 * S::IW4 + cq;

  Stager<S, VEC4> st;
  st.fetch(I, Wx, Wy, (wg / tiles_x) * S::TH, (wg % tiles_x) * S::TW);
  st.commit(tile);
  lds_barrier();

  float f[K][K];
  load_filter<K>(F, m_begin, f);
  for (int t = wg; t < ntiles; t += nwg) {
    const int y0 = (t / tiles_x) * S::TH;
    const int x0 = (t % tiles_x) * S::TW;
    const int tn = t + nwg;
    const bool more = tn < ntiles;
    if (more) st.fetch(I, Wx, Wy, (tn / tiles_x) * S::TH, (tn % tiles_x) * S::TW);

    for (int m = m_begin; m < m_end; ++m) {
      if (m != m_begin) load_filter<K>(F, m, f);
      apply_filter<K, R, NT, L>(rowp, f, O + (size_t)m * Hout * Wout, y0 + row0,
                                x0 + cq * kW, Hout, Wout);
    }
    if (m_end - m_begin > 1) load_filter<K>(F, m_begin, f);

    lds_barrier();  // every wave is done reading this tile
    if (more) st.commit(tile);
    lds_barrier();  // the next tile is in LDS
  }
}

// ---------------------------------------------------------------------------
// Matrix-core variant: banded filter rows on v_mfma_f32_4x4x1f32
// ---------------------------------------------------------------------------
// The instruction runs 16 independent 4x4 outer products per wave: lane
// 4b + i supplies A[b][i], lane 4b + j supplies B[b][j], and lane 4b + j
// receives D[b][i][j] in its register i.  Block b is a 4 x 4 output patch:
// D[b][i][j] = O[y_b + j][x_b + i].  For filter row r, step t adds
// A[i] * B[j] with A[i] = F[r][t - i] (zero outside 0..K-1) and
// B[j] = I[y_b + j + r][x_b + t]; the K + 3 steps t = 0..K+2 of a row add
// each of its K taps to all 16 outputs, so K of every K + 3 products are
// useful (79% at K = 11).  A is the same for every block: a banded copy of
// the filter, K x (K + 3) values per lane, held in accumulation registers
// (the instruction reads its A operand from them directly).
//
// Sixteen blocks side by side make a 4-row x 64-column patch, and a wave
// owns a column of P = 4 patches (16 rows x 64 columns; the four waves of a
// workgroup make a 16 x 256 tile).  It streams the
// input rows of that column through registers once: lane 4b + j holds
// input row u + j (four steps t at a time, one 16-byte LDS read), which is
// row j + r of patch p for r = u - 4p, so one read feeds every patch with
// 0 <= u - 4p < K (about K / 4 independent accumulation chains at once).

template <int K>
struct MfmaTileShape {
  static constexpr int P = 4;                   // patches (4 rows each) per wave column
  static constexpr int TH = 4 * P;              // output rows per tile
  static constexpr int IH = TH + K - 1;
  static constexpr int NT = K + 3;              // steps per filter row
  static constexpr int NQ = (NT + 3) / 4;       // 16-byte reads per input row
  static constexpr int IW4 = kLanes + NQ - 1;   // float4 staged per row (256 + K - 1 floats used)
  // Row stride = 2 (mod 8) float4: the 8 lanes (2 blocks x 4 rows) of one
  // 128-byte LDS access then touch 8 different 16-byte bank groups.
  static constexpr int LW4 = IW4 + (10 - IW4 % 8) % 8;
  static constexpr int BUF4 = IH * LW4;         // one tile buffer, float4
  static constexpr int LDS = 2 * BUF4 * 16 + 4 * K * NT * 4;
};

// Two workgroups per compute unit (the two tile buffers and the band fit
// twice in LDS; accumulators, band and input rows in 2 x 128 registers).
template <int K> struct MfmaOcc { static constexpr int value = 2; };

typedef float mf4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void *lds_ptr;

// Direct global->LDS copy of 16 bytes per lane: lane l's float4 from `src`
// lands at dst + l (dst is wave-uniform).
__device__ __forceinline__ void dma_f128(const float *src, float4 *dst) {
  __builtin_amdgcn_global_load_lds(src, (lds_ptr)dst, 16, 0, 0);
}

// The A operands of filter m: every thread stages its share of the banded
// table band[i][r][t] = F[m][r][t - i] in LDS, then each lane copies row
// i = lane % 4 into registers.  Two barriers; the caller must not be
// reading `band` (a K x (K + 3) x 4 float LDS array).
template <int K>
__device__ __forceinline__ void load_band(const float *__restrict__ F, int m, int lane,
                                          float *band, float (&a)[K][K + 3]) {
  constexpr int NT = K + 3;
  constexpr int P = MfmaTileShape<K>::P;
  const float *Fm = F + (size_t)m * K * K;
  for (int idx = threadIdx.x; idx < 4 * K * NT; idx += kBlock) {
    const int t = idx % NT;
    const int r = (idx / NT) % K;
    const int s = t - idx / (K * NT);
    band[idx] = (s >= 0 && s < K) ? Fm[r * K + s] : 0.f;
  }
  __syncthreads();
  const float *row = band + (lane & 3) * K * NT;
#pragma unroll
  for (int r = 0; r < K; ++r)
#pragma unroll
    for (int t = 0; t < NT; ++t) a[r][t] = row[r * NT + t];
  // The first KA rows go to accumulation registers, the rest to ordinary
  // vector registers (the instruction takes A from either): with the patch
  // accumulators that keeps each file within the 128 registers a wave has
  // when two workgroups share a compute unit.
  constexpr int KA = (128 - 8 * P) / NT < K ? (128 - 8 * P) / NT : K;
#pragma unroll
  for (int r = 0; r < K; ++r)
#pragma unroll
    for (int t = 0; t < NT; ++t) {
      if (r < KA)
        asm volatile("" : "+a"(a[r][t]));
      else
        asm volatile("" : "+v"(a[r][t]));
    }
  __syncthreads();
}

// Stage the tile at (y0, x0) into `buf` with direct global->LDS copies (no
// registers): wave w copies rows w, w + 4, ...  Rows and columns past the
// map re-read its last row / last float4; they feed only outputs that are
// never stored.
template <int K>
__device__ __forceinline__ void stage_tile(const float *__restrict__ I, int Wx, int Wy, int y0,
                                           int x0, float4 *buf, int wave, int lane) {
  using S = MfmaTileShape<K>;
  for (int row = wave; row < S::IH; row += kWaves) {
    const float *srow = I + (size_t)min(y0 + row, Wy - 1) * Wx;
#pragma unroll
    for (int c = 0; c < S::IW4; c += kLanes) {
      const int ix = c + lane;
      if (c + kLanes <= S::IW4 || ix < S::IW4)
        dma_f128(srow + min(x0 + 4 * ix, Wx - 4), buf + row * S::LW4 + c);
    }
  }
}

template <int K>
__global__ __launch_bounds__(kBlock, (MfmaOcc<K>::value)) void single_mfma(
    const float *__restrict__ I, const float *__restrict__ F, float *__restrict__ O,
    int Wx, int Wy, int M, int tiles_x, int ntiles, int m_per_block) {
  using S = MfmaTileShape<K>;
  constexpr int NT = S::NT, NQ = S::NQ, LW4 = S::LW4, P = S::P;
  // Two tile buffers as separate LDS objects (see the loop below).
  __shared__ float4 tile0[S::BUF4];
  __shared__ float4 tile1[S::BUF4];
  __shared__ float band[4 * K * NT];
  DCONV_POISON(poison_lds(tile0, S::BUF4), poison_lds(tile1, S::BUF4),
               poison_lds(band, 4 * K * NT));

  const int Hout = Wy - K + 1;
  const int Wout = Wx - K + 1;
  const int nwg = gridDim.x;
  const int wg = xcd_remap(blockIdx.x, nwg);
  if (wg >= ntiles) return;
  const int m_begin = blockIdx.y * m_per_block;
  const int m_end = min(M, m_begin + m_per_block);

  const int lane = threadIdx.x & (kLanes - 1);
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x / kLanes);
  const int blk = lane >> 2;   // block: output columns 4 * blk .. +3 of a patch
  const int q4 = lane & 3;     // output row of the lane (B, D roles)

  float a[K][NT];
  load_band<K>(F, m_begin, lane, band, a);
  stage_tile<K>(I, Wx, Wy, (wg / tiles_x) * S::TH, (wg % tiles_x) * kTileW, tile0, wave, lane);
  // One tile: wait for its copies, start the next tile's copies into the
  // other buffer, compute.  The wait is the compiler's own instruction (not
  // inline assembly), so it knows every copy has landed; and since the two
  // buffers are distinct LDS objects fixed at compile time in each call, it
  // can tell that the copies just started cannot alias this tile's reads and
  // adds no wait for them before the compute (with one array indexed at run
  // time it waited for all copies in flight, serialising copy and compute).
  auto step = [&](int t, const float4 *tile, float4 *next) {
    const int y0 = (t / tiles_x) * S::TH;
    const int x0 = (t % tiles_x) * kTileW;
    // Tile t is in `tile` once this wave's copies (and stores) have
    // completed and every wave has passed the barrier; every wave is then
    // also done with `next`, which takes the next tile's copies while this
    // one is computed.
    __builtin_amdgcn_s_waitcnt(kWaitVmcnt0);
    lds_barrier();
    const int tn = t + nwg;
    if (tn < ntiles)
      stage_tile<K>(I, Wx, Wy, (tn / tiles_x) * S::TH, (tn % tiles_x) * kTileW, next, wave, lane);

    for (int m = m_begin; m < m_end; ++m) {
      if (m != m_begin) load_band<K>(F, m, lane, band, a);
      float *Om = O + (size_t)m * Hout * Wout;
      // Input rows u = 0 .. 4P + K - 5 of this wave's column (row u + j in
      // lane 4b + j); output patch p (rows 4p .. 4p + 3) takes row u with
      // filter row u - 4p and is stored after its last row, u = 4p + K - 1.
      constexpr int U = 4 * P + K - 4;
      const float4 *src = tile + q4 * LW4 + wave * 16 + blk;
      const int gx = x0 + 4 * (wave * 16 + blk);
      // Two accumulators per patch (even and odd steps t) keep at least two
      // independent chains in flight where only one patch takes a row.
      mf4 acc[P][2];
#pragma unroll
      for (int p = 0; p < P; ++p) acc[p][0] = acc[p][1] = (mf4){0.f, 0.f, 0.f, 0.f};
      float4 cb[NQ], nb[NQ];
#pragma unroll
      for (int q = 0; q < NQ; ++q) cb[q] = src[q];
#pragma unroll
      for (int u = 0; u < U; ++u) {
        if (u + 1 < U) {
#pragma unroll
          for (int q = 0; q < NQ; ++q) nb[q] = src[(u + 1) * LW4 + q];
        }
#pragma unroll
        for (int q = 0; q < NQ; ++q)
#pragma unroll
          for (int e = 0; e < 4; ++e) {
            if (4 * q + e >= NT) continue;
            const float bv = e == 0 ? cb[q].x : e == 1 ? cb[q].y : e == 2 ? cb[q].z : cb[q].w;
#pragma unroll
            for (int p = 0; p < P; ++p) {
              const int r = u - 4 * p;
              if (r >= 0 && r < K)
                acc[p][e & 1] = __builtin_amdgcn_mfma_f32_4x4x1f32(a[r][4 * q + e], bv,
                                                                   acc[p][e & 1], 0, 0, 0);
            }
          }
#pragma unroll
        for (int p = 0; p < P; ++p) {
          if (u != 4 * p + K - 1) continue;
          // Patch p is complete: this lane holds output row y0 + 4p + q4,
          // columns gx .. gx + 3.
          const int gy = y0 + 4 * p + q4;
          if (gy >= Hout) continue;
          float *orow = Om + (size_t)gy * Wout + gx;
          const mf4 v = acc[p][0] + acc[p][1];
          if (gx + 4 <= Wout) {
            __builtin_nontemporal_store((vf4u){v[0], v[1], v[2], v[3]},
                                        reinterpret_cast<vf4u *>(orow));
          } else {
#pragma unroll
            for (int w = 0; w < 4; ++w)
              if (gx + w < Wout) __builtin_nontemporal_store(v[w], orow + w);
          }
        }
#pragma unroll
        for (int p = 0; p < P; ++p) asm volatile("" : "+a"(acc[p][0]), "+a"(acc[p][1]));
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int q = 0; q < NQ; ++q) cb[q] = nb[q];
      }
    }
    if (m_end - m_begin > 1) load_band<K>(F, m_begin, lane, band, a);
  };
  for (int t = wg; t < ntiles; t += 2 * nwg) {
    step(t, tile0, tile1);
    if (t + nwg >= ntiles) break;
    step(t + nwg, tile1, tile0);
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

// Persistent workgroups: as many as fit on the chip at once.  Filters reuse
// the staged tile; they are split over workgroups only as far as needed to
// fill the chip when there are fewer tiles than slots (or into `force_splits`
// groups when that is given, for the candidate plans).
void plan_persistent(int Wx, int Wy, int K, int M, int num_cu, int th, int tw, int occupancy,
                     SinglePlan *p, int force_splits = 0) {
  const int Hout = Wy - K + 1, Wout = Wx - K + 1;
  p->tile_h = th;
  p->tile_w = tw;
  p->tiles_x = (Wout + tw - 1) / tw;
  p->tiles_y = (Hout + th - 1) / th;
  const int ntiles = p->tiles_x * p->tiles_y;
  const int slots = occupancy * num_cu;
  int splits = force_splits > 0 ? force_splits : (slots + ntiles - 1) / ntiles;
  if (splits > M) splits = M;
  if (splits < 1) splits = 1;
  p->m_per_block = (M + splits - 1) / splits;
  p->grid_z = (M + p->m_per_block - 1) / p->m_per_block;
  int per_split = slots / p->grid_z;
  if (per_split < 1) per_split = 1;
  p->grid = ntiles < per_split ? ntiles : per_split;
  p->block = kBlock;
}

template <int K, bool VEC4>
void plan_tiled(int Wx, int Wy, int M, int num_cu, SinglePlan *p) {
  constexpr int R = Rows<K, VEC4>::value;
  using S = TileShape<K, R>;
  p->kernel = VEC4 ? 0 : 2;
  p->rows = R;
  p->lanes = kLanes;
  if constexpr (VEC4 && K <= kNarrowMaxK) {
    // Narrow maps: lanes in row groups over 64-column tiles.
    if (Wx - K + 1 <= kNarrowMaxWout) {
      using SN = TileShape<K, R, kNarrowLanes>;
      p->lanes = kNarrowLanes;
      plan_persistent(Wx, Wy, K, M, num_cu, SN::TH, SN::TW, Occupancy<K, VEC4>::value, p);
      p->lds_bytes = SN::LDS;
      return;
    }
  }
  plan_persistent(Wx, Wy, K, M, num_cu, S::TH, S::TW, Occupancy<K, VEC4>::value, p);
  p->lds_bytes = S::LDS;
  if constexpr (R > kShortRows) {
    // Fewer tall tiles than compute units (a small map with few filters):
    // short tiles, twice as many (1024 x 1024, K = 7, M = 1: 128 tall tiles
    // left half the chip idle).
    if ((int64_t)p->tiles_x * p->tiles_y * p->grid_z < num_cu) {
      using SS = TileShape<K, kShortRows>;
      p->rows = kShortRows;
      plan_persistent(Wx, Wy, K, M, num_cu, SS::TH, SS::TW, Occupancy<K, VEC4>::value, p);
      p->lds_bytes = SS::LDS;
    }
  }
}

// Matrix-core kernels exist for K = kMfmaMinK .. kMaxTiledK.
constexpr int kMfmaMinK = 5;

template <int K>
void plan_mfma(int Wx, int Wy, int M, int num_cu, SinglePlan *p) {
  using S = MfmaTileShape<K>;
  p->kernel = 3;
  p->rows = 8;
  plan_persistent(Wx, Wy, K, M, num_cu, S::TH, kTileW, MfmaOcc<K>::value, p);
  p->lds_bytes = S::LDS;
}

// Non-temporal output stores, except where rows of O do not start on
// 16-byte boundaries, each workgroup writes four or more filters per tile
// and the output is larger than the L2s together: there ordinary stores,
// which L2 merges into whole lines, measured faster (1024 x 1024 map, K = 3,
// 32 filters: 31.6 vs 39.7 us; 2048 x 2048, 4 filters: 15.4 vs 19.1 us).
// With one or two filters per workgroup or aligned rows the non-temporal
// stores are as fast or faster (4096 x 4096, K = 3, M = 1: 22.3 vs 26.3 us),
// and on small outputs (112 x 112, 128 filters) slightly faster.  The
// ordinary-store kernels exist for K <= kTemporalMaxK (the filter sizes of
// the many-filter layers).
constexpr int kTemporalMaxK = 5;
constexpr int64_t kTemporalMinBytes = 32ll << 20;
bool use_nt_stores(const SinglePlan &p, const float *O, int Wx, int Wy, int M) {
  const int Hout = Wy - p.K + 1, Wout = Wx - p.K + 1;
  const bool aligned_rows = Wout % 4 == 0 && (reinterpret_cast<uintptr_t>(O) & 15) == 0;
  const int64_t out_bytes = (int64_t)M * Hout * Wout * 4;
  return aligned_rows || p.m_per_block < 4 || p.K > kTemporalMaxK ||
         out_bytes < kTemporalMinBytes;
}

template <int K, bool VEC4, int R>
void launch_vector(const SinglePlan &p, const float *I, const float *F, float *O, int Wx, int Wy,
                   int M, bool nt, hipStream_t s) {
  const int ntiles = p.tiles_x * p.tiles_y;
  if constexpr (VEC4 && K <= kNarrowMaxK) {
    if (p.lanes == kNarrowLanes) {
      hipLaunchKernelGGL((single_tiled<K, R, VEC4, true, kNarrowLanes>), dim3(p.grid, p.grid_z),
                         dim3(kBlock), 0, s, I, F, O, Wx, Wy, M, p.tiles_x, ntiles,
                         p.m_per_block);
      return;
    }
  }
  if constexpr (K <= kTemporalMaxK) {
    if (!nt) {
      hipLaunchKernelGGL((single_tiled<K, R, VEC4, false, kLanes>), dim3(p.grid, p.grid_z),
                         dim3(kBlock), 0, s, I, F, O, Wx, Wy, M, p.tiles_x, ntiles,
                         p.m_per_block);
      return;
    }
  }
  hipLaunchKernelGGL((single_tiled<K, R, VEC4, true, kLanes>), dim3(p.grid, p.grid_z),
                     dim3(kBlock), 0, s, I, F, O, Wx, Wy, M, p.tiles_x, ntiles, p.m_per_block);
}

template <int K>
hipError_t launch_tiled(const SinglePlan &p, const float *I, const float *F, float *O,
                        int Wx, int Wy, int M, hipStream_t s) {
  const int ntiles = p.tiles_x * p.tiles_y;
  if constexpr (K >= kMfmaMinK) {
    if (p.kernel == 3) {
      hipLaunchKernelGGL(single_mfma<K>, dim3(p.grid, p.grid_z), dim3(kBlock), 0, s, I, F, O, Wx,
                         Wy, M, p.tiles_x, ntiles, p.m_per_block);
      return hipGetLastError();
    }
  }
  const bool nt = use_nt_stores(p, O, Wx, Wy, M);
  constexpr int RA = Rows<K, true>::value, RU = Rows<K, false>::value;
  if (p.kernel == 0) {
    if (RA > kShortRows && p.rows == kShortRows)
      launch_vector<K, true, kShortRows>(p, I, F, O, Wx, Wy, M, nt, s);
    else
      launch_vector<K, true, RA>(p, I, F, O, Wx, Wy, M, nt, s);
  } else {
    if (RU > kShortRows && p.rows == kShortRows)
      launch_vector<K, false, kShortRows>(p, I, F, O, Wx, Wy, M, nt, s);
    else
      launch_vector<K, false, RU>(p, I, F, O, Wx, Wy, M, nt, s);
  }
  return hipGetLastError();
}

}  // namespace

int plan_single(int Wx, int Wy, int K, int M, int num_cu, bool aligned, int variant,
                SinglePlan *p) {
  *p = SinglePlan{};
  p->K = K;
  // 16-byte aligned rows: whole float4 staging loads.
  const bool vec4 = aligned && (Wx % 4 == 0);
  // The matrix-core kernel needs float4 staging.  On a 4096 x 4096 map it
  // is level with the vector kernel at K = 7 (ahead in a sequence of
  // launches of all filter sizes, behind in repeats of K = 7 alone) and
  // slower at K = 5 (31 vs 28 us), K = 9 (54 vs 47 us) and K = 11 (72 vs
  // 63 us), so the automatic choice takes it at K = 7 only.
  const bool can_mfma = vec4 && K >= kMfmaMinK && K <= kMaxTiledK;
  if (variant == DCONV_VARIANT_MFMA && !can_mfma) return DCONV_EUNSUPPORTED;
  const bool mfma =
      variant == DCONV_VARIANT_MFMA || (variant == DCONV_VARIANT_AUTO && can_mfma && K == 7);
  switch (K) {
#define DCONV_PLAN_K(k)                                              \
  case k:                                                            \
    if (mfma) plan_mfma<(k >= kMfmaMinK ? k : kMfmaMinK)>(Wx, Wy, M, num_cu, p); \
    else if (vec4) plan_tiled<k, true>(Wx, Wy, M, num_cu, p);        \
    else plan_tiled<k, false>(Wx, Wy, M, num_cu, p);                 \
    return DCONV_OK;
    DCONV_PLAN_K(1) DCONV_PLAN_K(2) DCONV_PLAN_K(3) DCONV_PLAN_K(4) DCONV_PLAN_K(5)
    DCONV_PLAN_K(6) DCONV_PLAN_K(7) DCONV_PLAN_K(8) DCONV_PLAN_K(9) DCONV_PLAN_K(10)
    DCONV_PLAN_K(11)
#undef DCONV_PLAN_K
    default:
      break;
  }
  const int64_t total = (int64_t)M * (Wy - K + 1) * (Wx - K + 1);
  p->kernel = 1;  // generic
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
  return DCONV_OK;
}

namespace {

// The filter divisions tried for one tile shape: 1, 2, 4, ... groups up to
// M, M itself, and the planner's own (enough groups to fill the chip).
void add_splits(int Wx, int Wy, int K, int M, int num_cu, int occupancy, const SinglePlan &base,
                std::vector<SinglePlan> &out) {
  const int Hout = Wy - K + 1, Wout = Wx - K + 1;
  const int ntiles = ((Wout + base.tile_w - 1) / base.tile_w) * ((Hout + base.tile_h - 1) / base.tile_h);
  const int slots = occupancy * num_cu;
  std::vector<int> splits;
  for (int s = 1; s < M; s *= 2) splits.push_back(s);
  splits.push_back(M);
  splits.push_back((slots + ntiles - 1) / ntiles);
  const size_t first = out.size();
  for (int s : splits) {
    SinglePlan p = base;
    plan_persistent(Wx, Wy, K, M, num_cu, base.tile_h, base.tile_w, occupancy, &p, s);
    bool dup = false;
    for (size_t i = first; i < out.size(); ++i)
      dup = dup || (out[i].m_per_block == p.m_per_block && out[i].grid == p.grid &&
                    out[i].grid_z == p.grid_z);
    if (!dup) out.push_back(p);
  }
}

template <int K, bool VEC4>
void tiled_candidates(int Wx, int Wy, int M, int num_cu, std::vector<SinglePlan> &out) {
  constexpr int RA = Rows<K, VEC4>::value;
  constexpr int OCC = Occupancy<K, VEC4>::value;
  SinglePlan b{};
  b.kernel = VEC4 ? 0 : 2;
  b.K = K;
  b.block = kBlock;
  // tall (or the only) tiles
  b.rows = RA;
  b.lanes = kLanes;
  b.tile_h = TileShape<K, RA>::TH;
  b.tile_w = TileShape<K, RA>::TW;
  b.lds_bytes = TileShape<K, RA>::LDS;
  add_splits(Wx, Wy, K, M, num_cu, OCC, b, out);
  if constexpr (RA > kShortRows) {
    b.rows = kShortRows;
    b.tile_h = TileShape<K, kShortRows>::TH;
    b.tile_w = TileShape<K, kShortRows>::TW;
    b.lds_bytes = TileShape<K, kShortRows>::LDS;
    add_splits(Wx, Wy, K, M, num_cu, OCC, b, out);
  }
  if constexpr (VEC4 && K <= kNarrowMaxK) {
    using SN = TileShape<K, RA, kNarrowLanes>;
    b.rows = RA;
    b.lanes = kNarrowLanes;
    b.tile_h = SN::TH;
    b.tile_w = SN::TW;
    b.lds_bytes = SN::LDS;
    add_splits(Wx, Wy, K, M, num_cu, OCC, b, out);
  }
}

template <int K>
void mfma_candidates(int Wx, int Wy, int M, int num_cu, std::vector<SinglePlan> &out) {
  using S = MfmaTileShape<K>;
  SinglePlan b{};
  b.kernel = 3;
  b.K = K;
  b.rows = 8;
  b.lanes = kLanes;
  b.block = kBlock;
  b.tile_h = S::TH;
  b.tile_w = kTileW;
  b.lds_bytes = S::LDS;
  add_splits(Wx, Wy, K, M, num_cu, MfmaOcc<K>::value, b, out);
}

}  // namespace

int single_candidates(int Wx, int Wy, int K, int M, int num_cu, bool aligned, int variant,
                      std::vector<SinglePlan> &out) {
  out.clear();
  if (num_cu <= 0) num_cu = 256;
  const bool vec4 = aligned && (Wx % 4 == 0);
  const bool valu = variant != DCONV_VARIANT_MFMA;
  const bool mfma = variant != DCONV_VARIANT_VALU && vec4 && K >= kMfmaMinK && K <= kMaxTiledK;
  if (K > kMaxTiledK) {
    if (!valu) return DCONV_EUNSUPPORTED;
    SinglePlan p;
    plan_single(Wx, Wy, K, M, num_cu, aligned, DCONV_VARIANT_VALU, &p);
    out.push_back(p);
    return DCONV_OK;
  }
  switch (K) {
#define DCONV_CANDIDATES_K(k)                                                    \
  case k:                                                                        \
    if (valu) {                                                                  \
      if (vec4) tiled_candidates<k, true>(Wx, Wy, M, num_cu, out);               \
      else tiled_candidates<k, false>(Wx, Wy, M, num_cu, out);                   \
    }                                                                            \
    if (mfma) mfma_candidates<(k >= kMfmaMinK ? k : kMfmaMinK)>(Wx, Wy, M, num_cu, out); \
    break;
    DCONV_CANDIDATES_K(1) DCONV_CANDIDATES_K(2) DCONV_CANDIDATES_K(3) DCONV_CANDIDATES_K(4)
    DCONV_CANDIDATES_K(5) DCONV_CANDIDATES_K(6) DCONV_CANDIDATES_K(7) DCONV_CANDIDATES_K(8)
    DCONV_CANDIDATES_K(9) DCONV_CANDIDATES_K(10) DCONV_CANDIDATES_K(11)
#undef DCONV_CANDIDATES_K
    default:
      break;
  }
  return out.empty() ? DCONV_EUNSUPPORTED : DCONV_OK;
}

void export_single_plan(const SinglePlan &p, dconv_plan *out) {
  *out = dconv_plan{};
  out->variant = p.kernel == 3 ? DCONV_VARIANT_MFMA : DCONV_VARIANT_VALU;
  out->kernel = p.kernel;
  out->tile_m = p.m_per_block;
  out->tile_h = p.tile_h;
  out->tile_w = p.tile_w;
  out->chunk_c = 1;
  out->waves_c = 1;
  out->grid_x = p.grid;
  out->grid_y = p.grid_z;
  out->grid_z = 1;
  out->block = p.block;
  out->lds_bytes = p.lds_bytes;
}

hipError_t launch_single(const SinglePlan &p, const float *I, const float *F, float *O,
                         int Wx, int Wy, int M, hipStream_t s) {
  if (p.kernel == 1) {  // generic
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
