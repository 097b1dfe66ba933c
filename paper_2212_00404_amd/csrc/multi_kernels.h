// Multi-channel direct convolution (paper, Section 2.1, Eq. 1; Section 3.2):
// the kernels, their workgroup shapes and launch templates.  The planner and
// launch_multi are in multi.hip; the matrix-core kernels are instantiated
// per filter size in multi_mfma_k*.hip.
//
// C input maps I[C][Wy][Wx], M filters F[M][C][K][K], output O[M][Hout][Wout].
//
// Work division (Section 2.3 lists splitting along the filters m, along the
// map and along the channels): a workgroup owns a tile of filters x output
// pixels and sums over a range of channels.  Channels are consumed in stages
// of CC channels: the filter slice F[m0:m0+MT][c0:c0+CC] (MT contiguous runs
// of CC*K*K floats, the filter layout of Section 2.3) and the input halo tile
// I[c0:c0+CC][y0:y0+tpy+K-1][x0:x0+tpx+K-1] are staged in LDS, then reduced
// into register accumulators.  This is the role the paper's stride-fixed
// blocks play (a filter segment along the channel axis plus the map lines it
// needs), re-sized for gfx950's 160 KB LDS and 64-wide waves.
//
// Maps of 7x7 or 14x14 pixels give far fewer output tiles than the 256
// compute units.  As the paper does (Section 2.3 rejects dividing the channel
// sum over processors: extra global traffic and synchronisation), the sum
// stays inside one workgroup: small maps take small tiles (16 filters x 16
// pixels) and up to 16 waves per workgroup, each wave summing its own share
// of every stage's channels; the shares are added through LDS in a fixed
// order.  The library needs no device memory beyond the caller's tensors.
//
// Two inner products are provided:
//   * MFMA: the stage is an implicit GEMM  acc[m][p] += A[m][k] * B[k][p]
//     with A = filter slice and B = the im2col view of the staged input
//     (k = channel, filter row, filter column), fed to
//     v_mfma_f32_32x32x2_f32 (32 x 32 tiles; lanes 0-31 and 32-63 supply two
//     channels c, c+1 at one (r, s)) or v_mfma_f32_16x16x4_f32 (16 x 16
//     tiles; the four 16-lane groups supply channels c .. c+3).
//   * VALU: one output pixel per lane and MR filters per wave, with the
//     filter values wave-uniform in scalar registers and one fp32 FMA per
//     term (packed fp32 FMAs are not used).
#pragma once
#include <type_traits>
#include <utility>
#include <vector>

#include "internal.h"

namespace dconv {

struct TileArgs {
  int C, M, Wx, Wy;
  int tpy, tpx;       // output tile rows x cols
  int tiles_x;        // output tiles along x
  int ntiles;         // output tiles per map
  int mtiles;         // filter tiles
  int IH, IW, ICS;    // staged input tile rows, columns, channel stride
  long long *trace;   // stage-trace records (trace builds only; null otherwise)
};

// The launchers of the matrix-core kernels for one filter size each,
// compiled in separate translation units (multi_mfma_k*.hip).
#define DCONV_MFMA_LAUNCHER(K)                                                              \
  hipError_t launch_mfma_k##K(const MultiPlan &p, const float *I, const float *F, float *O, \
                              const TileArgs &a, hipStream_t st)
DCONV_MFMA_LAUNCHER(1);
DCONV_MFMA_LAUNCHER(2);
DCONV_MFMA_LAUNCHER(3);
DCONV_MFMA_LAUNCHER(4);
DCONV_MFMA_LAUNCHER(5);
DCONV_MFMA_LAUNCHER(6);
DCONV_MFMA_LAUNCHER(7);
DCONV_MFMA_LAUNCHER(8);
DCONV_MFMA_LAUNCHER(9);
DCONV_MFMA_LAUNCHER(10);
DCONV_MFMA_LAUNCHER(11);

namespace {

typedef float floatx16 __attribute__((ext_vector_type(16)));

constexpr int kBlock = 256;

// a * b for 0 <= a, b < 2^24 with a product below 2^32: one full-rate
// 24-bit multiply (a 32-bit one issues at a quarter of the rate).
__device__ __forceinline__ int mul24(int a, int b) { return (int)__umul24(a, b); }

// n / d for 0 <= n < 2^16 and 1 <= d < 2^16 using a float reciprocal inv
// within one ulp of 1/d (the hardware's approximate reciprocal, rcp(d)):
// the truncated product is then off by at most one, which the remainder
// test corrects.
__device__ __forceinline__ float rcp(int d) { return __builtin_amdgcn_rcpf((float)d); }
__device__ __forceinline__ int fdiv(int n, int d, float inv) {
  int q = __float2int_rz((float)n * inv);
  int r = n - q * d;
  if (r >= d) { ++q; }
  if (r < 0) { --q; }
  return q;
}

// Stage input channels [c0, c0+CC) of rows [py0, py0+IH) and columns
// [px0, px0+IW) into Is[cl*ICS + iy*IW + ix]; zero outside the map or past
// c_end.  Consecutive threads take consecutive columns (coalesced rows), and
// each thread issues kBatch loads before its first LDS write so that they
// are in flight together.
__device__ __forceinline__ void stage_input(float *__restrict__ Is, const float *__restrict__ I,
                                            int CC, int c0, int c_end, int py0, int px0,
                                            int IH, int IW, int ICS, int Wx, int Wy) {
  constexpr int kBatch = 8;
  const int per_c = IH * IW;
  const int total = CC * per_c;
  const float inv_pc = rcp(per_c);
  const float inv_iw = rcp(IW);
  for (int base = threadIdx.x; base < total; base += kBlock * kBatch) {
    float v[kBatch];
    int dst[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j) {
      const int idx = base + j * kBlock;
      v[j] = 0.f;
      dst[j] = -1;
      if (idx < total) {
        const int cl = fdiv(idx, per_c, inv_pc);
        const int rem = idx - cl * per_c;
        const int iy = fdiv(rem, IW, inv_iw);
        const int ix = rem - iy * IW;
        const int c = c0 + cl;
        const int gy = py0 + iy;
        const int gx = px0 + ix;
        dst[j] = cl * ICS + rem;
        if (c < c_end && gy < Wy && gx < Wx) v[j] = I[((size_t)c * Wy + gy) * Wx + gx];
      }
    }
#pragma unroll
    for (int j = 0; j < kBatch; ++j)
      if (dst[j] >= 0) Is[dst[j]] = v[j];
  }
}


// Decompose the (remapped) linear block id into output tile and filter tile.
// Output tiles vary fastest, so workgroups sharing a filter slice run close
// together (and, after the remap, on one XCD's L2).
__device__ __forceinline__ void block_coords(const TileArgs &a, int &tile, int &mt) {
  const int b = xcd_remap(blockIdx.x, a.ntiles * a.mtiles);
  tile = b % a.ntiles;
  mt = b / a.ntiles;
}

// ---------------------------------------------------------------------------
// MFMA implicit-GEMM kernel
// ---------------------------------------------------------------------------
typedef __attribute__((address_space(3))) void *lds_void_ptr;

// Barrier for LDS hand-over inside a workgroup (waits for this wave's LDS
// operations, not for its outstanding global memory operations).
__device__ __forceinline__ void lds_barrier() {
  asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

// Wait until this wave's direct global->LDS loads have landed in LDS.
__device__ __forceinline__ void wait_lds_dma() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// Direct global->LDS copy of one float per lane (gfx950 global_load_lds):
// lane l of the wave writes lds_row[l]; lds_row must be wave-uniform.
__device__ __forceinline__ void dma_f32(const float *src, float *lds_row) {
  __builtin_amdgcn_global_load_lds(src, (lds_void_ptr)lds_row, 4, 0, 0);
}

// The same copies (4 bytes per lane, or 16: lane l's four floats land at
// lds[4l .. 4l+3], 4-byte alignment suffices for both sides) addressed as a
// wave-uniform base plus a 32-bit per-lane byte offset, with a constant byte
// offset OFF (0 <= OFF < 4096) added to both addresses: lane l copies 4 (16)
// bytes from base + voff + OFF to lds + OFF + 4l (16l).  This is one instruction with the base in scalar
// registers and the LDS address in M0 (shared by copies that differ only
// in OFF): no 64-bit vector arithmetic per copy.  The empty asm statement
// keeps the offset a 32-bit value at its use, so the scalar-base form is
// selected.
template <int OFF>
__device__ __forceinline__ void dma_f32_at(const float *base, uint32_t voff, float *lds) {
  static_assert(OFF >= 0 && OFF < 4096, "immediate offset");
  asm volatile("" : "+v"(voff));
  __builtin_amdgcn_global_load_lds(
      reinterpret_cast<const float *>(reinterpret_cast<const char *>(base) + voff),
      (lds_void_ptr)lds, 4, OFF, 0);
}
template <int OFF>
__device__ __forceinline__ void dma_f128_at(const float *base, uint32_t voff, float *lds) {
  static_assert(OFF >= 0 && OFF < 4096, "immediate offset");
  asm volatile("" : "+v"(voff));
  __builtin_amdgcn_global_load_lds(
      reinterpret_cast<const float *>(reinterpret_cast<const char *>(base) + voff),
      (lds_void_ptr)lds, 16, OFF, 0);
}

constexpr int ceil_div(int a, int b) { return (a + b - 1) / b; }

// The two fp32 matrix instructions.  MF x MF output tile per instruction,
// KG lane groups each supplying one k value (lanes KG-group g = lane / MF,
// row / column = lane % MF), NV accumulator registers per lane.
template <int MF> struct Mfma;
template <> struct Mfma<32> {
  typedef float acc __attribute__((ext_vector_type(16)));
  static constexpr int KG = 2, NV = 16;
  static __device__ __forceinline__ acc mac(float a, float b, acc c) {
    return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
  }
  // Row (filter within the 32) held by accumulator register v of `lane`;
  // the column (pixel) is lane % 32.
  static __device__ __forceinline__ int row(int lane, int v) {
    return 8 * (v >> 2) + 4 * (lane >> 5) + (v & 3);
  }
};
template <> struct Mfma<16> {
  typedef float acc __attribute__((ext_vector_type(4)));
  static constexpr int KG = 4, NV = 4;
  static __device__ __forceinline__ acc mac(float a, float b, acc c) {
    return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
  }
  // Row held by register v of `lane`; the column is lane % 16.
  static __device__ __forceinline__ int row(int lane, int v) { return 4 * (lane >> 4) + v; }
};

// Staged geometry, in floats.
//  * Filter rows: FROW = CC*K*K values per filter, copied in 64-lane chunks;
//    row pitch FP = FROW rounded up to odd, so the lanes that read one
//    k-column of MF filters hit MF different banks.
//  * Input planes: ICS floats per channel = the largest (tpy+K-1)*(tpx+K-1)
//    over output tiles of at most PT pixels, K*(PT+K-1) (a 1 x PT or PT x 1
//    tile), rounded up to whole 64-lane chunks so a plane is copied with
//    unmasked chunks.  With 32x32 tiles, planes of at most 32 floats (K = 1,
//    32-pixel tiles) take 32, and one 64-lane copy then fills two channels.
//    With 16x16 tiles 16 floats are added, so that the lane groups reading
//    neighbouring channels in one half-wave start 16 banks apart.
constexpr int mfma_fp(int K, int CC) { return (CC * K * K) | 1; }
constexpr int mfma_ics(int K, int PT, int MF) {
  return MF == 32 && K * (PT + K - 1) <= 32 ? 32
                                             : 64 * ceil_div(K * (PT + K - 1), 64) + (MF == 16 ? 16 : 0);
}
// Filter rows are copied by the NW waves in blocks of MT/NW consecutive
// rows, each block followed by a 64-float gap (see the kernel's issue()).
constexpr int mfma_fblk(int K, int MT, int CC, int NW) { return (MT / NW) * mfma_fp(K, CC) + 64; }
constexpr int mfma_buf_floats(int K, int MT, int PT, int CC, int NW, int MF) {
  return NW * mfma_fblk(K, MT, CC, NW) + CC * mfma_ics(K, PT, MF);
}
// Channels per stage, a multiple of G = KG*WC (one k value per lane group of
// every wave group and k-step): the largest such count, at most 64, whose
// two stage buffers fit in 80 KB (two four-wave workgroups per CU; an
// eight-wave workgroup fills a CU's SIMDs with two waves each on its own,
// and longer stages measured no faster).
//   A deep shape instead takes the largest power-of-two multiple of G, up to
// 256 channels, whose two buffers fit in 160 KB (one workgroup per CU): for
// small tiles with little work per channel (K = 1, small maps), where each
// stage costs about one load latency whatever its size.
// Shapes that only split the channel sum (every wave covers the whole tile,
// WC waves): each wave stages its own channels in a region of its own, MT
// filter rows of CCW*K*K floats, then its CCW input planes; the stage sizes
// are multiples of 4*WC channels, so that a wave's filter rows are whole
// float4, and deep ones stop at 128 channels (the next stage's copies then
// overlap the current stage's MFMAs; 2-3% faster at K = 1 than one stage of
// 256).
// A wave's filter rows: CCW*K*K floats (a multiple of 4), at a pitch of an
// odd number of float4 so that the rows read together start in different
// banks.
constexpr int mfma_frwp(int FRW) { return (FRW / 4) % 2 == 1 ? FRW : FRW + 4; }
// The input part of a wave's region (PRIV): CCW planes of ICS floats, then
// room for the reads of never-stored pixels past the last plane (PT + 4
// floats; see the kernel).
constexpr int mfma_inreg(int K, int PT, int MF, int CCW) {
  return CCW * mfma_ics(K, PT, MF) + PT + 4;
}
// A wave's whole region, in floats: a multiple of 64 (256 bytes), so that
// every wave's copies land at the same alignment.
constexpr int mfma_rw(int K, int MT, int PT, int CCW, int MF) {
  return (MT * mfma_frwp(CCW * K * K) + mfma_inreg(K, PT, MF, CCW) + 63) / 64 * 64;
}
constexpr int mfma_buf_floats_priv(int K, int MT, int PT, int CC, int WC, int MF) {
  return WC * mfma_rw(K, MT, PT, CC / WC, MF);
}
constexpr int mfma_cc_priv(int K, int MT, int PT, int G, int WC, bool DEEP, int MF) {
  int best = G;
  if (DEEP) {
    for (int cc = G; cc <= 128; cc *= 2)
      if (2 * mfma_buf_floats_priv(K, MT, PT, cc, WC, MF) * 4 <= 160 * 1024) best = cc;
    return best;
  }
  for (int cc = G; cc <= 64; cc += G)
    if (2 * mfma_buf_floats_priv(K, MT, PT, cc, WC, MF) * 4 <= 80 * 1024) best = cc;
  return best;
}
constexpr int mfma_cc(int K, int MT, int PT, int G, int NW, bool DEEP, int MF) {
  int best = G;
  if (DEEP) {
    for (int cc = G; cc <= 256; cc *= 2)
      if (2 * mfma_buf_floats(K, MT, PT, cc, NW, MF) * 4 <= 160 * 1024) best = cc;
    return best;
  }
  for (int cc = G; cc <= 64; cc += G)
    if (2 * mfma_buf_floats(K, MT, PT, cc, NW, MF) * 4 <= 80 * 1024) best = cc;
  return best;
}

template <int K, int MF, int MB, int NB, int WM, int WN, int WC, bool DEEP>
struct MfmaCfg {
  static constexpr int KK = K * K;
  static constexpr int KG = Mfma<MF>::KG;
  static constexpr int NV = Mfma<MF>::NV;
  static constexpr int NW = WM * WN * WC;   // waves per workgroup
  static constexpr int MT = MF * MB * WM;   // filters per workgroup
  static constexpr int PT = MF * NB * WN;   // pixel lanes per workgroup tile
  // Each wave stages only the channels it sums (see the kernel)
  static constexpr bool PRIV = WM == 1 && WN == 1;
  static constexpr int CC = PRIV ? mfma_cc_priv(K, MT, PT, 4 * WC, WC, DEEP, MF)
                                 : mfma_cc(K, MT, PT, KG * WC, NW, DEEP, MF);  // channels per stage
  static constexpr int CCW = CC / WC;       // channels per wave group per stage
  static constexpr int FROW = CC * KK;      // staged floats per filter
  static constexpr int FP = mfma_fp(K, CC);
  static constexpr int NCF = ceil_div(FROW, 64);       // 64-lane chunks per filter row
  static constexpr int RPW = MT / NW;                  // filter rows copied per wave
  static constexpr int FBLK = mfma_fblk(K, MT, CC, NW);  // LDS stride of a wave's row block
  static constexpr int F_FLOATS = NW * FBLK;
  static constexpr int ICS = mfma_ics(K, PT, MF);
  static constexpr bool PAIR = ICS == 32;              // two input planes per 64-lane copy
  static constexpr int NCI = PAIR ? 1 : ICS / 64;      // most chunks an input plane needs
  // PRIV: a wave's region of RW floats in a stage buffer: MT filter rows of
  // FRW floats at pitch FRWP (FREG floats, copied as NF4W 16-byte chunks and
  // NTW 4-byte ones), then its CCW input planes
  static constexpr int FRW = CCW * KK;
  static constexpr int FRWP = mfma_frwp(FRW);          // row pitch
  static constexpr int FREG = MT * FRWP;
  static constexpr int NF4W = FREG / 256;
  static constexpr int NTW = ceil_div(FREG - 256 * NF4W, 64);
  // PRIV input copies: NC4 16-byte chunks, then NT4 4-byte ones (masked)
  static constexpr int NC4 = CCW * ICS / 256;
  static constexpr int NT4 = ceil_div(CCW * ICS - 256 * NC4, 64);
  static constexpr int RW = mfma_rw(K, MT, PT, CCW, MF);
  static constexpr int BUF = PRIV ? NW * RW : F_FLOATS + CC * ICS;      // one stage buffer
  static constexpr int ACC = NV * 64;                  // floats of one accumulator tile
  static constexpr int RED = (WC - 1) * WM * WN * MB * NB * ACC;
  static constexpr int BUF0 = BUF > RED ? BUF : RED;   // buffer 0 also holds the WC sums
  static constexpr int LDS_BYTES = (BUF0 + BUF) * 4;
  static_assert(NW == 4 || NW == 8 || NW == 16, "four, eight or sixteen waves per workgroup");
  static_assert(CCW % KG == 0, "each k-step takes one channel per lane group");
  static_assert(MT % NW == 0, "filter rows are shared out over the waves");
  static_assert(!PRIV || FRW % 4 == 0, "16-byte copies of a wave's filter rows");
};

// fn(integral_constant<int, B>), fn(... B + 1), ..., fn(... E - 1).
template <int B, int E, class Fn>
__device__ __forceinline__ void static_for(Fn &&fn) {
  if constexpr (B < E) {
    fn(std::integral_constant<int, B>{});
    static_for<B + 1, E>(fn);
  }
}



// Stage pipeline: while the MFMAs consume stage s from one LDS buffer, the
// filter slice and input tile of stage s+1 stream into the other buffer with
// direct global->LDS loads (no registers, no LDS write instructions).  The
// per-lane source offsets of a stage are fixed for the whole kernel, so a
// full stage of the shared layout is issued as unmasked 64-lane copies:
// lanes that fall outside the map or past a filter row are pointed at valid
// elements whose values only reach outputs that are never stored (or the
// padding of a row); the private layout below masks its 4-byte tail chunks.
//   Shapes that only split the channel sum (PRIV: WC waves each covering
// the whole tile) share nothing between waves: each wave copies only the
// channels it sums into a region of its own and waits only for its own
// copies, with no barrier between stages, so the waves drift apart and some
// issue copies while others run MFMAs (the shared stage's barrier made
// every wave wait for the slowest one's copies before any MFMA; on the
// benchmark layers most plans of these shapes run 5-30% faster so).  Such a
// wave issues the next stage's copies halfway through the current stage's
// MFMAs, not before them (a further 2% on average).
template <int K, int MF, int MB, int NB, int WM, int WN, int WC, bool DEEP>
__global__ __launch_bounds__(64 * WM * WN * WC) void multi_mfma(const float *__restrict__ I,
                                                               const float *__restrict__ F,
                                                               float *__restrict__ O, TileArgs a) {
  using Cfg = MfmaCfg<K, MF, MB, NB, WM, WN, WC, DEEP>;
#ifdef DCONV_STAGE_TRACE
  const long long tr_clock0 = clock64();
  const long long tr_wall0 = wall_clock64();
#endif
  using Op = Mfma<MF>;
  using acc_t = typename Op::acc;
  constexpr int KK = Cfg::KK, MT = Cfg::MT, CC = Cfg::CC, CCW = Cfg::CCW, FROW = Cfg::FROW;
  constexpr int FP = Cfg::FP, ICS = Cfg::ICS, F_FLOATS = Cfg::F_FLOATS;
  constexpr int NCF = Cfg::NCF, NCI = Cfg::NCI, RPW = Cfg::RPW, FBLK = Cfg::FBLK;
  constexpr int NW = Cfg::NW, NTHR = 64 * NW, KG = Cfg::KG, NV = Cfg::NV, ACC = Cfg::ACC;
  constexpr bool PAIR = Cfg::PAIR;
  __shared__ float buf0[Cfg::BUF0];
  __shared__ float buf1[Cfg::BUF];
  DCONV_POISON(poison_lds(buf0, Cfg::BUF0), poison_lds(buf1, Cfg::BUF));

  int tile, mt;
  block_coords(a, tile, mt);
  const int py0 = (tile / a.tiles_x) * a.tpy;
  const int px0 = (tile % a.tiles_x) * a.tpx;
  const int m0 = mt * MT;
  const int c_end = a.C;
  const int Hout = a.Wy - K + 1;
  const int Wout = a.Wx - K + 1;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wc = wave % WC;
  const int wmn = wave / WC;
  const int wm = wmn % WM;
  const int wn = wmn / WM;
  const int col = lane % MF;   // filter row of A / pixel of B this lane supplies
  // Stage trace (trace builds): lane 0 of wave 0 and of the last wave writes
  // the shader clock into word idx of its record.
  [[maybe_unused]] const int tr_sel = wave == 0 ? 0 : (wave == NW - 1 ? 1 : -1);
  auto mark = [&](int idx) __attribute__((always_inline)) {
#ifdef DCONV_STAGE_TRACE
    const long long t = clock64();
    if (a.trace && tr_sel >= 0 && lane == 0)
      a.trace[((size_t)blockIdx.x * 2 + tr_sel) * kStageTraceWords + idx] = t;
#else
    (void)idx;
#endif
  };
#ifdef DCONV_STAGE_TRACE
  if (a.trace && tr_sel >= 0 && lane == 0) {
    long long *rec = a.trace + ((size_t)blockIdx.x * 2 + tr_sel) * kStageTraceWords;
    rec[0] = tr_wall0;
    rec[1] = tr_clock0;
  }
#endif
  const int grp = lane / MF;   // which of the KG channels of a k-step

  constexpr bool PRIV = Cfg::PRIV;
  constexpr int RW = Cfg::RW, FRW = Cfg::FRW, FRWP = Cfg::FRWP, FREG = Cfg::FREG;
  constexpr int NF4W = Cfg::NF4W, NTW = Cfg::NTW;
  int a_base[MB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb) {
    const int row = wm * MF * MB + mb * MF + col;
    if constexpr (PRIV)
      a_base[mb] = wave * RW + row * FRWP + grp * KK;
    else
      a_base[mb] = (row / RPW) * FBLK + (row % RPW) * FP + (wc * CCW + grp) * KK;
  }
  // PRIV input planes (IN4: where the map is at least one padded row wide
  // and the tile's padded plane fits the plane stride): rows at pitch IWP
  // (IW rounded up to 4), copied 16 bytes per lane, staged from map column
  // sx, the tile's first column moved left so that no 16-byte read leaves
  // the map (the valid pixels' columns stay inside the staged window;
  // never-stored pixels may read past it, inside the wave's region).
  // Otherwise (and on the shared layout) rows at pitch IW from the tile's
  // first column, copied 4 bytes per lane.
  constexpr int NC4 = Cfg::NC4, NT4 = Cfg::NT4;
  const int IWP = (a.IW + 3) & ~3;
  const bool in4 = PRIV && a.Wx >= IWP && a.IH * IWP <= ICS && a.Wx * a.Wy < (1 << 24);
  const int ipitch = in4 ? IWP : a.IW;
  const int sx = in4 ? min(px0, a.Wx - IWP) : px0;
  // Divisions by run-time tile sizes through a float reciprocal (fdiv): the
  // integer division sequence costs tens of instructions per lane.
  const float inv_tpx = rcp(a.tpx);
  int b_base[NB];
  const int npix = a.tpy * a.tpx;
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int p = wn * MF * NB + nb * MF + col;
    int off = 0;  // padding lanes read pixel (0, 0); their results are dropped
    if (p < npix) {
      const int ty = fdiv(p, a.tpx, inv_tpx);
      off = mul24(ty, ipitch) + (p - mul24(ty, a.tpx)) + (px0 - sx);
    }
    if constexpr (PRIV)
      b_base[nb] = wave * RW + FREG + grp * ICS + off;
    else
      b_base[nb] = F_FLOATS + (wc * CCW + grp) * ICS + off;
  }
  // One input address per filter row r: every B read of a stage is then
  // b_row[nb][r] plus a compile-time offset (channel group and column).
  int b_row[NB][K];
#pragma unroll
  for (int nb = 0; nb < NB; ++nb)
#pragma unroll
    for (int r = 0; r < K; ++r) b_row[nb][r] = b_base[nb] + r * ipitch;

  // Per-lane source offsets of one input plane, chunk j covers plane elements
  // [64j, 64j+64): element e is row e / IW, column e % IW of the halo tile,
  // clamped into the map.  PAIR: one chunk covers two planes, lanes 0-31
  // element e = lane of the first and lanes 32-63 element lane - 32 of the
  // next channel (one map further).
  const int plane = a.IH * a.IW;
  const int nci = PAIR ? 1 : (plane + 63) >> 6;
  // (Not used by the 16-byte input copies of private stages.)
  int ioff[NCI];
  const float inv_iw = rcp(a.IW);
  if (!in4) {
#pragma unroll
    for (int j = 0; j < NCI; ++j) {
      int e = PAIR ? (lane & 31) : 64 * j + lane;
      if (e >= plane) e = 0;
      const int iy = fdiv(e, a.IW, inv_iw);
      const int gy = min(py0 + iy, a.Wy - 1);
      const int gx = min(px0 + (e - iy * a.IW), a.Wx - 1);
      ioff[j] = gy * a.Wx + gx;
    }
  } else {
#pragma unroll
    for (int j = 0; j < NCI; ++j) ioff[j] = 0;
  }
  // Filter rows.  Rows of at least 256 floats whose length is a multiple of
  // 4 (F128) start with NF4 16-byte-per-lane copies (1 KB per instruction,
  // about 1.6x the bytes per clock of 4-byte copies), chunk q covering row
  // elements [256q, 256q+256); the rest of a row, from T = 256 * NF4, goes in
  // NT 64-lane chunks of 4-byte copies.  The last chunk's lanes past FROW
  // land on the row's padding float or at position e of the next row's slot
  // and copy that row's element e (element 0 for a padding float): they
  // write what the next row's own copy writes, so the order of the two
  // copies does not matter.  For the last row of a wave's block they land
  // in the 64-float gap after the block and re-read the row's first
  // element.  Every copy runs on all 64 lanes (each lane picks its source),
  // with no branch around it.
  constexpr bool F128 = FROW % 4 == 0 && FROW >= 256;
  constexpr int NF4 = F128 ? FROW / 256 : 0;
  constexpr int T = 256 * NF4;
  constexpr int NT = ceil_div(FROW - T, 64);
  // The overhang stays within the next row's elements (short rows: the last
  // chunk is masked instead) and, for a block's last row, within the gap.
  constexpr bool FSPILL = T + 64 * NT <= FROW + FP;
  static_assert(T + 64 * NT <= FP + 64, "overhang of a block's last row fits the gap");
  const size_t plane_elems = (size_t)a.Wy * a.Wx;
  // PAIR: lanes 32-63 copy the next channel's plane
  const size_t pair_off = PAIR ? (size_t)(lane >> 5) * plane_elems : 0;
  const size_t frow_stride = (size_t)a.C * KK;
  const int e_last = T + 64 * (NT - 1) + lane;
  const bool f_spill = e_last >= FROW;
  int e_next = e_last - FP;
  if (e_next < 0 || e_next >= FROW) e_next = 0;
  // source of the last chunk relative to the row start: within a block
  // (times the row distance for the spilling lanes), and for its last row
  const int ofs_last = f_spill ? e_next : e_last;
  const int ofs_last_end = f_spill ? 0 : e_last;
  // The per-lane parts of every source address of a full stage, as 32-bit
  // byte offsets from a wave-uniform base (a filter row or an input plane):
  // each copy is then one instruction with a scalar base and no 64-bit
  // vector arithmetic.  The planner keeps C*K*K and Wx*Wy under 2^29, so
  // the offsets fit.
  const uint32_t vo4 = 4u * lane;
  const uint32_t vo16 = 16u * lane;
  const uint32_t vo_next = 4u * (uint32_t)(f_spill ? frow_stride + e_next : e_last);
  const uint32_t vo_same = 4u * (uint32_t)ofs_last;
  const uint32_t vo_end = 4u * (uint32_t)ofs_last_end;
  uint32_t vo_in[NCI];
#pragma unroll
  for (int j = 0; j < NCI; ++j) vo_in[j] = 4u * (uint32_t)(pair_off + ioff[j]);

  acc_t acc[MB][NB];
#pragma unroll
  for (int mb = 0; mb < MB; ++mb)
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
      for (int v = 0; v < NV; ++v) acc[mb][nb][v] = 0.f;

  // The copies of one full stage, as ND slots in a fixed order: the RPW
  // filter rows of this wave (SF copies each: NF4 16-byte chunks, NT - 1
  // plain 4-byte chunks, then the last chunk with its overhang), then the
  // input planes cl = wave, wave + NW, ... (PAIR: pairs from 2 * wave) in
  // NCI chunks each.
  //   Filter row r goes to buf[(r / RPW)*FBLK + (r % RPW)*FP + e], input
  // planes to buf[F_FLOATS + cl*ICS + e].  Rows past M (last filter tile
  // only) are clamped to filter M-1: they only feed outputs that are never
  // stored; a clamped row's spilling lanes re-read that same row, which is
  // also what the next slot holds.
  constexpr int SF = NF4 + NT;
  constexpr int ND_F = RPW * SF;
  constexpr int PL = PAIR ? ceil_div(CC, 2 * NW) : ceil_div(CC, NW);
  constexpr int ND = ND_F + PL * NCI;
  auto issue_slot = [&](int c0, float *buf, auto S) __attribute__((always_inline)) {
    constexpr int s = decltype(S)::value;
    if constexpr (s < ND_F) {
      constexpr int i = s / SF, q = s % SF;
      const int r = m0 + wave * RPW + i;
      const float *src = F + ((size_t)min(r, a.M - 1) * a.C + c0) * KK;
      float *dst = buf + wave * FBLK + i * FP;
      if constexpr (q < NF4 || q < SF - 1) {
        // chunk q starts at row element e; the copies of a row share a
        // base (and M0) per 4 KB of the row, the rest goes in the offset
        // (the last 4-byte chunk, which may spill into the next row, below)
        constexpr int e = q < NF4 ? 256 * q : T + 64 * (q - NF4);
        constexpr int g = e / 1024;
        if constexpr (q < NF4)
          dma_f128_at<4 * (e - 1024 * g)>(src + 1024 * g, vo16, dst + 1024 * g);
        else
          dma_f32_at<4 * (e - 1024 * g)>(src + 1024 * g, vo4, dst + 1024 * g);
      } else if constexpr (FSPILL) {
        // spilling lanes read the next row (the same row once r + 1 is
        // clamped to M - 1); a block's last row keeps them on its own start
        const uint32_t vo = i + 1 < RPW ? (r + 1 < a.M ? vo_next : vo_same) : vo_end;
        dma_f32_at<0>(src, vo, dst + T + 64 * (NT - 1));
      } else {
        if (!f_spill) dma_f32_at<0>(src, 4u * (uint32_t)e_last, dst + T + 64 * (NT - 1));
      }
    } else {
      constexpr int u = s - ND_F, t = u / NCI, jj = u % NCI;
      if constexpr (PAIR) {
        // channel pairs (cl, cl + 1), cl even; CC is even
        const int cl = 2 * wave + t * 2 * NW;
        if (cl < CC)
          dma_f32_at<0>(I + (size_t)(c0 + cl) * plane_elems, vo_in[0], buf + F_FLOATS + cl * ICS);
      } else {
        const int cl = wave + t * NW;
        if (cl < CC && jj < nci)
          dma_f32_at<0>(I + (size_t)(c0 + cl) * plane_elems, vo_in[jj],
                        buf + F_FLOATS + cl * ICS + 64 * jj);
      }
    }
  };
  auto issue_slots = [&](int c0, float *buf, auto B, auto E) __attribute__((always_inline)) {
    static_for<decltype(B)::value, decltype(E)::value>([&](auto S) { issue_slot(c0, buf, S); });
  };

  // Partial stage (the channel range ends inside it): copy the nc channels
  // present and zero the rest, which meet valid outputs.
  auto issue_partial = [&](int c0, float *buf) __attribute__((always_inline)) {
    const int nc = c_end - c0;
    const int flen = nc * KK;
    for (int i = 0; i < RPW; ++i) {
      const int r = wave * RPW + i;
      const float *src = F + ((size_t)min(m0 + r, a.M - 1) * a.C + c0) * KK + lane;
      float *dst = buf + wave * FBLK + i * FP;
      for (int q = 0; q < NCF; ++q)
        if (64 * q + lane < flen) dma_f32(src + 64 * q, dst + 64 * q);
    }
    if constexpr (PAIR) {
      // the second plane of the last pair only where that channel exists
      for (int cl = 2 * wave; cl < nc; cl += 2 * NW)
        if (cl + (lane >> 5) < nc)
          dma_f32(I + (size_t)(c0 + cl) * plane_elems + pair_off + ioff[0],
                  buf + F_FLOATS + cl * ICS);
    } else {
      for (int cl = wave; cl < nc; cl += NW) {
        const float *src = I + (size_t)(c0 + cl) * plane_elems;
        float *dst = buf + F_FLOATS + cl * ICS;
#pragma unroll
        for (int j = 0; j < NCI; ++j)
          if (j < nci) dma_f32(src + ioff[j], dst + 64 * j);
      }
    }
    const int fz = FROW - flen;
    for (int idx = threadIdx.x; idx < MT * fz; idx += NTHR) {
      const int r = idx / fz;
      buf[(r / RPW) * FBLK + (r % RPW) * FP + flen + (idx - r * fz)] = 0.f;
    }
    for (int idx = threadIdx.x; idx < (CC - nc) * ICS; idx += NTHR)
      buf[F_FLOATS + nc * ICS + idx] = 0.f;
  };
  // PRIV: per-lane offsets of this wave's filter copies, relative to filter
  // m0's first channel of the wave: 16-byte chunk j covers region floats
  // [256j, 256j+256), 4-byte chunk t floats [256*NF4W + 64t, +64) (lanes past
  // FREG masked off).  Rows past M are clamped to M-1.
  // (The planner keeps C*K*K below 2^24 for these shapes.)
  const int ckk = a.C * KK;
  uint32_t vf4[NF4W > 0 ? NF4W : 1];
  uint32_t vft[NTW > 0 ? NTW : 1];
  bool ft_ok[NTW > 0 ? NTW : 1];
  if constexpr (PRIV) {
#pragma unroll
    for (int j = 0; j < NF4W; ++j) {
      const int e = 256 * j + 4 * lane;
      const int row = e / FRWP;
      int eo = e - row * FRWP;
      if (eo >= FRW) eo = 0;  // the row's padding float4: any element of the row
      const int rr = min(m0 + row, a.M - 1) - m0;
      vf4[j] = 4u * (uint32_t)(mul24(rr, ckk) + eo);
    }
#pragma unroll
    for (int t = 0; t < NTW; ++t) {
      int e = 256 * NF4W + 64 * t + lane;
      ft_ok[t] = e < FREG;
      if (!ft_ok[t]) e = 0;
      const int row = e / FRWP;
      int eo = e - row * FRWP;
      if (eo >= FRW) eo = 0;
      const int rr = min(m0 + row, a.M - 1) - m0;
      vft[t] = 4u * (uint32_t)(mul24(rr, ckk) + eo);
    }
  }
  // PRIV, IN4: per-lane offsets of the input copies, relative to the wave's
  // first channel: 16-byte chunk j covers region floats [256j, 256j+256) of
  // the CCW planes (plane i at i*ICS, rows at pitch IWP), 4-byte chunk t
  // floats [256*NC4 + 64t, +64) (lanes past the planes masked off); lanes on
  // a plane's padding read plane 0's first element.  vpl4/vplt: the lane's
  // plane.  The planner keeps CCW*Wx*Wy below 2^30.
  uint32_t vin4[NC4 > 0 ? NC4 : 1], vint[NT4 > 0 ? NT4 : 1];
  int vpl4[NC4 > 0 ? NC4 : 1], vplt[NT4 > 0 ? NT4 : 1];
  bool it_ok[NT4 > 0 ? NT4 : 1];
  const float inv_iwp = rcp(IWP);
  const int plane_i = a.Wx * a.Wy;   // below 2^24 where IN4 holds
  auto in_src = [&](int e, uint32_t &vo, int &pl) __attribute__((always_inline)) {
    int i = e / ICS;
    const int pe = e - i * ICS;
    int row = fdiv(pe, IWP, inv_iwp);
    int cx = pe - mul24(row, IWP);
    if (i >= CCW || row >= a.IH) i = row = cx = 0;
    const int gy = min(py0 + row, a.Wy - 1);
    vo = 4u * (uint32_t)(mul24(i, plane_i) + mul24(gy, a.Wx) + sx + cx);
    pl = i;
  };
  if constexpr (PRIV) {
    if (in4) {
#pragma unroll
      for (int j = 0; j < NC4; ++j) in_src(256 * j + 4 * lane, vin4[j], vpl4[j]);
#pragma unroll
      for (int t = 0; t < NT4; ++t) {
        const int e = 256 * NC4 + 64 * t + lane;
        it_ok[t] = e < CCW * ICS;
        in_src(it_ok[t] ? e : 0, vint[t], vplt[t]);
      }
    }
  }
  // PRIV: this wave's channels [cw, cw + CCW) of the stage at c0 into its own
  // region of buf (channels past c_end zeroed).
  // IN4 is the run-time in4 as a compile-time constant: the stage loop is
  // instantiated once per copy form, so no branch on it sits between the
  // MFMAs.
  auto issue_priv = [&](int c0, float *buf, auto IN4) __attribute__((always_inline)) {
    constexpr bool use4 = decltype(IN4)::value;
    const int cw = c0 + wc * CCW;
    float *reg = buf + wave * RW;
    const int nc = min(CCW, c_end - cw);
    if (nc == CCW) {
      const float *fsrc = F + ((size_t)m0 * a.C + cw) * KK;
      static_for<0, NF4W>([&](auto J) {
        constexpr int j = decltype(J)::value;
        dma_f128_at<0>(fsrc, vf4[j], reg + 256 * j);
      });
      static_for<0, NTW>([&](auto TT) {
        constexpr int t = decltype(TT)::value;
        if (ft_ok[t]) dma_f32_at<0>(fsrc, vft[t], reg + 256 * NF4W + 64 * t);
      });
      if constexpr (use4) {
        static_for<0, NC4>([&](auto J) {
          constexpr int j = decltype(J)::value;
          dma_f128_at<0>(I + (size_t)cw * plane_elems, vin4[j], reg + FREG + 256 * j);
        });
        static_for<0, NT4>([&](auto TT) {
          constexpr int t = decltype(TT)::value;
          if (it_ok[t])
            dma_f32_at<0>(I + (size_t)cw * plane_elems, vint[t], reg + FREG + 256 * NC4 + 64 * t);
        });
      } else if constexpr (PAIR) {
#pragma unroll
        for (int i = 0; i < CCW; i += 2)
          dma_f32_at<0>(I + (size_t)(cw + i) * plane_elems, vo_in[0], reg + FREG + i * ICS);
      } else {
#pragma unroll
        for (int i = 0; i < CCW; ++i)
#pragma unroll
          for (int jj = 0; jj < NCI; ++jj)
            if (jj < nci)
              dma_f32_at<0>(I + (size_t)(cw + i) * plane_elems, vo_in[jj],
                            reg + FREG + i * ICS + 64 * jj);
      }
    } else {
      const int ncp = nc > 0 ? nc : 0;
      const int flen = ncp * KK;
      for (int row = 0; row < MT; ++row) {
        const float *src = F + ((size_t)min(m0 + row, a.M - 1) * a.C + cw) * KK;
        for (int e = lane; e < FRW; e += 64) {
          if (e < flen)
            dma_f32(src + e, reg + row * FRWP + (e - lane));
          else
            reg[row * FRWP + e] = 0.f;
        }
      }
      if (use4 && ncp > 0) {
        // planes past the last channel re-read channel cw + ncp - 1: their
        // filter values are zero, so they add nothing
        static_for<0, NC4>([&](auto J) {
          constexpr int j = decltype(J)::value;
          const int over = vpl4[j] - (ncp - 1);
          const uint32_t vo =
              over > 0 ? vin4[j] - 4u * (uint32_t)((size_t)over * plane_elems) : vin4[j];
          dma_f128_at<0>(I + (size_t)cw * plane_elems, vo, reg + FREG + 256 * j);
        });
        static_for<0, NT4>([&](auto TT) {
          constexpr int t = decltype(TT)::value;
          const int over = vplt[t] - (ncp - 1);
          const uint32_t vo =
              over > 0 ? vint[t] - 4u * (uint32_t)((size_t)over * plane_elems) : vint[t];
          if (it_ok[t]) dma_f32_at<0>(I + (size_t)cw * plane_elems, vo, reg + FREG + 256 * NC4 + 64 * t);
        });
      } else if constexpr (PAIR) {
        for (int i = 0; i < CCW; i += 2) {
          if (i + (lane >> 5) < ncp)
            dma_f32(I + (size_t)(cw + i) * plane_elems + pair_off + ioff[0], reg + FREG + i * ICS);
          else
            reg[FREG + i * ICS + lane] = 0.f;
        }
      } else {
        for (int i = 0; i < CCW; ++i) {
          if (i < ncp) {
            const float *src = I + (size_t)(cw + i) * plane_elems;
#pragma unroll
            for (int j = 0; j < NCI; ++j)
              if (j < nci) dma_f32(src + ioff[j], reg + FREG + i * ICS + 64 * j);
          } else {
            for (int e = lane; e < ICS; e += 64) reg[FREG + i * ICS + e] = 0.f;
          }
        }
      }
    }
  };
  // A whole stage at once (the first stages, and partial stages).
  auto issue = [&](int c0, float *buf, auto IN4) __attribute__((always_inline)) {
    if constexpr (PRIV)
      issue_priv(c0, buf, IN4);
    else if (c_end - c0 >= CC)
      issue_slots(c0, buf, std::integral_constant<int, 0>{}, std::integral_constant<int, ND>{});
    else
      issue_partial(c0, buf);
  };

  // The stage's k-steps (channel group cg, filter row r, filter column s) run
  // in NCH chunks of L with one chunk of operand look-ahead from LDS.  The
  // empty asm statements on the accumulators and the scheduling barriers
  // keep the compiler from hoisting every LDS read of the stage into
  // registers.  (Issuing the next stage's copies a few at a time between
  // these chunks instead of all before them measured 3-13% slower.)
  // `mid` runs halfway through the chunks (the private stages' copies).
  auto compute = [&](const float *buf, auto &&mid) __attribute__((always_inline)) {
    constexpr int NQ = (CCW / KG) * KK;
    // chunks of 3 where they divide the k-steps and 4 do not (K = 3): 0.5%
    // faster on average over the K = 3 plans
    constexpr int L = (NQ % 4 != 0 && NQ % 3 == 0) ? 3 : 4;
    constexpr int NCH = (NQ + L - 1) / L;
    float ca[L][MB], cb[L][NB], na[L][MB], nbv[L][NB];
    auto load_chunk = [&](int ch, float (&av)[L][MB], float (&bv)[L][NB]) {
#pragma unroll
      for (int l = 0; l < L; ++l) {
        const int q = ch * L + l;
        if (q < NQ) {
          const int cg = q / KK, r = (q % KK) / K, s = q % K;
#pragma unroll
          for (int mb = 0; mb < MB; ++mb) av[l][mb] = buf[a_base[mb] + KG * cg * KK + r * K + s];
#pragma unroll
          for (int nb = 0; nb < NB; ++nb) bv[l][nb] = buf[b_row[nb][r] + KG * cg * ICS + s];
        }
      }
    };
    load_chunk(0, ca, cb);
    static_for<0, NCH>([&](auto CH) {
      constexpr int ch = decltype(CH)::value;
      // The look-ahead reads are issued between the two halves of this
      // chunk's MFMAs: late enough that waiting for them at the start of the
      // next chunk costs nothing, early enough to be in flight for half a
      // chunk.  Scheduling barriers keep the order.
      if constexpr (ch == NCH / 2) {
        __builtin_amdgcn_sched_barrier(0);
        mid();
        __builtin_amdgcn_sched_barrier(0);
      }
#pragma unroll
      for (int l = 0; l < L; ++l) {
        if (l == L / 2) {
          __builtin_amdgcn_sched_barrier(0);
          if (ch + 1 < NCH) load_chunk(ch + 1, na, nbv);
          __builtin_amdgcn_sched_barrier(0);
        }
        if (ch * L + l < NQ) {
#pragma unroll
          for (int mb = 0; mb < MB; ++mb)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) acc[mb][nb] = Op::mac(ca[l][mb], cb[l][nb], acc[mb][nb]);
        }
      }
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) asm volatile("" : "+a"(acc[mb][nb]));
      __builtin_amdgcn_sched_barrier(0);
#pragma unroll
      for (int l = 0; l < L; ++l) {
#pragma unroll
        for (int mb = 0; mb < MB; ++mb) ca[l][mb] = na[l][mb];
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) cb[l][nb] = nbv[l][nb];
      }
    });
  };

  // Two stage buffers: while stage s is computed from one, the copies of
  // stage s+1 land in the other.  Before computing a stage, wait for this
  // wave's copies of it, then the barrier: every wave's copies have landed,
  // and every wave is done with the other buffer, which the next stage's
  // copies refill (PRIV: no barrier; a wave's own reads of the other buffer
  // completed in its previous stage).  Each buffer is named as the LDS object itself where it
  // is used (not a pointer chosen at run time), which is what lets the
  // compiler leave the copies to one buffer in flight while the other is
  // read.  (Tried and not kept, no faster on any layer: a third and a
  // fourth buffer; the copies of stage s+2 spread between the MFMA chunks
  // of stage s over three buffers; waves that only copy beside waves that
  // only compute; a stage order rotated per output tile.)
  auto stage = [&](auto J, int cs, auto IN4) __attribute__((always_inline)) {
    constexpr int j = decltype(J)::value;
    float *cur = j == 0 ? buf0 : buf1;
    float *nxt = j == 0 ? buf1 : buf0;
    const int st = cs / CC;
    const int tw = st < kStageTraceStages ? 6 + 5 * st : -1;
    if (tw >= 0) mark(tw);
    wait_lds_dma();
    if (tw >= 0) mark(tw + 1);
    if constexpr (!PRIV) lds_barrier();
    if (tw >= 0) mark(tw + 2);
    if constexpr (PRIV) {
      if (tw >= 0) mark(tw + 3);
      compute(cur, [&]() { if (cs + CC < c_end) issue(cs + CC, nxt, IN4); });
    } else {
      if (cs + CC < c_end) issue(cs + CC, nxt, IN4);
      if (tw >= 0) mark(tw + 3);
      compute(cur, []() {});
    }
    if (tw >= 0) mark(tw + 4);
  };
  auto run_stages = [&](auto IN4) __attribute__((always_inline)) {
    mark(2);
    issue(0, buf0, IN4);
    mark(3);
    for (int c0 = 0; c0 < c_end; c0 += 2 * CC) {
      stage(std::integral_constant<int, 0>{}, c0, IN4);
      if (c0 + CC >= c_end) break;
      stage(std::integral_constant<int, 1>{}, c0 + CC, IN4);
    }
  };
  if (PRIV && in4)
    run_stages(std::true_type{});
  else
    run_stages(std::false_type{});

  // Fixed-order sum of the WC channel groups through LDS: group 0 adds the
  // partial tiles of groups 1, 2, ..., WC-1 in that order.
  if constexpr (WC > 1) {
    float *red = buf0;
    lds_barrier();  // every wave is done with the stage buffers
    if (wc > 0) {
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int v = 0; v < NV; ++v)
            red[((((wc - 1) * WM * WN + wmn) * MB + mb) * NB + nb) * ACC + v * 64 + lane] =
                acc[mb][nb][v];
    }
    lds_barrier();
    if (wc != 0) return;
#pragma unroll
    for (int g = 1; g < WC; ++g)
#pragma unroll
      for (int mb = 0; mb < MB; ++mb)
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
          for (int v = 0; v < NV; ++v)
            acc[mb][nb][v] += red[((((g - 1) * WM * WN + wmn) * MB + mb) * NB + nb) * ACC + v * 64 + lane];
  }

  mark(4);
#ifdef DCONV_STAGE_TRACE
  if (a.trace && tr_sel >= 0 && lane == 0)
    a.trace[((size_t)blockIdx.x * 2 + tr_sel) * kStageTraceWords + 5] = wall_clock64();
#endif
#pragma unroll
  for (int nb = 0; nb < NB; ++nb) {
    const int p = wn * MF * NB + nb * MF + col;
    if (p >= npix) continue;
    const int ty = fdiv(p, a.tpx, inv_tpx);
    const int gy = py0 + ty;
    const int gx = px0 + (p - ty * a.tpx);
    if (gy >= Hout || gx >= Wout) continue;
    const size_t pix = (size_t)gy * Wout + gx;
#pragma unroll
    for (int mb = 0; mb < MB; ++mb)
#pragma unroll
      for (int v = 0; v < NV; ++v) {
        const int m = m0 + wm * MF * MB + mb * MF + Op::row(lane, v);
        if (m < a.M) O[(size_t)m * Hout * Wout + pix] = acc[mb][nb][v];
      }
  }
}

// ---------------------------------------------------------------------------
// VALU kernel: lane = output pixel, wave = MR filters, fp32 FMA per term
// ---------------------------------------------------------------------------
// KT > 0: compile-time filter size; KT == 0: any K (loops not unrolled).
template <int KT, int MR, int WC, int CC>
__global__ __launch_bounds__(kBlock) void multi_valu(const float *__restrict__ I,
                                                     const float *__restrict__ F,
                                                     float *__restrict__ O, TileArgs a,
                                                     int Krt) {
  constexpr int CCW = CC / WC;
  constexpr int WMV = 4 / WC;     // filter groups per workgroup
  constexpr int MT = MR * WMV;
  const int K = KT > 0 ? KT : Krt;
  const int KK = K * K;
  extern __shared__ float lds[];
  float *Is = lds;

  int tile, mt;
  block_coords(a, tile, mt);
  const int py0 = (tile / a.tiles_x) * a.tpy;
  const int px0 = (tile % a.tiles_x) * a.tpx;
  const int c_end = a.C;
  const int Hout = a.Wy - K + 1;
  const int Wout = a.Wx - K + 1;

  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
  const int wc = wave % WC;
  const int wm = wave / WC;
  const int mbase = mt * MT + wm * MR;

  const int npix = a.tpy * a.tpx;
  int boff = 0;
  if (lane < npix) {
    const int ty = lane / a.tpx;
    boff = ty * a.IW + (lane - ty * a.tpx);
  }

  // Filter rows read with wave-uniform addresses (scalar loads); filters past
  // M are clamped to M-1 and their results dropped.
  const float *Fm[MR];
#pragma unroll
  for (int mr = 0; mr < MR; ++mr) Fm[mr] = F + (size_t)min(mbase + mr, a.M - 1) * a.C * KK;

  float acc[MR];
#pragma unroll
  for (int mr = 0; mr < MR; ++mr) acc[mr] = 0.f;

  for (int c0 = 0; c0 < c_end; c0 += CC) {
    stage_input(Is, I, CC, c0, c_end, py0, px0, a.IH, a.IW, a.ICS, a.Wx, a.Wy);
    __syncthreads();
    for (int cl = wc * CCW; cl < (wc + 1) * CCW; ++cl) {
      const int c = min(c0 + cl, a.C - 1);  // staged input is zero past c_end
      const float *Ic = Is + cl * a.ICS + boff;
      if constexpr (KT > 0) {
#pragma unroll
        for (int r = 0; r < KT; ++r) {
          float f[MR][KT];
#pragma unroll
          for (int mr = 0; mr < MR; ++mr)
#pragma unroll
            for (int s = 0; s < KT; ++s) f[mr][s] = Fm[mr][(size_t)c * KK + r * KT + s];
#pragma unroll
          for (int s = 0; s < KT; ++s) {
            const float v = Ic[r * a.IW + s];
#pragma unroll
            for (int mr = 0; mr < MR; ++mr) acc[mr] = __builtin_fmaf(v, f[mr][s], acc[mr]);
          }
        }
      } else {
        for (int r = 0; r < K; ++r)
          for (int s = 0; s < K; ++s) {
            const float v = Ic[r * a.IW + s];
#pragma unroll
            for (int mr = 0; mr < MR; ++mr)
              acc[mr] = __builtin_fmaf(v, Fm[mr][(size_t)c * KK + r * K + s], acc[mr]);
          }
      }
    }
    __syncthreads();
  }

  if constexpr (WC > 1) {
    float *red = lds;
    if (wc > 0) {
#pragma unroll
      for (int mr = 0; mr < MR; ++mr) red[(((wc - 1) * WMV + wm) * MR + mr) * 64 + lane] = acc[mr];
    }
    __syncthreads();
    if (wc != 0) return;
#pragma unroll
    for (int g = 1; g < WC; ++g)
#pragma unroll
      for (int mr = 0; mr < MR; ++mr) acc[mr] += red[(((g - 1) * WMV + wm) * MR + mr) * 64 + lane];
  }

  if (lane >= npix) return;
  const int ty = lane / a.tpx;
  const int gy = py0 + ty;
  const int gx = px0 + (lane - ty * a.tpx);
  if (gy >= Hout || gx >= Wout) return;
  const size_t pix = (size_t)gy * Wout + gx;
#pragma unroll
  for (int mr = 0; mr < MR; ++mr)
    if (mbase + mr < a.M) O[(size_t)(mbase + mr) * Hout * Wout + pix] = acc[mr];
}

// Any size: one output per thread, operands read through the caches.  Used
// when no tiled kernel's LDS footprint fits (very large filters).
__global__ __launch_bounds__(256) void multi_generic(const float *__restrict__ I,
                                                     const float *__restrict__ F,
                                                     float *__restrict__ O, int C, int M, int Wx,
                                                     int Wy, int K) {
  const int Hout = Wy - K + 1;
  const int Wout = Wx - K + 1;
  const int64_t total = (int64_t)M * Hout * Wout;
  const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (idx >= total) return;
  const int x = (int)(idx % Wout);
  const int64_t my = idx / Wout;
  const int y = (int)(my % Hout);
  const int m = (int)(my / Hout);
  float acc = 0.f;
  for (int c = 0; c < C; ++c) {
    const float *Fc = F + ((int64_t)m * C + c) * K * K;
    for (int r = 0; r < K; ++r) {
      const float *irow = I + ((int64_t)c * Wy + y + r) * Wx + x;
      for (int s = 0; s < K; ++s) acc = __builtin_fmaf(irow[s], Fc[r * K + s], acc);
    }
  }
  O[idx] = acc;
}

// Dynamic LDS per workgroup the planner may request (gfx950: 160 KB per CU).
constexpr int kMaxLds = 160 * 1024;

// Kernels are allowed the full LDS once per instance, before their first
// launch (thread-safe static initialisation).
template <typename Kern>
hipError_t allow_full_lds(Kern kern) {
  static const hipError_t e = hipFuncSetAttribute(
      reinterpret_cast<const void *>(kern), hipFuncAttributeMaxDynamicSharedMemorySize, kMaxLds);
  return e;
}

// ---------------------------------------------------------------------------
// Kernel table
// ---------------------------------------------------------------------------
// Each family has a few workgroup shapes; the planner picks one per call.
// MF: 32 (v_mfma_f32_32x32x2_f32) or 16 (v_mfma_f32_16x16x4_f32) tiles.
struct MfmaShape { int MF, MB, NB, WM, WN, WC; bool deep; };
constexpr MfmaShape kMfmaShapes[] = {
    {32, 1, 1, 2, 1, 2, false},  // 64 filters x 32 pixels, channel sum split over 2 wave pairs
    {32, 1, 2, 1, 2, 2, false},  // 32 x 128, channel sum split over 2 wave pairs
    {32, 1, 1, 2, 2, 1, false},  // 64 x 64
    {32, 1, 2, 2, 2, 1, false},  // 64 x 128
    {32, 2, 2, 2, 2, 1, false},  // 128 x 128
    {32, 1, 2, 1, 1, 4, false},  // 32 x 64, channel sum split over 4 waves
    {32, 1, 1, 2, 2, 2, false},  // 64 x 64, eight waves, channel sum split over 2 wave groups
    {32, 1, 1, 2, 4, 1, false},  // 64 x 128, eight waves
    {32, 1, 1, 1, 1, 4, true},   // 32 x 32, channel sum split over 4 waves, deep stages
    {32, 1, 1, 1, 1, 8, true},   // 32 x 32, eight waves splitting the channel sum, deep stages
    {16, 1, 1, 1, 1, 16, true},  // 16 x 16, sixteen waves splitting the channel sum, deep stages
    {16, 1, 1, 1, 1, 8, false},  // 16 x 16, eight waves splitting the channel sum
    {16, 1, 1, 1, 1, 4, false},  // 16 x 16, four waves splitting the channel sum
    {16, 1, 1, 2, 1, 4, false},  // 32 x 16, eight waves (four per 16 filters)
    {16, 1, 1, 1, 2, 4, false},  // 16 x 32, eight waves (four per 16 pixels)
    {16, 1, 2, 1, 1, 8, false},  // 16 x 32, eight waves splitting the channel sum
};
constexpr int kNumMfma = sizeof(kMfmaShapes) / sizeof(kMfmaShapes[0]);

struct ValuShape { int MR, WC, CC; };
constexpr ValuShape kValuShapes[] = {
    {8, 4, 16},  // 8 filters x 64 pixels, channel sum split over 4 waves
    {8, 1, 8},   // 32 filters x 64 pixels
};
constexpr int kNumValu = sizeof(kValuShapes) / sizeof(kValuShapes[0]);

template <int K, int S>
using ShapeCfg = MfmaCfg<K, kMfmaShapes[S].MF, kMfmaShapes[S].MB, kMfmaShapes[S].NB,
                         kMfmaShapes[S].WM, kMfmaShapes[S].WN, kMfmaShapes[S].WC,
                         kMfmaShapes[S].deep>;

template <int K, int S>
hipError_t launch_mfma_shape(const MultiPlan &p, const float *I, const float *F, float *O,
                             const TileArgs &a, hipStream_t st) {
  constexpr MfmaShape sh = kMfmaShapes[S];
  // Shapes whose stage buffers exceed the LDS for this K are never planned
  // (the candidate list drops them) and are not instantiated.
  if constexpr (ShapeCfg<K, S>::LDS_BYTES > kMaxLds) {
    return hipErrorInvalidValue;
  } else {
    auto kern = multi_mfma<K, sh.MF, sh.MB, sh.NB, sh.WM, sh.WN, sh.WC, sh.deep>;
    hipLaunchKernelGGL(kern, dim3(p.grid_x), dim3(64 * sh.WM * sh.WN * sh.WC), 0, st, I, F, O, a);
    return hipGetLastError();
  }
}

template <int K, int... S>
hipError_t launch_mfma_k(const MultiPlan &p, const float *I, const float *F, float *O,
                         const TileArgs &a, hipStream_t st, std::integer_sequence<int, S...>) {
  hipError_t e = hipErrorInvalidValue;
  ((p.kernel == S ? (e = launch_mfma_shape<K, S>(p, I, F, O, a, st), 0) : 0), ...);
  return e;
}

template <int K>
hipError_t launch_mfma_k(const MultiPlan &p, const float *I, const float *F, float *O,
                         const TileArgs &a, hipStream_t st) {
  return launch_mfma_k<K>(p, I, F, O, a, st, std::make_integer_sequence<int, kNumMfma>{});
}

template <int KT, int S>
hipError_t launch_valu_shape(const MultiPlan &p, const float *I, const float *F, float *O,
                             const TileArgs &a, hipStream_t st) {
  constexpr ValuShape sh = kValuShapes[S];
  auto kern = multi_valu<KT, sh.MR, sh.WC, sh.CC>;
  if (hipError_t e = allow_full_lds(kern); e != hipSuccess) return e;
  hipLaunchKernelGGL(kern, dim3(p.grid_x), dim3(kBlock), p.lds_bytes, st, I, F, O, a, p.K);
  return hipGetLastError();
}

template <int KT>
hipError_t launch_valu_k(const MultiPlan &p, const float *I, const float *F, float *O,
                         const TileArgs &a, hipStream_t st) {
  switch (p.kernel) {
    case 0: return launch_valu_shape<KT, 0>(p, I, F, O, a, st);
    case 1: return launch_valu_shape<KT, 1>(p, I, F, O, a, st);
    default: return hipErrorInvalidValue;
  }
}

}  // namespace
}  // namespace dconv
