// Multi-channel direct convolution: the planner (workgroup shape, output
// tile, channels per stage, time model) and launch_multi (paper, Section 3.2).
#include <algorithm>
#include <cmath>
#include <vector>

#include "multi_kernels.h"

namespace dconv {
#ifdef DCONV_STAGE_TRACE
long long *g_stage_trace = nullptr;
#endif
namespace {

// ---------------------------------------------------------------------------
// Planner
// ---------------------------------------------------------------------------
constexpr int kMfmaMaxK = 11;
constexpr int kGenericKernel = 99;

struct TileChoice { int tpy, tpx, tiles_x, tiles_y; int64_t lanes; };

// Rectangular output tiles of at most `cap` pixels; pick the shape that
// wastes the fewest pixel lanes over the whole map.  Ties go first (K > 1)
// to a tile whose input row, padded to whole float4s, still fits in the
// map width (the condition for 16-byte input copies), then to the wider
// tile, for coalesced rows.
TileChoice choose_tile(int Hout, int Wout, int cap, int K) {
  const int Wx = Wout + K - 1;
  const auto row_fits = [&](int tpx) { return K > 1 && ((tpx + K - 1 + 3) & ~3) <= Wx; };
  TileChoice best{1, 1, Wout, Hout, INT64_MAX};
  for (int tpx = 1; tpx <= cap && tpx <= Wout; ++tpx) {
    int tpy = cap / tpx;
    if (tpy > Hout) tpy = Hout;
    if (tpy < 1) continue;
    const int tx = (Wout + tpx - 1) / tpx;
    const int ty = (Hout + tpy - 1) / tpy;
    const int64_t lanes = (int64_t)tx * ty * cap;
    const bool fits = row_fits(tpx), bfits = row_fits(best.tpx);
    if (lanes < best.lanes ||
        (lanes == best.lanes && (fits > bfits || (fits == bfits && tpx > best.tpx))))
      best = TileChoice{tpy, tpx, tx, ty, lanes};
  }
  return best;
}

struct Candidate {
  int kernel, MT, PT, WC, CC;
  int mf;             // MFMA tile (32 or 16); 0 for the vector family
  int ops_per_kstep;  // MFMAs per wave per k-step; VALU: FMAs per lane per (c, r, s)
  int lds_fixed;      // static LDS bytes (MFMA family), 0 if it depends on the tile
  int red_floats;     // LDS floats for the in-workgroup channel-group sum
  int waves;          // waves per workgroup
};

template <int S>
int shape_lds_bytes(int K) {
  switch (K) {
    case 1: return ShapeCfg<1, S>::LDS_BYTES;
    case 2: return ShapeCfg<2, S>::LDS_BYTES;
    case 3: return ShapeCfg<3, S>::LDS_BYTES;
    case 4: return ShapeCfg<4, S>::LDS_BYTES;
    case 5: return ShapeCfg<5, S>::LDS_BYTES;
    case 6: return ShapeCfg<6, S>::LDS_BYTES;
    case 7: return ShapeCfg<7, S>::LDS_BYTES;
    case 8: return ShapeCfg<8, S>::LDS_BYTES;
    case 9: return ShapeCfg<9, S>::LDS_BYTES;
    case 10: return ShapeCfg<10, S>::LDS_BYTES;
    case 11: return ShapeCfg<11, S>::LDS_BYTES;
    default: return INT32_MAX;
  }
}

template <int S>
int shape_cc(int K) {
  switch (K) {
    case 1: return ShapeCfg<1, S>::CC;
    case 2: return ShapeCfg<2, S>::CC;
    case 3: return ShapeCfg<3, S>::CC;
    case 4: return ShapeCfg<4, S>::CC;
    case 5: return ShapeCfg<5, S>::CC;
    case 6: return ShapeCfg<6, S>::CC;
    case 7: return ShapeCfg<7, S>::CC;
    case 8: return ShapeCfg<8, S>::CC;
    case 9: return ShapeCfg<9, S>::CC;
    case 10: return ShapeCfg<10, S>::CC;
    case 11: return ShapeCfg<11, S>::CC;
    default: return 0;
  }
}

// The compile-time configuration of shape i at filter size K (the kernels'
// own constants, so the planner and the kernels cannot disagree).
template <int... S>
void shape_consts(int i, int K, int &cc, int &lds, std::integer_sequence<int, S...>) {
  ((i == S ? (cc = shape_cc<S>(K), lds = shape_lds_bytes<S>(K), 0) : 0), ...);
}

Candidate mfma_candidate(int i, int K) {
  const MfmaShape s = kMfmaShapes[i];
  const int MT = s.MF * s.MB * s.WM, PT = s.MF * s.NB * s.WN;
  const int NW = s.WM * s.WN * s.WC;
  int cc = 0, lds = 0;
  shape_consts(i, K, cc, lds, std::make_integer_sequence<int, kNumMfma>{});
  const int red = (s.WC - 1) * s.WM * s.WN * s.MB * s.NB * s.MF * s.MF;
  return Candidate{i, MT, PT, s.WC, cc, s.MF, s.MB * s.NB, lds, red, NW};
}

// Matrix-core shapes whose waves each stage their own channels (every wave
// covers the whole tile, the channel sum split over the waves:
// MfmaCfg::PRIV).
bool private_stages(const Candidate &cd) { return cd.mf > 0 && cd.waves == cd.WC; }

Candidate valu_candidate(int i) {
  const ValuShape s = kValuShapes[i];
  return Candidate{i, s.MR * (4 / s.WC), 64, s.WC, s.CC, 0, s.MR,
                   0, (s.WC - 1) * (4 / s.WC) * s.MR * 64, 4};
}

// Rough time model in GPU clock cycles, used only to rank candidates.
//   work:  inner-product plus per-stage bookkeeping cycles of the busiest CU
//          (co-resident workgroups share its four SIMDs; a SIMD with a
//          single wave issues its MFMAs less densely than one with two);
//          splitting the channels over WC wave groups adds their LDS
//          reduction at the end
//   chain: a workgroup's stages cannot run faster than the load latency
//          (the MFMA family overlaps the next stage's loads with the current
//          stage; the VALU family pays the latency every stage); `occ`
//          co-resident workgroups overlap each other's chains
//   copy:  the bytes a CU stages into LDS, at the rate one CU's vector
//          memory path delivers them
// Shapes whose waves stage their own channels (no barrier between stages)
// have their own stage cost and copy rate.  The constants were fitted to
// exhaustive timings of every matrix-core candidate plan of 21 benchmark
// layers and 48 seeded random layers on an MI355X, the six bench-step
// layers weighted five times (a factor for several accumulator tiles per
// wave fitted to 1 and was dropped).  With the tile rule of choose_tile the
// model picks the fastest plan on all six bench-step layers, is 1.4% above
// the fastest on average over all 69 (23% at worst) and 2.4% on 24 other
// random layers (13% at worst).  The MFMA terms are empirical
// weights, not instruction latencies.
double estimate(const Candidate &cd, bool mfma, int C, int M, int Wx, int Wy, int K, int num_cu,
                const TileChoice &t, int64_t lds_bytes) {
  const int64_t ntiles = (int64_t)t.tiles_x * t.tiles_y;
  const int64_t mtiles = (M + cd.MT - 1) / cd.MT;
  const int64_t blocks = ntiles * mtiles;
  const int stages = (C + cd.CC - 1) / cd.CC;
  const int kk = K * K;
  // Fitted per family: the matrix-core kernels on every layer with their
  // eight-wave and deep shapes, the vector kernels on the same layers.
  constexpr double kMfma32Cycles = 64.3;  // one 32x32x2 MFMA per wave (issue: 64)
  constexpr double kMfma16Cycles = 18.0;  // one 16x16x4 MFMA per wave (issue: 32)
  constexpr double kOneWavePerSimd = 1.13; // MFMA cycles factor with one wave per SIMD
  constexpr double kWcReduction = 69.0;   // per extra wave group
  constexpr double kLaunch = 2000.0;
  // Private stages, and among them those whose input planes go 16 bytes per
  // lane (the kernel's in4 condition), have their own copy rate and stage
  // cost.
  const bool priv = mfma && private_stages(cd);
  const int ics = priv ? mfma_ics(K, cd.PT, cd.mf) : 0;
  const int ih = t.tpy + K - 1, iwp = (t.tpx + K - 1 + 3) & ~3;
  const bool in4 = priv && Wx >= iwp && ih * iwp <= ics && (int64_t)Wx * Wy < (1 << 24);
  const double kCopyBytesPerClock = in4 ? 12.1 : priv ? 12.8 : 11.7;
  const double kStageOverhead = mfma ? (in4 ? 294.0 : priv ? 410.0 : 652.0) : 300.0;
  const double kLatency = mfma ? 11.0 : 2000.0;
  constexpr int kMaxWaves = 8;            // co-resident waves per CU the model counts
  int occ = (int)(160 * 1024 / (lds_bytes > 0 ? lds_bytes : 1));
  if (occ > kMaxWaves / cd.waves) occ = kMaxWaves / cd.waves;
  if (occ < 1) occ = 1;
  const int64_t per_cu = (blocks + num_cu - 1) / num_cu;
  const int64_t rounds = (per_cu + occ - 1) / occ;
  const int64_t waves_per_simd = cd.waves / 4 * (per_cu < occ ? per_cu : occ);
  const int kg = cd.mf == 16 ? 4 : 2;
  const double mcyc = cd.mf == 16 ? kMfma16Cycles : kMfma32Cycles;
  const double per_stage =
      (mfma ? (double)(cd.CC / cd.WC / kg) * kk * cd.ops_per_kstep * mcyc * cd.waves / 4 *
                  (waves_per_simd < 2 ? kOneWavePerSimd : 1.0)
            : (double)(cd.CC / cd.WC) * kk * cd.ops_per_kstep * 4.0) +
      kStageOverhead;
  const double work = (double)per_cu * stages * per_stage;
  const double stage_chain = mfma ? (per_stage > kLatency ? per_stage : kLatency)
                                  : per_stage + kLatency;
  const double chain = (double)rounds * stages * stage_chain;
  // Bytes staged per workgroup: the filter slice and the input halo tile of
  // every channel.
  const double staged = 4.0 * C * ((double)cd.MT * kk + (t.tpy + K - 1.0) * (t.tpx + K - 1.0));
  // the copy rate grows a little with the waves on a CU issuing copies
  const double wpc = (double)cd.waves * (per_cu < occ ? per_cu : occ);
  const double copy =
      mfma ? (double)per_cu * staged / (kCopyBytesPerClock * std::pow(wpc / 8.0, 0.05)) : 0.0;
  double tm = work > chain ? work : chain;
  if (copy > tm) tm = copy;
  tm += (cd.WC - 1) * kWcReduction + kLatency + kLaunch;
  // Private stages: in a last stage of fewer than CC channels the waves past
  // them get none; the time grows by kIdleWaves times the share of wave
  // stages left idle (fitted afterwards; it changes the plan of one
  // benchmark layer of the 93 timed, a 1x1 layer with 64 channels).
  if (priv) {
    constexpr double kIdleWaves = 0.5;
    const int rem = C % cd.CC ? C % cd.CC : cd.CC;
    const int ccw = cd.CC / cd.WC;
    const int active = std::min(cd.WC, (rem + ccw - 1) / ccw);
    tm *= 1.0 + kIdleWaves * (double)(cd.WC - active) / cd.WC / stages;
  }
  return tm;
}

// Every workgroup shape of one family whose LDS footprint fits, with the
// time model's estimate, in a fixed order.
void enumerate_family(int C, int M, int Wx, int Wy, int K, bool mfma, int num_cu,
                      std::vector<std::pair<double, MultiPlan>> &out) {
  const int Hout = Wy - K + 1, Wout = Wx - K + 1;
  // The matrix-core kernels address a filter row and an input plane with
  // 32-bit byte offsets per lane.
  if (mfma && ((int64_t)C * K * K >= (int64_t(1) << 29) || (int64_t)Wx * Wy >= (int64_t(1) << 29)))
    return;
  const int n = mfma ? kNumMfma : kNumValu;
  for (int i = 0; i < n; ++i) {
    const Candidate cd = mfma ? mfma_candidate(i, K) : valu_candidate(i);
    // per-wave copies: filter offsets span MT filter rows, input offsets a
    // wave's CC/WC planes; both are 32-bit (and C*K*K goes through a 24-bit
    // multiply)
    if (mfma && private_stages(cd) &&
        ((int64_t)C * K * K >= (int64_t(1) << 24) ||
         (int64_t)cd.MT * C * K * K >= (int64_t(1) << 30) ||
         (int64_t)(cd.CC / cd.WC) * Wx * Wy >= (int64_t(1) << 30)))
      continue;
    const TileChoice t = choose_tile(Hout, Wout, cd.PT, K);
    const int IH = t.tpy + K - 1, IW = t.tpx + K - 1;
    int64_t lds_bytes = cd.lds_fixed;
    if (!mfma) {
      const int64_t stage = (int64_t)cd.CC * IH * IW;
      lds_bytes = 4 * (stage > cd.red_floats ? stage : cd.red_floats);
    }
    if (lds_bytes > kMaxLds) continue;
    const double tm = estimate(cd, mfma, C, M, Wx, Wy, K, num_cu, t, lds_bytes);
    MultiPlan p{};
    p.variant = mfma ? DCONV_VARIANT_MFMA : DCONV_VARIANT_VALU;
    p.kernel = i;
    p.K = K;
    p.tile_m = cd.MT;
    p.tpy = t.tpy;
    p.tpx = t.tpx;
    p.tiles_x = t.tiles_x;
    p.tiles_y = t.tiles_y;
    p.chunk_c = cd.CC;
    p.waves_c = cd.WC;
    p.grid_x = (int)((int64_t)t.tiles_x * t.tiles_y * ((M + cd.MT - 1) / cd.MT));
    p.grid_y = 1;
    p.grid_z = 1;
    p.block = 64 * cd.waves;
    p.lds_bytes = (int)lds_bytes;
    out.emplace_back(tm, p);
  }
  if (out.empty() && !mfma) {
    // No tiled shape fits in LDS: one output per thread from the caches.
    const int64_t total = (int64_t)M * Hout * Wout;
    MultiPlan p{};
    p.variant = DCONV_VARIANT_VALU;
    p.kernel = kGenericKernel;
    p.K = K;
    p.tile_m = 1;
    p.tpy = 1;
    p.tpx = 1;
    p.tiles_x = Wout;
    p.tiles_y = Hout;
    p.chunk_c = C;
    p.waves_c = 1;
    p.grid_x = (int)((total + 255) / 256);
    p.grid_y = p.grid_z = 1;
    p.block = 256;
    p.lds_bytes = 0;
    out.emplace_back(0.0, p);
  }
}

int plan_family(int C, int M, int Wx, int Wy, int K, bool mfma, int num_cu, MultiPlan *best) {
  std::vector<std::pair<double, MultiPlan>> all;
  enumerate_family(C, M, Wx, Wy, K, mfma, num_cu, all);
  if (all.empty()) return DCONV_EUNSUPPORTED;
  size_t b = 0;
  for (size_t k = 1; k < all.size(); ++k)
    if (all[k].first < all[b].first) b = k;
  *best = all[b].second;
  return DCONV_OK;
}

}  // namespace

int plan_multi(int C, int M, int Wx, int Wy, int K, int variant, int num_cu, MultiPlan *p) {
  if (num_cu <= 0) num_cu = 256;
  if (variant == DCONV_VARIANT_MFMA) {
    if (K > kMfmaMaxK) return DCONV_EUNSUPPORTED;
    return plan_family(C, M, Wx, Wy, K, true, num_cu, p);
  }
  if (variant == DCONV_VARIANT_VALU) return plan_family(C, M, Wx, Wy, K, false, num_cu, p);
  // Automatic: the matrix cores deliver twice the fp32 rate of unpacked
  // vector FMAs, so they are preferred wherever a kernel exists.
  if (K <= kMfmaMaxK && plan_family(C, M, Wx, Wy, K, true, num_cu, p) == DCONV_OK) return DCONV_OK;
  return plan_family(C, M, Wx, Wy, K, false, num_cu, p);
}

void export_multi_plan(const MultiPlan &p, dconv_plan *out) {
  *out = dconv_plan{};
  out->variant = p.variant;
  out->kernel = p.kernel;
  out->tile_m = p.tile_m;
  out->tile_h = p.tpy;
  out->tile_w = p.tpx;
  out->chunk_c = p.chunk_c;
  out->waves_c = p.waves_c;
  out->grid_x = p.grid_x;
  out->grid_y = p.grid_y;
  out->grid_z = p.grid_z;
  out->block = p.block;
  out->lds_bytes = p.lds_bytes;
}

int multi_candidates(int C, int M, int Wx, int Wy, int K, int variant, int num_cu,
                     std::vector<MultiPlan> &out) {
  if (num_cu <= 0) num_cu = 256;
  std::vector<std::pair<double, MultiPlan>> all;
  if ((variant == DCONV_VARIANT_AUTO || variant == DCONV_VARIANT_MFMA) && K <= kMfmaMaxK)
    enumerate_family(C, M, Wx, Wy, K, true, num_cu, all);
  if (variant == DCONV_VARIANT_AUTO || variant == DCONV_VARIANT_VALU)
    enumerate_family(C, M, Wx, Wy, K, false, num_cu, all);
  out.clear();
  for (const auto &e : all) out.push_back(e.second);
  return out.empty() ? DCONV_EUNSUPPORTED : DCONV_OK;
}

hipError_t launch_multi(const MultiPlan &p, const float *I, const float *F, float *O, int C,
                        int M, int Wx, int Wy, hipStream_t st) {
  TileArgs a{};
  a.C = C;
  a.M = M;
  a.Wx = Wx;
  a.Wy = Wy;
  a.tpy = p.tpy;
  a.tpx = p.tpx;
  a.tiles_x = p.tiles_x;
  a.ntiles = p.tiles_x * p.tiles_y;
  a.mtiles = (M + p.tile_m - 1) / p.tile_m;
  a.IH = p.tpy + p.K - 1;
  a.IW = p.tpx + p.K - 1;
  a.ICS = a.IH * a.IW;
#ifdef DCONV_STAGE_TRACE
  a.trace = g_stage_trace;
#endif
  if (p.kernel == kGenericKernel) {
    hipLaunchKernelGGL(multi_generic, dim3(p.grid_x), dim3(256), 0, st, I, F, O, C, M, Wx, Wy, p.K);
    return hipGetLastError();
  }
  if (p.variant == DCONV_VARIANT_MFMA) {
    switch (p.K) {
      case 1: return launch_mfma_k1(p, I, F, O, a, st);
      case 2: return launch_mfma_k2(p, I, F, O, a, st);
      case 3: return launch_mfma_k3(p, I, F, O, a, st);
      case 4: return launch_mfma_k4(p, I, F, O, a, st);
      case 5: return launch_mfma_k5(p, I, F, O, a, st);
      case 6: return launch_mfma_k6(p, I, F, O, a, st);
      case 7: return launch_mfma_k7(p, I, F, O, a, st);
      case 8: return launch_mfma_k8(p, I, F, O, a, st);
      case 9: return launch_mfma_k9(p, I, F, O, a, st);
      case 10: return launch_mfma_k10(p, I, F, O, a, st);
      case 11: return launch_mfma_k11(p, I, F, O, a, st);
      default: return hipErrorInvalidValue;
    }
  }
  switch (p.K) {
    case 1: return launch_valu_k<1>(p, I, F, O, a, st);
    case 2: return launch_valu_k<2>(p, I, F, O, a, st);
    case 3: return launch_valu_k<3>(p, I, F, O, a, st);
    case 4: return launch_valu_k<4>(p, I, F, O, a, st);
    case 5: return launch_valu_k<5>(p, I, F, O, a, st);
    case 6: return launch_valu_k<6>(p, I, F, O, a, st);
    case 7: return launch_valu_k<7>(p, I, F, O, a, st);
    default: return launch_valu_k<0>(p, I, F, O, a, st);
  }
}

}  // namespace dconv
