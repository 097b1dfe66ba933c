// The paper's partition model (host only; no device code).
//
// Section 2.2 and Table 1: how much work and how much data in flight a
// processor needs to hide its global-memory latency (N_FMA and V_s).
// Section 3.1: how a single-channel convolution is divided over the
// processors (filters along m in P map pieces, or map along y in Q filter
// pieces).  Section 3.2: the stride-fixed block of the multi-channel kernel
// (segment S, W'x, W'y, M').
//
// The functions evaluate the formulas for any device description, so the
// same code reproduces Table 1 for the paper's GPU and gives the
// corresponding figures for an MI355X.
#include <algorithm>
#include <cmath>
#include <cstdint>
#include <vector>

#include "internal.h"

#define DCONV_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

int64_t ceil_div64(int64_t a, int64_t b) { return (a + b - 1) / b; }

bool valid_device(const dconv_device_params *d) {
  return d->latency_clk > 0 && d->bandwidth_gbs > 0 && d->clock_mhz > 0 && d->num_cu > 0 &&
         d->lanes_per_cu > 0 && d->ops_per_clk_lane > 0 && d->wave_size > 0 &&
         d->word_bytes > 0 && d->onchip_bytes > 0;
}

}  // namespace

// Section 2.2 / Table 1.
DCONV_EXPORT int dconv_model_latency(const dconv_device_params *dev, dconv_latency_model *out) {
  if (!dev || !out) return DCONV_ENULL;
  if (!valid_device(dev)) return DCONV_EINVAL;
  *out = dconv_latency_model{};
  const double lat = dev->latency_clk;
  // Work that keeps every lane busy for one latency: latency x lanes x the
  // per-lane rate (Table 1 counts 2 per clock per core).
  out->n_fma = (long long)std::llround(lat * dev->lanes_per_cu * dev->ops_per_clk_lane);
  // Bytes the memory delivers per clock, rounded down to whole bytes.
  out->bytes_per_clk = (int)std::floor(dev->bandwidth_gbs * 1e9 / (dev->clock_mhz * 1e6));
  // Bytes that must be in flight to cover one latency.
  out->data_bytes = (long long)std::llround((double)out->bytes_per_clk * lat);
  // One word per thread, rounded up to whole warps / wavefronts, then spread
  // over the processors and rounded up to whole warps again.
  const int64_t threads = (int64_t)std::ceil((double)out->data_bytes / dev->word_bytes);
  out->threads_total = ceil_div64(threads, dev->wave_size) * dev->wave_size;
  const int64_t per_cu = ceil_div64(out->threads_total, dev->num_cu);
  out->waves_per_cu = (int)ceil_div64(per_cu, dev->wave_size);
  out->threads_per_cu = out->waves_per_cu * dev->wave_size;
  out->bytes_per_cu = out->threads_per_cu * dev->word_bytes;
  out->v_s = (long long)out->bytes_per_cu * dev->num_cu;
  return DCONV_OK;
}

// Section 3.1: D1/Th1 (filters divided along m over the processors, the map
// streamed in P pieces along y) and D2/Th2 (map divided along y over the
// processors, the filters streamed in Q pieces), the bounds on P and Q, the
// smallest admissible values, and the choice of the method with the smaller
// on-chip footprint.
DCONV_EXPORT int dconv_model_single(const dconv_device_params *dev, const dconv_latency_model *lm,
                                    int Wx, int Wy, int K, int M, dconv_single_split *out) {
  if (!dev || !lm || !out) return DCONV_ENULL;
  if (!valid_device(dev) || Wx < 1 || Wy < 1 || K < 1 || M < 1 || K > Wx || K > Wy)
    return DCONV_EINVAL;
  *out = dconv_single_split{};
  const int64_t N = dev->num_cu, KK = (int64_t)K * K, w = dev->word_bytes;
  const double S = dev->onchip_bytes;
  const double nfma = (double)lm->n_fma;
  const int64_t m_per = ceil_div64(M, N);
  const int64_t y_per = ceil_div64(Wy, N);

  // Upper bounds: at least N_FMA operations per data set.
  int64_t p_hi = (int64_t)std::floor((double)(KK * m_per) * Wy * Wx / nfma);
  if (p_hi > Wy) p_hi = Wy;
  int64_t q_hi = (int64_t)std::floor((double)(KK * M) * y_per * Wx / nfma);
  if (q_hi > M) q_hi = M;
  // Lower bounds: the data set fits in on-chip memory.
  const double p_den = S - (double)w * KK * m_per + (double)(1 - K) * w * Wx;
  const double q_den = S - (double)w * Wx * (y_per + K - 1);
  int64_t p_lo = p_den > 0 ? (int64_t)std::ceil((double)w * Wy * Wx / p_den) : INT64_MAX;
  int64_t q_lo = q_den > 0 ? (int64_t)std::ceil((double)w * M * KK / q_den) : INT64_MAX;
  if (p_lo < 1) p_lo = 1;
  if (q_lo < 1) q_lo = 1;
  // The closed-form bounds divide Wy and M by P and Q exactly; the data set
  // holds whole lines and whole filters, so step up to the first factor whose
  // rounded-up piece fits.
  auto d1 = [&](int64_t P) { return (KK * m_per + (ceil_div64(Wy, P) + K - 1) * (int64_t)Wx) * w; };
  auto d2 = [&](int64_t Q) { return (KK * ceil_div64(M, Q) + (y_per + K - 1) * (int64_t)Wx) * w; };
  if (p_lo != INT64_MAX)
    while (p_lo <= p_hi && d1(p_lo) > dev->onchip_bytes) ++p_lo;
  if (q_lo != INT64_MAX)
    while (q_lo <= q_hi && d2(q_lo) > dev->onchip_bytes) ++q_lo;
  out->p_lo = p_lo == INT64_MAX ? -1 : (long long)p_lo;
  out->p_hi = (long long)p_hi;
  out->q_lo = q_lo == INT64_MAX ? -1 : (long long)q_lo;
  out->q_hi = (long long)q_hi;
  // The smallest admissible value, else 1.
  const bool p_ok = p_lo != INT64_MAX && p_lo <= p_hi;
  const bool q_ok = q_lo != INT64_MAX && q_lo <= q_hi;
  const int64_t P = p_ok ? p_lo : 1;
  const int64_t Q = q_ok ? q_lo : 1;
  out->p_admissible = p_ok;
  out->q_admissible = q_ok;

  out->D1 = d1(P);
  out->Th1 = KK * m_per * ceil_div64(Wy, P) * (int64_t)Wx;
  out->D2 = d2(Q);
  out->Th2 = KK * ceil_div64(M, Q) * y_per * (int64_t)Wx;
  // Both methods meet the requirements; the smaller footprint is kept.
  if (out->D1 < out->D2) {
    out->method = 1;
    out->P = (int)P;
    out->Q = 1;
  } else {
    out->method = 2;
    out->P = 1;
    out->Q = (int)Q;
  }
  return DCONV_OK;
}

// Section 3.2: for a segment of S bytes of each filter along the channels and
// W'x map pixels, W'y = ceil(S / (K * word)) map lines feed the segment; the
// smallest M' with M' * (S / word) * W'x >= N_FMA keeps the units busy, and a
// data set may use at most half of the on-chip memory (the other half holds
// the prefetched next set).
DCONV_EXPORT int dconv_model_multi(const dconv_device_params *dev, const dconv_latency_model *lm,
                                   int K, int S, int Wxp, dconv_multi_block *out) {
  if (!dev || !lm || !out) return DCONV_ENULL;
  if (!valid_device(dev) || K < 1 || S < dev->word_bytes || S % dev->word_bytes != 0 || Wxp < 1)
    return DCONV_EINVAL;
  *out = dconv_multi_block{};
  const int64_t w = dev->word_bytes;
  out->S = S;
  out->Wx_p = Wxp;
  out->Wy_p = (int)ceil_div64(S, (int64_t)K * w);
  // M' >= N_FMA * word / (S * W'x)
  out->M_p = (int)std::max<int64_t>(1, ceil_div64(lm->n_fma * w, (int64_t)S * Wxp));
  out->set_bytes = (long long)S * out->M_p + (long long)out->Wy_p * Wxp * w;
  out->fits = out->set_bytes * 2 <= dev->onchip_bytes;
  out->fma_per_set = (long long)out->M_p * (S / w) * Wxp;
  return DCONV_OK;
}

// Section 3.2 applied to this library's multi-channel plans: among the
// candidates that keep the channel sum inside one workgroup (the paper does
// not split it across processors), keep those whose stage gives each compute
// unit at least N_FMA multiply-adds (co-resident workgroups, as many as the
// LDS holds, each contribute their stage), take the fewest filters per
// workgroup (the smallest M', the most parallelism), then the most pixels per
// tile (the largest W'x).  If no candidate reaches N_FMA, the one with the
// most work per compute unit is taken.
DCONV_EXPORT int dconv_plan_multi_paper(int C, int M, int Wx, int Wy, int K,
                                        const dconv_device_params *dev, dconv_plan *out) {
  if (!dev || !out) return DCONV_ENULL;
  if (!valid_device(dev)) return DCONV_EINVAL;
  if (C < 1 || M < 1 || K < 1 || Wx < 1 || Wy < 1 || K > Wx || K > Wy) return DCONV_EINVAL;
  dconv_latency_model lm;
  int rc = dconv_model_latency(dev, &lm);
  if (rc != DCONV_OK) return rc;
  std::vector<dconv::MultiPlan> all;
  rc = dconv::multi_candidates(C, M, Wx, Wy, K, DCONV_VARIANT_AUTO, dev->num_cu, all);
  if (rc != DCONV_OK) return rc;
  int best = -1, fallback = -1;
  double best_work = -1.0;
  for (int i = 0; i < (int)all.size(); ++i) {
    const dconv::MultiPlan &p = all[i];
    const int64_t per_wg = (int64_t)p.tile_m * p.chunk_c * K * K * p.tpy * p.tpx;
    // Co-resident workgroups: as many as the on-chip memory holds, at most
    // 2048 threads per compute unit.
    const int64_t max_wg = 2048 / p.block;
    int64_t occ = p.lds_bytes > 0 ? dev->onchip_bytes / p.lds_bytes : max_wg;
    if (occ > max_wg) occ = max_wg;
    if (occ < 1) occ = 1;
    const int64_t wgs_per_cu = (p.grid_x + dev->num_cu - 1) / dev->num_cu;
    if (occ > wgs_per_cu) occ = wgs_per_cu;
    const double work = (double)per_wg * occ;
    if (work > best_work) {
      best_work = work;
      fallback = i;
    }
    if (work < (double)lm.n_fma) continue;
    if (best < 0) {
      best = i;
      continue;
    }
    const dconv::MultiPlan &b = all[best];
    if (p.tile_m < b.tile_m ||
        (p.tile_m == b.tile_m && p.tpy * p.tpx > b.tpy * b.tpx))
      best = i;
  }
  if (best < 0) best = fallback;
  if (best < 0) return DCONV_EUNSUPPORTED;
  dconv::export_multi_plan(all[best], out);
  return DCONV_OK;
}

// Section 3.1 applied to this library's single-map plans for a device
// described by `dev`: the model's method decides how the work is divided.
//   Method 1 (filters divided over the N processors, each walking the map in
// P pieces along y): the vector-kernel candidate whose number of filter
// groups is closest to min(M, N), then whose tile height is closest to a
// P-th of the output rows.
//   Method 2 (the map divided along y over the processors, every processor
// applying all M filters, Q at a time): among the candidates that keep all
// filters in one group, the one whose tile height is closest to an N-th of
// the output rows, then the one with the most workgroups.
DCONV_EXPORT int dconv_plan_single_paper(int Wx, int Wy, int K, int M,
                                         const dconv_device_params *dev, dconv_plan *out) {
  if (!dev || !out) return DCONV_ENULL;
  if (!valid_device(dev)) return DCONV_EINVAL;
  if (M < 1 || K < 1 || Wx < 1 || Wy < 1 || K > Wx || K > Wy) return DCONV_EINVAL;
  dconv_latency_model lm;
  int rc = dconv_model_latency(dev, &lm);
  if (rc != DCONV_OK) return rc;
  dconv_single_split sp;
  if ((rc = dconv_model_single(dev, &lm, Wx, Wy, K, M, &sp)) != DCONV_OK) return rc;
  std::vector<dconv::SinglePlan> all;
  rc = dconv::single_candidates(Wx, Wy, K, M, dev->num_cu, true, DCONV_VARIANT_VALU, all);
  if (rc != DCONV_OK) return rc;
  const int64_t Hout = (int64_t)Wy - K + 1;
  const int64_t N = dev->num_cu;
  int best = -1;
  auto dist = [](int64_t a, int64_t b) { return a > b ? a - b : b - a; };
  for (int i = 0; i < (int)all.size(); ++i) {
    const dconv::SinglePlan &p = all[i];
    if (best < 0) {
      best = i;
      continue;
    }
    const dconv::SinglePlan &b = all[best];
    if (sp.method == 1) {
      const int64_t groups = std::min<int64_t>(M, N);
      const int64_t rows = ceil_div64(Hout, sp.P);
      const int64_t dg = dist(p.grid_z, groups), dgb = dist(b.grid_z, groups);
      const int64_t dr = dist(p.tile_h, rows), drb = dist(b.tile_h, rows);
      if (dg < dgb || (dg == dgb && (dr < drb || (dr == drb && p.tile_w > b.tile_w)))) best = i;
    } else {
      const int64_t rows = ceil_div64(Hout, N);
      const bool one = p.grid_z == 1, oneb = b.grid_z == 1;
      const int64_t dr = dist(p.tile_h, rows), drb = dist(b.tile_h, rows);
      if ((one && !oneb) ||
          (one == oneb && (dr < drb || (dr == drb && (int64_t)p.grid * p.grid_z >
                                                         (int64_t)b.grid * b.grid_z))))
        best = i;
    }
  }
  dconv::export_single_plan(all[best], out);
  return DCONV_OK;
}
