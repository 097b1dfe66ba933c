// C ABI of libdconv: argument validation, planning and launch (the host side
// of the library; the kernels live in single.hip and multi.hip).
//
// Every entry point validates its arguments before touching the HIP runtime,
// so NULL pointers and bad sizes are reported without a device.
#include <climits>
#include <cstdint>
#include <mutex>
#include <vector>

#include "internal.h"

#define DCONV_EXPORT extern "C" __attribute__((visibility("default")))

namespace {

// Compute-unit count per device, read once per process; immutable afterwards.
std::once_flag g_props_once;
std::vector<int> g_num_cu;

void read_props() {
  int n = 0;
  if (hipGetDeviceCount(&n) != hipSuccess || n < 0) n = 0;
  g_num_cu.assign(n, 0);
  for (int d = 0; d < n; ++d) {
    int cu = 0;
    if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, d) == hipSuccess)
      g_num_cu[d] = cu;
  }
  (void)hipGetLastError();
}

// Returns DCONV_OK and the current device's CU count, or DCONV_EHIP.
int current_num_cu(int *num_cu) {
  std::call_once(g_props_once, read_props);
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) {
    (void)hipGetLastError();
    return DCONV_EHIP;
  }
  if (dev < 0 || dev >= (int)g_num_cu.size() || g_num_cu[dev] <= 0) return DCONV_EHIP;
  *num_cu = g_num_cu[dev];
  return DCONV_OK;
}

// Sizes of Eq. 1: C, M, K >= 1, 1 <= K <= min(Wx, Wy) (valid mode needs at
// least one output), and every tensor indexable with 32-bit element offsets.
int validate_sizes(int C, int M, int Wx, int Wy, int K) {
  if (C < 1 || M < 1 || K < 1 || Wx < 1 || Wy < 1 || K > Wx || K > Wy) return DCONV_EINVAL;
  const int64_t Hout = (int64_t)Wy - K + 1;
  const int64_t Wout = (int64_t)Wx - K + 1;
  const int64_t in = (int64_t)C * Wy * Wx;
  const int64_t f = (int64_t)M * C * K * K;
  const int64_t out = (int64_t)M * Hout * Wout;
  if (in > INT_MAX || f > INT_MAX || out > INT_MAX) return DCONV_ERANGE;
  return DCONV_OK;
}

// Whether two plans are the same, field by field.
bool same_plan(const dconv_plan &a, const dconv_plan &b) {
  return a.variant == b.variant && a.kernel == b.kernel && a.tile_m == b.tile_m &&
         a.tile_h == b.tile_h && a.tile_w == b.tile_w && a.chunk_c == b.chunk_c &&
         a.waves_c == b.waves_c && a.grid_x == b.grid_x && a.grid_y == b.grid_y &&
         a.grid_z == b.grid_z && a.block == b.block && a.lds_bytes == b.lds_bytes;
}

}  // namespace

DCONV_EXPORT int dconv_single_variant(const float *I, const float *F, float *O, int Wx, int Wy,
                                      int K, int M, int variant, void *stream) {
  if (!I || !F || !O) return DCONV_ENULL;
  if (variant != DCONV_VARIANT_AUTO && variant != DCONV_VARIANT_VALU &&
      variant != DCONV_VARIANT_MFMA)
    return DCONV_EINVAL;
  int rc = validate_sizes(1, M, Wx, Wy, K);
  if (rc != DCONV_OK) return rc;
  int num_cu = 0;
  if ((rc = current_num_cu(&num_cu)) != DCONV_OK) return rc;
  dconv::SinglePlan p;
  rc = dconv::plan_single(Wx, Wy, K, M, num_cu, (reinterpret_cast<uintptr_t>(I) & 15) == 0,
                          variant, &p);
  if (rc != DCONV_OK) return rc;
  // A launch error still pending from earlier work in this thread is
  // cleared first, so DCONV_EHIP reports this call's launch only.
  (void)hipGetLastError();
  const hipError_t e = dconv::launch_single(p, I, F, O, Wx, Wy, M, (hipStream_t)stream);
  return e == hipSuccess ? DCONV_OK : DCONV_EHIP;
}

DCONV_EXPORT int dconv_single(const float *I, const float *F, float *O, int Wx, int Wy, int K,
                              int M, void *stream) {
  return dconv_single_variant(I, F, O, Wx, Wy, K, M, DCONV_VARIANT_AUTO, stream);
}

DCONV_EXPORT int dconv_plan_single_candidates(int Wx, int Wy, int K, int M, int variant,
                                              int num_cu, dconv_plan *out, int capacity,
                                              int *count) {
  if (!count || (capacity > 0 && !out)) return DCONV_ENULL;
  if (capacity < 0) return DCONV_EINVAL;
  if (variant != DCONV_VARIANT_AUTO && variant != DCONV_VARIANT_VALU &&
      variant != DCONV_VARIANT_MFMA)
    return DCONV_EINVAL;
  int rc = validate_sizes(1, M, Wx, Wy, K);
  if (rc != DCONV_OK) return rc;
  std::vector<dconv::SinglePlan> all;
  rc = dconv::single_candidates(Wx, Wy, K, M, num_cu > 0 ? num_cu : 256, true, variant, all);
  *count = (int)all.size();
  if (rc != DCONV_OK) return rc;
  for (int i = 0; i < capacity && i < (int)all.size(); ++i)
    dconv::export_single_plan(all[i], out + i);
  return DCONV_OK;
}

DCONV_EXPORT int dconv_single_with_plan(const float *I, const float *F, float *O, int Wx, int Wy,
                                        int K, int M, const dconv_plan *plan, void *stream) {
  if (!I || !F || !O || !plan) return DCONV_ENULL;
  int rc = validate_sizes(1, M, Wx, Wy, K);
  if (rc != DCONV_OK) return rc;
  int num_cu = 0;
  if ((rc = current_num_cu(&num_cu)) != DCONV_OK) return rc;
  std::vector<dconv::SinglePlan> all;
  const bool aligned = (reinterpret_cast<uintptr_t>(I) & 15) == 0;
  if (dconv::single_candidates(Wx, Wy, K, M, num_cu, aligned, DCONV_VARIANT_AUTO, all) !=
      DCONV_OK)
    return DCONV_EINVAL;
  for (const auto &p : all) {
    dconv_plan e;
    dconv::export_single_plan(p, &e);
    if (same_plan(e, *plan)) {
      (void)hipGetLastError();  // report this launch only
      const hipError_t err = dconv::launch_single(p, I, F, O, Wx, Wy, M, (hipStream_t)stream);
      return err == hipSuccess ? DCONV_OK : DCONV_EHIP;
    }
  }
  return DCONV_EINVAL;
}

namespace {

// Launch a multi-channel plan.  A launch error still pending from earlier
// work in this thread is cleared first, so DCONV_EHIP reports this call's
// launch only.
int run_multi(const dconv::MultiPlan &p, const float *I, const float *F, float *O, int C, int M,
              int Wx, int Wy, hipStream_t st) {
  (void)hipGetLastError();
  const hipError_t e = dconv::launch_multi(p, I, F, O, C, M, Wx, Wy, st);
  return e == hipSuccess ? DCONV_OK : DCONV_EHIP;
}


}  // namespace

DCONV_EXPORT int dconv_multi_variant(const float *I, const float *F, float *O, int C, int M,
                                     int Wx, int Wy, int K, int variant, void *stream) {
  if (!I || !F || !O) return DCONV_ENULL;
  if (variant != DCONV_VARIANT_AUTO && variant != DCONV_VARIANT_VALU &&
      variant != DCONV_VARIANT_MFMA)
    return DCONV_EINVAL;
  int rc = validate_sizes(C, M, Wx, Wy, K);
  if (rc != DCONV_OK) return rc;
  int num_cu = 0;
  if ((rc = current_num_cu(&num_cu)) != DCONV_OK) return rc;
  dconv::MultiPlan p;
  if ((rc = dconv::plan_multi(C, M, Wx, Wy, K, variant, num_cu, &p)) != DCONV_OK) return rc;
  return run_multi(p, I, F, O, C, M, Wx, Wy, (hipStream_t)stream);
}

#ifdef DCONV_STAGE_TRACE
// Trace builds only (not declared in dconv.h): register the buffer the
// multi-channel matrix-core kernel writes its stage-trace records to
// (2 * grid_x * kStageTraceWords long longs, device memory), or NULL.
DCONV_EXPORT void dconv_debug_stage_trace(long long *buf) { dconv::g_stage_trace = buf; }
#endif

DCONV_EXPORT int dconv_multi_with_plan(const float *I, const float *F, float *O, int C, int M,
                                       int Wx, int Wy, int K, const dconv_plan *plan,
                                       void *stream) {
  if (!I || !F || !O || !plan) return DCONV_ENULL;
  int rc = validate_sizes(C, M, Wx, Wy, K);
  if (rc != DCONV_OK) return rc;
  int num_cu = 0;
  if ((rc = current_num_cu(&num_cu)) != DCONV_OK) return rc;
  std::vector<dconv::MultiPlan> all;
  if (dconv::multi_candidates(C, M, Wx, Wy, K, DCONV_VARIANT_AUTO, num_cu, all) != DCONV_OK)
    return DCONV_EINVAL;
  for (const auto &p : all) {
    dconv_plan e;
    dconv::export_multi_plan(p, &e);
    if (same_plan(e, *plan)) return run_multi(p, I, F, O, C, M, Wx, Wy, (hipStream_t)stream);
  }
  return DCONV_EINVAL;
}

DCONV_EXPORT int dconv_plan_multi_candidates(int C, int M, int Wx, int Wy, int K, int variant,
                                             int num_cu, dconv_plan *out, int capacity,
                                             int *count) {
  if (!count || (capacity > 0 && !out)) return DCONV_ENULL;
  if (capacity < 0) return DCONV_EINVAL;
  if (variant != DCONV_VARIANT_AUTO && variant != DCONV_VARIANT_VALU &&
      variant != DCONV_VARIANT_MFMA)
    return DCONV_EINVAL;
  int rc = validate_sizes(C, M, Wx, Wy, K);
  if (rc != DCONV_OK) return rc;
  std::vector<dconv::MultiPlan> all;
  rc = dconv::multi_candidates(C, M, Wx, Wy, K, variant, num_cu, all);
  *count = (int)all.size();
  if (rc != DCONV_OK) return rc;
  for (int i = 0; i < capacity && i < (int)all.size(); ++i) dconv::export_multi_plan(all[i], out + i);
  return DCONV_OK;
}

DCONV_EXPORT int dconv_multi(const float *I, const float *F, float *O, int C, int M, int Wx,
                             int Wy, int K, void *stream) {
  return dconv_multi_variant(I, F, O, C, M, Wx, Wy, K, DCONV_VARIANT_AUTO, stream);
}

DCONV_EXPORT const char *dconv_strerror(int status) {
  switch (status) {
    case DCONV_OK: return "success";
    case DCONV_ENULL: return "a required pointer is NULL";
    case DCONV_EINVAL:
      return "invalid size, variant or plan (need C, M, K >= 1 and K <= min(Wx, Wy); a plan "
             "must be one of the candidates for these sizes)";
    case DCONV_ERANGE: return "a tensor has more than 2^31-1 elements";
    case DCONV_EHIP: return "the HIP runtime reported an error";
    case DCONV_EUNSUPPORTED: return "the requested kernel family cannot run this shape";
    default: return "unknown status";
  }
}

DCONV_EXPORT int dconv_plan_single_variant(int Wx, int Wy, int K, int M, int variant,
                                           int num_cu, dconv_plan *out) {
  if (!out) return DCONV_ENULL;
  if (variant != DCONV_VARIANT_AUTO && variant != DCONV_VARIANT_VALU &&
      variant != DCONV_VARIANT_MFMA)
    return DCONV_EINVAL;
  int rc = validate_sizes(1, M, Wx, Wy, K);
  if (rc != DCONV_OK) return rc;
  dconv::SinglePlan p;
  rc = dconv::plan_single(Wx, Wy, K, M, num_cu > 0 ? num_cu : 256, true, variant, &p);
  if (rc != DCONV_OK) return rc;
  dconv::export_single_plan(p, out);
  return DCONV_OK;
}

DCONV_EXPORT int dconv_plan_single(int Wx, int Wy, int K, int M, int num_cu, dconv_plan *out) {
  return dconv_plan_single_variant(Wx, Wy, K, M, DCONV_VARIANT_AUTO, num_cu, out);
}

DCONV_EXPORT int dconv_plan_multi(int C, int M, int Wx, int Wy, int K, int variant, int num_cu,
                                  dconv_plan *out) {
  if (!out) return DCONV_ENULL;
  if (variant != DCONV_VARIANT_AUTO && variant != DCONV_VARIANT_VALU &&
      variant != DCONV_VARIANT_MFMA)
    return DCONV_EINVAL;
  int rc = validate_sizes(C, M, Wx, Wy, K);
  if (rc != DCONV_OK) return rc;
  dconv::MultiPlan p;
  if ((rc = dconv::plan_multi(C, M, Wx, Wy, K, variant, num_cu > 0 ? num_cu : 256, &p)) !=
      DCONV_OK)
    return rc;
  dconv::export_multi_plan(p, out);
  return DCONV_OK;
}
