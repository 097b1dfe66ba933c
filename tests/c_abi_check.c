/* A plain C99 caller of libdconv's C interface, without a GPU: the header
 * compiles as C, the library links from C, arguments are validated before
 * any HIP call (documented status codes), the host-side planners answer, and
 * the Section 2.2 latency model reproduces the paper's Table 1 for the
 * GTX 1080 Ti.  Exit status 0 when every check holds; each failure prints a
 * line naming the check. */
#include <stdio.h>
#include <string.h>

#include "dconv.h"

static int failures = 0;

static void check(int ok, const char *what) {
  if (!ok) {
    printf("FAIL %s\n", what);
    ++failures;
  }
}

int main(void) {
  /* Placeholders that are never dereferenced: validation rejects first. */
  const float *I = (const float *)0x1000, *F = (const float *)0x2000;
  float *O = (float *)0x3000;

  check(dconv_single(NULL, F, O, 8, 8, 3, 1, NULL) == DCONV_ENULL, "single NULL I");
  check(dconv_single(I, F, NULL, 8, 8, 3, 1, NULL) == DCONV_ENULL, "single NULL O");
  check(dconv_multi(I, NULL, O, 2, 2, 8, 8, 3, NULL) == DCONV_ENULL, "multi NULL F");
  check(dconv_single(I, F, O, 8, 8, 9, 1, NULL) == DCONV_EINVAL, "single K > Wx");
  check(dconv_single(I, F, O, 8, 8, 0, 1, NULL) == DCONV_EINVAL, "single K = 0");
  check(dconv_multi(I, F, O, 0, 2, 8, 8, 3, NULL) == DCONV_EINVAL, "multi C = 0");
  check(dconv_multi(I, F, O, 2, 0, 8, 8, 3, NULL) == DCONV_EINVAL, "multi M = 0");
  check(dconv_single_variant(I, F, O, 8, 8, 3, 1, 7, NULL) == DCONV_EINVAL, "single bad variant");
  check(dconv_single(I, F, O, 40000, 40000, 1, 2, NULL) == DCONV_ERANGE, "single output > 2^31-1");
  check(dconv_multi(I, F, O, 65536, 32768, 1, 1, 1, NULL) == DCONV_ERANGE, "multi input > 2^31-1");

  {
    int codes[] = {DCONV_OK, DCONV_ENULL, DCONV_EINVAL, DCONV_ERANGE,
                   DCONV_EHIP, DCONV_EUNSUPPORTED};
    size_t i;
    for (i = 0; i < sizeof(codes) / sizeof(codes[0]); ++i) {
      const char *s = dconv_strerror(codes[i]);
      check(s != NULL && strcmp(s, "unknown status") != 0, "strerror of a status code");
    }
    check(strcmp(dconv_strerror(12345), "unknown status") == 0, "strerror of an unknown code");
  }

  {
    dconv_plan p;
    check(dconv_plan_single(4096, 4096, 11, 1, 256, &p) == DCONV_OK, "plan single");
    check(p.grid_x * p.grid_y >= 256 && p.block == 256 && p.lds_bytes <= 160 * 1024,
          "plan single fills 256 CUs within LDS");
    check(dconv_plan_multi(512, 512, 9, 9, 3, DCONV_VARIANT_AUTO, 256, &p) == DCONV_OK,
          "plan multi");
    check(p.lds_bytes <= 160 * 1024 && p.grid_x >= 1, "plan multi within LDS");
    check(p.waves_c >= 1 && p.block % (64 * p.waves_c) == 0 && p.block <= 1024,
          "plan multi: wave groups of the channel sum inside one workgroup");
    check(dconv_plan_single_variant(4097, 64, 7, 1, DCONV_VARIANT_MFMA, 256, &p) ==
              DCONV_EUNSUPPORTED,
          "matrix-core single-map plan refused for rows not a multiple of 4 floats");
  }

  {
    /* Table 1 of the paper: GTX 1080 Ti, 258-clock latency, 484 GB/s at
     * 1480 MHz, 28 SMs of 128 cores, 2 flops per clock, 32-thread warps. */
    dconv_device_params d = {258.0, 484.0, 1480.0, 28, 128, 2, 32, 4, 98304};
    dconv_latency_model m;
    check(dconv_model_latency(&d, &m) == DCONV_OK, "latency model");
    check(m.n_fma == 66048, "Table 1 N_FMA = 66,048");
    check(m.bytes_per_clk == 327, "Table 1 327 bytes per clock");
    check(m.data_bytes == 84366, "Table 1 84,366 bytes in flight");
    check(m.threads_total == 21120, "21,120 threads");
    check(m.threads_per_cu == 768 && m.waves_per_cu == 24, "768 threads, 24 warps per SM");
    check(m.v_s == 86016, "Table 1 V_s = 86,016 bytes");
    check(dconv_model_latency(NULL, &m) == DCONV_ENULL, "latency model NULL");
  }

  {
    /* The host planners over a sweep of shapes (under the sanitizer build
     * this walks every planning path): every candidate list, the planners'
     * choices and the paper-rule plans, which must be among the candidates. */
    static const int Ks[] = {1, 2, 3, 5, 7, 9, 11, 13};
    static const int Ws[] = {1, 7, 9, 16, 30, 61, 114, 257, 1030};
    static const int Ms[] = {1, 3, 64, 130, 512};
    static const int Cs[] = {1, 5, 64, 513};
    dconv_device_params mi = {900.0, 8000.0, 2400.0, 256, 64, 2, 32, 4, 160 * 1024};
    dconv_plan cand[256], p, pp;
    size_t a, b, c, d;
    mi.wave_size = 64;
    for (a = 0; a < sizeof(Ks) / sizeof(Ks[0]); ++a)
      for (b = 0; b < sizeof(Ws) / sizeof(Ws[0]); ++b)
        for (c = 0; c < sizeof(Ms) / sizeof(Ms[0]); ++c) {
          const int K = Ks[a], W = Ws[b], M = Ms[c];
          int n = 0, i, found = 0;
          if (K > W) continue;
          check(dconv_plan_single_candidates(W, W + 3, K, M, DCONV_VARIANT_AUTO, 256, cand, 256,
                                             &n) == DCONV_OK && n >= 1 && n <= 256,
                "single candidates");
          check(dconv_plan_single(W, W + 3, K, M, 256, &p) == DCONV_OK, "plan single (sweep)");
          for (i = 0; i < n; ++i) found |= memcmp(&cand[i], &p, sizeof p) == 0;
          check(found, "the single planner's plan is a candidate");
          check(dconv_plan_single_paper(W, W + 3, K, M, &mi, &pp) == DCONV_OK, "single paper plan");
          for (d = 0; d < sizeof(Cs) / sizeof(Cs[0]); ++d) {
            const int C = Cs[d];
            int v;
            for (v = DCONV_VARIANT_AUTO; v <= DCONV_VARIANT_MFMA; ++v) {
              const int rc = dconv_plan_multi(C, M, W + 2, W, K, v, 256, &p);
              check(rc == DCONV_OK || (v == DCONV_VARIANT_MFMA && rc == DCONV_EUNSUPPORTED),
                    "plan multi (sweep)");
            }
            check(dconv_plan_multi_candidates(C, M, W + 2, W, K, DCONV_VARIANT_AUTO, 256, cand, 256,
                                              &n) == DCONV_OK && n >= 1,
                  "multi candidates");
            check(dconv_plan_multi_paper(C, M, W + 2, W, K, &mi, &pp) == DCONV_OK,
                  "multi paper plan");
          }
        }
  }

  if (failures == 0) printf("ok\n");
  return failures == 0 ? 0 : 1;
}
