/* The fp64 oracle (oracle/dconv_oracle.c) under AddressSanitizer and
 * UndefinedBehaviorSanitizer: a sweep of shapes (1x1 maps, K = W, tails,
 * several channels and filters) on one and on several threads, with and
 * without the sum of |I*F|, plus the rejected sizes.  Checks invariants that
 * need no second implementation: an all-ones filter on an all-ones input
 * gives C*K*K exactly, sum |I*F| >= |O|, and the single- and multi-threaded
 * runs agree bit for bit.  Prints "ok" and exits 0 when every check holds. */
#include <math.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int oracle_conv_f64(const float *I, const float *F, int C, int M, int Wx, int Wy, int K,
                    double *O, double *A, int nthreads);

static int failures = 0;
static void check(int ok, const char *what) {
  if (!ok) {
    printf("FAIL %s\n", what);
    ++failures;
  }
}

int main(void) {
  static const int shapes[][5] = {{1, 1, 1, 1, 1}, {2, 3, 5, 4, 2}, {3, 2, 7, 7, 7},
                                  {1, 4, 9, 3, 3}, {5, 1, 11, 13, 4}, {4, 3, 16, 9, 5}};
  size_t s;
  unsigned seed = 12345u;
  for (s = 0; s < sizeof(shapes) / sizeof(shapes[0]); ++s) {
    const int C = shapes[s][0], M = shapes[s][1], Wx = shapes[s][2], Wy = shapes[s][3],
              K = shapes[s][4];
    const int Hout = Wy - K + 1, Wout = Wx - K + 1;
    const size_t ni = (size_t)C * Wy * Wx, nf = (size_t)M * C * K * K, no = (size_t)M * Hout * Wout;
    float *I = malloc(ni * sizeof(float)), *F = malloc(nf * sizeof(float));
    float *I1 = malloc(ni * sizeof(float)), *F1 = malloc(nf * sizeof(float));
    double *O = malloc(no * sizeof(double)), *A = malloc(no * sizeof(double));
    double *O2 = malloc(no * sizeof(double)), *A2 = malloc(no * sizeof(double));
    size_t i;
    for (i = 0; i < ni; ++i) {
      seed = seed * 1103515245u + 12345u;
      I[i] = (float)((int)(seed >> 16) % 7 - 3);
      I1[i] = 1.0f;
    }
    for (i = 0; i < nf; ++i) {
      seed = seed * 1103515245u + 12345u;
      F[i] = (float)((int)(seed >> 16) % 7 - 3) * 0.5f;
      F1[i] = 1.0f;
    }
    check(oracle_conv_f64(I, F, C, M, Wx, Wy, K, O, A, 1) == 0, "oracle runs");
    check(oracle_conv_f64(I, F, C, M, Wx, Wy, K, O2, A2, 3) == 0, "oracle runs on 3 threads");
    check(memcmp(O, O2, no * sizeof(double)) == 0 && memcmp(A, A2, no * sizeof(double)) == 0,
          "thread count does not change the result");
    for (i = 0; i < no; ++i) check(A[i] >= fabs(O[i]), "sum |I*F| >= |O|");
    check(oracle_conv_f64(I, F, C, M, Wx, Wy, K, O2, NULL, 2) == 0, "oracle without A");
    check(oracle_conv_f64(I1, F1, C, M, Wx, Wy, K, O, NULL, 1) == 0, "ones");
    for (i = 0; i < no; ++i) check(O[i] == (double)C * K * K, "all-ones filter on all-ones input");
    free(I); free(F); free(I1); free(F1); free(O); free(A); free(O2); free(A2);
  }
  {
    float x = 1.0f;
    double o;
    check(oracle_conv_f64(&x, &x, 0, 1, 1, 1, 1, &o, NULL, 1) == -2, "C < 1 rejected");
    check(oracle_conv_f64(&x, &x, 1, 1, 1, 1, 2, &o, NULL, 1) == -2, "K > W rejected");
  }
  if (failures == 0) printf("ok\n");
  return failures == 0 ? 0 : 1;
}
