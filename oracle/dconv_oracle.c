/*
 * Reference oracle for direct valid-mode stride-1 2-D convolution.
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the plain, slow CPU definition that
 * the GPU library is checked against.  Only the test suite, the smoke check
 * and the CPU-baseline leg of the benchmark may build, load or call it; the
 * library itself never does, and the two share no code.
 *
 * What it computes (paper, Section 2.1, Eq. 1; Eq. 2 is the case C = 1):
 *
 *   O^m(x, y) = sum_{ch} sum_{i=0}^{K-1} sum_{j=0}^{K-1} I^ch(x+i, y+j) * F^{ch,m}(i, j)
 *
 *   for x in [0, Wx-K+1), y in [0, Wy-K+1), every filter m and channel ch.
 *
 * Readings taken where the paper leaves the storage open:
 *   - x is the width coordinate and is the fastest-varying index of a map, so
 *     I^ch(x, y) lives at I[ch][y][x] (row-major [C][Wy][Wx]).
 *   - The filter follows the same convention as the map: F^{ch,m}(i, j) lives
 *     at F[m][ch][j][i], i.e. the filter row index goes with the y offset and
 *     the column index with the x offset.  Filters are stored channel first,
 *     then filter number (Section 2.3), giving F[M][C][K][K].
 *   - Indices are 0-based; no flip is applied (Eq. 1 has none), so this is a
 *     cross-correlation.
 *   - Output O[M][Wy-K+1][Wx-K+1], row-major.
 *
 * Arithmetic: every product of two fp32 values is exact in fp64 and the sum is
 * accumulated in fp64 in the fixed order ch, j, i.  Alongside the value the
 * oracle returns A = sum |I * F| per output, which scales the tolerance for
 * results computed in fp32.
 *
 * Build: gcc -O2 -ffp-contract=off -fopenmp -shared -fPIC (see oracle/build.py).
 * The OpenMP loop only splits the independent outputs between threads; each
 * output is still summed by one thread in the order above.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/*
 * oracle_conv_f64
 *   I  : C*Wy*Wx input values, layout [C][Wy][Wx]
 *   F  : M*C*K*K filter values, layout [M][C][K][K]
 *   O  : M*Hout*Wout outputs (fp64), layout [M][Hout][Wout]
 *   A  : same shape as O, receives sum |I*F| per output (may be NULL)
 *   nthreads : OpenMP threads to use (<= 0: one thread)
 * Returns 0, or -2 if a size is out of range (nothing is written then).
 */
int oracle_conv_f64(const float *I, const float *F, int C, int M, int Wx,
                    int Wy, int K, double *O, double *A, int nthreads) {
  if (C < 1 || M < 1 || K < 1 || K > Wx || K > Wy)
    return -2;
  const int64_t Hout = (int64_t)Wy - K + 1;
  const int64_t Wout = (int64_t)Wx - K + 1;
  const int64_t rows = (int64_t)M * Hout;
  if (nthreads < 1)
    nthreads = 1;

#pragma omp parallel for schedule(static) num_threads(nthreads)
  for (int64_t row = 0; row < rows; ++row) {
    const int64_t m = row / Hout;
    const int64_t y = row % Hout;
    for (int64_t x = 0; x < Wout; ++x) {
      double acc = 0.0;
      double absacc = 0.0;
      for (int64_t ch = 0; ch < C; ++ch) {
        for (int64_t j = 0; j < K; ++j) {     /* offset along y */
          for (int64_t i = 0; i < K; ++i) {   /* offset along x */
            const double v = (double)I[(ch * Wy + (y + j)) * Wx + (x + i)];
            const double f = (double)F[((m * C + ch) * K + j) * K + i];
            const double p = v * f;
            acc += p;
            absacc += fabs(p);
          }
        }
      }
      O[(m * Hout + y) * Wout + x] = acc;
      if (A)
        A[(m * Hout + y) * Wout + x] = absacc;
    }
  }
  return 0;
}

/* Number of OpenMP threads available to this library (1 when compiled without OpenMP). */
int oracle_max_threads(void) {
#ifdef _OPENMP
  return omp_get_max_threads();
#else
  return 1;
#endif
}
