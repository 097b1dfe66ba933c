/*
 * libdconv: direct valid-mode stride-1 2-D convolution in fp32 on AMD Instinct
 * MI355X (gfx950).
 *
 * Operation (Chang, Onishi, Maruyama, "Fast convolution kernels on Pascal GPU
 * with high memory efficiency", Section 2.1, Eq. 1; Eq. 2 is the C = 1 case):
 *
 *   O[m][y][x] = sum_{c<C} sum_{r<K} sum_{s<K} I[c][y+r][x+s] * F[m][c][r][s]
 *
 *   for m < M, y < Hout = Wy-K+1, x < Wout = Wx-K+1.
 *
 * The paper writes the input as I^ch(x+i, y+j) with x the width coordinate
 * and the filter as F^{ch,m}(i, j).  This library stores maps with x fastest
 * and stores filters with the same convention, so the filter row index r is
 * the y offset j and the column index s is the x offset i.  No flip is
 * applied (a cross-correlation, as in CNN frameworks).  All indices are
 * 0-based.
 *
 * Layouts (row-major, contiguous, fp32, device memory):
 *   single: I[Wy][Wx]     F[M][K][K]     O[M][Hout][Wout]
 *   multi:  I[C][Wy][Wx]  F[M][C][K][K]  O[M][Hout][Wout]
 * Filters are stored channel first and filter number second (Section 2.3).
 *
 * Ownership and semantics common to every compute call:
 *   - I, F and O are device pointers owned by the caller; O must not overlap
 *     I or F.  Every element of O is written (O is not accumulated into).
 *   - Work is enqueued on `stream` (a hipStream_t; NULL is the null stream)
 *     and the call returns without waiting.  Faults during execution surface
 *     at the caller's next synchronisation.
 *   - Arguments are validated before any HIP call, so invalid sizes or NULL
 *     pointers never touch the device.
 *   - Results are accumulated in fp32 in a fixed order for a given shape and
 *     device, so repeated calls give bitwise identical output.
 *   - Calls on different streams may run concurrently; the library keeps no
 *     state that two calls share except an immutable per-device property
 *     cache and the per-(device, stream) workspace of dconv_multi.
 *   - Nothing is printed and the library never aborts.
 */
#ifndef DCONV_H
#define DCONV_H

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes returned by every call. */
#define DCONV_OK 0
#define DCONV_ENULL (-1)        /* a required pointer is NULL */
#define DCONV_EINVAL (-2)       /* C, M or K < 1, K > Wx, K > Wy, or bad variant */
#define DCONV_ERANGE (-3)       /* a tensor has more than 2^31-1 elements */
#define DCONV_EHIP (-4)         /* the HIP runtime reported an error */
#define DCONV_EUNSUPPORTED (-5) /* the forced variant cannot run this shape */
#define DCONV_ENOMEM (-6)       /* a stream-ordered workspace could not be allocated */

/* Kernel families for dconv_multi_variant / dconv_plan_multi. */
#define DCONV_VARIANT_AUTO 0 /* the planner's choice */
#define DCONV_VARIANT_VALU 1 /* direct convolution on the fp32 vector FMA units */
#define DCONV_VARIANT_MFMA 2 /* implicit GEMM over C*K*K on the fp32 matrix cores */

/*
 * dconv_single -- Eq. 2: one input map, M filters.
 *   I : device, Wy*Wx floats      F : device, M*K*K floats
 *   O : device, M*(Wy-K+1)*(Wx-K+1) floats, written
 *   Wx, Wy : map width (x, fastest) and height;  K : filter size;  M : filters
 *   stream : hipStream_t or NULL
 * Returns DCONV_OK, or DCONV_ENULL / DCONV_EINVAL / DCONV_ERANGE (nothing
 * launched), or DCONV_EHIP if a launch failed.
 */
int dconv_single(const float *I, const float *F, float *O, int Wx, int Wy, int K,
                 int M, void *stream);

/*
 * dconv_multi -- Eq. 1: C input maps, M filters of C channels each.
 *   I : device, C*Wy*Wx floats    F : device, M*C*K*K floats
 *   O : device, M*(Wy-K+1)*(Wx-K+1) floats, written
 *   note the argument order (C, M, Wx, Wy, K) differs from dconv_single
 * When the planner splits the channel sum across workgroups the partial
 * sums go to a workspace the library keeps per (device, stream): it is taken
 * from the device's default memory pool with a stream-ordered allocation the
 * first time a stream needs it (or needs more), reused by later calls on that
 * stream, and kept until the process ends; DCONV_ENOMEM if the allocation
 * fails.  The partial sums are added in a fixed order, so results stay
 * deterministic.  Other returns as for dconv_single.
 */
int dconv_multi(const float *I, const float *F, float *O, int C, int M, int Wx,
                int Wy, int K, void *stream);

/*
 * dconv_multi_variant -- dconv_multi with the kernel family forced
 * (DCONV_VARIANT_AUTO, _VALU or _MFMA), for A/B measurement of the vector
 * and matrix-core paths.  DCONV_EUNSUPPORTED if the forced family has no
 * kernel for this K (the matrix-core family covers K <= 7).
 */
int dconv_multi_variant(const float *I, const float *F, float *O, int C, int M,
                        int Wx, int Wy, int K, int variant, void *stream);

/* Human-readable text for a status code; never NULL, static storage. */
const char *dconv_strerror(int status);

/*
 * Launch plan, as chosen by the planner (host logic only, no device access).
 * Paper, Section 2.3 and Section 3: the work is divided among compute units
 * along the filters (m), along the map (x, y) and, for maps too small to fill
 * the chip, along the channels with a fixed-order sum of the partial results.
 */
typedef struct dconv_plan {
  int variant;          /* DCONV_VARIANT_VALU or DCONV_VARIANT_MFMA */
  int kernel;           /* internal kernel instance id (diagnostics) */
  int tile_m;           /* filters per workgroup */
  int tile_h, tile_w;   /* output rows and columns per workgroup tile */
  int chunk_c;          /* channels staged in LDS per pipeline step */
  int split_c;          /* channel groups summed across workgroups (1: none) */
  int grid_x, grid_y, grid_z;
  int block;            /* threads per workgroup */
  int lds_bytes;        /* LDS per workgroup */
  long long workspace_bytes; /* stream-ordered scratch (0: none) */
} dconv_plan;

/*
 * dconv_plan_single / dconv_plan_multi -- report the plan a call with these
 * sizes would use on a device with `num_cu` compute units (<= 0: 256).
 * Validation is the same as for the compute calls.  `out` must not be NULL.
 */
int dconv_plan_single(int Wx, int Wy, int K, int M, int num_cu, dconv_plan *out);
int dconv_plan_multi(int C, int M, int Wx, int Wy, int K, int variant, int num_cu,
                     dconv_plan *out);

#ifdef __cplusplus
}
#endif

#endif /* DCONV_H */
