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
 *   - The library allocates no device memory and needs no workspace: every
 *     call reads and writes the caller's three tensors only (and the latency
 *     probe its own two arguments).
 *   - Calls on different streams may run concurrently; the library keeps no
 *     state that two calls share except an immutable per-device property
 *     cache (compute-unit counts, read once).
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

/* Kernel families for the *_variant calls and the plans. */
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
 * dconv_single_variant -- dconv_single with the kernel family forced:
 * DCONV_VARIANT_VALU (vector FMAs), DCONV_VARIANT_MFMA (the fp32 matrix
 * cores on a banded form of each filter row) or DCONV_VARIANT_AUTO (the
 * planner's choice, what dconv_single does).  DCONV_EUNSUPPORTED if the
 * matrix-core family is forced where it has no kernel (K < 5, K > 11, or an
 * input whose rows are not 16-byte aligned: I not 16-byte aligned or Wx not
 * a multiple of 4).  Other returns as for dconv_single.
 */
int dconv_single_variant(const float *I, const float *F, float *O, int Wx, int Wy, int K,
                         int M, int variant, void *stream);

/*
 * dconv_multi -- Eq. 1: C input maps, M filters of C channels each.
 *   I : device, C*Wy*Wx floats    F : device, M*C*K*K floats
 *   O : device, M*(Wy-K+1)*(Wx-K+1) floats, written
 *   note the argument order (C, M, Wx, Wy, K) differs from dconv_single
 * The channel sum of every output stays inside one workgroup (Section 2.3
 * rejects dividing it over processors); where a workgroup's waves split a
 * stage's channels, their partial sums are added through LDS in a fixed
 * order, so results are deterministic.  Returns as for dconv_single.
 */
int dconv_multi(const float *I, const float *F, float *O, int C, int M, int Wx,
                int Wy, int K, void *stream);

/*
 * dconv_multi_variant -- dconv_multi with the kernel family forced
 * (DCONV_VARIANT_AUTO, _VALU or _MFMA), for A/B measurement of the vector
 * and matrix-core paths.  DCONV_EUNSUPPORTED if the forced family has no
 * kernel for this K (the matrix-core family covers K <= 11).
 */
int dconv_multi_variant(const float *I, const float *F, float *O, int C, int M,
                        int Wx, int Wy, int K, int variant, void *stream);

/* Human-readable text for a status code; never NULL, static storage. */
const char *dconv_strerror(int status);

/*
 * Launch plan, as chosen by the planner (host logic only, no device access).
 * Paper, Section 2.3 and Section 3: the work is divided among compute units
 * along the filters (m) and along the map (x, y); the channel sum of an
 * output is never divided among workgroups, only among the waves of one.
 */
typedef struct dconv_plan {
  int variant;          /* DCONV_VARIANT_VALU or DCONV_VARIANT_MFMA */
  int kernel;           /* internal kernel instance id (diagnostics) */
  int tile_m;           /* filters per workgroup */
  int tile_h, tile_w;   /* output rows and columns per workgroup tile */
  int chunk_c;          /* channels staged in LDS per pipeline step */
  int waves_c;          /* wave groups of a workgroup that split each stage's
                           channels (their sums added through LDS; 1: none) */
  int grid_x, grid_y, grid_z;
  int block;            /* threads per workgroup */
  int lds_bytes;        /* LDS per workgroup */
} dconv_plan;

/*
 * dconv_plan_single / dconv_plan_multi -- report the plan a call with these
 * sizes would use on a device with `num_cu` compute units (<= 0: 256).
 * Validation is the same as for the compute calls.  `out` must not be NULL.
 */
int dconv_plan_single(int Wx, int Wy, int K, int M, int num_cu, dconv_plan *out);
/* The plan dconv_single_variant would use (the input assumed 16-byte aligned). */
int dconv_plan_single_variant(int Wx, int Wy, int K, int M, int variant, int num_cu,
                              dconv_plan *out);
int dconv_plan_multi(int C, int M, int Wx, int Wy, int K, int variant, int num_cu,
                     dconv_plan *out);

/*
 * dconv_plan_multi_candidates -- every plan of a kernel family (both
 * families for DCONV_VARIANT_AUTO) that fits a device with `num_cu` compute
 * units: each workgroup shape, in a fixed order.  dconv_plan_multi returns
 * one of them (the planner's estimate is the smallest).  Writes min(count, capacity) plans to `out` (may be NULL when
 * capacity is 0) and the total to *count.  For autotuning (Section 3 divides
 * the work by rules; these are the alternatives the rules choose from).
 */
int dconv_plan_multi_candidates(int C, int M, int Wx, int Wy, int K, int variant, int num_cu,
                                dconv_plan *out, int capacity, int *count);

/*
 * dconv_multi_with_plan -- dconv_multi with a plan chosen by the caller, which
 * must equal (field by field) one of the candidates dconv_plan_multi_candidates
 * returns for these sizes on the current device; DCONV_EINVAL otherwise.
 * Semantics and returns as for dconv_multi.
 */
int dconv_multi_with_plan(const float *I, const float *F, float *O, int C, int M, int Wx,
                          int Wy, int K, const dconv_plan *plan, void *stream);

/*
 * dconv_plan_single_candidates -- every single-map plan for these sizes on a
 * device with `num_cu` compute units (<= 0: 256), the input assumed 16-byte
 * aligned with Wx a multiple of 4 (as dconv_plan_single_variant): each tile
 * shape of the vector kernel (tall or short tiles, 64 or 16 lanes across a
 * row) and, for DCONV_VARIANT_AUTO / _MFMA with K in 5..11, the matrix-core
 * kernel, crossed with the division of the M filters into groups of
 * workgroups (Section 3.1 divides the filters over processors, or the map).
 * Fixed order; dconv_plan_single returns one of them.  Writes
 * min(count, capacity) plans to `out` (may be NULL when capacity is 0) and
 * the total to *count.
 */
int dconv_plan_single_candidates(int Wx, int Wy, int K, int M, int variant, int num_cu,
                                 dconv_plan *out, int capacity, int *count);

/*
 * dconv_single_with_plan -- dconv_single with a plan chosen by the caller,
 * which must equal (field by field) one of the candidates for these sizes on
 * the current device and for the alignment of I (a 16-byte-aligned input
 * with Wx a multiple of 4 has the candidates of
 * dconv_plan_single_candidates; other inputs have the single-float staging
 * kernel's); DCONV_EINVAL otherwise.  Semantics and returns as for
 * dconv_single.
 */
int dconv_single_with_plan(const float *I, const float *F, float *O, int Wx, int Wy, int K,
                           int M, const dconv_plan *plan, void *stream);

/*
 * The paper's partition model (host arithmetic only, no device access).
 *
 * Section 2.2 and Table 1: to hide a global-memory latency of L clocks a
 * processor needs N_FMA = L x lanes x (operations per lane per clock) of work
 * per data set, or the memory must have V_s bytes in flight: the bytes it
 * delivers per clock (bandwidth / clock, rounded down) times L, fetched one
 * word per thread (rounded up to whole warps/wavefronts), spread over the
 * processors and rounded up to whole warps/wavefronts again.  Table 1 (GTX 1080 Ti: L = 258, 484 GB/s, 1480 MHz, 28
 * SMs of 128 cores, 2 per core per clock, warps of 32, 4-byte words, 96 KB
 * shared memory) gives N_FMA = 66,048, 327 B/clock, 84,366 B, 21,120
 * threads, 768 threads = 24 warps = 3,072 B per SM, V_s = 86,016 B.
 */
typedef struct dconv_device_params {
  double latency_clk;    /* global-memory latency, clock cycles */
  double bandwidth_gbs;  /* memory bandwidth, 1e9 bytes per second */
  double clock_mhz;      /* the clock the latency is counted in */
  int num_cu;            /* processors (SMs, compute units) */
  int lanes_per_cu;      /* arithmetic lanes per processor */
  int ops_per_clk_lane;  /* per lane per clock, as the paper counts for N_FMA */
  int wave_size;         /* threads per warp / wavefront */
  int word_bytes;        /* bytes each thread fetches per load */
  int onchip_bytes;      /* shared memory / LDS per processor */
} dconv_device_params;

typedef struct dconv_latency_model {
  long long n_fma;       /* N_FMA */
  int bytes_per_clk;     /* transmission rate */
  long long data_bytes;  /* bytes in flight over one latency */
  long long threads_total; /* data_bytes / word_bytes, rounded up to whole waves */
  int threads_per_cu;    /* threads_total / num_cu, rounded up to whole waves */
  int waves_per_cu;
  int bytes_per_cu;      /* threads_per_cu x word_bytes */
  long long v_s;         /* V_s = bytes_per_cu x num_cu */
} dconv_latency_model;

/* Section 2.2 / Table 1.  DCONV_ENULL, or DCONV_EINVAL if a field is <= 0. */
int dconv_model_latency(const dconv_device_params *dev, dconv_latency_model *out);

/*
 * Section 3.1, single-channel division of an Wx x Wy map and M K x K filters
 * over the processors.  Method 1: filters divided along m, the map streamed
 * in P pieces along y; on-chip data D1 = (K^2 ceil(M/N) + (ceil(Wy/P)+K-1) Wx)
 * x word, work Th1 = K^2 ceil(M/N) ceil(Wy/P) Wx.  Method 2: map divided along
 * y, filters streamed in Q pieces; D2 = (K^2 ceil(M/Q) + (ceil(Wy/N)+K-1) Wx)
 * x word, Th2 = K^2 ceil(M/Q) ceil(Wy/N) Wx.  P and Q are bounded above by
 * Th >= N_FMA (and by Wy, M) and below by D <= on-chip bytes; the smallest
 * admissible value is taken (1 if none), and the method with the smaller D
 * is kept (the other factor is reset to 1).
 */
typedef struct dconv_single_split {
  int method;                 /* 1 or 2 */
  int P, Q;                   /* the chosen factors */
  long long D1, D2;           /* bytes, at the admissible (or unit) P and Q */
  long long Th1, Th2;         /* multiply-adds per data set */
  long long p_lo, p_hi;       /* bounds on P (p_lo = -1: on-chip bound unreachable) */
  long long q_lo, q_hi;       /* bounds on Q */
  int p_admissible, q_admissible;
} dconv_single_split;

int dconv_model_single(const dconv_device_params *dev, const dconv_latency_model *lm, int Wx,
                       int Wy, int K, int M, dconv_single_split *out);

/*
 * Section 3.2, the stride-fixed block of the multi-channel kernel: a segment
 * of S bytes of each filter along the channels (S a multiple of the word),
 * W'x map pixels, W'y = ceil(S / (K x word)) map lines, the smallest M' with
 * M' x (S / word) x W'x >= N_FMA, and whether the data set
 * S x M' + W'y x W'x x word fits in half the on-chip memory.
 */
typedef struct dconv_multi_block {
  int S, Wx_p, Wy_p, M_p;
  long long set_bytes;
  long long fma_per_set;
  int fits;
} dconv_multi_block;

int dconv_model_multi(const dconv_device_params *dev, const dconv_latency_model *lm, int K,
                      int S, int Wxp, dconv_multi_block *out);

/*
 * dconv_plan_multi_paper -- the Section 3.2 rules applied to this library's
 * multi-channel plans for a device described by `dev` (its num_cu and
 * onchip_bytes included): among the candidates that keep the channel sum
 * inside a workgroup (the paper does not split it across processors), those
 * whose stage gives each compute unit at least N_FMA multiply-adds (the
 * co-resident workgroups, as many as the on-chip memory holds, counted
 * together); of these the fewest filters per workgroup (smallest M'), then
 * the most pixels per tile (largest W'x).  If none reaches N_FMA, the
 * candidate with the most work per compute unit.  For comparison with the
 * library's own planner and with exhaustive search; `out` can be passed to
 * dconv_multi_with_plan when dev->num_cu is the device's count.
 */
int dconv_plan_multi_paper(int C, int M, int Wx, int Wy, int K, const dconv_device_params *dev,
                           dconv_plan *out);

/*
 * dconv_plan_single_paper -- the Section 3.1 division applied to this
 * library's single-map plans for a device described by `dev`
 * (dconv_model_single decides the method).  Method 1, filters divided over
 * the processors and the map walked in P pieces: the vector-kernel candidate
 * whose number of filter groups is closest to min(M, num_cu), then whose tile
 * height is closest to Hout / P.  Method 2, the map divided over the
 * processors and all filters applied by each: among the candidates with one
 * filter group, the tile height closest to Hout / num_cu, then the most
 * workgroups.  For comparison with the library's planner and with exhaustive
 * search; `out` can be passed to dconv_single_with_plan when dev->num_cu is
 * the device's count and the input is 16-byte aligned with Wx % 4 == 0.
 */
int dconv_plan_single_paper(int Wx, int Wy, int K, int M, const dconv_device_params *dev,
                            dconv_plan *out);

/*
 * dconv_probe_latency -- measure the latency the model above takes as input
 * (Section 2.2 uses a pointer-chasing measurement).  One lane follows
 * j <- chain[j] from j = 0 for `steps` dependent loads; the caller's chain
 * (device memory, every entry a valid index into it) sets the footprint and
 * so which level of the memory hierarchy is measured.  Writes to the device
 * array out[3]: elapsed shader clock cycles (s_memtime), elapsed ticks of the
 * constant 100 MHz counter (s_memrealtime), and the final index.  Enqueued on
 * `stream`; read `out` after synchronising.
 */
int dconv_probe_latency(const int *chain, int steps, long long *out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* DCONV_H */
