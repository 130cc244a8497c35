/*
 * mpq.h - C ABI of the MI355X (gfx950) multipoint quantization library.
 *
 * Multipoint quantization (Liu, Ye, Zhou, Liu, "Post-training Quantization
 * with Multiple Points: Mixed Precision without Mixed Precision") replaces
 * each output channel's weight vector w (length d) of a linear or conv layer
 * by a sum  sum_{i<n} a_i * q_i  of n low-bit integer vectors q_i with fp32
 * scales a_i (Sec. 3.2, Eq. (4)).
 *
 * Conventions shared by every entry point
 *  - Array arguments are DEVICE pointers (hipMalloc memory or ROCm torch
 *    tensors) unless the comment says HOST.  Arrays are dense, row-major.
 *  - The caller owns every buffer.  The library keeps no pointer after the
 *    stream work of a call has completed.  Outputs must not alias inputs.
 *  - Calls enqueue work on `stream` (a hipStream_t; NULL = default stream)
 *    and return without waiting for it.  Argument checks are synchronous and
 *    happen before anything is enqueued; on an error nothing is enqueued.
 *  - Results are deterministic: identical inputs give bitwise identical
 *    outputs.  Calls on distinct streams may run concurrently.
 *  - Every call returns an MPQ_* status; mpq_last_error() describes the
 *    last failure of the calling thread.  No C++ exception crosses the ABI.
 *  - Inputs must be finite.
 *
 * Codes and scales (readings of the paper, shared with the test oracle)
 *  - bits b in [2, 8]; codes are the integers [-M, M] with M = 2^(b-1) - 1,
 *    i.e. the symmetric set of Eq. (1) with its 2M+1 points, B = 0 and the
 *    step K * eps_b folded into the scale.  -2^(b-1) is never produced.
 *  - Rounding to the nearest code (Eq. (2)) breaks exact half-way ties to
 *    the even integer.
 */
#ifndef MPQ_H
#define MPQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MPQ_OK 0
#define MPQ_ERR_INVALID_ARG (-1) /* a null pointer, a size or value out of range */
#define MPQ_ERR_SHAPE (-2)       /* d (with n_grid) too large for one workgroup's LDS */
#define MPQ_ERR_HIP (-3)         /* a HIP runtime call failed; see mpq_last_error() */
#define MPQ_ERR_NOMEM (-4)       /* device scratch allocation failed (or exceeded the
                                    MPQ_WORKSPACE_LIMIT environment variable: a cap in
                                    bytes on each scratch allocation, checked before
                                    any HIP call; unset means no cap) */

#define MPQ_MAX_BITS 8
#define MPQ_MAX_POINTS 64
#define MPQ_MAX_GRID 4096
#define MPQ_MAX_ERR_DIM 16777216   /* c_out and n of mpq_output_error */
#define MPQ_MAX_ERR_D 4194272      /* d of mpq_output_error (128 rows of the residual below 2 GiB) */
#define MPQ_MAX_INT_DIM 131072     /* d of mpq_integer_forward */

/*
 * mpq_fit_layer - greedy multipoint fit of every channel of a layer
 * (Sec. 3.2, Eq. (6)-(10), Algorithm 1, with the stopping rule of
 * Algorithm 2 / Eq. (12)).
 *
 * For each channel k (row W[k], length d), independently:
 *   r = w; n = 0
 *   loop:
 *     stop if n == max_points, or ||r||^2 == 0,
 *       or (n >= 1 and ||r||^2 <= tol * ||w||^2)
 *     candidate scales a_g = fl32(fl32(max_j |r_j|) * c_g / M), g = 1..G
 *     (products and quotient in fp64; Algorithm 1 sets the search grid up
 *     afresh from the residual at every step)
 *     a* = argmin_g || r - a_g * clip(round(r / a_g), -M, M) ||^2
 *          (Eq. (9); exactly equal errors: the smallest g; a candidate that
 *          rounds to 0 in fp32 is skipped, and if all do the fit stops)
 *     q* = clip(round(r / a*), -M, M)      (Eq. (10), fp64 quotient)
 *     r  = r - a* q*  (fp64)               (Eq. (7)); n += 1
 *   The stopping rule reads Algorithm 2's output-error threshold for an
 *   isotropic calibration distribution (E[x x^T] = I gives
 *   E (r . x)^2 = ||r||^2), relative to ||w||^2.  A nonzero channel always
 *   gets at least one point; an all-zero channel gets none.
 *
 * Arguments
 *   W          [c_out][d] fp32 weights (input).
 *   c_out, d   c_out >= 0 (0: nothing to do), d >= 1.
 *   bits       2..8.
 *   max_points 1..MPQ_MAX_POINTS: the per-channel cap on n.
 *   grid_host  HOST array of n_grid multipliers c_g, strictly ascending,
 *              each in (0, 1]; NULL selects c_g = g / n_grid (g = 1..n_grid,
 *              rounded to fp32).  Read before the call returns.
 *   n_grid     1..MPQ_MAX_GRID: number of candidate scales G.
 *   tol        relative stopping tolerance, finite and >= 0.
 *   codes      [c_out][max_points][d] int8 (output).  Rows at or after a
 *              channel's count are zero.
 *   scales     [c_out][max_points] fp32 (output), zero after the count.
 *   counts     [c_out] int32 (output): the number of points n of each channel.
 *   err_opt    NULL or [c_out][max_points] fp32 (output): ||r||^2 after
 *              each point (fp64 sum rounded to fp32), zero after the count.
 *   stream     hipStream_t or NULL.
 * Errors: MPQ_ERR_INVALID_ARG, MPQ_ERR_SHAPE (see mpq_fit_max_dim),
 *         MPQ_ERR_NOMEM, MPQ_ERR_HIP.
 */
int mpq_fit_layer(const float *W, int64_t c_out, int64_t d, int bits, int max_points,
                  const float *grid_host, int n_grid, float tol, int8_t *codes,
                  float *scales, int32_t *counts, float *err_opt, void *stream);

/*
 * How mpq_fit_layer evaluates Eq. (9): for d <= 32768 it counts, per element
 * and code level k, the candidates whose boundary (k + 1/2) a_g lies below
 * |r_j|, accumulates exact integer histograms, and gets every candidate's
 * error from ||r||^2 - 2 a A(g) + a^2 B(g) in fp64 (A, B: suffix sums), in
 * O(d M + G) per step; candidates whose error bound overlaps the minimum are
 * re-evaluated directly in fp64.  Longer channels use the dense search of
 * mpq_fit_layer_dense.
 *
 * mpq_fit_layer_dense - mpq_fit_layer with the dense candidate search:
 * every (element, candidate) pair is evaluated in fp32 on the residual
 * staged in LDS, with fp64 sums of 16-element blocks, in O(d G) per step.
 * Same arguments, outputs and errors as mpq_fit_layer; the two agree except
 * where the top-2 candidate errors lie within fp32 rounding of each other.
 */
int mpq_fit_layer_dense(const float *W, int64_t c_out, int64_t d, int bits, int max_points,
                        const float *grid_host, int n_grid, float tol, int8_t *codes,
                        float *scales, int32_t *counts, float *err_opt, void *stream);

/*
 * mpq_fit_max_dim - largest channel length d that mpq_fit_layer accepts for
 * n_grid candidates on the current device: the larger of 32768 (the
 * histogram search keeps a channel's residual in the registers of one
 * workgroup) and the dense search's limit (the residual staged in the LDS of
 * one workgroup).  Returns a negative MPQ_* status on failure.
 */
int64_t mpq_fit_max_dim(int n_grid);

/*
 * mpq_output_error - output error of the quantized layer on a calibration
 * batch (Sec. 3.3, Eq. (12)):
 *   err[k] = (1/n) sum_t ( (w_k - w~_k) . x_t )^2,
 *   ref[k] = (1/n) sum_t ( w_k . x_t )^2          (if ref_opt != NULL)
 * where w~_k = sum_{i<counts[k]} scales[k][i] * codes[k][i] and x_t is
 * column t of X.  The difference w_k - w~_k is formed in fp64 and rounded
 * to fp32; each fp32 product is summed from six products of the operands'
 * exact three-piece bf16 splits on the bf16 matrix cores, with fp32
 * accumulation (within one rounding of the fp32 product of an fp32 MFMA);
 * the sum over the batch is fp64.
 *
 * Arguments
 *   W, codes, scales, counts   as produced for mpq_fit_layer (inputs);
 *                              counts[k] in [0, max_points].
 *   c_out, d, max_points       as for mpq_fit_layer.
 *   X          [d][n] fp32 calibration inputs (input), n >= 1.
 *   c_out and n are at most MPQ_MAX_ERR_DIM, d at most MPQ_MAX_ERR_D.
 *   err        [c_out] fp32 (output).
 *   ref_opt    NULL or [c_out] fp32 (output).
 * Errors: MPQ_ERR_INVALID_ARG, MPQ_ERR_NOMEM, MPQ_ERR_HIP.
 */
int mpq_output_error(const float *W, const int8_t *codes, const float *scales,
                     const int32_t *counts, int64_t c_out, int64_t d, int max_points,
                     const float *X, int64_t n, float *err, float *ref_opt, void *stream);

/*
 * mpq_output_error_noalloc - mpq_output_error for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc).  Same arguments, kernels and results
 * (bitwise those of mpq_output_error on the same inputs); the call
 * allocates nothing.  Its workspace (the residual rows in tiles, row
 * partials and per-K-range outputs) is a fixed array of MPQ_NOALLOC_BYTES
 * per device, held by the library from the moment its code loads on that
 * device until the process ends.  A call whose workspace would exceed it
 * (about 4 ceil(c_out / 128) 128 ceil(d / 32) 32 bytes for the residual,
 * doubled with ref_opt, plus 8 c_out ceil(n / 128) and, for long d,
 * 4 c_out n per K range) returns MPQ_ERR_SHAPE before anything is enqueued.
 * Every call on one device shares that device's array and leaves its
 * contents behind: calls that overlap on one device (on different streams,
 * or from different threads before the first finishes) race and must be
 * ordered by the caller.  Errors: MPQ_ERR_INVALID_ARG, MPQ_ERR_SHAPE,
 * MPQ_ERR_HIP.
 */
#define MPQ_NOALLOC_BYTES (64 << 20)
int mpq_output_error_noalloc(const float *W, const int8_t *codes, const float *scales,
                             const int32_t *counts, int64_t c_out, int64_t d, int max_points,
                             const float *X, int64_t n, float *err, float *ref_opt, void *stream);

/*
 * mpq_reconstruct - the quantized weights of Eq. (4):
 *   W_hat[k][j] = fl32( sum_{i<counts[k]} scales[k][i] * codes[k][i][j] ),
 * summed in fp64 in point order.
 *   codes [c_out][max_points][d] int8, scales [c_out][max_points] fp32,
 *   counts [c_out] int32 in [0, max_points] (inputs); W_hat [c_out][d] fp32
 *   (output).
 * Errors: MPQ_ERR_INVALID_ARG, MPQ_ERR_HIP.
 */
int mpq_reconstruct(const int8_t *codes, const float *scales, const int32_t *counts,
                    int64_t c_out, int64_t d, int max_points, float *W_hat, void *stream);

/*
 * Batched calls: one call covers the layers of a network.  Each layer is
 * described by an mpq_layer (a HOST array of them is passed; the pointers in
 * it are DEVICE pointers); every call reads only the fields it names.  The
 * result is the same as calling the single-layer entry point on each layer
 * in order, on the same stream.  Layers whose channel lengths select the
 * same kernel share one launch, so a whole network costs a handful of
 * launches.  Arguments are checked for every layer before anything is
 * enqueued.
 */
typedef struct mpq_layer {
    const float *W;       /* [c_out][d] fp32 weights                               */
    int64_t c_out, d;
    int8_t *codes;        /* [c_out][max_points][d]                                */
    float *scales;        /* [c_out][max_points]                                   */
    int32_t *counts;      /* [c_out]                                               */
    float *fit_err;       /* mpq_fit_layers: NULL or [c_out][max_points] (err_opt) */
    const float *X;       /* mpq_output_error_layers: [d][n] calibration inputs    */
    int64_t n;            /* mpq_output_error_layers: columns of X                 */
    float *out_err;       /* mpq_output_error_layers: [c_out]                      */
    float *out_ref;       /* mpq_output_error_layers: NULL or [c_out]              */
    float *W_hat;         /* mpq_reconstruct_layers: [c_out][d]                    */
    float *fit_xerr;      /* mpq_fit_layers_calib: [c_out][max_points]             */
    float *offsets;       /* NULL, or [c_out]: asymmetric codes (mpq_fit_options.asym):
                             written by the fit, read by mpq_output_error_layers and
                             mpq_reconstruct_layers (w~ = offset + sum a q)      */
} mpq_layer;

/* mpq_fit_layer on every layer (reads W, c_out, d, codes, scales, counts,
 * fit_err).  All layers share bits, max_points, the grid and tol. */
int mpq_fit_layers(const mpq_layer *layers, int n_layers, int bits, int max_points,
                   const float *grid_host, int n_grid, float tol, void *stream);

/* mpq_output_error on every layer (reads W, c_out, d, codes, scales, counts,
 * X, n, out_err, out_ref). */
int mpq_output_error_layers(const mpq_layer *layers, int n_layers, int max_points, void *stream);

/* mpq_reconstruct on every layer (reads c_out, d, codes, scales, counts,
 * W_hat). */
int mpq_reconstruct_layers(const mpq_layer *layers, int n_layers, int max_points, void *stream);

/*
 * mpq_quantize_layers - the whole path for a network in one call: the fit of
 * every layer (mpq_fit_layers), then, for each layer with out_err != NULL,
 * its output error (Eq. (12), as mpq_output_error_layers; X, n, out_err and
 * out_ref are read) and, for each layer with W_hat != NULL, its quantized
 * weights (Eq. (4), as mpq_reconstruct_layers).  The outputs are bitwise
 * those of the three batched calls made in that order on the same stream.
 * The fit launches run side by side (as in mpq_fit_layers), with the upload
 * of the output error's descriptor tables beside them; a fit launch of at
 * least 2e6 weights other than the longest one is followed on its stream by
 * its layers' reconstruction; every fit also writes its layers' rows of the
 * output error's residual D (bitwise what the output error would form from
 * the stored points).  Then the
 * output errors of all layers run as one batch while the remaining layers
 * are reconstructed beside them.  The streams are the caller's and
 * library-owned ones joined back to it.
 * The fit is symmetric: the layers' offsets fields are ignored.
 * Arguments as for mpq_fit_layers; every layer is checked before anything is
 * enqueued.
 */
int mpq_quantize_layers(const mpq_layer *layers, int n_layers, int bits, int max_points,
                        const float *grid_host, int n_grid, float tol, void *stream);

/*
 * mpq_fit_layer_calib - the greedy fit of mpq_fit_layer with Algorithm 2's
 * stopping rule on a calibration batch (Sec. 3.3, Eq. (12)) instead of the
 * isotropic one.  For each channel k, after each point n >= 1:
 *   e_n = (1/n_cols) sum_t ( (w_k - w~_k,n) . x_t )^2     (x_t: column t of X)
 * is computed as mpq_output_error does (fp64 difference rounded to fp32,
 * fp32 products from bf16 pieces, fp64 sum over the batch), and the channel stops once
 *   e_n <= thr,  thr = eps * (1/n_cols) sum_t (w_k . x_t)^2   (relative != 0)
 *                thr = eps                                  (relative == 0),
 * or at max_points, or when its residual is zero.  The points themselves
 * are Algorithm 1's, which does not see X: a channel's points are the first
 * ones mpq_fit_layer would choose with tol = 0.  A nonzero channel gets at
 * least one point.
 *
 * The fit runs one step at a time: step s takes point s + 1 of every channel
 * still going, then scores those channels' output error on the batch (only
 * theirs), so the work follows the points each channel actually takes.
 *
 * Arguments as for mpq_fit_layer (tol replaced by eps and relative), plus
 *   X          [d][n] fp32 calibration inputs (input), 1 <= n <= MPQ_MAX_ERR_DIM.
 *   eps        threshold, finite and >= 0 (relative or absolute).
 *   relative   nonzero: thr relative to the output error of w itself.
 *   xerr       [c_out][max_points] fp32 (output): e_n after each point n,
 *              zero after the count.
 *   c_out <= MPQ_MAX_ERR_DIM; d within the histogram search (d <= 32768,
 *   else MPQ_ERR_SHAPE).
 * Errors: MPQ_ERR_INVALID_ARG, MPQ_ERR_SHAPE, MPQ_ERR_NOMEM, MPQ_ERR_HIP.
 */
int mpq_fit_layer_calib(const float *W, int64_t c_out, int64_t d, int bits, int max_points,
                        const float *grid_host, int n_grid, const float *X, int64_t n, float eps,
                        int relative, int8_t *codes, float *scales, int32_t *counts, float *err_opt,
                        float *xerr, void *stream);

/* mpq_fit_layer_calib on every layer (reads W, c_out, d, codes, scales,
 * counts, fit_err, X, n, fit_xerr).  Each step's fits run side by side and
 * its output errors run as one batch over all layers. */
int mpq_fit_layers_calib(const mpq_layer *layers, int n_layers, int bits, int max_points,
                         const float *grid_host, int n_grid, float eps, int relative, void *stream);

/*
 * mpq_fit_layers_ex - mpq_fit_layers with options (opt == NULL: exactly
 * mpq_fit_layers).
 *   refit     nonzero: once a point's codes q are fixed (Eq. (10) at the
 *             scale Eq. (9) chose), its scale becomes the least-squares
 *             scale for them, fl32(<r, q> / <q, q>) (fp64 sums), and the
 *             residual of Eq. (7) uses that scale.  A variant of Algorithm 1
 *             (which keeps the searched scale).
 *   calib     nonzero: the stopping rule of mpq_fit_layers_calib with eps and
 *             relative (reads X, n and fit_xerr of every layer; tol unused).
 *   clip_grid 0, or the number Gc of clipping factors of Eq. (13) (the paper
 *             uses 20, K in [0.05 : 0.05 : 1] * max|w|): point 1 of each
 *             channel is the naive quantization, at the code step
 *             fl32(fl32(max|w|) * fl32(j / Gc) / M), j = 1..Gc, whose output
 *             error on the layer's X is smallest (ties: the smallest j); the
 *             points after it follow Algorithm 1 with the stopping rule.
 *             Reads X and n of every layer; c_out * Gc <= MPQ_MAX_ERR_DIM.
 *             Cannot be combined with refit.
 *   asym      nonzero: asymmetric per-channel codes (Eq. (1) with B != 0): the
 *             offset beta = fl32((max_j w_j + min_j w_j) / 2) is written to the
 *             layer's offsets [c_out] (must not be NULL), the points fit
 *             w - beta, and w~ = beta + sum a q.  The stopping rules still
 *             compare with w's own error (||w||^2, or w's output energy).
 *             With either stopping rule and refit; not with clip_grid or
 *             paper_eta.  The batched output error and reconstruction add the
 *             offsets of layers whose offsets are not NULL.
 *   paper_eta 0, or eta > 0: the candidate scales of each step are the
 *             paper's own grid (Eq. (11), Def. 1): a = g * gamma,
 *             g = 1 .. floor(2 M ||r|| / gamma), gamma = min(Delta_r / M, eta),
 *             Delta_r half the smallest positive difference of the |r_j|
 *             (none: gamma = eta); the paper uses eta = 2^-10.  The grid is
 *             searched exactly without enumerating it; the chosen scale is
 *             stored as fl32(g * gamma), and the point's codes and residual
 *             use that value.  grid_host and n_grid are ignored.  Only with
 *             the isotropic stopping rule (not with refit, calib,
 *             clip_grid, asym or gate); d <= 32768 (else MPQ_ERR_SHAPE;
 *             channels past 8192 keep their sorted magnitudes in a stream-
 *             ordered scratch of about 8 (2 d) bytes for each of up to 1024
 *             channels in flight).
 *   gate      nonzero: Algorithm 2's naive first point (Sec. 3.3).  Each
 *             channel is first quantized naively, a_N = fl32(fl32(max|w|) / M)
 *             (the candidate c = 1), q = [w / a_N]_Q; if that point already
 *             meets the threshold of the stopping rule (isotropic:
 *             ||w - a_N q||^2 <= tol ||w||^2; calib: its output error
 *             e <= thr), it is the channel's only point; otherwise it is
 *             discarded and Algorithm 1 runs from w (max_points bounds
 *             Algorithm 1 only).  Without it point 1 is always Algorithm 1's.
 *             Not with clip_grid or paper_eta; with calib not with asym.
 * refit, calib and clip_grid need the histogram search for every layer
 * (d <= 32768; else MPQ_ERR_SHAPE).  Errors as for mpq_fit_layers /
 * mpq_fit_layers_calib.
 */
typedef struct mpq_fit_options {
    int refit;
    int calib;
    float eps;
    int relative;
    int clip_grid;
    float paper_eta;
    int asym;
    int gate;
} mpq_fit_options;
int mpq_fit_layers_ex(const mpq_layer *layers, int n_layers, int bits, int max_points,
                      const float *grid_host, int n_grid, float tol, const mpq_fit_options *opt,
                      void *stream);

/*
 * Deployment arithmetic (Sec. 3.4).
 *
 * mpq_integer_scales - the integer scales of Eq. (14):
 *   A[k][i] = nearest integer to 2^p * scales[k][i] (ties to even; 2^p a is
 *   exact in fp64) for i < counts[k], 0 after the count.  A value beyond
 *   the 32-bit range is clamped to +-(2^31 - 1); if n_clamped_opt is not
 *   NULL, the number of clamped values is added to it (a DEVICE uint64 the
 *   caller zeroes).
 *   scales [c_out][max_points] fp32, counts [c_out] int32 in [0, max_points]
 *   (inputs); A [c_out][max_points] int32 (output); 0 <= p <= 62.
 * Errors: MPQ_ERR_INVALID_ARG, MPQ_ERR_HIP.
 */
int mpq_integer_scales(const float *scales, const int32_t *counts, int64_t c_out, int max_points, int p,
                       int32_t *A, unsigned long long *n_clamped_opt, void *stream);

/*
 * mpq_integer_forward - a multipoint layer's integer dot products on a batch
 * of integer activations (Eq. (15), Steps 1-3).  For channel k and column t:
 *   Step 1  z_i = q_{k,i} . x_t   for i < counts[k], in 32-bit accumulators
 *           (int8 MFMA; exact for codes in [-127, 127], as the fit writes
 *           them, any int8 activations and d <= MPQ_MAX_INT_DIM)
 *   Step 2  s = sum_{i < counts[k]} A[k][i] * z_i, in 64 bits
 *   Step 3  Y[k][t] = s >> p, an arithmetic right shift (floor(s / 2^p))
 * Y is exact while |s| < 2^63 (e.g. |A| < 2^31 and counts[k] * d * 128 * 128
 * < 2^32).  Codes past a channel's count, and their A, are not read.
 *
 * Arguments
 *   codes    [c_out][max_points][d] int8 (the fit's codes), A [c_out][max_points]
 *            int32 (mpq_integer_scales), counts [c_out] int32 in [0, max_points].
 *   X        [n][d] int8: column t of the batch is the contiguous row X[t]
 *            (signed activation integers; the batch is stored transposed
 *            with respect to mpq_output_error's fp32 X).
 *   Y        [c_out][n] int64 (output).
 *   c_out, n >= 0; 1 <= d <= MPQ_MAX_INT_DIM; codes and X each below 2^31
 *   bytes; 0 <= p <= 62.
 * Errors: MPQ_ERR_INVALID_ARG, MPQ_ERR_HIP.
 */
int mpq_integer_forward(const int8_t *codes, const int32_t *A, const int32_t *counts, int64_t c_out,
                        int64_t d, int max_points, const int8_t *X, int64_t n, int p, int64_t *Y,
                        void *stream);

/* mpq_integer_forward on a list of layers (HOST array; DEVICE pointers),
 * with one launch per 32 layers.  All layers share max_points and p. */
typedef struct mpq_int_layer {
    const int8_t *codes;    /* [c_out][max_points][d] */
    const int32_t *A;       /* [c_out][max_points]    */
    const int32_t *counts;  /* [c_out]                */
    int64_t c_out, d;
    const int8_t *X;        /* [n][d]                 */
    int64_t n;
    int64_t *Y;             /* [c_out][n]             */
} mpq_int_layer;
int mpq_integer_forward_layers(const mpq_int_layer *layers, int n_layers, int max_points, int p,
                               void *stream);

/*
 * Per-launch timing (instrumentation, not part of the method).  While it is
 * enabled, every kernel launch of the library is bracketed by two HIP events
 * recorded on the stream the kernel runs on (a call may run independent
 * launches on library-owned streams, joined back to the caller's stream).
 *
 * mpq_timing_enable(on): drops the records collected so far and turns the
 *   recording on (on != 0) or off.  Returns MPQ_OK.
 * mpq_timing_only(name): while the recording is on, record only the
 *   launches of the kernel of this name (a HOST string of up to 63 bytes, as
 *   mpq_timing_read reports it), so that timing one kernel adds no events
 *   around the others; NULL or "" records every launch again.  Returns MPQ_OK,
 *   or MPQ_ERR_INVALID_ARG for a longer name.
 * mpq_timing_read(out, cap): waits for the recorded events, writes up to cap
 *   records (HOST array) in launch order and returns the number of records
 *   (which may exceed cap), or MPQ_ERR_INVALID_ARG.  ms is -1 for a record
 *   whose events could not be read.
 * mpq_fit_kernel_of(d, bits, n_grid, default_grid, name, cap): writes to the
 *   HOST buffer name (cap bytes) the kernel name under which mpq_fit_layer
 *   records the fit of channels of length d (default_grid: grid_host ==
 *   NULL).  Returns an MPQ_* status.
 */
typedef struct mpq_kernel_time {
    char name[64];
    float ms;
} mpq_kernel_time;

int mpq_timing_enable(int on);
int mpq_timing_only(const char *name);
int mpq_timing_read(mpq_kernel_time *out, int cap);
int mpq_fit_kernel_of(int64_t d, int bits, int n_grid, int default_grid, char *name, int cap);

/* Text of the calling thread's last failure ("" if none).  The pointer stays
 * valid until the thread's next failing call. */
const char *mpq_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* MPQ_H */
