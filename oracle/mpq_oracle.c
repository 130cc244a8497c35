/*
 * Oracle for the per-channel greedy multipoint fit, its output error and
 * its reconstruction.  Plain, slow, fp64.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * benchmark's CPU-baseline leg load this library.  The HIP library never
 * links, includes or calls it, and it shares no code with the HIP library.
 *
 * What it computes (Liu, Ye, Zhou, Liu, "Post-training Quantization with
 * Multiple Points: Mixed Precision without Mixed Precision"):
 *   Sec. 3.1, Eq. (1)-(3): the symmetric b-bit set and nearest rounding.
 *   Sec. 3.2, Eq. (4)-(10) and Algorithm 1: approximate a channel w by
 *     sum_i a_i * q_i, adding one (a, q) pair per step, each fitted to the
 *     current residual; a by grid search over candidate scales (Eq. (9)),
 *     q as the rounding of r / a (Eq. (8), (10)); residual by Eq. (7).
 *   Sec. 3.3, Eq. (12) and Algorithm 2: output error on a calibration
 *     batch; points are added until the error falls below a threshold.
 *   Sec. 3.4, Eq. (14)-(15): integer scales A_i = [2^p a_i] and the layer's
 *     integer dot products in three steps (point products in 32-bit
 *     accumulators, the A_i-weighted sum, a shift by p).
 *
 * Readings taken where the paper is silent, ambiguous or garbled (the same
 * readings bind the HIP library):
 *   Q1/K1  Codes are the integers [-M, M], M = 2^(b-1) - 1 (Eq. (1) with
 *          B = 0 and K * eps_b folded into the scale a).
 *   R1     Nearest rounding breaks exact half-way ties to even.
 *   G1/G2  Candidate scales: a_g = fl32(m * c_g / M) with m = fl32(max|r|)
 *          recomputed at every step and multipliers 0 < c_1 < ... < c_G <= 1
 *          (default c_g = g / G).  Products and the quotient are fp64.
 *   T1     Among exactly equal candidate errors the smallest g wins.
 *   S1-S3  Stop after n points when n == max_points, or ||r||^2 == 0, or
 *          every candidate scale rounds to zero in fp32 (zero candidates
 *          are skipped in the search), or n >= 1
 *          and ||r||^2 <= tol * ||w||^2 (the output error of Eq. (12) under
 *          an isotropic calibration distribution).  A nonzero channel
 *          always gets at least one point; an all-zero channel gets none.
 *   S4     Algorithm 2 on a calibration batch X [d][N] (oracle_fit_calib):
 *          after n >= 1 points the channel's output error
 *          e_n = (1/N) sum_t ((w - sum_{i<n} a_i q_i) . x_t)^2 (Eq. (12)) is
 *          compared with a threshold thr, eps itself (the paper's absolute
 *          epsilon) or eps * (1/N) sum_t (w . x_t)^2 (relative); the fit
 *          stops when e_n <= thr (Algorithm 2 applies Algorithm 1 while
 *          e > eps), or at max_points, ||r||^2 == 0 or no nonzero scale.
 *          The points are still chosen by Eq. (9): Algorithm 1 fits the
 *          residual, Algorithm 2 only decides how many points to take.
 *   F1     Variant (gate != 0), Algorithm 2's first step: the channel is
 *          first quantized naively, w~ = a_N [w / a_N]_Q with the max-abs
 *          code step a_N = fl32(fl32(max|w|) / M) (fp64 quotient; the
 *          candidate c = 1 of reading G2); if its error already meets the
 *          threshold of the rule in force (S1: ||w - w~||^2 <= tol ||w||^2;
 *          S4: e <= thr on the batch), it is the channel's only point;
 *          otherwise it is discarded and Algorithm 1 runs from r_1 = w as
 *          without the gate (the cap max_points bounds Algorithm 1 only).  Without the
 *          gate (the default) point 1 is Algorithm 1's grid search from the
 *          start, so a channel whose naive point would pass can get a
 *          different first point, and under S4 more points.
 *   A1     No refit of a once q is fixed (the method as printed).
 *   A2     Variant (refit != 0): once q is fixed by Eq. (10) at the searched
 *          a*, the point's scale is the least-squares one for that q,
 *          a = fl32(<r, q> / <q, q>) (fp64 sums in index order), and the
 *          residual of Eq. (7) uses it.
 *   E1     Output error: mean over the N columns of X of ((w - w~) . x)^2.
 *   P1     Scales are stored as fp32 values (exactly the candidate value).
 *   C1     Variant (clip != 0): the clipping of Eq. (13) per channel (the set
 *          of weights sharing K is one channel).  K runs over
 *          [0.05 : 0.05 : 1] * max|w|, i.e. the candidate scales a_j =
 *          fl32(fl32(max|w|) c_j / M), c_j = fl32(j / 20); the first point is
 *          (a_j, [w / a_j]_Q) for the j whose output error on X is smallest
 *          (ties: the smallest j; zero scales skipped); Algorithm 1 then
 *          continues from that point with the stopping rule, as the paper
 *          fixes K before adding points.
 *   D1     Def. 1's minimal gap: half the smallest difference | |t_i| - |t_j| |
 *          over pairs with |t_i| != |t_j| (the printed constraint t_i != t_j
 *          would make it zero for t_i = -t_j); none such: no gap.
 *   G3     Variant (paper_grid != 0), Eq. (11) with eta: the candidates of a
 *          step are a_g = g * gamma (fp64), g = 1 .. floor(2 M ||r|| / gamma),
 *          gamma = min(Delta_r / M, eta) in fp64 (no gap: gamma = eta); the
 *          scale 0 is left out (Theorem 1 searches (0 : gamma : 2M||r||]).
 *          The chosen scale is stored as fl32(a_g) (P1) and the point's codes
 *          (Eq. (10)) and residual use that stored value.
 *          The grid's argmin of Eq. (9) is found without enumerating it: the
 *          codes are constant between consecutive breakpoints |r_j| / (k+1/2),
 *          where E is a convex quadratic, so the argmin is one of the three
 *          grid points around a breakpoint or one of the two next to the
 *          vertex A / B of the piece that holds such a point; every such
 *          candidate is evaluated by Eq. (9) and the smallest error wins
 *          (ties: the smallest g).
 *   B2     Variant (asym != 0), the asymmetric set of Eq. (1) with B != 0
 *          per channel: the offset beta = fl32((max_j w_j + min_j w_j) / 2)
 *          (fp64 midpoint) takes B's place, the points fit w - beta
 *          (Algorithm 1 on the centred weights, r_1 = w - beta), and
 *          w~ = beta + sum_i a_i q_i.  The stopping rules still compare the
 *          error of w~ with w's own (||w||^2, or the output energy of w).
 *   I1     Eq. (14) rounds 2^p a_i to the nearest integer with ties to even
 *          (R1); a value outside the 32-bit range is clamped to
 *          [-(2^31 - 1), 2^31 - 1] and counted.
 *   B1     Step 3's "shift by p bits" is a division by 2^p: an arithmetic
 *          right shift of the 64-bit sum, i.e. the floor of sum / 2^p.
 *   I2     Activations are signed integers held in int8, one vector of d per
 *          column of the batch; Step 2 sums in 64 bits.
 *
 * Pins (tests/oracle_pins.py) tie every function here to the paper, exact
 * arithmetic, brute force or library routines; the only part left without
 * one ("parity unpinned") is the exponential rate of Theorem 1, whose
 * constants the paper does not give.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* Eq. (1): [-1 : eps_b : 1] with eps_b = 1 / (2^(b-1) - 1) has 2M+1 points,
 * M = 2^(b-1) - 1. */
int oracle_levels(int bits) { return (1 << (bits - 1)) - 1; }

/* Eq. (2): nearest point of the integer code set {-M..M} to t.  nearbyint
 * rounds to nearest with ties to even in the default rounding mode (R1);
 * clipping to [-M, M] then gives the nearest point of the bounded set. */
static double nearest_code(double t, int M)
{
    double q = nearbyint(t);
    if (q > (double)M) q = (double)M;
    if (q < -(double)M) q = -(double)M;
    return q;
}

/* Default candidate multipliers c_g = g / G, g = 1..G (reading G1). */
void oracle_default_grid(int G, float *c)
{
    for (int g = 0; g < G; ++g) c[g] = (float)((double)(g + 1) / (double)G);
}

/* Candidate scales of one step (reading G2):
 * a_g = fl32( fl32(max|r|) * c_g / M ). */
void oracle_candidate_scales(const double *r, int64_t d, int M,
                             const float *c, int G, float *a)
{
    double mx = 0.0;
    for (int64_t j = 0; j < d; ++j) {
        double v = fabs(r[j]);
        if (v > mx) mx = v;
    }
    float m = (float)mx;
    for (int g = 0; g < G; ++g)
        a[g] = (float)((double)m * (double)c[g] / (double)M);
}

/* Eq. (8): for a fixed scale a the best code vector is [r / a]_Q. */
void oracle_codes(const double *r, int64_t d, double a, int M, int8_t *q)
{
    for (int64_t j = 0; j < d; ++j) q[j] = (int8_t)nearest_code(r[j] / a, M);
}

/* Objective of Eq. (9): || r - a [r / a]_Q ||^2, summed in index order. */
double oracle_scale_error(const double *r, int64_t d, double a, int M)
{
    double e = 0.0;
    for (int64_t j = 0; j < d; ++j) {
        double t = r[j] - a * nearest_code(r[j] / a, M);
        e += t * t;
    }
    return e;
}

static double sum_sq(const double *r, int64_t d)
{
    double s = 0.0;
    for (int64_t j = 0; j < d; ++j) s += r[j] * r[j];
    return s;
}

/* Eq. (9) by grid search: errors of all G candidates, best index by T1.
 * A candidate whose fp32 scale is zero is not a scale and is skipped
 * (E = +inf); returns -1 when every candidate is zero. */
static int grid_search(const double *r, int64_t d, const float *a, int G, int M,
                       double *E)
{
    int best = -1;
    for (int g = 0; g < G; ++g) {
        E[g] = a[g] == 0.0f ? INFINITY : oracle_scale_error(r, d, (double)a[g], M);
        if (a[g] != 0.0f && (best < 0 || E[g] < E[best])) best = g;
    }
    return best;
}

/* Stopping rule S1-S3 with n points taken so far and Er = ||r||^2. */
static int should_stop(int n, int P, double Er, double Ew, double tol)
{
    if (n >= P) return 1;
    if (Er == 0.0) return 1;
    if (n >= 1 && Er <= tol * Ew) return 1;
    return 0;
}

/* The calibration-batch stopping rule S4: batch X [d][N], threshold eps,
 * relative != 0 for eps times the channel's full-precision output energy. */
typedef struct {
    const float *X;
    int64_t N;
    double eps;
    int relative;
} calib_rule;

/* Eq. (12) for one channel: (1/N) sum_t (v . x_t)^2, every sum in index
 * order, fp64. */
static double calib_error(const double *v, int64_t d, const float *X, int64_t N)
{
    double s = 0.0;
    for (int64_t t = 0; t < N; ++t) {
        double y = 0.0;
        for (int64_t j = 0; j < d; ++j) y += v[j] * (double)X[j * N + t];
        s += y * y;
    }
    return s / (double)N;
}

/* ------------------------------------------------------------------------
 * Eq. (11): the paper's own grid (readings D1, G3).
 * ------------------------------------------------------------------------ */

static int cmp_desc(const void *x, const void *y)
{
    double a = *(const double *)x, b = *(const double *)y;
    return (a < b) - (a > b);
}

/* Def. 1 (reading D1): half the smallest positive difference of |r_j|;
 * 0 when all magnitudes are equal.  work [d]. */
double oracle_min_gap(const double *r, int64_t d, double *work)
{
    for (int64_t j = 0; j < d; ++j) work[j] = fabs(r[j]);
    qsort(work, (size_t)d, sizeof(double), cmp_desc);
    double gap = 0.0;
    for (int64_t j = 1; j < d; ++j) {
        double diff = work[j - 1] - work[j];
        if (diff > 0.0 && (gap == 0.0 || diff < gap)) gap = diff;
    }
    return gap / 2.0;
}

/* Eq. (11): the step gamma and the number of grid points (reading G3). */
void oracle_paper_grid(const double *r, int64_t d, int M, double eta, double *work, double *gamma,
                       int64_t *count)
{
    double gap = oracle_min_gap(r, d, work);
    double g = gap > 0.0 ? gap / (double)M : eta;
    if (g > eta) g = eta;
    *gamma = g;
    *count = (int64_t)floor(2.0 * (double)M * sqrt(sum_sq(r, d)) / g);
}

/* A = sum |r_j| |q_j| and B = sum q_j^2 of the codes at scale a. */
static void codes_ab(const double *r, int64_t d, double a, int M, double *A, double *B)
{
    double sa = 0.0, sb = 0.0;
    for (int64_t j = 0; j < d; ++j) {
        double q = fabs(nearest_code(r[j] / a, M));
        sa += fabs(r[j]) * q;
        sb += q * q;
    }
    *A = sa;
    *B = sb;
}

/* The grid argmin of Eq. (9) over a_g = g gamma, 1 <= g <= count (reading
 * G3).  Returns the chosen g (0 if there is none) and its error in *Ebest. */
int64_t oracle_paper_grid_search(const double *r, int64_t d, int M, double gamma, int64_t count,
                                 double *Ebest)
{
    int64_t best = 0;
    double Eb = INFINITY;
    /* evaluate grid point g (and, with vertex != 0, the points nearest the
     * vertex of its piece) */
    for (int64_t j = 0; j < d; ++j) {
        for (int k = 0; k < M; ++k) {
            double b = fabs(r[j]) / ((double)k + 0.5);     /* a breakpoint */
            if (b == 0.0) continue;
            /* the grid points next to the breakpoint; one of them lies inside
             * each piece it bounds (a grid point exactly at b belongs to one
             * side by the rounding tie) */
            int64_t g0 = (int64_t)floor(b / gamma);
            int64_t around[3] = {g0 - 1, g0, g0 + 1};
            for (int u = 0; u < 3; ++u) {
                int64_t g = around[u];
                if (g < 1 || g > count) continue;
                int64_t cand[3] = {g, 0, 0};
                double a = (double)g * gamma;
                {
                    double A, B;
                    codes_ab(r, d, a, M, &A, &B);
                    if (B > 0.0) {
                        int64_t gv = (int64_t)floor((A / B) / gamma);
                        cand[1] = gv;
                        cand[2] = gv + 1;
                    }
                }
                for (int c = 0; c < 3; ++c) {
                    int64_t h = cand[c];
                    if (h < 1 || h > count) continue;
                    double E = oracle_scale_error(r, d, (double)h * gamma, M);    /* Eq. (9) */
                    if (E < Eb || (E == Eb && h < best)) { Eb = E; best = h; }
                }
            }
        }
    }
    *Ebest = Eb;
    return best;
}

/* Verifier only: how far an fp32 evaluation of Eq. (12) may lie from the
 * fp64 value when the outputs of the batch nearly cancel.  The other side
 * rounds v to fp32 and sums each length-d product in fp32; the usual
 * probabilistic model of those rounding errors (independent, zero mean)
 * puts column t's error below beta_t = 4 u sqrt(d) ||v o x_t||_2, u = 2^-24,
 * and e's below (2/N) sqrt(sum_t (y_t beta_t)^2) + (1/N) sum_t beta_t^2.
 * For a batch of many columns this is far below 1e-5 e. */
static double calib_slack(const double *v, int64_t d, const float *X, int64_t N)
{
    double a = 0.0, b = 0.0;
    const double lam = 4.0 * 0x1p-24 * sqrt((double)d);
    for (int64_t t = 0; t < N; ++t) {
        double y = 0.0, q = 0.0;
        for (int64_t j = 0; j < d; ++j) {
            const double p = (double)X[j * N + t] * v[j];
            y += p;
            q += p * p;
        }
        const double beta = lam * sqrt(q);
        a += (y * beta) * (y * beta);
        b += beta * beta;
    }
    return (2.0 * sqrt(a) + b) / (double)N;
}

/* Threshold of S4 for a channel whose residual is still w (r = w). */
static double calib_threshold(const calib_rule *cal, const double *w, int64_t d)
{
    return cal->relative ? cal->eps * calib_error(w, d, cal->X, cal->N) : cal->eps;
}

/* Reading C1's inputs, with per-thread work arrays. */
typedef struct {
    const float *X;
    int64_t N;
    const float *c;   /* [G] the multipliers j / G */
    int G;
    float *a;         /* [G] work */
    double *e;        /* [G] work */
    double *D;        /* [2 d] work */
} clip_rule;

/* S4 with n points taken: stop at P, at a zero residual, or once the output
 * error e of the n >= 1 points is at most thr. */
static int calib_should_stop(int n, int P, double Er, double e, double thr)
{
    if (n >= P || Er == 0.0) return 1;
    if (n >= 1 && e <= thr) return 1;
    return 0;
}

/* Algorithm 1 with the stopping rule, one channel.  codes [P][d], scales [P],
 * err [P] (||r||^2 after each point).  cal: NULL for S1-S3, else S4 with
 * xerr [P] (NULL or the output error after each point).  Returns the number
 * of points. */
/* Reading A2: the least-squares scale of the codes q for the residual r. */
static double refit_scale(const double *r, const int8_t *q, int64_t d)
{
    double rq = 0.0, qq = 0.0;
    for (int64_t j = 0; j < d; ++j) {
        rq += r[j] * (double)q[j];
        qq += (double)q[j] * (double)q[j];
    }
    return rq / qq;
}

/* Reading C1: the clipping candidates of a channel and their output errors
 * on X [d][N] (Eq. (13) for one channel); returns the chosen index, or -1
 * if every candidate scale is zero.  a [clipG], e [clipG], D [d] work. */
static int clip_choose(const float *w, int64_t d, int M, const float *cc, int clipG, const float *X,
                       int64_t N, float *a, double *e, double *D, int8_t *q)
{
    for (int64_t j = 0; j < d; ++j) D[j] = (double)w[j];
    oracle_candidate_scales(D, d, M, cc, clipG, a);
    int best = -1;
    for (int g = 0; g < clipG; ++g) {
        e[g] = INFINITY;
        if (a[g] == 0.0f) continue;
        oracle_codes(D, d, (double)a[g], M, q);
        double *R = D + d;                                   /* w - a q, fp64 */
        for (int64_t j = 0; j < d; ++j) R[j] = (double)w[j] - (double)a[g] * (double)q[j];
        e[g] = calib_error(R, d, X, N);                      /* Eq. (12) / (13) */
        if (best < 0 || e[g] < e[best]) best = g;
    }
    return best;
}

static int fit_channel(const float *w, int64_t d, int M, int P, const float *c,
                       int G, double tol, const calib_rule *cal, int refit, const clip_rule *clip,
                       double eta, double *gwork, int asym, int gate, float *offset,
                       int8_t *codes, float *scales, double *err, double *xerr, double *r,
                       float *a, double *E)
{
    for (int64_t j = 0; j < d; ++j) r[j] = (double)w[j];   /* r_1 = w, Eq. (7) */
    double Ew = sum_sq(r, d);
    double thr = cal ? calib_threshold(cal, r, d) : 0.0;
    if (asym) {                                             /* B2: r_1 = w - beta */
        double mx = (double)w[0], mn = (double)w[0];
        for (int64_t j = 1; j < d; ++j) {
            if ((double)w[j] > mx) mx = (double)w[j];
            if ((double)w[j] < mn) mn = (double)w[j];
        }
        const float beta = (float)((mx + mn) / 2.0);   /* B2: the midpoint */
        *offset = beta;
        for (int64_t j = 0; j < d; ++j) r[j] = (double)w[j] - (double)beta;   /* B2 */
    }
    double e = 0.0;                                         /* S4: e_n */
    int n = 0;
    if (clip && !asym && Ew > 0.0 && P >= 1) {              /* C1: the first point */
        int g = clip_choose(w, d, M, clip->c, clip->G, clip->X, clip->N, clip->a, clip->e,
                            clip->D, codes);
        if (g >= 0) {
            double as = (double)clip->a[g];
            oracle_codes(r, d, as, M, codes);
            for (int64_t j = 0; j < d; ++j) r[j] = r[j] - as * (double)codes[j];
            scales[0] = clip->a[g];
            n = 1;
            err[0] = sum_sq(r, d);
            if (cal) {
                e = calib_error(r, d, cal->X, cal->N);
                if (xerr) xerr[0] = e;
            }
        }
    }
    if (gate && !clip && Ew > 0.0 && P >= 1) {              /* F1: Algorithm 2's naive point */
        const float one = 1.0f;
        float aN;
        oracle_candidate_scales(r, d, M, &one, 1, &aN);    /* a_N = fl32(m / M) */
        if (aN != 0.0f) {
            double *R = gwork;                              /* r_1 - a_N [r_1 / a_N]_Q */
            oracle_codes(r, d, (double)aN, M, codes);
            for (int64_t j = 0; j < d; ++j) R[j] = r[j] - (double)aN * (double)codes[j];
            const double EN = sum_sq(R, d);
            const double eN = cal ? calib_error(R, d, cal->X, cal->N) : 0.0;
            if (cal ? eN <= thr : EN <= tol * Ew) {            /* Algorithm 2's test */
                memcpy(r, R, sizeof(double) * (size_t)d);  /* kept: the only point */
                scales[0] = aN;
                err[0] = EN;
                if (cal && xerr) xerr[0] = eN;
                return 1;
            }
            memset(codes, 0, (size_t)d);                    /* discarded: Algorithm 1 from w */
        }
    }
    for (;;) {
        double Er = sum_sq(r, d);
        if (cal ? calib_should_stop(n, P, Er, e, thr) : should_stop(n, P, Er, Ew, tol)) break;
        float a_pt;
        if (eta > 0.0) {                                    /* G3: Eq. (11)'s grid */
            double gamma, Eb;
            int64_t cnt;
            oracle_paper_grid(r, d, M, eta, gwork, &gamma, &cnt);
            int64_t g = oracle_paper_grid_search(r, d, M, gamma, cnt, &Eb);
            a_pt = (float)((double)g * gamma);
            if (g < 1 || a_pt == 0.0f) break;               /* S3: no scale */
        } else {
            oracle_candidate_scales(r, d, M, c, G, a);
            int g = grid_search(r, d, a, G, M, E);          /* Eq. (9)  */
            if (g < 0) break;                               /* S3: no scale */
            a_pt = a[g];
        }
        double as = (double)a_pt;
        int8_t *q = codes + (int64_t)n * d;
        oracle_codes(r, d, as, M, q);                       /* Eq. (10) */
        if (refit) {                                        /* A2 */
            a_pt = (float)refit_scale(r, q, d);
            as = (double)a_pt;
        }
        for (int64_t j = 0; j < d; ++j) r[j] = r[j] - as * (double)q[j]; /* Eq. (7) */
        scales[n] = a_pt;
        n += 1;
        err[n - 1] = sum_sq(r, d);
        if (cal) {
            e = calib_error(r, d, cal->X, cal->N);          /* Eq. (12) */
            if (xerr) xerr[n - 1] = e;
        }
    }
    return n;
}

static int n_threads_or_default(int nt)
{
#ifdef _OPENMP
    return nt > 0 ? nt : omp_get_max_threads();
#else
    (void)nt;
    return 1;
#endif
}

/* Free-running fit of a layer W [C][d].  grid: NULL for the default.
 * Outputs: codes [C][P][d] int8, scales [C][P], counts [C], err [C][P]
 * (may be NULL), and with cal the output error after each point, xerr
 * [C][P] (may be NULL).  Slots at or after a channel's count are zero. */
static int fit_layer(const float *W, int64_t C, int64_t d, int bits, int P,
                     const float *grid, int G, double tol, const calib_rule *cal, int refit,
                     const float *clipX, int64_t clipN, int clipG, double eta, int gate,
                     float *offsets, int8_t *codes, float *scales, int32_t *counts, double *err,
                     double *xerr, int n_threads)
{
    int M = oracle_levels(bits);
    float *c = (float *)malloc(sizeof(float) * (size_t)G);
    float *cc = (float *)malloc(sizeof(float) * (size_t)(clipG > 0 ? clipG : 1));
    if (!c || !cc) { free(c); free(cc); return -1; }
    if (grid) memcpy(c, grid, sizeof(float) * (size_t)G);
    else oracle_default_grid(G, c);
    if (clipG > 0) oracle_default_grid(clipG, cc);
    memset(codes, 0, (size_t)(C * P * d));
    memset(scales, 0, sizeof(float) * (size_t)(C * P));
    if (err) memset(err, 0, sizeof(double) * (size_t)(C * P));
    if (xerr) memset(xerr, 0, sizeof(double) * (size_t)(C * P));
    int nt = n_threads_or_default(n_threads);
    int fail = 0;
#pragma omp parallel num_threads(nt)
    {
        double *r = (double *)malloc(sizeof(double) * (size_t)d);
        float *a = (float *)malloc(sizeof(float) * (size_t)G);
        double *E = (double *)malloc(sizeof(double) * (size_t)G);
        double *e = (double *)malloc(sizeof(double) * (size_t)P);
        double *xe = (double *)malloc(sizeof(double) * (size_t)P);
        clip_rule cl = {clipX, clipN, cc, clipG, NULL, NULL, NULL};
        if (clipG > 0) {
            cl.a = (float *)malloc(sizeof(float) * (size_t)clipG);
            cl.e = (double *)malloc(sizeof(double) * (size_t)clipG);
            cl.D = (double *)malloc(sizeof(double) * (size_t)(2 * d));
        }
        double *gw = (double *)malloc(sizeof(double) * (size_t)d);
        if (!r || !a || !E || !e || !xe || !gw || (clipG > 0 && (!cl.a || !cl.e || !cl.D))) {
#pragma omp atomic write
            fail = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t k = 0; k < C; ++k) {
                memset(e, 0, sizeof(double) * (size_t)P);
                memset(xe, 0, sizeof(double) * (size_t)P);
                float beta = 0.0f;
                int n = fit_channel(W + k * d, d, M, P, c, G, tol, cal, refit,
                                    clipG > 0 ? &cl : NULL, eta, gw, offsets != NULL, gate, &beta,
                                    codes + k * P * d, scales + k * P, e, xe, r, a, E);
                if (offsets) offsets[k] = beta;
                counts[k] = n;
                if (err) memcpy(err + k * P, e, sizeof(double) * (size_t)P);
                if (xerr) memcpy(xerr + k * P, xe, sizeof(double) * (size_t)P);
            }
        }
        free(r); free(a); free(E); free(e); free(xe); free(gw);
        free(cl.a); free(cl.e); free(cl.D);
    }
    free(c);
    free(cc);
    return fail ? -1 : 0;
}

int oracle_fit(const float *W, int64_t C, int64_t d, int bits, int P,
               const float *grid, int G, double tol, int8_t *codes,
               float *scales, int32_t *counts, double *err, int n_threads)
{
    return fit_layer(W, C, d, bits, P, grid, G, tol, NULL, 0, NULL, 0, 0, 0.0, 0, NULL, codes,
                     scales, counts, err, NULL, n_threads);
}

/* The fit with its options: calib == 0 for the stopping rule S1 with tol,
 * else S4 on X [d][N] with eps / relative; refit != 0 for reading A2;
 * clipG > 0 for reading C1 on X with clipG candidates (the paper's 20);
 * eta > 0 for the paper's grid of Eq. (11) (reading G3; the paper's 2^-10)
 * instead of the G-point grid; gate != 0 for Algorithm 2's naive first
 * point (reading F1; not with clipG). */
int oracle_fit_ex(const float *W, int64_t C, int64_t d, int bits, int P, const float *grid, int G,
                  double tol, const float *X, int64_t N, int calib, double eps, int relative,
                  int refit, int clipG, double eta, int gate, float *offsets, int8_t *codes,
                  float *scales, int32_t *counts, double *err, double *xerr, int n_threads)
{
    calib_rule cal = {X, N, eps, relative};
    return fit_layer(W, C, d, bits, P, grid, G, tol, calib ? &cal : NULL, refit, X, N, clipG, eta,
                     gate, offsets, codes, scales, counts, err, calib ? xerr : NULL, n_threads);
}

/* The fit with the stopping rule S4 on the calibration batch X [d][N]. */
int oracle_fit_calib(const float *W, int64_t C, int64_t d, int bits, int P,
                     const float *grid, int G, const float *X, int64_t N, double eps,
                     int relative, int8_t *codes, float *scales, int32_t *counts,
                     double *err, double *xerr, int n_threads)
{
    calib_rule cal = {X, N, eps, relative};
    return fit_layer(W, C, d, bits, P, grid, G, 0.0, &cal, 0, NULL, 0, 0, 0.0, 0, NULL, codes,
                     scales, counts, err, xerr, n_threads);
}

/* ------------------------------------------------------------------------
 * Lockstep verifier.  For each listed channel it replays the outputs of
 * another implementation step by step on its own fp64 residual and checks:
 *  V1 the chosen scale is a candidate of the step and its error is the
 *     minimum, or within 1e-6 relative of it (a "candidate tie");
 *  V2 the codes equal [r / a]_Q except at elements whose r / a lies within
 *     1e-6 * max(1, |r / a|) of a half-integer, where either neighbour is
 *     accepted (a "code tie");
 *  V3 the stop decision agrees, except when ||r||^2 / (tol ||w||^2) is
 *     within 1e-6 of 1 (a "stop tie");
 *  V4 the per-point ||r||^2 (if given) agrees within 1e-5 relative (plus
 *     one fp32 subnormal quantum, as it is an fp32 output) or equals the
 *     fp32 rounding of the fp64 value;
 * and that every slot at or after the count is zero.  After each accepted
 * step it continues from the other implementation's (a, q).
 * With the calibration rule S4 (oracle_verify_calib), V3 is S4's decision,
 * tied when |e_n - thr| is within 1e-5 thr plus the fp32 evaluation
 * allowances of e_n and thr (calib_slack: the other side evaluates Eq. (12)
 * with fp32 products and sums), and
 *  V4x the per-point output error (if given) agrees with the fp64 e_n as
 *     V4 asks of ||r||^2, plus the allowance of e_n.
 * With the refit of reading A2 (oracle_verify_ex, refit != 0), V1 and V2 ask
 * instead that the codes be those of the best candidate, or of a candidate
 * within 1e-6 relative of it (a candidate tie), up to code ties, and that
 * the scale be the least-squares scale of those codes (fl32 of the fp64
 * quotient, or one fp32 ulp from it: the sums may run in another order).
 * With the clipping of reading C1 (clipG > 0), the first point's scale must
 * be a clipping candidate whose output error is within 1e-5 relative plus
 * the fp32 evaluation allowance (calib_slack) of the smallest one, and its
 * codes Eq. (10)'s at that scale (up to code ties).
 * With Algorithm 2's naive first point (reading F1, gate != 0), point 1 may
 * be the naive point (a_N, [r_1 / a_N]_Q) only if the stopping rule holds
 * for it (or its error is within the stop-tie band of the threshold, a
 * "stop tie"); then the channel must stop there.  If the rule holds and the
 * other side took another first point, the status is 10.
 * status: 0 ok, 1 count, 2 scale not a candidate, 3 scale not optimal,
 *         4 code, 5 nonzero unused slot, 6 err value, 7 bad count range,
 *         8 output-error value, 9 offset (reading B2), 10 the naive-point
 *         decision of reading F1.
 * ------------------------------------------------------------------------ */

/* V4 / V4x for one fp32 output: 1e-5 relative plus slack, one fp32
 * subnormal quantum (2^-149: the most an fp32 value below the normal range
 * can be off by), or exactly fl32 of the fp64 value (which is +inf above the
 * fp32 range).
 * Tracks the largest relative deviation of normal values in *emax. */
static int fp32_value_ok(double got, double ref, double slack, double *emax)
{
    double dev = fabs(got - ref);
    if (ref >= 0x1p-126 && dev / ref > *emax) *emax = dev / ref;
    return got == (double)(float)ref || dev <= 1e-5 * ref + slack + 0x1p-149;
}

/* V2 for one point: do the codes q equal [r / a]_Q except at code ties?
 * Adds the ties to *ties; returns 0 on a mismatch. */
static int codes_agree(const double *r, int64_t d, double as, int M, const int8_t *q, int *ties)
{
    int qt = 0;
    for (int64_t j = 0; j < d; ++j) {
        double t = r[j] / as;
        int qr = (int)nearest_code(t, M);
        int qo = (int)q[j];
        if (qo != qr) {
            double fl = floor(t);
            double half = fabs(t - (fl + 0.5));
            int lo = (int)nearest_code(fl, M), hi = (int)nearest_code(fl + 1.0, M);
            if (half <= 1e-6 * fmax(1.0, fabs(t)) && (qo == lo || qo == hi)) qt++;
            else return 0;
        }
    }
    *ties += qt;
    return 1;
}

static int verify_layer(const float *W, int64_t C, int64_t d, int bits, int P,
                        const float *grid, int G, double tol, const calib_rule *cal, int refit,
                        const float *clipX, int64_t clipN, int clipG, double eta, int gate,
                        const float *offsets,
                        const int8_t *codes, const float *scales, const int32_t *counts,
                        const float *err, const float *xerr, const int64_t *chan,
                        int64_t n_chan, int32_t *status, int32_t *cand_ties,
                        int32_t *code_ties, int32_t *stop_ties, double *err_relmax,
                        int n_threads)
{
    int M = oracle_levels(bits);
    float *c = (float *)malloc(sizeof(float) * (size_t)G);
    float *cc = (float *)malloc(sizeof(float) * (size_t)(clipG > 0 ? clipG : 1));
    if (!c || !cc) { free(c); free(cc); return -1; }
    if (grid) memcpy(c, grid, sizeof(float) * (size_t)G);
    else oracle_default_grid(G, c);
    if (clipG > 0) oracle_default_grid(clipG, cc);
    int nt = n_threads_or_default(n_threads);
    int fail = 0;
    (void)C;
#pragma omp parallel num_threads(nt)
    {
        double *r = (double *)malloc(sizeof(double) * (size_t)d);
        float *a = (float *)malloc(sizeof(float) * (size_t)G);
        double *E = (double *)malloc(sizeof(double) * (size_t)G);
        double *gw = (double *)malloc(sizeof(double) * (size_t)d);
        clip_rule cl = {clipX, clipN, cc, clipG, NULL, NULL, NULL};
        int8_t *cq = NULL;
        if (clipG > 0) {
            cl.a = (float *)malloc(sizeof(float) * (size_t)clipG);
            cl.e = (double *)malloc(sizeof(double) * (size_t)clipG);
            cl.D = (double *)malloc(sizeof(double) * (size_t)(2 * d));
            cq = (int8_t *)malloc((size_t)d);
        }
        if (!r || !a || !E || !gw || (clipG > 0 && (!cl.a || !cl.e || !cl.D || !cq))) {
#pragma omp atomic write
            fail = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t s = 0; s < n_chan; ++s) {
                int64_t k = chan[s];
                const float *w = W + k * d;
                const int8_t *qk = codes + k * P * d;
                const float *ak = scales + k * P;
                const float *ek = err ? err + k * P : NULL;
                const float *xk = (cal && xerr) ? xerr + k * P : NULL;
                int st = 0, ct = 0, qt = 0, stt = 0;
                double emax = 0.0;
                int n_other = counts[k];
                if (n_other < 0 || n_other > P) st = 7;
                for (int64_t j = 0; j < d; ++j) r[j] = (double)w[j];
                double Ew = sum_sq(r, d);
                double thr = cal ? calib_threshold(cal, r, d) : 0.0;
                double thr_slack = (cal && cal->relative) ? cal->eps * calib_slack(r, d, cal->X, cal->N) : 0.0;
                if (offsets) {   /* B2: the other side's offset is the midpoint, exactly */
                    double mx = (double)w[0], mn = (double)w[0];
                    for (int64_t j = 1; j < d; ++j) {
                        if ((double)w[j] > mx) mx = (double)w[j];
                        if ((double)w[j] < mn) mn = (double)w[j];
                    }
                    const float beta = (float)((mx + mn) / 2.0);
                    if (offsets[k] != beta) st = 9;
                    for (int64_t j = 0; j < d; ++j) r[j] = (double)w[j] - (double)beta;
                }
                double e = 0.0;   /* S4: output error of the points so far */
                for (int n = 0; st == 0; ++n) {
                    double Er = sum_sq(r, d);
                    /* err and xerr are fp32 outputs (V4, V4x) */
                    if (n >= 1 && ek && !fp32_value_ok((double)ek[n - 1], Er, 0.0, &emax)) {
                        st = 6;
                        break;
                    }
                    /* S4: e and the threshold carry the fp32 evaluation
                     * allowance (calib_slack) */
                    const double e_slack = (cal && n >= 1) ? calib_slack(r, d, cal->X, cal->N) : 0.0;
                    if (n >= 1 && xk && !fp32_value_ok((double)xk[n - 1], e, e_slack, &emax)) {
                        st = 8;
                        break;
                    }
                    oracle_candidate_scales(r, d, M, c, G, a);
                    int gbest = -1;
                    int stop_ref = cal ? calib_should_stop(n, P, Er, e, thr)
                                       : should_stop(n, P, Er, Ew, tol);
                    double pg_gamma = 0.0, pg_E = INFINITY;   /* G3 */
                    int64_t pg_cnt = 0, pg_best = 0;
                    if (!stop_ref && eta > 0.0) {
                        oracle_paper_grid(r, d, M, eta, gw, &pg_gamma, &pg_cnt);
                        pg_best = oracle_paper_grid_search(r, d, M, pg_gamma, pg_cnt, &pg_E);
                        stop_ref = pg_best < 1 || (float)((double)pg_best * pg_gamma) == 0.0f;
                        gbest = stop_ref ? -1 : 0;
                    } else if (!stop_ref) {
                        gbest = grid_search(r, d, a, G, M, E);
                        stop_ref = gbest < 0;
                    }
                    int stop_other = (n == n_other);
                    if (stop_ref != stop_other) {
                        double lim = cal ? thr : tol * Ew;
                        double ratio = lim > 0 ? (cal ? e : Er) / lim : INFINITY;
                        int near = cal ? fabs(e - thr) <= 1e-5 * thr + e_slack + thr_slack
                                       : fabs(ratio - 1.0) <= 1e-6;
                        if (n >= 1 && n < P && Er != 0.0 && near) {
                            stt++;
                        } else { st = 1; break; }
                    }
                    if (stop_other) break;
                    if (n == 0 && gate && clipG == 0 && Ew > 0.0) {
                        /* F1: the naive point, kept only if the rule holds for it */
                        const float one = 1.0f;
                        float aN;
                        oracle_candidate_scales(r, d, M, &one, 1, &aN);
                        if (aN != 0.0f) {
                            double *R = gw;
                            for (int64_t j = 0; j < d; ++j)
                                R[j] = r[j] - (double)aN * nearest_code(r[j] / (double)aN, M);
                            const double EN = sum_sq(R, d);
                            const double eN = cal ? calib_error(R, d, cal->X, cal->N) : 0.0;
                            const int pass = cal ? eN <= thr : EN <= tol * Ew;
                            int nearN = 0;
                            if (cal) {
                                nearN = fabs(eN - thr) <= 1e-5 * thr +
                                                              calib_slack(R, d, cal->X, cal->N) +
                                                              thr_slack;
                            } else if (tol * Ew > 0.0) {
                                nearN = fabs(EN / (tol * Ew) - 1.0) <= 1e-6;
                            }
                            int qtN = 0;
                            const int kept = ak[0] == aN && codes_agree(r, d, (double)aN, M, qk, &qtN);
                            if (kept && (pass || nearN)) {
                                qt += qtN;
                                if (!pass) stt++;
                                for (int64_t j = 0; j < d; ++j) r[j] = r[j] - (double)aN * (double)qk[j];
                                if (cal) e = calib_error(r, d, cal->X, cal->N);
                                continue;
                            }
                            if (pass && !nearN) { st = 10; break; }
                            if (pass) stt++;   /* discarded within the stop-tie band */
                        }
                    }
                    /* V1 */
                    if (gbest < 0) {           /* the other side went on past a stop */
                        if (eta > 0.0) { st = 1; break; }
                        gbest = grid_search(r, d, a, G, M, E);
                        if (gbest < 0) { st = 1; break; }
                    }
                    float ao = ak[n];
                    const int8_t *q = qk + (int64_t)n * d;
                    double as = (double)ao;
                    int cbest = (clipG > 0 && n == 0)
                                    ? clip_choose(w, d, M, cc, clipG, clipX, clipN, cl.a, cl.e, cl.D, cq)
                                    : -1;
                    if (eta > 0.0) {
                        /* G3: fl32 of a grid point g gamma whose error is the
                         * smallest, or within 1e-6 relative of it */
                        const int64_t g0 = llround(as / pg_gamma);
                        double Eo = INFINITY;
                        for (int64_t h = g0 - 2; h <= g0 + 2; ++h) {
                            if (h < 1 || h > pg_cnt || (float)((double)h * pg_gamma) != ao) continue;
                            const double Eh = oracle_scale_error(r, d, (double)h * pg_gamma, M);
                            if (Eh < Eo) Eo = Eh;
                        }
                        if (Eo == INFINITY) { st = 2; break; }
                        if (Eo > pg_E) {
                            if (Eo <= (1.0 + 1e-6) * pg_E) ct++;
                            else { st = 3; break; }
                        }
                        if (!codes_agree(r, d, as, M, q, &qt)) { st = 4; break; }
                    } else if (cbest >= 0) {
                        /* C1: a clipping candidate within the evaluation allowance of the best */
                        int go = -1;
                        for (int g = 0; g < clipG; ++g)
                            if (cl.a[g] == ao && ao != 0.0f) { go = g; break; }
                        if (go < 0) { st = 2; break; }
                        if (go != cbest) {
                            double *R = cl.D + d;
                            for (int64_t j = 0; j < d; ++j)
                                R[j] = (double)w[j] - (double)cl.a[go] * (double)q[j];
                            const double sg = calib_slack(R, d, clipX, clipN);
                            if (cl.e[go] <= cl.e[cbest] * (1.0 + 1e-5) + sg) ct++;
                            else { st = 3; break; }
                        }
                        if (!codes_agree(r, d, as, M, q, &qt)) { st = 4; break; }
                    } else if (refit) {
                        /* A2: codes of the best candidate or a tied one, then
                         * the least-squares scale of those codes */
                        int got = codes_agree(r, d, (double)a[gbest], M, q, &qt) ? gbest : -1;
                        for (int g = 0; g < G && got < 0; ++g) {
                            if (g == gbest || a[g] == 0.0f || !(E[g] <= (1.0 + 1e-6) * E[gbest]))
                                continue;
                            if (codes_agree(r, d, (double)a[g], M, q, &qt)) { got = g; ct++; }
                        }
                        if (got < 0) { st = 4; break; }
                        const double aref = refit_scale(r, q, d);
                        if (!(ao == (float)aref || fabs(as - aref) <= 0x1p-23 * fabs(aref))) {
                            st = 2;
                            break;
                        }
                    } else {
                        int go = -1;
                        for (int g = 0; g < G; ++g)
                            if (a[g] == ao && ao != 0.0f) { go = g; break; }
                        if (go < 0) { st = 2; break; }
                        if (go != gbest) {
                            if (E[go] <= (1.0 + 1e-6) * E[gbest]) ct++;
                            else { st = 3; break; }
                        }
                        /* V2, then continue from the other side's (a, q) */
                        if (!codes_agree(r, d, as, M, q, &qt)) { st = 4; break; }
                    }
                    for (int64_t j = 0; j < d; ++j) r[j] = r[j] - as * (double)q[j];
                    if (cal) e = calib_error(r, d, cal->X, cal->N);
                }
                /* unused slots must be zero */
                if (st == 0) {
                    for (int n = n_other; n < P && st == 0; ++n) {
                        if (ak[n] != 0.0f) st = 5;
                        if (ek && ek[n] != 0.0f) st = 5;
                        if (xk && xk[n] != 0.0f) st = 5;
                        for (int64_t j = 0; j < d && st == 0; ++j)
                            if (qk[(int64_t)n * d + j] != 0) st = 5;
                    }
                }
                status[s] = st; cand_ties[s] = ct; code_ties[s] = qt;
                stop_ties[s] = stt; err_relmax[s] = emax;
            }
        }
        free(r); free(a); free(E); free(gw);
        free(cl.a); free(cl.e); free(cl.D); free(cq);
    }
    free(c);
    free(cc);
    return fail ? -1 : 0;
}

int oracle_verify(const float *W, int64_t C, int64_t d, int bits, int P,
                  const float *grid, int G, double tol, const int8_t *codes,
                  const float *scales, const int32_t *counts, const float *err,
                  const int64_t *chan, int64_t n_chan, int32_t *status,
                  int32_t *cand_ties, int32_t *code_ties, int32_t *stop_ties,
                  double *err_relmax, int n_threads)
{
    return verify_layer(W, C, d, bits, P, grid, G, tol, NULL, 0, NULL, 0, 0, 0.0, 0, NULL, codes,
                        scales, counts, err, NULL, chan, n_chan, status, cand_ties, code_ties,
                        stop_ties, err_relmax, n_threads);
}

/* The lockstep check of a fit with its options (as oracle_fit_ex). */
int oracle_verify_ex(const float *W, int64_t C, int64_t d, int bits, int P, const float *grid,
                     int G, double tol, const float *X, int64_t N, int calib, double eps,
                     int relative, int refit, int clipG, double eta, int gate,
                     const float *offsets, const int8_t *codes, const float *scales,
                     const int32_t *counts, const float *err, const float *xerr,
                     const int64_t *chan, int64_t n_chan, int32_t *status, int32_t *cand_ties,
                     int32_t *code_ties, int32_t *stop_ties, double *err_relmax, int n_threads)
{
    calib_rule cal = {X, N, eps, relative};
    return verify_layer(W, C, d, bits, P, grid, G, tol, calib ? &cal : NULL, refit, X, N, clipG, eta,
                        gate, offsets, codes, scales, counts, err, calib ? xerr : NULL, chan, n_chan,
                        status, cand_ties, code_ties, stop_ties, err_relmax, n_threads);
}

/* The lockstep check of a fit with the calibration rule S4; xerr [C][P] is
 * the other side's output error after each point (NULL: not checked). */
int oracle_verify_calib(const float *W, int64_t C, int64_t d, int bits, int P,
                        const float *grid, int G, const float *X, int64_t N, double eps,
                        int relative, const int8_t *codes, const float *scales,
                        const int32_t *counts, const float *err, const float *xerr,
                        const int64_t *chan, int64_t n_chan, int32_t *status,
                        int32_t *cand_ties, int32_t *code_ties, int32_t *stop_ties,
                        double *err_relmax, int n_threads)
{
    calib_rule cal = {X, N, eps, relative};
    return verify_layer(W, C, d, bits, P, grid, G, 0.0, &cal, 0, NULL, 0, 0, 0.0, 0, NULL, codes,
                        scales, counts, err, xerr, chan, n_chan, status, cand_ties, code_ties,
                        stop_ties, err_relmax, n_threads);
}

/* Residual D = w - sum_{i<n} a_i q_i of one channel, summed in point order
 * (Eq. (7); the same sequence of fp64 operations as the fit). */
static void channel_residual(const float *w, float beta, const int8_t *q, const float *a,
                             int n, int64_t d, double *D)
{
    for (int64_t j = 0; j < d; ++j) D[j] = (double)w[j] - (double)beta;
    for (int i = 0; i < n; ++i)
        for (int64_t j = 0; j < d; ++j)
            D[j] = D[j] - (double)a[i] * (double)q[(int64_t)i * d + j];
}

/* Eq. (12): err[k] = (1/N) sum_n ((w_k - w~_k) . x_n)^2 and, if ref is not
 * NULL, ref[k] = (1/N) sum_n (w_k . x_n)^2, for the listed channels
 * (chan == NULL: all C channels, outputs indexed by channel).  Every dot
 * product sums over j in index order and the squares over n in column
 * order; X is first copied to column-contiguous rows, and four columns'
 * dot products run side by side, which changes no operation of any sum. */
int oracle_output_error_ex(const float *W, const float *offsets, const int8_t *codes,
                           const float *scales, const int32_t *counts, int64_t C, int64_t d, int P,
                           const float *X, int64_t N, const int64_t *chan,
                           int64_t n_chan, double *err, double *ref, int n_threads)
{
    int nt = n_threads_or_default(n_threads);
    int64_t cnt = chan ? n_chan : C;
    float *Xt = (float *)malloc(sizeof(float) * (size_t)(N * d));   /* Xt[n][j] = X[j][n] */
    if (!Xt) return -1;
    for (int64_t j = 0; j < d; ++j)
        for (int64_t n = 0; n < N; ++n) Xt[n * d + j] = X[j * N + n];
    int fail = 0;
#pragma omp parallel num_threads(nt)
    {
        double *D = (double *)malloc(sizeof(double) * (size_t)d);
        if (!D) {
#pragma omp atomic write
            fail = 1;
        } else {
#pragma omp for schedule(dynamic, 1)
            for (int64_t s = 0; s < cnt; ++s) {
                int64_t k = chan ? chan[s] : s;
                const float *w = W + k * d;
                channel_residual(w, offsets ? offsets[k] : 0.0f, codes + k * P * d, scales + k * P,
                                 counts[k], d, D);
                double se = 0.0, sr = 0.0;
                int64_t n = 0;
                for (; n + 4 <= N; n += 4) {
                    double y[4] = {0.0, 0.0, 0.0, 0.0}, yr[4] = {0.0, 0.0, 0.0, 0.0};
                    const float *x0 = Xt + n * d;
                    for (int64_t j = 0; j < d; ++j) {
                        for (int u = 0; u < 4; ++u) {
                            double x = (double)x0[u * d + j];
                            y[u] += D[j] * x;
                            yr[u] += (double)w[j] * x;
                        }
                    }
                    for (int u = 0; u < 4; ++u) {
                        se += y[u] * y[u];
                        sr += yr[u] * yr[u];
                    }
                }
                for (; n < N; ++n) {
                    double y = 0.0, yr = 0.0;
                    for (int64_t j = 0; j < d; ++j) {
                        double x = (double)Xt[n * d + j];
                        y += D[j] * x;
                        yr += (double)w[j] * x;
                    }
                    se += y * y;
                    sr += yr * yr;
                }
                err[s] = se / (double)N;
                if (ref) ref[s] = sr / (double)N;
            }
        }
        free(D);
    }
    free(Xt);
    return fail ? -1 : 0;
}

int oracle_output_error(const float *W, const int8_t *codes, const float *scales,
                        const int32_t *counts, int64_t C, int64_t d, int P,
                        const float *X, int64_t N, const int64_t *chan,
                        int64_t n_chan, double *err, double *ref, int n_threads)
{
    return oracle_output_error_ex(W, NULL, codes, scales, counts, C, d, P, X, N, chan, n_chan, err,
                                  ref, n_threads);
}

/* Eq. (4): w~ = sum_{i<n} a_i q_i (plus the offset of reading B2, first),
 * accumulated in fp64 in point order and rounded once to fp32. */
void oracle_reconstruct_ex(const float *offsets, const int8_t *codes, const float *scales,
                           const int32_t *counts, int64_t C, int64_t d, int P, float *W_hat)
{
    for (int64_t k = 0; k < C; ++k) {
        const int8_t *q = codes + k * P * d;
        const float *a = scales + k * P;
        for (int64_t j = 0; j < d; ++j) {
            double s = offsets ? (double)offsets[k] : 0.0;
            for (int i = 0; i < counts[k]; ++i)
                s = s + (double)a[i] * (double)q[(int64_t)i * d + j];
            W_hat[k * d + j] = (float)s;
        }
    }
}

/* ------------------------------------------------------------------------
 * Sec. 3.4: deployment arithmetic.
 * ------------------------------------------------------------------------ */

/* Eq. (14), reading I1: A_i = nearest integer to 2^p a_i (ties to even) for
 * the points i < counts[k] of each channel, zero after the count.  2^p a_i is
 * exact in fp64.  Returns the number of values clamped to the 32-bit range. */
int64_t oracle_integer_scales(const float *scales, const int32_t *counts, int64_t C, int P, int p,
                              int32_t *A)
{
    const double lim = 2147483647.0;
    int64_t clamped = 0;
    for (int64_t k = 0; k < C; ++k) {
        for (int i = 0; i < P; ++i) {
            double v = 0.0;
            if (i < counts[k]) {
                v = rint(ldexp((double)scales[k * P + i], p));   /* round to nearest, ties even */
                if (v > lim) { v = lim; ++clamped; }
                if (v < -lim) { v = -lim; ++clamped; }
            }
            A[k * P + i] = (int32_t)v;
        }
    }
    return clamped;
}

/* Eq. (15), Steps 1-3, for channel k and column t of the batch (X [N][d]):
 *   Step 1: z_i = q_i . x_t for every point i < counts[k], each in a 32-bit
 *           accumulator;
 *   Step 2: s = sum_{i < counts[k]} A_i z_i, in 64 bits;
 *   Step 3: y = s shifted right by p (reading B1: floor(s / 2^p)).
 * Y [C][N] int64.  Returns -1 if some z_i leaves the 32-bit range or some s
 * the 64-bit range (checked with 128-bit arithmetic), else 0. */
int oracle_integer_forward(const int8_t *codes, const int32_t *A, const int32_t *counts, int64_t C,
                           int64_t d, int P, const int8_t *X, int64_t N, int p, int64_t *Y)
{
    int bad = 0;
    for (int64_t k = 0; k < C; ++k) {
        for (int64_t t = 0; t < N; ++t) {
            __int128 s = 0;
            for (int i = 0; i < counts[k]; ++i) {
                const int8_t *q = codes + (k * P + i) * d;
                int64_t z = 0;
                for (int64_t j = 0; j < d; ++j) z += (int64_t)q[j] * (int64_t)X[t * d + j];
                if (z > INT32_MAX || z < INT32_MIN) bad = 1;
                s += (__int128)A[k * P + i] * (__int128)z;
            }
            if (s > (__int128)INT64_MAX || s < (__int128)INT64_MIN) bad = 1;
            Y[k * N + t] = (int64_t)s >> p;   /* arithmetic shift: floor division */
        }
    }
    return bad ? -1 : 0;
}

void oracle_reconstruct(const int8_t *codes, const float *scales, const int32_t *counts, int64_t C,
                        int64_t d, int P, float *W_hat)
{
    oracle_reconstruct_ex(NULL, codes, scales, counts, C, d, P, W_hat);
}
