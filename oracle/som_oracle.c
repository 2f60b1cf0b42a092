/*
 * som_oracle.c -- plain fp64 CPU oracle for online self-organizing-map (SOM)
 * training and evaluation.
 *
 * TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
 * CPU-baseline leg of the benchmark may load this file's library.  It shares
 * no code, header, table or helper with the HIP library: everything below is
 * written out again from the definitions it cites.
 *
 * What it computes (Kohonen's standard, per-sample SOM as stated in Sec. 5A of
 * the paper; the GPU training procedure of Sec. 6C; the evaluation of Sec. 6D
 * and Sec. 8A/8B):
 *
 *   for each step t, with sample x = X[order[t]]:
 *     D_u   = sum_j (x_j - w_uj)^2                 squared Euclidean distance
 *     c     = smallest u with D_u = min D          best-matching unit (BMU)
 *     h_u   = lr(t) * exp(-|pos(u) - pos(c)|^2 / (2 sigma(t)^2))
 *     w_uj <- w_uj + h_u * (x_j - w_uj)            Eq. (1), every unit u
 *
 * All state is double precision.  Inputs X (fp32) are widened exactly.
 * Loops run in plain index order; the only parallelism is OpenMP over
 * independent units (distance and update) or independent samples
 * (evaluation), whose per-item arithmetic is unchanged by it, so the result
 * does not depend on the thread count.
 *
 * Readings of points the paper leaves open (each is listed with its reason in
 * the design notes):
 *   - neighbourhood: Gaussian of the squared lattice distance with the
 *     learning rate folded in (Eq. (1) puts lr inside h);
 *   - sigma = 0 gives a Kronecker delta at the BMU; sigma = +inf gives h = lr
 *     for every unit;
 *   - decay: linear (1-p) a + p b or exponential a^(1-p) b^p interpolation
 *     between endpoint values a, b at p = t / (T - 1) (p = 0 when T = 1);
 *     equal endpoints give that value;
 *   - lattice: rectangular (row, col) = (u / cols, u % cols), or hexagonal
 *     with odd rows shifted by half a unit and rows sqrt(3)/2 apart;
 *     Euclidean lattice distance, no wrap-around;
 *   - QE: mean unsquared Euclidean distance from each sample to its BMU;
 *   - TE: fraction of samples whose first and second BMUs are not lattice
 *     neighbours (lattice distance > 1); 0 for a single-unit map.
 *
 * Build: gcc -O2 -fopenmp -ffp-contract=off -shared -fPIC (no fast-math).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

#define ORACLE_OK 0
#define ORACLE_E_ARG 1

#define ORACLE_RECT 0
#define ORACLE_HEX 1

#define ORACLE_LINEAR 0
#define ORACLE_EXPONENTIAL 1

typedef struct {
    double lr0, lr1;
    int32_t lr_decay;
    double sigma0, sigma1;
    int32_t sigma_decay;
} som_oracle_schedule;

/* ------------------------------------------------------------------------
 * SplitMix64 (Steele, Lea and Flood, "Fast splittable pseudorandom number
 * generators", OOPSLA 2014), in its counter form: the i-th output (i = 0, 1,
 * ...) of the generator seeded with s is mix(s + (i + 1) * golden_gamma).
 * ---------------------------------------------------------------------- */
static uint64_t oracle_splitmix64(uint64_t seed, uint64_t i)
{
    uint64_t z = seed + (i + 1u) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

void som_oracle_splitmix64(uint64_t seed, int64_t count, uint64_t *out)
{
    for (int64_t i = 0; i < count; ++i)
        out[i] = oracle_splitmix64(seed, (uint64_t)i);
}

/* U[0,1) on the grid k * 2^-24: the top 24 bits of each SplitMix64 output.
 * Every value is exact in fp32 and fp64.  Element i of a rows*cols*d map is
 * W[u][j] with i = u * d + j. */
void som_oracle_init_uniform(uint64_t seed, int64_t count, double *out)
{
    for (int64_t i = 0; i < count; ++i)
        out[i] = (double)(oracle_splitmix64(seed, (uint64_t)i) >> 40)
                 * (1.0 / 16777216.0);
}

/* Fisher-Yates shuffle of [0, n) for epoch e.  The epoch's stream seed is
 * the e-th SplitMix64 output of `seed`; the k-th swap (j = n-1 down to 1)
 * takes the k-th output r of that stream and picks position
 * floor(r * (j + 1) / 2^64) (multiply-high range reduction). */
void som_oracle_shuffle(uint64_t seed, int64_t epoch, int64_t n, int32_t *out)
{
    uint64_t es = oracle_splitmix64(seed, (uint64_t)epoch);
    for (int64_t i = 0; i < n; ++i)
        out[i] = (int32_t)i;
    uint64_t k = 0;
    for (int64_t j = n - 1; j >= 1; --j, ++k) {
        uint64_t r = oracle_splitmix64(es, k);
        uint64_t pick = (uint64_t)(((unsigned __int128)r * (uint64_t)(j + 1)) >> 64);
        int32_t tmp = out[j];
        out[j] = out[pick];
        out[pick] = tmp;
    }
}

/* ------------------------------------------------------------------------
 * Schedule: learning rate and radius at global step t of T (Sec. 6D says
 * both decay; the linear and exponential forms are the workload's).
 * ---------------------------------------------------------------------- */
static double oracle_decay(double a, double b, int32_t kind, double p)
{
    if (a == b)
        return a;
    /* Both forms are written so that p = 0 gives a and p = 1 gives b
     * exactly: (1-p)a + pb and a^(1-p) b^p. */
    if (kind == ORACLE_LINEAR)
        return (1.0 - p) * a + p * b;
    return pow(a, 1.0 - p) * pow(b, p);
}

void som_oracle_schedule_at(int64_t t, int64_t T, const som_oracle_schedule *s,
                            double *lr, double *sigma)
{
    double p = (T > 1) ? (double)t / (double)(T - 1) : 0.0;
    *lr = oracle_decay(s->lr0, s->lr1, s->lr_decay, p);
    *sigma = oracle_decay(s->sigma0, s->sigma1, s->sigma_decay, p);
}

/* ------------------------------------------------------------------------
 * Lattice geometry.
 * ---------------------------------------------------------------------- */
void som_oracle_position(int32_t topology, int32_t cols, int64_t u,
                         double *py, double *px)
{
    int64_t r = u / cols, c = u % cols;
    if (topology == ORACLE_HEX) {
        *px = (double)c + ((r % 2) ? 0.5 : 0.0);
        *py = (double)r * (sqrt(3.0) / 2.0);
    } else {
        *px = (double)c;
        *py = (double)r;
    }
}

static double oracle_lattice_sq(int32_t topology, int32_t cols, int64_t a, int64_t b)
{
    double ya, xa, yb, xb;
    som_oracle_position(topology, cols, a, &ya, &xa);
    som_oracle_position(topology, cols, b, &yb, &xb);
    return (ya - yb) * (ya - yb) + (xa - xb) * (xa - xb);
}

/* h for every unit, BMU c: Eq. (1)'s h_ck with the Gaussian kernel. */
void som_oracle_neighbourhood(int32_t rows, int32_t cols, int32_t topology,
                              int64_t c, double lr, double sigma, double *h)
{
    int64_t N = (int64_t)rows * cols;
    for (int64_t u = 0; u < N; ++u) {
        if (sigma == 0.0) {
            h[u] = (u == c) ? lr : 0.0;
        } else if (isinf(sigma)) {
            h[u] = lr;
        } else {
            double g = oracle_lattice_sq(topology, cols, u, c);
            h[u] = lr * exp(-g / (2.0 * sigma * sigma));
        }
    }
}

/* ------------------------------------------------------------------------
 * Competition: squared Euclidean distance of x to every prototype, and the
 * best-matching unit (lowest index among equal minima).
 * ---------------------------------------------------------------------- */
static void oracle_distances(const double *W, int64_t N, int64_t d,
                             const double *x, double *D, int nthreads)
{
#pragma omp parallel for schedule(static) num_threads(nthreads) if (nthreads > 1)
    for (int64_t u = 0; u < N; ++u) {
        const double *w = W + u * d;
        double s = 0.0;
        for (int64_t j = 0; j < d; ++j) {
            double diff = x[j] - w[j];
            s += diff * diff;
        }
        D[u] = s;
    }
}

static int64_t oracle_argmin(const double *D, int64_t N, int64_t skip)
{
    int64_t best = -1;
    for (int64_t u = 0; u < N; ++u) {
        if (u == skip)
            continue;
        if (best < 0 || D[u] < D[best])
            best = u;
    }
    return best;
}

void som_oracle_distances(const double *W, int64_t N, int64_t d,
                          const float *x, double *D)
{
    double *xd = (double *)malloc((size_t)d * sizeof(double));
    for (int64_t j = 0; j < d; ++j)
        xd[j] = (double)x[j];
    oracle_distances(W, N, d, xd, D, 1);
    free(xd);
}

/* ------------------------------------------------------------------------
 * Training: nsteps online steps, global step indices step0 .. step0+nsteps-1
 * of a schedule that spans T = total_steps steps.  order[k] is the sample of
 * local step k.  W (N x d, row-major, u = r * cols + c) is updated in place.
 * bmu_trace (nullable) receives the BMU of each step.
 * ---------------------------------------------------------------------- */
int som_oracle_train(double *W, int32_t rows, int32_t cols, int32_t topology,
                     int64_t d, const float *X, int64_t n, const int32_t *order,
                     int64_t nsteps, int64_t step0, int64_t total_steps,
                     const som_oracle_schedule *s, int32_t *bmu_trace,
                     int nthreads)
{
    if (!W || !X || !order || !s || rows <= 0 || cols <= 0 || d <= 0 || n <= 0 ||
        nsteps < 0 || step0 < 0 || total_steps < step0 + nsteps)
        return ORACLE_E_ARG;
    if (nthreads < 1)
        nthreads = 1;
    int64_t N = (int64_t)rows * cols;
    double *x = (double *)malloc((size_t)d * sizeof(double));
    double *D = (double *)malloc((size_t)N * sizeof(double));
    double *h = (double *)malloc((size_t)N * sizeof(double));
    if (!x || !D || !h) {
        free(x); free(D); free(h);
        return ORACLE_E_ARG;
    }
    for (int64_t k = 0; k < nsteps; ++k) {
        int64_t i = order[k];
        if (i < 0 || i >= n) {
            free(x); free(D); free(h);
            return ORACLE_E_ARG;
        }
        for (int64_t j = 0; j < d; ++j)
            x[j] = (double)X[i * d + j];
        double lr, sigma;
        som_oracle_schedule_at(step0 + k, total_steps, s, &lr, &sigma);

        oracle_distances(W, N, d, x, D, nthreads);
        int64_t c = oracle_argmin(D, N, -1);
        if (bmu_trace)
            bmu_trace[k] = (int32_t)c;

        som_oracle_neighbourhood(rows, cols, topology, c, lr, sigma, h);
#pragma omp parallel for schedule(static) num_threads(nthreads) if (nthreads > 1)
        for (int64_t u = 0; u < N; ++u) {
            double *w = W + u * d;
            double hu = h[u];
            for (int64_t j = 0; j < d; ++j)
                w[j] = w[j] + hu * (x[j] - w[j]);
        }
    }
    free(x); free(D); free(h);
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------
 * Training with near ties decided by a coin.  The same online steps as
 * som_oracle_train, except at a step whose second-smallest distance D2
 * exceeds the smallest D1 by at most tie_rel * D1: there the BMU is the
 * first or the second unit as bit 63 of SplitMix64(seed, global step) says
 * (1 = the second).  Two units that close are a tie at any precision that
 * cannot resolve tie_rel, so each such training is as valid as the plain
 * one; an ensemble of them over seeds measures how far the end of training
 * moves when runs part at near ties.  With tie_rel = 0 only exact ties
 * (D2 = D1) are candidates, and those flip too.  *flips (nullable) receives
 * the number of steps at which the second unit was taken.
 * ---------------------------------------------------------------------- */
int som_oracle_train_near_tie(double *W, int32_t rows, int32_t cols, int32_t topology,
                              int64_t d, const float *X, int64_t n, const int32_t *order,
                              int64_t nsteps, int64_t step0, int64_t total_steps,
                              const som_oracle_schedule *s, double tie_rel,
                              uint64_t seed, int64_t *flips, int nthreads)
{
    if (!W || !X || !order || !s || rows <= 0 || cols <= 0 || d <= 0 || n <= 0 ||
        nsteps < 0 || step0 < 0 || total_steps < step0 + nsteps || !(tie_rel >= 0.0))
        return ORACLE_E_ARG;
    if (nthreads < 1)
        nthreads = 1;
    int64_t N = (int64_t)rows * cols;
    double *x = (double *)malloc((size_t)d * sizeof(double));
    double *D = (double *)malloc((size_t)N * sizeof(double));
    double *h = (double *)malloc((size_t)N * sizeof(double));
    if (!x || !D || !h) {
        free(x); free(D); free(h);
        return ORACLE_E_ARG;
    }
    int64_t nflip = 0;
    for (int64_t k = 0; k < nsteps; ++k) {
        int64_t i = order[k];
        if (i < 0 || i >= n) {
            free(x); free(D); free(h);
            return ORACLE_E_ARG;
        }
        for (int64_t j = 0; j < d; ++j)
            x[j] = (double)X[i * d + j];
        double lr, sigma;
        som_oracle_schedule_at(step0 + k, total_steps, s, &lr, &sigma);

        oracle_distances(W, N, d, x, D, nthreads);
        int64_t c = oracle_argmin(D, N, -1);
        if (N > 1) {
            int64_t c2 = oracle_argmin(D, N, c);
            if (D[c2] - D[c] <= tie_rel * D[c] &&
                (oracle_splitmix64(seed, (uint64_t)(step0 + k)) >> 63)) {
                c = c2;
                ++nflip;
            }
        }

        som_oracle_neighbourhood(rows, cols, topology, c, lr, sigma, h);
#pragma omp parallel for schedule(static) num_threads(nthreads) if (nthreads > 1)
        for (int64_t u = 0; u < N; ++u) {
            double *w = W + u * d;
            double hu = h[u];
            for (int64_t j = 0; j < d; ++j)
                w[j] = w[j] + hu * (x[j] - w[j]);
        }
    }
    if (flips)
        *flips = nflip;
    free(x); free(D); free(h);
    return ORACLE_OK;
}

/* ------------------------------------------------------------------------
 * Evaluation over all n samples with fixed weights: first and second BMU,
 * their squared distances, quantization error and topographic error.
 * Any output pointer may be NULL.
 * ---------------------------------------------------------------------- */
int som_oracle_evaluate(const double *W, int32_t rows, int32_t cols,
                        int32_t topology, int64_t d, const float *X, int64_t n,
                        int32_t *c1, int32_t *c2, double *d1, double *d2,
                        double *qe, double *te, int nthreads)
{
    if (!W || !X || rows <= 0 || cols <= 0 || d <= 0 || n <= 0)
        return ORACLE_E_ARG;
    if (nthreads < 1)
        nthreads = 1;
    int64_t N = (int64_t)rows * cols;
    double *dist1 = (double *)malloc((size_t)n * sizeof(double));
    unsigned char *err = (unsigned char *)malloc((size_t)n);
#pragma omp parallel num_threads(nthreads) if (nthreads > 1)
    {
        double *x = (double *)malloc((size_t)d * sizeof(double));
        double *D = (double *)malloc((size_t)N * sizeof(double));
#pragma omp for schedule(static)
        for (int64_t i = 0; i < n; ++i) {
            for (int64_t j = 0; j < d; ++j)
                x[j] = (double)X[i * d + j];
            oracle_distances(W, N, d, x, D, 1);
            int64_t a = oracle_argmin(D, N, -1);
            int64_t b = (N > 1) ? oracle_argmin(D, N, a) : -1;
            dist1[i] = D[a];
            err[i] = (b >= 0) && (sqrt(oracle_lattice_sq(topology, cols, a, b)) > 1.0 + 1e-9);
            if (c1) c1[i] = (int32_t)a;
            if (c2) c2[i] = (int32_t)b;
            if (d1) d1[i] = D[a];
            if (d2) d2[i] = (b >= 0) ? D[b] : INFINITY;
        }
        free(x);
        free(D);
    }
    double sq = 0.0, st = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        sq += sqrt(dist1[i]);
        st += err[i] ? 1.0 : 0.0;
    }
    if (qe) *qe = sq / (double)n;
    if (te) *te = st / (double)n;
    free(dist1);
    free(err);
    return ORACLE_OK;
}
