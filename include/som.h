/*
 * som.h -- C ABI of libsom, an MI355X (gfx950) library for online
 * self-organizing-map (SOM) training on high-dimensional document vectors.
 *
 * The method (paper Sec. 5A, Eq. (1); GPU procedure Sec. 6C): a map of
 * rows x cols units, each with a prototype w_u of length d, is trained one
 * sample x at a time.  Every step computes the squared Euclidean distance of x
 * to every prototype, takes the best-matching unit (BMU) c as the arg-min
 * (lowest index among equal minima), and moves every prototype toward x:
 *
 *     w_u <- w_u + h_u (x - w_u),  h_u = lr(t) exp(-|pos(u) - pos(c)|^2 / (2 sigma(t)^2))
 *
 * while the learning rate lr and the neighbourhood radius sigma decay over
 * the steps (Sec. 6D).  The trained map then assigns each document to its BMU
 * (Sec. 8A) and is scored by its quantization error (Sec. 6D, Sec. 8B).
 *
 * Conventions shared by every call:
 *   - Every call returns a som_status.  No call throws or aborts.
 *   - Arguments are validated before any device work; a call that returns
 *     SOM_E_ARG has enqueued nothing and changed nothing.
 *   - Data pointers named "device" must point into device memory (hipMalloc
 *     or a torch CUDA tensor) that covers the stated extent; the library
 *     checks both and returns SOM_E_ARG otherwise.  They stay owned by the
 *     caller and must stay valid until the map's stream reaches the end of
 *     the call.
 *   - Calls are ordered on the map's stream (som_set_stream) and return
 *     after enqueueing, except where a call says it synchronizes.  A device
 *     error inside an asynchronous call (for example a bad sample index in a
 *     caller-supplied order, or a training kernel whose grid barrier timed
 *     out) is reported by the next synchronizing call on that map.
 *   - A map is not thread-safe: use one map per host thread.
 *   - Floating point: prototypes and data are fp32; distances are fp32 sums;
 *     the schedule (lr and log2(e) / (2 sigma^2) per step) is evaluated in
 *     fp64 and rounded once to fp32; the neighbourhood factor of every unit
 *     is then lr * exp2(-g * log2(e) / (2 sigma^2)) in fp32 (the hardware
 *     exp2, denormal results flushed to zero), g the squared lattice
 *     distance; QE and TE are accumulated in fp64.
 *   - Memory cap: SOM_MAX_BYTES (environment, decimal bytes, default 64 GiB,
 *     read at every call) bounds each buffer a map allocates: the prototypes
 *     (som_create), the evaluation scratch (candidate lists; three per-sample
 *     arrays), the sparse and batch work buffers.  A call that would exceed
 *     it returns SOM_E_OOM before allocating, and the map stays usable.
 *   - Failure-path switches (environment, for tests of the error paths only):
 *     SOM_DEBUG_EXCHANGE_TIMEOUT_US bounds each grid-exchange wait of the
 *     training kernels (default 20 s); SOM_DEBUG_ABSENT_WORKGROUP=1 makes
 *     som_train launch one workgroup fewer than its exchanges wait for, so
 *     every wait runs into that bound, every workgroup leaves its loop, and
 *     the next synchronizing call reports SOM_E_TIMEOUT.
 *   - Device pointer extents are checked against the allocation that holds
 *     the pointer (hipMemGetAddressRange).  Under a pooling allocator (for
 *     example torch's caching allocator) that allocation can be a larger
 *     pool segment, so the check is best effort: a pointer whose own tensor
 *     is shorter than the stated extent can still pass it.
 */
#ifndef SOM_H
#define SOM_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum som_status {
    SOM_OK = 0,
    SOM_E_ARG = 1,         /* invalid argument; nothing was done            */
    SOM_E_OOM = 2,         /* device allocation failed or over the cap      */
    SOM_E_DEVICE = 3,      /* HIP runtime error                             */
    SOM_E_LAUNCH = 4,      /* the cooperative grid cannot be co-resident    */
    SOM_E_TIMEOUT = 5,     /* a grid barrier did not complete in time       */
    SOM_E_UNSUPPORTED = 6, /* shape outside what the kernels are built for  */
    SOM_E_BAD_ORDER = 7,   /* a caller-supplied sample index was outside [0, n) */
    SOM_E_NONFINITE = 8    /* the training data held a NaN or an infinity   */
} som_status;

/* Lattice of the map.  RECT: unit u = r * cols + c sits at (r, c).  HEX
 * (the paper's choice, Sec. 6C): odd rows shifted by half a unit, rows
 * sqrt(3)/2 apart.  Lattice distance is Euclidean, without wrap-around. */
typedef enum som_topology { SOM_RECT = 0, SOM_HEX = 1 } som_topology;

/* Decay law of lr and sigma between their endpoint values a (step 0) and b
 * (step T-1), at p = t / (T - 1) (p = 0 when T = 1):
 *   LINEAR       (1 - p) a + p b
 *   EXPONENTIAL  a^(1-p) b^p            (needs a > 0 and b > 0)
 * Equal endpoints give that constant value (also +inf for sigma). */
typedef enum som_decay { SOM_DECAY_LINEAR = 0, SOM_DECAY_EXPONENTIAL = 1 } som_decay;

/* Training schedule (paper Sec. 6D: lr and the neighbourhood radius decay).
 *   lr0, lr1        learning rate at the first and last step; >= 0, finite.
 *   sigma0, sigma1  radius at the first and last step; >= 0 (+inf allowed for
 *                   a constant radius).  sigma = 0 makes h a Kronecker delta
 *                   at the BMU; sigma = +inf makes h = lr for every unit.
 *   shuffle_seed    used only when order == NULL: epoch e presents the
 *                   samples in a Fisher-Yates permutation drawn from the
 *                   e-th SplitMix64 output of shuffle_seed (see som_shuffle).
 *   order           NULL, or a device int32 array of epochs * n sample
 *                   indices, entry k being the sample of the call's step k.
 *   step0           global index of the call's first step (to resume).
 *   total_steps     T, the schedule's length; 0 means step0 + epochs * n.
 *                   Must be >= step0 + epochs * n.
 *   bmu_trace       NULL, or a device int32 array of epochs * n entries that
 *                   receives the BMU of every step.                            */
typedef struct som_schedule {
    double lr0;
    double lr1;
    int32_t lr_decay;
    double sigma0;
    double sigma1;
    int32_t sigma_decay;
    uint64_t shuffle_seed;
    const int32_t *order;
    int64_t step0;
    int64_t total_steps;
    int32_t *bmu_trace;
} som_schedule;

typedef struct som_map som_map;

/* Create a rows x cols map of d-dimensional fp32 prototypes on the current
 * HIP device and initialise them U[0,1): element i = u * d + j is the top
 * 24 bits of the i-th SplitMix64 output of `seed`, times 2^-24 (the paper's
 * principal-component plane initialisation, Sec. 6D, is som_init_linear).
 * The prototypes are owned by the map.  Topology starts as RECT and
 * the stream as the null stream.
 * Errors: SOM_E_ARG (rows, cols or d <= 0, rows * cols > 2^24 - 1,
 * rows * cols * d overflows, out == NULL), SOM_E_OOM, SOM_E_DEVICE.
 * Synchronizes the device once (initialisation). */
som_status som_create(int32_t rows, int32_t cols, int32_t d, uint64_t seed,
                      som_map **out);

/* Release the map and its device memory after the stream drains.  NULL is
 * a no-op. */
som_status som_destroy(som_map *map);

/* SOM_RECT or SOM_HEX; SOM_E_ARG otherwise. */
som_status som_set_topology(som_map *map, int32_t topology);

/* Order all later calls on `stream` (a hipStream_t, e.g. torch's
 * torch.cuda.current_stream().cuda_stream); NULL selects the null stream. */
som_status som_set_stream(som_map *map, void *stream);

/* Online training (paper Sec. 5A and 6C): epochs * n steps over the n x d
 * row-major fp32 device matrix X, as one persistent cooperative kernel that
 * keeps the whole per-sample loop on the device.  Stream-ordered.  When d is
 * not a multiple of 4 or X is not 16-byte aligned, X is first copied into a
 * buffer of n * roundup(d, 4) floats that the map keeps for later calls;
 * when the plan is the long-row kernel (som_train_plan variant 4) and the
 * prototypes' row pitch exceeds d, into a buffer of n rows of that pitch
 * (zero past d).
 * Errors: SOM_E_ARG (map, X or sched NULL, n <= 0, epochs <= 0, epochs * n
 * beyond 2^31 - 1, bad decay kind, lr < 0 or not finite, sigma < 0 or NaN,
 * exponential decay with a zero or infinite endpoint, total_steps too small,
 * X, order or bmu_trace not covering their extent), SOM_E_UNSUPPORTED
 * (d above the largest built kernel shape, or more units per workgroup than
 * the kernels' per-unit LDS state holds: 4096 per workgroup for d <= 256
 * and at least 690 otherwise, i.e. 1,048,576 and 176,640 units on 256
 * workgroups), SOM_E_LAUNCH, SOM_E_DEVICE.
 * An order entry outside [0, n) stops the kernel before any update and is
 * reported as SOM_E_BAD_ORDER by the next synchronizing call.  Every call
 * also scans all n * d floats of X once (a read of n * d * 4 bytes): a NaN
 * or an infinity anywhere in X likewise stops the kernel before any update
 * and is reported as SOM_E_NONFINITE (the first of the two errors raised
 * is the one reported). */
som_status som_train(som_map *map, const float *X, int64_t n, int32_t epochs,
                     const som_schedule *sched);

/* Online training from sparse samples: the same steps as som_train (Eq. (1)
 * of Sec. 5A, one BMU per step, lowest index on ties) for the n rows of a
 * CSR matrix, such as the L2-normalised TF-IDF vectors of Sec. 6B, at a
 * cost per step proportional to the row's non-zeros rather than to d.
 *   indptr   device int64 array of n + 1 offsets, indptr[0] = 0; row i is
 *            entries indptr[i] .. indptr[i+1] - 1 of indices and values.
 *   indices  device int32 array of indptr[n] feature indices, strictly
 *            increasing within each row, in [0, d).
 *   values   device fp32 array of indptr[n] values.
 * indices and values may be NULL when indptr[n] = 0.  The schedule fields
 * mean what they mean for som_train.
 * Internally each prototype is held as a scale times an fp64 vector stored
 * feature by feature ((d + 3) * roundup(rows * cols, 64) doubles, at most
 * 2^31 - 1 bytes for the vectors, plus 28 K + 40 bytes per step for the
 * padded entries, K = 16, 32 or 64 from the longest row; all kept by the
 * map for later calls), so a step reads and writes only the sample's
 * features; distances are evaluated in fp64 and rounded once to fp32 for
 * the BMU comparison.  The call synchronizes the stream twice to validate
 * the CSR structure before training, which is then stream-ordered.
 * Errors: as som_train, and SOM_E_ARG (indptr NULL or not covering n + 1
 * entries, indptr[0] != 0, a row with decreasing offsets or offsets past
 * indptr[n], indices not strictly increasing within a row or outside
 * [0, d), indices or values not covering indptr[n] entries),
 * SOM_E_UNSUPPORTED (a row with more than 64 non-zeros, more than 16,384
 * units, or (d + 1) * roundup(rows * cols, 64) * 8 above 2^31 - 1 bytes),
 * SOM_E_OOM (the buffers above beyond the map's memory cap).  The
 * indptr[n] values are scanned as som_train scans X (SOM_E_NONFINITE). */
som_status som_train_csr(som_map *map, const int64_t *indptr, const int32_t *indices,
                         const float *values, int64_t n, int32_t epochs,
                         const som_schedule *sched);

/* Batch-map training, the batch form of the SOM that Sec. 4 attributes to
 * earlier GPU SOMs ([25], [26]), beside the paper's online rule (Sec. 5A):
 * each of `epochs` epochs assigns all n rows of the device matrix X to
 * their BMUs (as som_bmu) and then sets every prototype to the
 * neighbourhood-weighted mean of the samples,
 *     w_u = sum_i h(u, c_i) x_i / sum_i h(u, c_i),
 * h(u, c) = exp(-|pos(u) - pos(c)|^2 / (2 sigma^2)) (a delta at the BMU for
 * sigma = 0, 1 everywhere for sigma = +inf); a unit whose weights all
 * vanish keeps its prototype.  sigma goes from sigma0 (first epoch) to
 * sigma1 (last epoch) by sigma_decay at p = e / (epochs - 1).  Everything
 * after the BMU is fp64: per-unit sample sums, then the lattice Gaussian as
 * a blur along the lattice columns and then along the rows (it factors over
 * the two axes).  Work memory of (2 + P) N (d + 1) + rows^2 + P cols^2
 * doubles (P = 1 for RECT, 3 for HEX) is kept by the map.  Stream-ordered.
 * Errors: SOM_E_ARG (map or X NULL, n <= 0 or above 2^31 - 1, epochs <= 0,
 * sigma < 0 or NaN, a bad decay kind, an exponential decay with a zero or
 * infinite endpoint, X not covering n * d floats), SOM_E_UNSUPPORTED (d
 * above 4,194,239), SOM_E_OOM, SOM_E_DEVICE. */
som_status som_train_batch(som_map *map, const float *X, int64_t n, int32_t epochs,
                           double sigma0, double sigma1, int32_t sigma_decay);

/* Batched BMU assignment (Sec. 8A): for each of the n rows of the device
 * matrix X, out_idx[i] = BMU index (lowest index among equal minima).
 * Candidates are ranked with fp32 matrix-core products
 * ||w||^2 - 2 x.w (the product split over ranges of d, and the ranges
 * summed in order, when there are too few samples to fill the chip
 * otherwise); the four best by that score are re-ranked by direct fp32
 * distances.  Scratch (candidate lists of 32 bytes per sample and unit
 * group, or 512 bytes per sample, range and 128 units of partial products
 * when d is split) is kept by the map.
 * out_idx is a device int32 array of n entries.  Stream-ordered. */
som_status som_bmu(som_map *map, const float *X, int64_t n, int32_t *out_idx);

/* As som_bmu, also writing the second BMU (out_idx2, -1 for a one-unit map)
 * and the squared distance to the BMU (out_d1, fp32).  Any of the three
 * outputs may be NULL.  Device arrays of n entries.  Stream-ordered. */
som_status som_bmu2(som_map *map, const float *X, int64_t n, int32_t *out_idx,
                    int32_t *out_idx2, float *out_d1);

/* As som_bmu2, for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same kernels and the same outputs, but no hipMalloc, hipFree or
 * allocating library routine is called.  The call's scratch (the
 * prototypes' squared norms, the BMUs when out_idx is NULL, the candidate
 * lists, and the partial products when the search splits d) lives in one
 * fixed 8 MiB array per device, held from the library's load until the
 * process ends.  The search takes the fastest shape whose scratch fits:
 *     roundup256(4 N) + (out_idx ? 0 : roundup256(4 n))
 *       + (split ? roundup256(512 S n T_u) : roundup256(32 n G))
 * bytes (N units; unsplit, G the unit groups whose candidate lists are kept
 * apart; split, S the ranges of d and T_u = ceil(N / 128) the unit tiles);
 * with G = 1 and no split the need is smallest, and a call whose inputs
 * need more than the array even then
 * returns SOM_E_UNSUPPORTED without launching anything.  The outputs equal
 * som_bmu2's whenever the same shape fits (the shape is chosen from the
 * sizes alone), and otherwise whenever a sample's best two units are not
 * tied with its fifth by score within rounding.
 * Every call on a device shares that device's array and overwrites what
 * it needs before reading it, so calls that overlap on one device (on
 * different streams, or from different host threads) race; order them.
 * The map's device must be the current device.  Stream-ordered.
 * Errors: as som_bmu2, and SOM_E_ARG (the map's device is not current),
 * SOM_E_UNSUPPORTED (scratch beyond the fixed array). */
som_status som_bmu2_noalloc(som_map *map, const float *X, int64_t n, int32_t *out_idx,
                            int32_t *out_idx2, float *out_d1);

/* Quantization error (Sec. 6D, Sec. 8B): mean over the n samples of the
 * unsquared Euclidean distance to the BMU, accumulated in fp64.  *out_qe is
 * a host double.  Synchronizes the stream. */
som_status som_quantization_error(som_map *map, const float *X, int64_t n,
                                  double *out_qe);

/* Topographic error: fraction of the n samples whose first and second BMUs
 * are not lattice neighbours (lattice distance > 1); 0 for a one-unit map.
 * *out_te is a host double.  Synchronizes the stream. */
som_status som_topographic_error(som_map *map, const float *X, int64_t n,
                                 double *out_te);

/* Evaluation in one pass (Sec. 8A, Sec. 6D, Sec. 8B): the BMU of every
 * one of the n rows of the device matrix X into out_idx (a device int32
 * array of n entries, or NULL), together with the quantization error
 * (*out_qe) and the topographic error (*out_te) of som_quantization_error
 * and som_topographic_error, from one batched BMU search instead of one
 * per quantity.  out_qe and out_te are host doubles; either may be NULL,
 * but not all three outputs.  Synchronizes the stream.
 * Errors: SOM_E_ARG (map or X NULL, n <= 0 or above 2^31 - 1, X or out_idx
 * not covering their extent, all outputs NULL), SOM_E_OOM, SOM_E_DEVICE. */
som_status som_evaluate(som_map *map, const float *X, int64_t n, int32_t *out_idx,
                        double *out_qe, double *out_te);

/* Copy the rows*cols x d prototypes (row-major, unit u = r * cols + c) out
 * to / in from `dst` / `src`, a host or device pointer of rows*cols*d floats.
 * Used to start from a given state and to checkpoint and resume.
 * Synchronize the stream. */
som_status som_get_weights(som_map *map, float *dst);
som_status som_set_weights(som_map *map, const float *src);

/* Wait for the map's stream and report any deferred device error. */
som_status som_synchronize(som_map *map);

/* rows, cols, d and topology of a map; any output may be NULL. */
som_status som_get_shape(const som_map *map, int32_t *rows, int32_t *cols,
                         int32_t *d, int32_t *topology);

/* The Fisher-Yates permutation of [0, n) that som_train uses for epoch
 * `epoch` when no order is given (host int32 array of n entries). */
som_status som_shuffle(uint64_t seed, int64_t epoch, int64_t n, int32_t *out);

/* The two largest principal components of the n x d row-major fp32 device
 * matrix X (paper Fig. 2 steps 3-4, Sec. 6D): eigenvalues lambda[0] >=
 * lambda[1] of the covariance (1/n) sum_i (x_i - mu)(x_i - mu)^T into the
 * host array lambda[2], and optionally the column means (mean) and the
 * unit eigenvectors (v1, v2; sign such that the component of largest
 * magnitude, lowest index on ties, is positive) into device arrays of d
 * floats.  Computed on the device (fp32 matrix-core covariance, fp64-reduced
 * subspace iteration until both residuals are below 2e-5 lambda[0], at most
 * 4000 iterations) with d * d + 144 d floats of work memory allocated for
 * the call; ordered on `stream` (a hipStream_t, NULL for the null stream),
 * which it synchronizes.
 * Errors: SOM_E_ARG (NULL X or lambda, n or d <= 0, pointers not covering
 * their extent), SOM_E_OOM, SOM_E_DEVICE. */
som_status som_pca2(const float *X, int64_t n, int32_t d, void *stream, double *lambda,
                    float *mean, float *v1, float *v2);

/* Map size and iteration count for m samples whose two largest
 * principal-component variances are lambda1 >= lambda2 (paper Fig. 2):
 * munits = ceil(5 sqrt(m)); r = sqrt(lambda1 / lambda2), or 1 when lambda1
 * = 0 or lambda2 * munits < lambda1; size1 = the nearest integer to
 * sqrt(munits / (r sqrt(3/4))) (the figure's garbled cube root read as the
 * square root of 3/4, the hexagonal row pitch), within [1, munits]; size2 =
 * ceil(munits / size1); rows = min(size1, size2), cols = max; iterations =
 * ceil(50 rows cols / m) * m * 4.  Host arithmetic; outputs may be NULL.
 * Errors: SOM_E_ARG (m <= 0, lambda2 < 0, lambda1 < lambda2, non-finite). */
som_status som_suggest_size(int64_t m, double lambda1, double lambda2, int32_t *rows,
                            int32_t *cols, int64_t *iterations);

/* Linear initialisation (Sec. 6D): the map's prototypes become a regular
 * grid in the plane through the mean mu of the n x d device matrix X spanned
 * by its two largest principal components (as som_pca2):
 *     w(r, c) = mu + a_c sqrt(lambda1) v1 + b_r sqrt(lambda2) v2,
 *     a_c = 2c / (cols - 1) - 1,  b_r = 2r / (rows - 1) - 1   (0 for one
 * column / row), so the longer side spans the first component over one
 * standard deviation either side.  Synchronizes the map's stream.
 * Errors: as som_pca2. */
som_status som_init_linear(som_map *map, const float *X, int64_t n);

/* Launch shape that som_train would use for this map: workgroups, threads
 * per workgroup, kernel variant (0 = prototypes streamed from memory once
 * per block of steps, 1 = prototypes held in LDS for the whole call, 2 / 3 =
 * the same with the pass over the prototypes overlapped with the grid
 * exchanges, 4 = as 2 for rows too long to keep the samples' slices in
 * registers: the pass walks the columns and loads each column slice of the
 * samples once for all rows) and steps per block (the number of consecutive samples whose
 * updates one pass over the prototypes applies).  Any output may be NULL. */
som_status som_train_plan(const som_map *map, int32_t *grid, int32_t *block,
                          int32_t *variant, int32_t *block_steps);

/* Memory reference for the roofline of som_train; not a step of the
 * method.  Rewrites the `bytes` bytes at the device pointer buf in place,
 * `passes` times, in one launch of `grid` workgroups of 256 threads:
 * workgroup b of G reads, scales by 1 and writes back its own contiguous
 * share of the buffer's 16-byte words (b / G to (b + 1) / G of them), as a
 * training workgroup streams its own range of prototype rows, so no
 * workgroup waits for another and the passes follow each other without a
 * gap.  The buffer's contents are unchanged.  Moves 2 * bytes * passes
 * bytes.  Ordered on `stream` (a hipStream_t, NULL for the null stream);
 * returns after enqueueing.
 * Errors: SOM_E_ARG (buf NULL or not 16-byte aligned, bytes <= 0 or not a
 * multiple of 16, passes <= 0, grid outside [1, 1024], buf not covering
 * `bytes`), SOM_E_DEVICE. */
som_status som_stream_inplace(void *buf, int64_t bytes, int32_t passes, int32_t grid,
                              void *stream);

/* Human-readable name of a status code (static storage). */
const char *som_status_string(som_status status);

#ifdef __cplusplus
}
#endif

#endif /* SOM_H */
