// Host runtime of libsom: the C ABI declared in include/som.h.
//
// Owns the map (prototypes in device memory, each row padded with zeros to
// the training kernel's lane slots, so rows are read as 16-byte vectors with
// no column bounds), validates every
// argument before any device work, builds the per-epoch sample order when
// the caller gives none, and launches the kernels on the map's stream.
#include "som.h"
#include "som_internal.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

#include <vector>

// Subspace iteration of the principal components: residual target relative
// to the largest eigenvalue, and an iteration cap.
static constexpr int kPcaMaxIters = 4000;
static constexpr double kPcaTol = 2e-5;

struct som_map {
    int32_t rows = 0, cols = 0, d = 0, topology = SOM_RECT;
    int32_t N = 0;
    int64_t ld = 0;  // row pitch in floats
    int device = 0;
    int num_cus = 0;
    hipStream_t stream = nullptr;
    float *W = nullptr;
    som::DevState *state = nullptr;
    unsigned long long *slots = nullptr;  // grid-exchange words
    // order staging for library-shuffled training
    int32_t *order_dev = nullptr;
    int64_t order_cap = 0;
    int32_t *order_host = nullptr;  // pinned
    hipEvent_t order_done = nullptr;
    // per-step schedule table of the current training call
    float2 *sched = nullptr;
    int64_t sched_cap = 0;
    // per-block sample products of the pipelined training kernel
    float *block_dots = nullptr;
    int64_t block_dots_cap = 0;
    // training copy of X with rows padded to a multiple of 4 floats (used
    // when d % 4 != 0 or X is not 16-byte aligned)
    float *xpad = nullptr;
    int64_t xpad_cap = 0;
    // sparse training: feature-major fp64 prototypes with their scales and
    // norms ((d + 1) * ldv + 2 * ldv doubles) and the per-step entries
    double *sv = nullptr;
    int64_t sv_cap = 0;
    uint32_t *soff = nullptr;
    double *sval = nullptr, *spv1 = nullptr, *spv2 = nullptr;
    som::SparseStep *sst = nullptr;
    int64_t soff_cap = 0, sval_cap = 0, spv1_cap = 0, spv2_cap = 0, sst_cap = 0;
    // batch-map work memory (som_batch.hip)
    double *bwork = nullptr;
    int64_t bwork_cap = 0;
    // evaluation scratch
    float *wnorm = nullptr;
    int32_t *cand = nullptr, *idx1 = nullptr, *idx2 = nullptr;
    int64_t cand_cap = 0;
    float *part = nullptr;
    int64_t part_cap = 0;
    float *d1 = nullptr;
    double *sums = nullptr;
    int64_t eval_cap = 0;
};

namespace {

constexpr uint64_t kMaxBytesDefault = 64ull << 30;  // per-map device memory cap

uint64_t max_bytes() {
    const char *e = getenv("SOM_MAX_BYTES");
    if (e && *e) {
        char *end = nullptr;
        unsigned long long v = strtoull(e, &end, 10);
        if (end && *end == '\0' && v > 0) return v;
    }
    return kMaxBytesDefault;
}

som_status from_hip(hipError_t e) {
    if (e == hipSuccess) return SOM_OK;
    if (e == hipErrorOutOfMemory || e == hipErrorMemoryAllocation) return SOM_E_OOM;
    if (e == hipErrorCooperativeLaunchTooLarge) return SOM_E_LAUNCH;
    return SOM_E_DEVICE;
}

// True when [p, p + bytes) lies inside one device allocation.
bool device_range_ok(const void *p, uint64_t bytes) {
    if (!p) return false;
    hipPointerAttribute_t attr;
    if (hipPointerGetAttributes(&attr, p) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    if (attr.type != hipMemoryTypeDevice && attr.type != hipMemoryTypeManaged) return false;
    hipDeviceptr_t base = nullptr;
    size_t size = 0;
    if (hipMemGetAddressRange(&base, &size, const_cast<void *>(p)) != hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    const uintptr_t b = reinterpret_cast<uintptr_t>(base);
    const uintptr_t q = reinterpret_cast<uintptr_t>(p);
    return q >= b && bytes <= size && q - b <= size - bytes;
}

bool schedule_ok(const som_schedule *s) {
    if (s->lr_decay != SOM_DECAY_LINEAR && s->lr_decay != SOM_DECAY_EXPONENTIAL) return false;
    if (s->sigma_decay != SOM_DECAY_LINEAR && s->sigma_decay != SOM_DECAY_EXPONENTIAL)
        return false;
    if (!(s->lr0 >= 0.0) || !(s->lr1 >= 0.0) || isinf(s->lr0) || isinf(s->lr1)) return false;
    if (!(s->sigma0 >= 0.0) || !(s->sigma1 >= 0.0)) return false;  // rejects NaN
    if (s->lr_decay == SOM_DECAY_EXPONENTIAL && s->lr0 != s->lr1 &&
        (s->lr0 == 0.0 || s->lr1 == 0.0))
        return false;
    if (s->sigma_decay == SOM_DECAY_EXPONENTIAL && s->sigma0 != s->sigma1 &&
        (s->sigma0 == 0.0 || s->sigma1 == 0.0 || isinf(s->sigma0) || isinf(s->sigma1)))
        return false;
    if (s->sigma_decay == SOM_DECAY_LINEAR && s->sigma0 != s->sigma1 &&
        (isinf(s->sigma0) || isinf(s->sigma1)))
        return false;
    return true;
}

uint64_t splitmix64_at(uint64_t seed, uint64_t i) {
    uint64_t z = seed + (i + 1u) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

void fisher_yates(uint64_t seed, int64_t epoch, int64_t n, int32_t *out) {
    const uint64_t es = splitmix64_at(seed, (uint64_t)epoch);
    for (int64_t i = 0; i < n; ++i) out[i] = (int32_t)i;
    uint64_t k = 0;
    for (int64_t j = n - 1; j >= 1; --j, ++k) {
        const uint64_t r = splitmix64_at(es, k);
        const uint64_t pick = (uint64_t)(((unsigned __int128)r * (uint64_t)(j + 1)) >> 64);
        const int32_t t = out[j];
        out[j] = out[pick];
        out[pick] = t;
    }
}

// Replace *p by a fresh device array of `count` elements.
template <typename T>
som_status grow(T **p, int64_t count) {
    if (*p) {
        hipError_t e = hipFree(*p);
        *p = nullptr;
        if (e != hipSuccess) return from_hip(e);
    }
    return from_hip(hipMalloc(reinterpret_cast<void **>(p), (size_t)count * sizeof(T)));
}

// Make *p hold at least `need` elements (waiting for the stream before a
// buffer it may still use is replaced).
template <typename T>
hipError_t ensure(som_map *m, T **p, int64_t *cap, int64_t need) {
    if (*cap >= need) return hipSuccess;
    hipError_t e = hipStreamSynchronize(m->stream);
    if (e == hipSuccess && *p) e = hipFree(*p);
    *p = nullptr;
    *cap = 0;
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(p), (size_t)need * sizeof(T));
    if (e == hipSuccess) *cap = need;
    return e;
}

// Evaluation scratch for n samples, ncand candidate-list entries (int32)
// and npart partial products.  A capacity is zeroed before its buffers are
// replaced and set again only once every one of them is allocated, so a
// failed allocation leaves no stale capacity behind a null or freed buffer.
som_status ensure_eval_scratch(som_map *m, int64_t n, int64_t ncand, int64_t npart = 0) {
    hipError_t e;
    som_status st;
    // the candidate lists, the partial products and the three per-sample
    // arrays, each against the cap
    if ((uint64_t)ncand * sizeof(int32_t) > max_bytes() ||
        (uint64_t)npart * sizeof(float) > max_bytes() ||
        (uint64_t)n * (2 * sizeof(int32_t) + sizeof(float)) > max_bytes())
        return SOM_E_OOM;
    if (ncand > m->cand_cap) {
        if ((e = hipStreamSynchronize(m->stream)) != hipSuccess) return from_hip(e);
        m->cand_cap = 0;
        if ((st = grow(&m->cand, ncand)) != SOM_OK) return st;
        m->cand_cap = ncand;
    }
    if (npart > m->part_cap) {
        if ((e = hipStreamSynchronize(m->stream)) != hipSuccess) return from_hip(e);
        m->part_cap = 0;
        if ((st = grow(&m->part, npart)) != SOM_OK) return st;
        m->part_cap = npart;
    }
    if (n <= m->eval_cap) return SOM_OK;
    if ((e = hipStreamSynchronize(m->stream)) != hipSuccess) return from_hip(e);
    m->eval_cap = 0;
    if ((st = grow(&m->idx1, n)) != SOM_OK) return st;
    if ((st = grow(&m->idx2, n)) != SOM_OK) return st;
    if ((st = grow(&m->d1, n)) != SOM_OK) return st;
    m->eval_cap = n;
    return SOM_OK;
}

som_status check_deferred(som_map *m) {
    som::DevState st;
    hipError_t e = hipMemcpy(&st, m->state, sizeof(st), hipMemcpyDeviceToHost);
    if (e != hipSuccess) return from_hip(e);
    if (st.status != 0) {
        const int32_t zero = 0;
        e = hipMemcpy(&m->state->status, &zero, sizeof(zero), hipMemcpyHostToDevice);
        if (e != hipSuccess) return from_hip(e);
        return (som_status)st.status;
    }
    return SOM_OK;
}

som_status run_eval(som_map *m, const float *X, int64_t n, int32_t *idx1,
                    int32_t *idx2, float *d1) {
    som::EvalArgs a{};
    a.W = m->W;
    a.ld = m->ld;
    a.N = m->N;
    a.d = m->d;
    a.rows = m->rows;
    a.cols = m->cols;
    a.topology = m->topology;
    a.X = X;
    a.n = n;
    if (!som::plan_bmu_candidates(&a, m->num_cus, max_bytes())) return SOM_E_OOM;
    som_status st = ensure_eval_scratch(m, n, som::bmu_cand_ints(a), som::bmu_part_floats(a));
    if (st != SOM_OK) return st;
    a.wnorm = m->wnorm;
    a.cand = m->cand;
    a.part = m->part;
    a.idx1 = idx1;
    a.idx2 = idx2;
    a.d1 = d1;
    a.x_vec4 = (m->d % 4 == 0) && (reinterpret_cast<uintptr_t>(X) % 16 == 0);
    hipError_t e = som::launch_row_sqnorm(m->W, m->ld, m->N, m->wnorm, m->stream);
    if (e == hipSuccess) e = som::launch_bmu_candidates(a, m->stream);
    if (e == hipSuccess) e = som::launch_bmu_rerank(a, m->stream);
    return from_hip(e);
}

bool eval_args_ok(som_map *m, const float *X, int64_t n) {
    if (!m || !X || n <= 0 || n > INT32_MAX) return false;
    return device_range_ok(X, (uint64_t)n * (uint64_t)m->d * sizeof(float));
}

}  // namespace

extern "C" {

const char *som_status_string(som_status s) {
    switch (s) {
        case SOM_OK: return "ok";
        case SOM_E_ARG: return "invalid argument";
        case SOM_E_OOM: return "out of device memory";
        case SOM_E_DEVICE: return "device error";
        case SOM_E_LAUNCH: return "cooperative grid cannot be co-resident";
        case SOM_E_TIMEOUT: return "grid barrier timed out";
        case SOM_E_UNSUPPORTED: return "shape not supported by the built kernels";
        case SOM_E_BAD_ORDER: return "sample order holds an index outside [0, n)";
        case SOM_E_NONFINITE: return "training data holds a NaN or an infinity";
    }
    return "unknown status";
}

som_status som_shuffle(uint64_t seed, int64_t epoch, int64_t n, int32_t *out) {
    if (!out || n <= 0 || n > INT32_MAX || epoch < 0) return SOM_E_ARG;
    fisher_yates(seed, epoch, n, out);
    return SOM_OK;
}

som_status som_create(int32_t rows, int32_t cols, int32_t d, uint64_t seed,
                      som_map **out) {
    if (!out || rows <= 0 || cols <= 0 || d <= 0) return SOM_E_ARG;
    *out = nullptr;
    const int64_t N = (int64_t)rows * cols;
    if (N > som::kMaxUnits) return SOM_E_ARG;
    // Rows padded to the training kernel's lane slots (zero padding) when a
    // kernel shape covers d; otherwise to 16 bytes (evaluation only).
    int64_t ld = som::train_row_pitch(d);
    if (ld == 0) ld = ((int64_t)d + 3) / 4 * 4;
    const uint64_t bytes = (uint64_t)N * (uint64_t)ld * sizeof(float);
    if (bytes / sizeof(float) / (uint64_t)ld != (uint64_t)N) return SOM_E_ARG;
    if (bytes > max_bytes()) return SOM_E_OOM;

    som_map *m = new (std::nothrow) som_map();
    if (!m) return SOM_E_OOM;
    m->rows = rows;
    m->cols = cols;
    m->d = d;
    m->N = (int32_t)N;
    m->ld = ld;
    hipError_t e = hipGetDevice(&m->device);
    if (e == hipSuccess)
        e = hipDeviceGetAttribute(&m->num_cus, hipDeviceAttributeMultiprocessorCount,
                                  m->device);
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&m->W), bytes);
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&m->state), sizeof(som::DevState));
    if (e == hipSuccess) e = hipMemset(m->state, 0, sizeof(som::DevState));
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&m->slots),
                      (size_t)som::kSlotWords * sizeof(unsigned long long));
    // prototype norms, roundup(N, 4) floats: the re-rank reads them as float4
    if (e == hipSuccess)
        e = hipMalloc(reinterpret_cast<void **>(&m->wnorm), (size_t)((N + 3) & ~3) * sizeof(float));
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&m->sums), 2 * sizeof(double));
    if (e == hipSuccess) e = hipEventCreateWithFlags(&m->order_done, hipEventDisableTiming);
    if (e == hipSuccess) e = som::launch_init_uniform(m->W, ld, m->N, d, seed, nullptr);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        som_destroy(m);
        return from_hip(e);
    }
    *out = m;
    return SOM_OK;
}

som_status som_destroy(som_map *m) {
    if (!m) return SOM_OK;
    if (m->stream) (void)hipStreamSynchronize(m->stream);
    else (void)hipDeviceSynchronize();
    (void)hipFree(m->W);
    (void)hipFree(m->state);
    (void)hipFree(m->slots);
    (void)hipFree(m->order_dev);
    if (m->order_host) (void)hipHostFree(m->order_host);
    if (m->order_done) (void)hipEventDestroy(m->order_done);
    (void)hipFree(m->sched);
    (void)hipFree(m->block_dots);
    (void)hipFree(m->xpad);
    (void)hipFree(m->bwork);
    (void)hipFree(m->sv);
    (void)hipFree(m->soff);
    (void)hipFree(m->sval);
    (void)hipFree(m->spv1);
    (void)hipFree(m->spv2);
    (void)hipFree(m->sst);
    (void)hipFree(m->wnorm);
    (void)hipFree(m->cand);
    (void)hipFree(m->part);
    (void)hipFree(m->idx1);
    (void)hipFree(m->idx2);
    (void)hipFree(m->d1);
    (void)hipFree(m->sums);
    delete m;
    return SOM_OK;
}

som_status som_set_topology(som_map *m, int32_t topology) {
    if (!m || (topology != SOM_RECT && topology != SOM_HEX)) return SOM_E_ARG;
    m->topology = topology;
    return SOM_OK;
}

som_status som_set_stream(som_map *m, void *stream) {
    if (!m) return SOM_E_ARG;
    m->stream = reinterpret_cast<hipStream_t>(stream);
    return SOM_OK;
}

som_status som_get_shape(const som_map *m, int32_t *rows, int32_t *cols, int32_t *d,
                         int32_t *topology) {
    if (!m) return SOM_E_ARG;
    if (rows) *rows = m->rows;
    if (cols) *cols = m->cols;
    if (d) *d = m->d;
    if (topology) *topology = m->topology;
    return SOM_OK;
}

static som::TrainArgs train_args(som_map *m, const float *X, int64_t n) {
    som::TrainArgs a{};
    a.W = m->W;
    a.ld = m->ld;
    a.N = m->N;
    a.d = m->d;
    a.rows = m->rows;
    a.cols = m->cols;
    a.topology = m->topology;
    a.X = X;
    a.n = n;
    a.slots = m->slots;
    a.state = m->state;
    a.xld = m->d;
    // Launch-shape overrides for tuning sweeps: workgroup count and variant
    // (1 = LDS-resident prototypes, 2 = streamed prototypes).
    const char *g = getenv("SOM_TRAIN_GRID");
    a.grid = (g && *g) ? atoi(g) : 0;
    if (a.grid < 0) a.grid = 0;
    if (a.grid > som::kMaxTrainGrid) a.grid = som::kMaxTrainGrid;
    // SOM_TRAIN_VARIANT: 1 LDS-resident, 2 streamed, 3 / 4 pipelined LDS /
    // streamed, 5 never pipelined.
    const char *v = getenv("SOM_TRAIN_VARIANT");
    a.variant = (v && *v) ? atoi(v) : 0;
    if (a.variant < 0 || a.variant > 5) a.variant = 0;
    // SOM_TRAIN_LDS_ROWS: rows per workgroup the pipelined streamed variant
    // keeps in LDS (at most what fits); unset = as many as fit.
    const char *lr = getenv("SOM_TRAIN_LDS_ROWS");
    a.lds_rows = (lr && *lr) ? atoi(lr) : -1;
    if (a.lds_rows < -1) a.lds_rows = -1;
    // SOM_TRAIN_BLOCK_M: steps per block (a pipelined shape the build has
    // for the row length, else the blocked kernel's instance of that length
    // if there is one, else the default choice).
    const char *bm = getenv("SOM_TRAIN_BLOCK_M");
    a.block_m = (bm && *bm) ? atoi(bm) : 0;
    if (a.block_m < 0) a.block_m = 0;
    // SOM_TRAIN_SWEEPERS: 3 or 4 sweeper waves in the pipelined kernel.
    const char *sw = getenv("SOM_TRAIN_SWEEPERS");
    a.sweepers = (sw && *sw) ? atoi(sw) : 0;
    if (a.sweepers != 3 && a.sweepers != 4) a.sweepers = 0;
    a.timeout_ticks = 100000000ull * 20;  // 20 s at the 100 MHz reference clock
    // SOM_DEBUG_EXCHANGE_TIMEOUT_US (failure-path tests): a shorter bound on
    // each exchange wait, in microseconds.
    const char *to = getenv("SOM_DEBUG_EXCHANGE_TIMEOUT_US");
    if (to && *to) {
        const long long us = atoll(to);
        if (us > 0 && us < 20000000) a.timeout_ticks = (uint64_t)us * 100;
    }
    return a;
}

// Principal components on the device; the vectors stay in *work (freed by
// the caller with hipFree).
static som_status pca_run(const float *X, int64_t n, int32_t d, hipStream_t stream,
                          double *lambda, float **work, float **mean) {
    *work = nullptr;
    *mean = nullptr;
    double *stats = nullptr;
    hipError_t e = hipMalloc(reinterpret_cast<void **>(work), som::pca_work_floats(d) * sizeof(float));
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(mean), (size_t)d * sizeof(float));
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&stats), 4 * sizeof(double));
    if (e == hipSuccess)
        e = som::pca_top2(X, n, d, *work, *mean, stats, kPcaMaxIters, kPcaTol, stream, lambda,
                          nullptr);
    (void)hipFree(stats);
    if (e != hipSuccess) {
        (void)hipFree(*work);
        (void)hipFree(*mean);
        *work = nullptr;
        *mean = nullptr;
        return from_hip(e);
    }
    return SOM_OK;
}

som_status som_pca2(const float *X, int64_t n, int32_t d, void *stream, double *lambda,
                    float *mean, float *v1, float *v2) {
    if (!X || !lambda || n <= 0 || d <= 0 || n > INT32_MAX) return SOM_E_ARG;
    if (!device_range_ok(X, (uint64_t)n * (uint64_t)d * sizeof(float))) return SOM_E_ARG;
    for (float *p : {mean, v1, v2})
        if (p && !device_range_ok(p, (uint64_t)d * sizeof(float))) return SOM_E_ARG;
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    float *work = nullptr, *mu = nullptr;
    som_status st = pca_run(X, n, d, s, lambda, &work, &mu);
    if (st != SOM_OK) return st;
    const float *V = som::pca_vectors(work, d);
    hipError_t e = hipSuccess;
    if (mean) e = hipMemcpyAsync(mean, mu, (size_t)d * 4, hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess && v1) e = hipMemcpyAsync(v1, V, (size_t)d * 4, hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess && v2)
        e = hipMemcpyAsync(v2, V + d, (size_t)d * 4, hipMemcpyDeviceToDevice, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    (void)hipFree(work);
    (void)hipFree(mu);
    return from_hip(e);
}

som_status som_suggest_size(int64_t m, double lambda1, double lambda2, int32_t *rows,
                            int32_t *cols, int64_t *iterations) {
    if (m <= 0 || !(lambda1 >= 0.0) || !(lambda2 >= 0.0) || lambda2 > lambda1 ||
        !isfinite(lambda1))
        return SOM_E_ARG;
    // Fig. 2: munits units, side ratio from the two largest variances.
    const double munits = ceil(5.0 * sqrt((double)m));
    if (munits > (double)INT32_MAX) return SOM_E_ARG;
    const double r = (lambda1 == 0.0 || lambda2 * munits < lambda1) ? 1.0 : sqrt(lambda1 / lambda2);
    double size1 = floor(sqrt(munits / (r * sqrt(0.75))) + 0.5);
    if (size1 < 1.0) size1 = 1.0;
    if (size1 > munits) size1 = munits;
    const double size2 = ceil(munits / size1);
    const double nr = size1 < size2 ? size1 : size2, nc = size1 < size2 ? size2 : size1;
    const double iters = ceil(50.0 * nr * nc / (double)m) * (double)m * 4.0;
    if (iters > 9.2e18) return SOM_E_ARG;
    if (rows) *rows = (int32_t)nr;
    if (cols) *cols = (int32_t)nc;
    if (iterations) *iterations = (int64_t)iters;
    return SOM_OK;
}

som_status som_init_linear(som_map *m, const float *X, int64_t n) {
    if (!m || !X || n <= 0 || n > INT32_MAX) return SOM_E_ARG;
    if (!device_range_ok(X, (uint64_t)n * (uint64_t)m->d * sizeof(float))) return SOM_E_ARG;
    double lambda[2];
    float *work = nullptr, *mu = nullptr;
    som_status st = pca_run(X, n, m->d, m->stream, lambda, &work, &mu);
    if (st != SOM_OK) return st;
    const float *V = som::pca_vectors(work, m->d);
    hipError_t e = som::launch_linear_init(m->W, m->ld, m->rows, m->cols, m->d, mu, V, V + m->d,
                                           lambda[0], lambda[1], m->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(m->stream);
    (void)hipFree(work);
    (void)hipFree(mu);
    if (e != hipSuccess) return from_hip(e);
    return check_deferred(m);
}

som_status som_train_plan(const som_map *m, int32_t *grid, int32_t *block,
                          int32_t *variant, int32_t *block_steps) {
    if (!m) return SOM_E_ARG;
    som::TrainArgs a = train_args(const_cast<som_map *>(m), nullptr, 1);
    som::TrainPlan p;
    hipError_t e = som::plan_train(a, m->num_cus, &p);
    if (e == hipErrorInvalidValue) return SOM_E_UNSUPPORTED;
    if (e != hipSuccess) return from_hip(e);
    if (grid) *grid = p.grid;
    if (block) *block = p.block;
    if (variant) *variant = p.variant;
    if (block_steps) *block_steps = p.block_m;
    return SOM_OK;
}

// The per-step inputs of a training call: the sample order (the library's
// shuffle when the schedule gives none, staged through pinned memory) and
// the schedule table; fills a's order, step and schedule fields.
static hipError_t stage_steps(som_map *m, const som_schedule *s, int64_t n, int64_t nsteps,
                              int64_t total, som::TrainArgs &a) {
    hipError_t e;
    const int32_t *order = s->order;
    if (!order) {
        // Library order: epoch e = t / n presents permutation e of [0, n).
        if (m->order_cap < nsteps) {
            e = hipStreamSynchronize(m->stream);
            if (e == hipSuccess && m->order_dev) e = hipFree(m->order_dev);
            m->order_dev = nullptr;
            if (e == hipSuccess && m->order_host) e = hipHostFree(m->order_host);
            m->order_host = nullptr;
            m->order_cap = 0;
            if (e == hipSuccess)
                e = hipMalloc(reinterpret_cast<void **>(&m->order_dev), (size_t)nsteps * 4);
            if (e == hipSuccess)
                e = hipHostMalloc(reinterpret_cast<void **>(&m->order_host), (size_t)nsteps * 4,
                                  hipHostMallocDefault);
            if (e != hipSuccess) return e;
            m->order_cap = nsteps;
        }
        e = hipEventSynchronize(m->order_done);  // previous upload has left the buffer
        if (e != hipSuccess) return e;
        std::vector<int32_t> perm((size_t)n);
        int64_t cur_epoch = -1;
        for (int64_t k = 0; k < nsteps; ++k) {
            const int64_t t = s->step0 + k;
            const int64_t ep = t / n;
            if (ep != cur_epoch) {
                fisher_yates(s->shuffle_seed, ep, n, perm.data());
                cur_epoch = ep;
            }
            m->order_host[k] = perm[(size_t)(t % n)];
        }
        e = hipMemcpyAsync(m->order_dev, m->order_host, (size_t)nsteps * 4,
                           hipMemcpyHostToDevice, m->stream);
        if (e == hipSuccess) e = hipEventRecord(m->order_done, m->stream);
        if (e != hipSuccess) return e;
        order = m->order_dev;
    }

    a.order = order;
    a.nsteps = nsteps;
    a.step0 = s->step0;
    a.total_steps = total;
    a.lr0 = s->lr0;
    a.lr1 = s->lr1;
    a.sigma0 = s->sigma0;
    a.sigma1 = s->sigma1;
    a.lr_decay = s->lr_decay;
    a.sigma_decay = s->sigma_decay;
    a.bmu_trace = s->bmu_trace;
    if (m->sched_cap < nsteps) {
        e = hipStreamSynchronize(m->stream);
        if (e == hipSuccess && m->sched) e = hipFree(m->sched);
        m->sched = nullptr;
        m->sched_cap = 0;
        if (e == hipSuccess)
            e = hipMalloc(reinterpret_cast<void **>(&m->sched), (size_t)nsteps * sizeof(float2));
        if (e != hipSuccess) return e;
        m->sched_cap = nsteps;
    }
    a.sched = m->sched;
    return hipSuccess;
}

// Checks shared by the training calls: step counts, schedule, order and
// trace extents.  Sets the call's step count and schedule length.
static bool train_call_ok(const som_schedule *s, int64_t n, int32_t epochs, int64_t *nsteps,
                          int64_t *total) {
    if (!s || n <= 0 || epochs <= 0) return false;
    if (n > INT32_MAX || (int64_t)epochs * n > INT32_MAX) return false;
    if (!schedule_ok(s)) return false;
    *nsteps = (int64_t)epochs * n;
    if (s->step0 < 0) return false;
    *total = s->total_steps == 0 ? s->step0 + *nsteps : s->total_steps;
    if (*total < s->step0 + *nsteps) return false;
    if (s->order && !device_range_ok(s->order, (uint64_t)*nsteps * sizeof(int32_t)))
        return false;
    if (s->bmu_trace && !device_range_ok(s->bmu_trace, (uint64_t)*nsteps * sizeof(int32_t)))
        return false;
    return true;
}

som_status som_train(som_map *m, const float *X, int64_t n, int32_t epochs,
                     const som_schedule *s) {
    int64_t nsteps = 0, total = 0;
    if (!m || !X || !train_call_ok(s, n, epochs, &nsteps, &total)) return SOM_E_ARG;
    if (!device_range_ok(X, (uint64_t)n * (uint64_t)m->d * sizeof(float))) return SOM_E_ARG;

    som::TrainArgs a = train_args(m, X, n);
    som::TrainPlan plan;
    hipError_t e = som::plan_train(a, m->num_cus, &plan);
    if (e == hipErrorInvalidValue) return SOM_E_UNSUPPORTED;
    if (e != hipSuccess) return from_hip(e);

    e = stage_steps(m, s, n, nsteps, total, a);
    if (e != hipSuccess) return from_hip(e);
    if (plan.variant >= 2) {
        const int64_t need = som::pipe_block_dots_floats(plan.block_m, nsteps);
        if (m->block_dots_cap < need) {
            e = hipStreamSynchronize(m->stream);
            if (e == hipSuccess && m->block_dots) e = hipFree(m->block_dots);
            m->block_dots = nullptr;
            m->block_dots_cap = 0;
            if (e == hipSuccess)
                e = hipMalloc(reinterpret_cast<void **>(&m->block_dots), (size_t)need * sizeof(float));
            if (e != hipSuccess) return from_hip(e);
            m->block_dots_cap = need;
        }
        a.block_dots = m->block_dots;
    }
    // The training kernels read sample rows as aligned float4; the long-row
    // kernel reads them as long as the prototypes' rows (zero past d).
    const bool full_rows = plan.cols_rmax > 0 && m->ld != (int64_t)m->d;
    if (m->d % 4 != 0 || reinterpret_cast<uintptr_t>(X) % 16 != 0 || full_rows) {
        const int64_t xld = full_rows ? m->ld : ((int64_t)m->d + 3) & ~(int64_t)3;
        if (m->xpad_cap < n * xld) {
            e = hipStreamSynchronize(m->stream);
            if (e == hipSuccess && m->xpad) e = hipFree(m->xpad);
            m->xpad = nullptr;
            m->xpad_cap = 0;
            if (e == hipSuccess)
                e = hipMalloc(reinterpret_cast<void **>(&m->xpad), (size_t)(n * xld) * sizeof(float));
            if (e != hipSuccess) return from_hip(e);
            m->xpad_cap = n * xld;
        }
        e = som::launch_pad_rows(X, n, m->d, m->xpad, xld, m->stream);
        if (e != hipSuccess) return from_hip(e);
        a.X = m->xpad;
        a.xld = xld;
    }
    a.grid = plan.grid;
    a.slot_spread = plan.slot_spread;
    // SOM_DEBUG_ABSENT_WORKGROUP=1 (failure-path tests): launch one workgroup
    // fewer than the exchanges wait for, so that every exchange wait of the
    // call runs into its time bound and the kernel ends with SOM_E_TIMEOUT.
    const char *ab = getenv("SOM_DEBUG_ABSENT_WORKGROUP");
    if (ab && ab[0] == '1' && ab[1] == '\0' && plan.grid > 1) plan.absent = 1;
    e = som::launch_prepare_train(a, m->sched, m->stream);
    if (e == hipSuccess) e = som::launch_scan_finite(X, n * m->d, m->state, m->stream);
    if (e == hipSuccess) e = som::launch_train(a, plan, m->stream);
    return from_hip(e);
}

som_status som_train_csr(som_map *m, const int64_t *indptr, const int32_t *indices,
                         const float *values, int64_t n, int32_t epochs, const som_schedule *s) {
    int64_t nsteps = 0, total = 0;
    if (!m || !indptr || !train_call_ok(s, n, epochs, &nsteps, &total)) return SOM_E_ARG;
    if (!device_range_ok(indptr, (uint64_t)(n + 1) * sizeof(int64_t))) return SOM_E_ARG;
    const int64_t ldv = ((int64_t)m->N + 63) & ~(int64_t)63;
    if (ldv / 64 > som::kSparseMaxGrid) return SOM_E_UNSUPPORTED;

    // The CSR structure: indptr[0] = 0, nnz = indptr[n], then every row on
    // the device (lengths, sorted unique indices in [0, d), longest row).
    int64_t ends[2] = {-1, -1};
    hipError_t e = hipMemcpyAsync(&ends[0], indptr, sizeof(int64_t), hipMemcpyDeviceToHost, m->stream);
    if (e == hipSuccess)
        e = hipMemcpyAsync(&ends[1], indptr + n, sizeof(int64_t), hipMemcpyDeviceToHost,
                           m->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(m->stream);
    if (e != hipSuccess) return from_hip(e);
    if (ends[0] != 0 || ends[1] < 0) return SOM_E_ARG;
    const int64_t nnz = ends[1];
    if (nnz > 0 && (!device_range_ok(indices, (uint64_t)nnz * sizeof(int32_t)) ||
                    !device_range_ok(values, (uint64_t)nnz * sizeof(float))))
        return SOM_E_ARG;
    e = som::launch_csr_check(indptr, indices, n, nnz, m->d, m->state, m->stream);
    som::DevState st{};
    if (e == hipSuccess)
        e = hipMemcpyAsync(&st, m->state, sizeof(st), hipMemcpyDeviceToHost, m->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(m->stream);
    if (e != hipSuccess) return from_hip(e);
    if (st.csr_bad) return SOM_E_ARG;
    if (st.csr_max_len > som::kSparseMaxNnz) return SOM_E_UNSUPPORTED;
    const int K = st.csr_max_len <= 16 ? 16 : st.csr_max_len <= 32 ? 32 : 64;

    som::TrainArgs a = train_args(m, nullptr, n);
    a.grid = (int32_t)(ldv / 64);
    a.slot_spread = a.grid <= 64 ? 16 : 4;
    // rows of V are addressed through one buffer resource of 2^31 - 1 bytes
    if (((uint64_t)m->d + 1) * (uint64_t)ldv * sizeof(double) > INT32_MAX)
        return SOM_E_UNSUPPORTED;
    const uint64_t vbytes = ((uint64_t)m->d + 3) * (uint64_t)ldv * sizeof(double);
    const uint64_t ebytes = ((uint64_t)nsteps + 1) * ((uint64_t)K * 28 + sizeof(som::SparseStep));
    if (vbytes + ebytes > max_bytes()) return SOM_E_OOM;
    e = stage_steps(m, s, n, nsteps, total, a);
    if (e == hipSuccess) e = ensure(m, &m->sv, &m->sv_cap, ((int64_t)m->d + 3) * ldv);
    // the call's steps and one padding step
    const int64_t nent = (nsteps + 1) * K;
    if (e == hipSuccess) e = ensure(m, &m->soff, &m->soff_cap, nent);
    if (e == hipSuccess) e = ensure(m, &m->sval, &m->sval_cap, nent);
    if (e == hipSuccess) e = ensure(m, &m->spv1, &m->spv1_cap, nent);
    if (e == hipSuccess) e = ensure(m, &m->spv2, &m->spv2_cap, nent);
    if (e == hipSuccess) e = ensure(m, &m->sst, &m->sst_cap, nsteps + 1);
    if (e != hipSuccess) return from_hip(e);

    som::SparseArgs sp{};
    sp.V = m->sv;
    sp.ldv = ldv;
    sp.S = m->sv + ((int64_t)m->d + 1) * ldv;
    sp.WW = sp.S + ldv;
    sp.K = K;
    sp.soff = m->soff;
    sp.sval = m->sval;
    sp.spv1 = m->spv1;
    sp.spv2 = m->spv2;
    sp.sst = m->sst;
    e = som::launch_prepare_train(a, m->sched, m->stream);
    if (e == hipSuccess && nnz > 0) e = som::launch_scan_finite(values, nnz, m->state, m->stream);
    if (e == hipSuccess) e = som::launch_sparse_steps(a, sp, indptr, indices, values, m->stream);
    if (e == hipSuccess) e = som::launch_sparse_enter(a, sp, m->stream);
    if (e == hipSuccess) e = som::launch_train_sparse(a, sp, m->stream);
    if (e == hipSuccess) e = som::launch_sparse_leave(a, sp, m->stream);
    return from_hip(e);
}

som_status som_train_batch(som_map *m, const float *X, int64_t n, int32_t epochs,
                           double sigma0, double sigma1, int32_t sigma_decay) {
    if (!m || !X || n <= 0 || n > INT32_MAX || epochs <= 0) return SOM_E_ARG;
    som_schedule s{};
    s.lr0 = s.lr1 = 1.0;
    s.lr_decay = SOM_DECAY_LINEAR;
    s.sigma0 = sigma0;
    s.sigma1 = sigma1;
    s.sigma_decay = sigma_decay;
    if (!schedule_ok(&s)) return SOM_E_ARG;
    if (!device_range_ok(X, (uint64_t)n * (uint64_t)m->d * sizeof(float))) return SOM_E_ARG;
    const size_t work = som::batch_work_doubles(m->rows, m->cols, m->d, m->topology);
    if (((uint64_t)m->d + 1 + 63) / 64 > 65535) return SOM_E_UNSUPPORTED;
    if ((uint64_t)work * sizeof(double) > max_bytes()) return SOM_E_OOM;
    hipError_t e = ensure(m, &m->bwork, &m->bwork_cap, (int64_t)work);
    if (e != hipSuccess) return from_hip(e);
    som_status st = ensure_eval_scratch(m, n, 0);
    if (st != SOM_OK) return st;
    for (int32_t ep = 0; ep < epochs; ++ep) {
        // the radius at p = ep / (epochs - 1), endpoints exact
        const double p = epochs > 1 ? (double)ep / (double)(epochs - 1) : 0.0;
        double sigma = sigma0;
        if (sigma0 != sigma1) {
            if (p == 1.0)
                sigma = sigma1;
            else if (p != 0.0)
                sigma = sigma_decay == SOM_DECAY_LINEAR
                            ? (1.0 - p) * sigma0 + p * sigma1
                            : pow(sigma0, 1.0 - p) * pow(sigma1, p);
        }
        st = run_eval(m, X, n, m->idx1, nullptr, nullptr);
        if (st != SOM_OK) return st;
        som::BatchArgs b{};
        b.bmu = m->idx1;
        b.X = X;
        b.n = n;
        b.d = m->d;
        b.rows = m->rows;
        b.cols = m->cols;
        b.topology = m->topology;
        b.sigma = sigma;
        b.work = m->bwork;
        b.W = m->W;
        b.ld = m->ld;
        e = som::launch_batch_epoch(b, m->stream);
        if (e != hipSuccess) return from_hip(e);
    }
    return SOM_OK;
}

som_status som_bmu2(som_map *m, const float *X, int64_t n, int32_t *out_idx,
                    int32_t *out_idx2, float *out_d1) {
    if (!eval_args_ok(m, X, n)) return SOM_E_ARG;
    if (out_idx && !device_range_ok(out_idx, (uint64_t)n * 4)) return SOM_E_ARG;
    if (out_idx2 && !device_range_ok(out_idx2, (uint64_t)n * 4)) return SOM_E_ARG;
    if (out_d1 && !device_range_ok(out_d1, (uint64_t)n * 4)) return SOM_E_ARG;
    som_status st = ensure_eval_scratch(m, n, 0);
    if (st != SOM_OK) return st;
    return run_eval(m, X, n, out_idx ? out_idx : m->idx1, out_idx2, out_d1);
}

som_status som_bmu2_noalloc(som_map *m, const float *X, int64_t n, int32_t *out_idx,
                            int32_t *out_idx2, float *out_d1) {
    if (!eval_args_ok(m, X, n)) return SOM_E_ARG;
    if (out_idx && !device_range_ok(out_idx, (uint64_t)n * 4)) return SOM_E_ARG;
    if (out_idx2 && !device_range_ok(out_idx2, (uint64_t)n * 4)) return SOM_E_ARG;
    if (out_d1 && !device_range_ok(out_d1, (uint64_t)n * 4)) return SOM_E_ARG;
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return from_hip(e);
    if (dev != m->device) return SOM_E_ARG;
    som::EvalArgs a{};
    a.W = m->W;
    a.ld = m->ld;
    a.N = m->N;
    a.d = m->d;
    a.rows = m->rows;
    a.cols = m->cols;
    a.topology = m->topology;
    a.X = X;
    a.n = n;
    // scratch layout: prototype norms | BMUs when out_idx is NULL | candidate
    // lists | partial products, each rounded up to 256 bytes; the search
    // takes the best shape that fits what the first two leave
    const auto round256 = [](uint64_t b) { return (b + 255) / 256 * 256; };
    const uint64_t norm_bytes = round256((uint64_t)m->N * 4);
    const uint64_t idx_bytes = out_idx ? 0 : round256((uint64_t)n * 4);
    if (norm_bytes + idx_bytes + 512 > som::kNoAllocScratchBytes) return SOM_E_UNSUPPORTED;
    if (!som::plan_bmu_candidates(&a, m->num_cus,
                                  som::kNoAllocScratchBytes - norm_bytes - idx_bytes - 512))
        return SOM_E_UNSUPPORTED;
    const uint64_t cand_bytes = round256((uint64_t)som::bmu_cand_ints(a) * 4);
    const uint64_t part_bytes = round256((uint64_t)som::bmu_part_floats(a) * 4);
    if (norm_bytes + idx_bytes + cand_bytes + part_bytes > som::kNoAllocScratchBytes)
        return SOM_E_UNSUPPORTED;
    void *base = nullptr;
    e = som::noalloc_scratch(&base);
    if (e != hipSuccess) return from_hip(e);
    unsigned char *p = static_cast<unsigned char *>(base);
    float *wnorm = reinterpret_cast<float *>(p);
    a.wnorm = wnorm;
    a.cand = reinterpret_cast<int32_t *>(p + norm_bytes + idx_bytes);
    a.part = part_bytes ? reinterpret_cast<float *>(p + norm_bytes + idx_bytes + cand_bytes)
                        : nullptr;
    a.idx1 = out_idx ? out_idx : reinterpret_cast<int32_t *>(p + norm_bytes);
    a.idx2 = out_idx2;
    a.d1 = out_d1;
    a.x_vec4 = (m->d % 4 == 0) && (reinterpret_cast<uintptr_t>(X) % 16 == 0);
    e = som::launch_row_sqnorm(m->W, m->ld, m->N, wnorm, m->stream);
    if (e == hipSuccess) e = som::launch_bmu_candidates(a, m->stream);
    if (e == hipSuccess) e = som::launch_bmu_rerank(a, m->stream);
    return from_hip(e);
}

som_status som_bmu(som_map *m, const float *X, int64_t n, int32_t *out_idx) {
    if (!out_idx) return SOM_E_ARG;
    return som_bmu2(m, X, n, out_idx, nullptr, nullptr);
}

static som_status qe_te(som_map *m, const float *X, int64_t n, int32_t *out_idx, double *qe,
                        double *te) {
    if (!eval_args_ok(m, X, n)) return SOM_E_ARG;
    if (out_idx && !device_range_ok(out_idx, (uint64_t)n * 4)) return SOM_E_ARG;
    som_status st = ensure_eval_scratch(m, n, 0);
    if (st != SOM_OK) return st;
    st = run_eval(m, X, n, out_idx ? out_idx : m->idx1, m->idx2, m->d1);
    if (st != SOM_OK) return st;
    hipError_t e = som::launch_qe_te_reduce(out_idx ? out_idx : m->idx1, m->idx2, m->d1, n,
                                            m->cols, m->topology, m->sums, m->stream);
    double h[2] = {0.0, 0.0};
    if (e == hipSuccess)
        e = hipMemcpyAsync(h, m->sums, sizeof(h), hipMemcpyDeviceToHost, m->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(m->stream);
    if (e != hipSuccess) return from_hip(e);
    st = check_deferred(m);
    if (st != SOM_OK) return st;
    if (qe) *qe = h[0] / (double)n;
    if (te) *te = h[1] / (double)n;
    return SOM_OK;
}

som_status som_quantization_error(som_map *m, const float *X, int64_t n, double *out_qe) {
    if (!out_qe) return SOM_E_ARG;
    return qe_te(m, X, n, nullptr, out_qe, nullptr);
}

som_status som_topographic_error(som_map *m, const float *X, int64_t n, double *out_te) {
    if (!out_te) return SOM_E_ARG;
    return qe_te(m, X, n, nullptr, nullptr, out_te);
}

som_status som_evaluate(som_map *m, const float *X, int64_t n, int32_t *out_idx,
                        double *out_qe, double *out_te) {
    if (!out_qe && !out_te && !out_idx) return SOM_E_ARG;
    return qe_te(m, X, n, out_idx, out_qe, out_te);
}

som_status som_stream_inplace(void *buf, int64_t bytes, int32_t passes, int32_t grid,
                              void *stream) {
    if (!buf || bytes <= 0 || bytes % 16 != 0 || passes <= 0 || grid <= 0 ||
        grid > som::kMaxTrainGrid)
        return SOM_E_ARG;
    if (reinterpret_cast<uintptr_t>(buf) % 16 != 0) return SOM_E_ARG;
    if (!device_range_ok(buf, (uint64_t)bytes)) return SOM_E_ARG;
    return from_hip(som::launch_stream_inplace(static_cast<float *>(buf), bytes, passes, grid,
                                               1.0f, reinterpret_cast<hipStream_t>(stream)));
}

som_status som_get_weights(som_map *m, float *dst) {
    if (!m || !dst) return SOM_E_ARG;
    hipError_t e = hipMemcpy2DAsync(dst, (size_t)m->d * 4, m->W, (size_t)m->ld * 4,
                                    (size_t)m->d * 4, (size_t)m->N, hipMemcpyDefault,
                                    m->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(m->stream);
    if (e != hipSuccess) return from_hip(e);
    return check_deferred(m);
}

som_status som_set_weights(som_map *m, const float *src) {
    if (!m || !src) return SOM_E_ARG;
    hipError_t e = hipMemcpy2DAsync(m->W, (size_t)m->ld * 4, src, (size_t)m->d * 4,
                                    (size_t)m->d * 4, (size_t)m->N, hipMemcpyDefault,
                                    m->stream);
    if (e == hipSuccess) e = hipStreamSynchronize(m->stream);
    if (e != hipSuccess) return from_hip(e);
    return check_deferred(m);
}

som_status som_synchronize(som_map *m) {
    if (!m) return SOM_E_ARG;
    hipError_t e = hipStreamSynchronize(m->stream);
    if (e != hipSuccess) return from_hip(e);
    return check_deferred(m);
}

}  // extern "C"
