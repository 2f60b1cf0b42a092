// Internal declarations shared by the host runtime (som_api.cpp) and the
// kernel translation units.  Not part of the public ABI (include/som.h).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace som {

// Threads per workgroup of the persistent training kernel.
constexpr int kTrainBlock = 256;
// Grid-exchange slot layout: 64-bit key = dist_bits << 32 | tag << 24 | unit.
constexpr int kUnitBits = 24;
constexpr int32_t kMaxUnits = (1 << kUnitBits) - 1;
// Each workgroup writes its key into kSlotReplicas copies of the slot array
// and polls the copy of its XCD (workgroup b runs on XCD b % 8), so each
// copy is read by one eighth of the grid; slots sit `slot_spread` u64 apart.
constexpr int kSlotReplicas = 8;
constexpr int kMaxTrainGrid = 1024;
constexpr int kMaxSlotSpread = 16;
constexpr int64_t kSlotReplicaStride = 2LL * kMaxTrainGrid * kMaxSlotSpread;  // u64
constexpr int64_t kSlotWords = kSlotReplicas * kSlotReplicaStride;

// Device-side status words of a map (one allocation, zeroed at creation).
struct DevState {
    int32_t status;     // sticky error code (som_status), cleared by the host
    int32_t order_bad;  // 1 if the current call's inputs are unusable: an order index
                        // outside [0, n), or a NaN or infinity in its samples
    int32_t csr_bad;    // 1 if the current call's CSR rows are malformed
    int32_t csr_max_len;  // longest CSR row of the current call
};

struct TrainArgs {
    float *W;               // N x ld, row-major, ld % 4 == 0, zero padding
    int64_t ld;             // row pitch in floats
    int32_t N, d, rows, cols, topology;
    const float *X;         // n x xld, row-major, 16-byte aligned, zero past d
    int64_t xld;            // row pitch of X in floats, a multiple of 4
    int64_t n;
    const int32_t *order;   // nsteps sample indices
    int64_t nsteps, step0, total_steps;
    double lr0, lr1, sigma0, sigma1;
    int32_t lr_decay, sigma_decay;
    const float2 *sched;    // nsteps (lr, log2(e) / (2 sigma^2)) of the call's steps
    float *block_dots;      // pipelined variant: per-block sample products
    int32_t *bmu_trace;     // nullable, nsteps entries
    unsigned long long *slots;  // kSlotWords exchange words
    int32_t slot_spread;        // u64 between consecutive workgroups' slots
    DevState *state;
    int32_t grid;           // requested workgroups (0 = planner's choice)
    int32_t variant;        // requested variant: 0 any, 1 LDS-resident, 2 streamed
    int32_t lds_rows;       // pipelined streamed variant: leading rows of each
                            // workgroup kept in LDS (-1 = planner's choice)
    int32_t block_m;        // pipelined kernel: requested block length (0 = any)
    int32_t sweepers;       // pipelined kernel: requested sweeper waves (0 = any, 3, 4)
    uint64_t timeout_ticks; // bound of one exchange wait, in 100 MHz ticks
};

struct TrainPlan {
    int32_t grid = 0;
    int32_t block = kTrainBlock;
    int32_t variant = 0;     // 0 streamed, 1 LDS-resident, 2 / 3 pipelined streamed / LDS,
                             // 4 pipelined streamed for long rows (column-walk sweep)
    int32_t block_m = 0;     // steps per block of the chosen kernel instance
    int32_t kslots = 0;      // float4 columns per lane (template instance)
    int32_t lds_rows = 0;    // pipelined streamed variant: rows per workgroup in LDS
    int32_t cols_rmax = 0;   // pipelined streamed variant for long rows (column-walk
                             // sweep): its row bound per workgroup, 0 otherwise
    int32_t slot_spread = 1;
    size_t lds_bytes = 0;
    int32_t absent = 0;      // workgroups left out of the launch (the failure-path
                             // tests' host-forced exchange timeout); 0 otherwise
};

// Squared lattice distance between units u and c of a map with `cols`
// columns.  RECT: unit r * cols + c sits at (r, c).  HEX: odd rows are
// shifted by half a unit and rows are sqrt(3)/2 apart.  No wrap-around.
__device__ inline double lattice_sq(int u, int c, int cols, int topology) {
    const int ru = u / cols, cu = u - ru * cols;
    const int rc = c / cols, cc = c - rc * cols;
    if (topology == 1) {
        const double pitch = 0.86602540378443864676;  // sqrt(3) / 2
        const double xu = cu + ((ru & 1) ? 0.5 : 0.0), xc = cc + ((rc & 1) ? 0.5 : 0.0);
        const double yu = ru * pitch, yc = rc * pitch;
        return (yu - yc) * (yu - yc) + (xu - xc) * (xu - xc);
    }
    const double dr = ru - rc, dc = cu - cc;
    return dr * dr + dc * dc;
}

// Row pitch (floats) of a d-dimensional map: d rounded up to the training
// kernel's lane slots (16-byte columns times lanes per row), so the sweep
// needs no column bounds; 0 when no training kernel covers d.
int64_t train_row_pitch(int32_t d);

// Pipelined training (som_train_pipe.hip): estimated microseconds per step
// of its best shape (1e300 if none fits), written into *plan.
double plan_train_pipe(const TrainArgs &a, int num_cus, int max_lds, TrainPlan *plan);
int64_t pipe_block_dots_floats(int m, int64_t nsteps);
hipError_t launch_train_pipe(const TrainArgs &a, const TrainPlan &plan, hipStream_t s);

// Host-side launchers (each translation unit owns its kernels).
hipError_t plan_train(const TrainArgs &a, int num_cus, TrainPlan *plan);
hipError_t launch_train(const TrainArgs &a, const TrainPlan &plan, hipStream_t s);

hipError_t launch_init_uniform(float *W, int64_t ld, int32_t N, int32_t d,
                               uint64_t seed, hipStream_t s);
// Before every training launch (a.grid and a.slot_spread set): zero the
// exchange slots in use and the order flag, then range-check the order
// (raising order_bad and the sticky status) and fill the per-step schedule
// table from the fp64 decay laws.
hipError_t launch_prepare_train(const TrainArgs &a, float2 *sched, hipStream_t s);
// After launch_prepare_train: flag (order_bad, status SOM_E_NONFINITE) a NaN
// or infinity among the `count` floats at x.
hipError_t launch_scan_finite(const float *x, int64_t count, DevState *state,
                              hipStream_t s);
// out[u] = |W[u]|^2 for the N rows of W.
hipError_t launch_row_sqnorm(const float *W, int64_t ld, int32_t N, float *out,
                             hipStream_t s);
// Copy the n x d rows of X into out, rows of xld floats (xld >= d, a
// multiple of 4), zero past d.
hipError_t launch_pad_rows(const float *X, int64_t n, int32_t d, float *out, int64_t xld,
                           hipStream_t s);

struct EvalArgs {
    const float *W;
    int64_t ld;
    int32_t N, d, rows, cols, topology;
    const float *X;
    int64_t n;
    const float *wnorm;     // N squared prototype norms (roundup(N, 4) floats allocated)
    int32_t *cand;          // n x ugroups x kCand (score bits, unit) pairs (scratch)
    int32_t ugroups;        // unit groups whose lists are kept apart
    int32_t group_units;    // units per group (a multiple of the unit tile)
    int32_t splits;         // ranges of d computed by separate workgroups (1: fused)
    int32_t split_len;      // columns per range (a multiple of the slice width)
    int32_t tiles_s, tiles_u;  // sample and unit tiles
    float *part;            // splits > 1: splits x n x (tiles_u x 128) partial products
    int32_t *idx1;          // n (required)
    int32_t *idx2;          // n (nullable)
    float *d1;              // n (nullable)
    int32_t x_vec4;
};
constexpr int kCand = 4;

// The candidate search's shape for n samples over N units on `num_cus`
// compute units (sets ugroups, group_units, splits, split_len, tiles_s,
// tiles_u): the fewest rounds of workgroups, among the shapes whose
// candidate lists and partial products fit in max_scratch_bytes.  False
// when none does.
bool plan_bmu_candidates(EvalArgs *a, int num_cus, uint64_t max_scratch_bytes);
// Scratch of a planned search: int32 entries of the candidate lists and
// floats of the partial products (0 for the fused form).
int64_t bmu_cand_ints(const EvalArgs &a);
int64_t bmu_part_floats(const EvalArgs &a);
hipError_t launch_bmu_candidates(const EvalArgs &a, hipStream_t s);
// Fixed per-device scratch of som_bmu2_noalloc (som_eval.hip): its device
// address on the current device, looked up once per device.
constexpr size_t kNoAllocScratchBytes = 8u << 20;
hipError_t noalloc_scratch(void **ptr);
hipError_t launch_bmu_rerank(const EvalArgs &a, hipStream_t s);
// QE and TE sums over n samples from (idx1, idx2, d1); writes 2 doubles.
hipError_t launch_qe_te_reduce(const int32_t *idx1, const int32_t *idx2,
                               const float *d1, int64_t n, int32_t cols,
                               int32_t topology, double *out2, hipStream_t s);

// Sparse-input training (som_sparse.hip).  Prototypes are held as
// w_u = S_u v_u with v stored feature-major in fp64, V[j * ldv + u], so a
// step touches only the rows of V at the sample's non-zero features.  Row d
// of V is a scratch row that the padding entries of a step point to.
constexpr int kSparseMaxNnz = 64;      // non-zeros per sample row
constexpr int kSparseMaxGrid = 256;    // workgroups of 64 units
struct SparseStep {
    double xx;       // |x_s|^2
    double xd1;      // x_{s-1} . x_s (0 for the call's first step)
    double xd2;      // x_{s-2} . x_s (0 for its first two steps)
    uint64_t both;   // bit q: entry q is a feature of x_{s-1} or x_{s-2}
    float lr, c2;    // the step's schedule entry (lr, log2(e) / (2 sigma^2))
};
constexpr int kSparseStepWords = (int)(sizeof(SparseStep) / 4);
struct SparseArgs {
    double *V;            // (d + 1) x ldv
    int64_t ldv;          // units rounded up to a multiple of 64
    double *S;            // ldv scales
    double *WW;           // ldv squared prototype norms |w_u|^2
    int32_t K;            // entries per step: 16, 32 or 64
    uint32_t *soff;       // nsteps x K: byte offset of the entry's row of V
    double *sval;         // nsteps x K values (0 for padding)
    double *spv1;         // nsteps x K: x_{s-1} at the entry's feature
    double *spv2;         // nsteps x K: x_{s-2} at the entry's feature
    SparseStep *sst;      // nsteps
};
// Per CSR row: lengths, sorted unique indices in [0, d); raises csr_bad and
// records the longest row in csr_max_len (both zeroed first).
hipError_t launch_csr_check(const int64_t *indptr, const int32_t *indices, int64_t n,
                            int64_t nnz, int32_t d, DevState *state, hipStream_t s);
// Per-step entries of the call's steps from the CSR rows and the order.
hipError_t launch_sparse_steps(const TrainArgs &a, const SparseArgs &sp, const int64_t *indptr,
                               const int32_t *indices, const float *values, hipStream_t s);
// W (N x ld fp32) into V, S = 1, WW = |w|^2, and back: W = S v.
hipError_t launch_sparse_enter(const TrainArgs &a, const SparseArgs &sp, hipStream_t s);
hipError_t launch_sparse_leave(const TrainArgs &a, const SparseArgs &sp, hipStream_t s);
hipError_t launch_train_sparse(const TrainArgs &a, const SparseArgs &sp, hipStream_t s);

// Batch-map training (som_batch.hip): one epoch after the BMUs are known.
struct BatchArgs {
    const int32_t *bmu;     // n BMU indices
    const float *X;         // n x d, row-major
    int64_t n;
    int32_t d, rows, cols, topology;
    double sigma;           // the epoch's radius
    double *work;           // batch_work_doubles(rows, cols, d, topology)
    float *W;               // N x ld prototypes, updated in place
    int64_t ld;
};
size_t batch_work_doubles(int32_t rows, int32_t cols, int32_t d, int32_t topology);
hipError_t launch_batch_epoch(const BatchArgs &b, hipStream_t s);

// In-place stream over `bytes` (a multiple of 16) of buf on `grid`
// workgroups, `passes` times, each word scaled by a (som_stream.hip).
hipError_t launch_stream_inplace(float *buf, int64_t bytes, int32_t passes, int32_t grid,
                                 float a, hipStream_t s);

// Principal components and linear initialisation (som_pca.hip).
constexpr int kPcaBlock = 8;  // subspace-iteration block
// Floats of work memory for pca_top2 (covariance d x d, iteration vectors,
// column partial sums).
size_t pca_work_floats(int32_t d);
// Two largest eigenvalues of the covariance of the n x d rows of X (host
// lambda[2]) and the column means (mean, d floats); the unit eigenvectors
// are left in pca_vectors(work, d) (columns 0 and 1, stride d).  stats: 4
// device doubles.  Iterates until both residuals are below tol * lambda1
// or max_iters; synchronizes the stream.
hipError_t pca_top2(const float *X, int64_t n, int32_t d, float *work, float *mean, double *stats,
                    int max_iters, double tol, hipStream_t s, double *lambda, int *iters);
const float *pca_vectors(const float *work, int32_t d);
hipError_t launch_linear_init(float *W, int64_t ld, int32_t rows, int32_t cols, int32_t d,
                              const float *mean, const float *v1, const float *v2, double lambda1,
                              double lambda2, hipStream_t s);

}  // namespace som
