// Persistent online-SOM training kernel for gfx950 (MI355X).
//
// One cooperative launch runs every step of a som_train call (paper Sec. 6C
// runs three kernels and a host round trip per sample; here the per-sample
// loop never leaves the device).  Each workgroup owns a fixed, contiguous
// range of prototype rows for the whole launch, so a row is only ever read
// and written by one workgroup (and so by one XCD and its L2).
//
// Step s of the call (global step t = step0 + s) with BMU c_s known:
//   1. h_u = lr(t) exp(-|pos(u) - pos(c_s)|^2 / (2 sigma(t)^2)) for the owned
//      rows, in fp64, rounded to fp32 (Eq. (1) with a Gaussian kernel);
//   2. one sweep over the owned rows that applies Eq. (1),
//      w <- fma(h, x_s, fma(-h, w, w)), and in the same pass accumulates
//      the squared distance of the updated row to the next sample x_{s+1};
//   3. the workgroup's (distance, unit) minimum goes to a grid exchange and
//      every workgroup reads all minima, so each learns c_{s+1} on its own.
// A distance-only sweep before step 0 gives c_0.
//
// The grid exchange uses one 64-bit slot per workgroup and parity,
// dist_bits << 32 | tag << 24 | unit, written and polled with relaxed
// device-scope atomics only.  The minimum over slots with the current tag is
// the minimum over (distance, unit): squared distances are non-negative, so
// their IEEE bits order like the values, and equal distances fall to the
// lowest unit.  Slots alternate by step parity, so a fast workgroup can
// publish step e+1 while a slow one still reads step e.  Every wait is
// bounded in time and also ends when any workgroup has flagged an error.
#include "som_internal.h"

#include <math.h>

namespace som {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = kTrainBlock / 64;
constexpr int32_t kStatusTimeout = 5;  // SOM_E_TIMEOUT

__device__ inline double decay_at(double a, double b, int kind, double p) {
    if (a == b) return a;
    if (kind == 0) return (1.0 - p) * a + p * b;
    return pow(a, 1.0 - p) * pow(b, p);
}

__device__ inline float wave_sum(float v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    return v;
}

__device__ inline unsigned long long u64_min(unsigned long long a, unsigned long long b) {
    return a < b ? a : b;
}

__device__ inline unsigned long long wave_min_u64(unsigned long long v) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        unsigned lo = __shfl_xor((unsigned)(v & 0xffffffffu), o, 64);
        unsigned hi = __shfl_xor((unsigned)(v >> 32), o, 64);
        v = u64_min(v, ((unsigned long long)hi << 32) | lo);
    }
    return v;
}

// Minimum of one value per thread over the workgroup; every thread gets it.
__device__ inline unsigned long long block_min_u64(unsigned long long v,
                                                   unsigned long long *red) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    v = wave_min_u64(v);
    if (lane == 0) red[wave] = v;
    __syncthreads();
    unsigned long long m = red[0];
#pragma unroll
    for (int w = 1; w < kWaves; ++w) m = u64_min(m, red[w]);
    __syncthreads();
    return m;
}

template <int K>
__device__ inline void load_sample(f4 (&x)[K], const TrainArgs &a, int64_t i,
                                   int64_t ld4) {
    const int tid = threadIdx.x;
    if (a.x_vec4) {
        const f4 *xr = reinterpret_cast<const f4 *>(a.X + i * a.d);
#pragma unroll
        for (int k = 0; k < K; ++k) {
            int64_t q = tid + (int64_t)kTrainBlock * k;
            x[k] = (q < ld4) ? xr[q] : f4{0.f, 0.f, 0.f, 0.f};
        }
    } else {
        const float *xr = a.X + i * a.d;
#pragma unroll
        for (int k = 0; k < K; ++k) {
            int64_t j = 4 * (tid + (int64_t)kTrainBlock * k);
            f4 v;
            v.x = (j + 0 < a.d) ? xr[j + 0] : 0.f;
            v.y = (j + 1 < a.d) ? xr[j + 1] : 0.f;
            v.z = (j + 2 < a.d) ? xr[j + 2] : 0.f;
            v.w = (j + 3 < a.d) ? xr[j + 3] : 0.f;
            x[k] = v;
        }
    }
}

__device__ inline int64_t sample_at(const TrainArgs &a, int64_t s) {
    int64_t i = a.order[s];
    // The order was range-checked before launch; keep every read in bounds.
    return (i >= 0 && i < a.n) ? i : 0;
}

// One pass over the workgroup's rows [r0, r0 + R).  UPD applies Eq. (1) with
// the factors in hs[]; DIST accumulates |xb - w|^2 of the (updated) rows
// into part[r * kWaves + wave].
template <int K, int U, bool UPD, bool DIST>
__device__ inline void sweep(f4 *__restrict__ W4, int64_t ld4, int r0, int R,
                             const f4 (&xa)[K], const f4 (&xb)[K],
                             const float *hs, float *part) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int rb = 0; rb < R; rb += U) {
        f4 w[U][K];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = rb + u;
            const f4 *row = W4 + (int64_t)(r0 + r) * ld4;
#pragma unroll
            for (int k = 0; k < K; ++k) {
                int64_t q = tid + (int64_t)kTrainBlock * k;
                w[u][k] = (r < R && q < ld4) ? row[q] : f4{0.f, 0.f, 0.f, 0.f};
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = rb + u;
            if (r < R) {
                f4 *row = W4 + (int64_t)(r0 + r) * ld4;
                const float h = UPD ? hs[r] : 0.f;
                float acc = 0.f;
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    int64_t q = tid + (int64_t)kTrainBlock * k;
                    f4 v = w[u][k];
                    if (UPD) {
                        v.x = fmaf(h, xa[k].x, fmaf(-h, v.x, v.x));
                        v.y = fmaf(h, xa[k].y, fmaf(-h, v.y, v.y));
                        v.z = fmaf(h, xa[k].z, fmaf(-h, v.z, v.z));
                        v.w = fmaf(h, xa[k].w, fmaf(-h, v.w, v.w));
                        if (q < ld4) row[q] = v;
                    }
                    if (DIST) {
                        f4 df = xb[k] - v;
                        acc = fmaf(df.x, df.x, acc);
                        acc = fmaf(df.y, df.y, acc);
                        acc = fmaf(df.z, df.z, acc);
                        acc = fmaf(df.w, df.w, acc);
                    }
                }
                if (DIST) {
                    acc = wave_sum(acc);
                    if (lane == 0) part[r * kWaves + wave] = acc;
                }
            }
        }
    }
}

// Workgroup minimum of (distance, unit) over the owned rows, as a packed key.
__device__ inline unsigned long long local_best(int r0, int R, const float *part,
                                                unsigned long long *red) {
    unsigned long long best = ~0ull;
    for (int r = threadIdx.x; r < R; r += kTrainBlock) {
        float D = part[r * kWaves + 0];
#pragma unroll
        for (int w = 1; w < kWaves; ++w) D += part[r * kWaves + w];
        unsigned long long key =
            ((unsigned long long)__float_as_uint(D) << 32) | (unsigned)(r0 + r);
        best = u64_min(best, key);
    }
    return block_min_u64(best, red);
}

// Grid exchange number e: publish this workgroup's key, wait for every
// workgroup's, return the winning unit (or -1 if the wait was abandoned).
__device__ inline int exchange(const TrainArgs &a, int64_t e, unsigned long long key,
                               unsigned long long *red) {
    const int tid = threadIdx.x, G = a.grid;
    const unsigned tag = 0x80u | (unsigned)((e >> 1) & 0x7f);
    unsigned long long *slots = a.slots + (e & 1) * (int64_t)G;
    if (tid == 0) {
        unsigned long long v = (key & 0xffffffff00000000ull) |
                               ((unsigned long long)tag << kUnitBits) |
                               (key & (unsigned long long)kMaxUnits);
        __hip_atomic_store(slots + blockIdx.x, v, __ATOMIC_RELAXED,
                           __HIP_MEMORY_SCOPE_AGENT);
    }
    unsigned long long m = ~0ull;
    int abort = 0;
    for (int i = tid; i < G && !abort; i += kTrainBlock) {
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        unsigned spins = 0;
        for (;;) {
            unsigned long long v = __hip_atomic_load(slots + i, __ATOMIC_RELAXED,
                                                     __HIP_MEMORY_SCOPE_AGENT);
            if (((unsigned)(v >> kUnitBits) & 0xffu) == tag) {
                m = u64_min(m, v);
                break;
            }
            if ((++spins & 63u) == 0) {
                if (__hip_atomic_load(&a.state->status, __ATOMIC_RELAXED,
                                      __HIP_MEMORY_SCOPE_AGENT) != 0) {
                    abort = 1;
                    break;
                }
                if (__builtin_amdgcn_s_memrealtime() - t0 > a.timeout_ticks) {
                    __hip_atomic_store(&a.state->status, kStatusTimeout,
                                       __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                    abort = 1;
                    break;
                }
            }
            __builtin_amdgcn_s_sleep(1);
        }
    }
    if (__syncthreads_or(abort)) return -1;
    m = block_min_u64(m, red);
    return (int)(m & (unsigned long long)kMaxUnits);
}

template <int K, int U>
__global__ __launch_bounds__(kTrainBlock, 1) void train_stream_kernel(TrainArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int G = a.grid, b = blockIdx.x;
    const int r0 = (int)(((int64_t)b * a.N) / G);
    const int r1 = (int)(((int64_t)(b + 1) * a.N) / G);
    const int R = r1 - r0;
    unsigned long long *red = reinterpret_cast<unsigned long long *>(smem);
    float *hs = reinterpret_cast<float *>(smem + 64);
    float *part = hs + ((R + 3) & ~3);

    if (a.state->order_bad) return;  // same value for every workgroup
    if (a.nsteps <= 0) return;

    const int64_t ld4 = a.ld / 4;
    f4 *W4 = reinterpret_cast<f4 *>(a.W);
    f4 xa[K], xb[K];
#pragma unroll
    for (int k = 0; k < K; ++k) xa[k] = f4{0.f, 0.f, 0.f, 0.f};

    // Prologue: distance-only sweep against the first sample gives c_0.
    load_sample<K>(xb, a, sample_at(a, 0), ld4);
    sweep<K, U, false, true>(W4, ld4, r0, R, xa, xb, hs, part);
    __syncthreads();
    int c = exchange(a, 0, local_best(r0, R, part, red), red);
    if (c < 0) return;

    const double T1 = (double)(a.total_steps - 1);
    for (int64_t s = 0; s < a.nsteps; ++s) {
        if (b == 0 && threadIdx.x == 0 && a.bmu_trace) a.bmu_trace[s] = c;
#pragma unroll
        for (int k = 0; k < K; ++k) xa[k] = xb[k];
        const bool has_next = s + 1 < a.nsteps;
        if (has_next) load_sample<K>(xb, a, sample_at(a, s + 1), ld4);

        // Schedule and neighbourhood factors of the owned rows (fp64).
        const int64_t t = a.step0 + s;
        const double p = (a.total_steps > 1) ? (double)t / T1 : 0.0;
        const double lr = decay_at(a.lr0, a.lr1, a.lr_decay, p);
        const double sg = decay_at(a.sigma0, a.sigma1, a.sigma_decay, p);
        for (int r = threadIdx.x; r < R; r += kTrainBlock) {
            const int u = r0 + r;
            double h;
            if (sg == 0.0) {
                h = (u == c) ? lr : 0.0;
            } else if (isinf(sg)) {
                h = lr;
            } else {
                h = lr * exp(-lattice_sq(u, c, a.cols, a.topology) / (2.0 * sg * sg));
            }
            hs[r] = (float)h;
        }
        __syncthreads();

        if (has_next) {
            sweep<K, U, true, true>(W4, ld4, r0, R, xa, xb, hs, part);
            __syncthreads();
            c = exchange(a, s + 1, local_best(r0, R, part, red), red);
            if (c < 0) return;
        } else {
            sweep<K, U, true, false>(W4, ld4, r0, R, xa, xb, hs, part);
        }
    }
}

template <int K>
constexpr int unroll_for() {
    return K <= 2 ? 8 : (K <= 4 ? 4 : (K <= 8 ? 2 : 1));
}

typedef void (*TrainKernel)(TrainArgs);

template <int K>
TrainKernel kernel_for() {
    return train_stream_kernel<K, unroll_for<K>()>;
}

struct Instance {
    int k;
    TrainKernel fn;
};

const Instance kInstances[] = {
    {1, kernel_for<1>()},   {2, kernel_for<2>()},   {3, kernel_for<3>()},
    {4, kernel_for<4>()},   {5, kernel_for<5>()},   {6, kernel_for<6>()},
    {8, kernel_for<8>()},   {10, kernel_for<10>()}, {12, kernel_for<12>()},
    {16, kernel_for<16>()},
};

const Instance *pick(int64_t ld4) {
    for (const Instance &in : kInstances)
        if ((int64_t)in.k * kTrainBlock >= ld4) return &in;
    return nullptr;
}

}  // namespace

hipError_t plan_train(const TrainArgs &a, int num_cus, TrainPlan *plan) {
    const Instance *in = pick(a.ld / 4);
    if (!in) return hipErrorInvalidValue;
    int grid = a.grid > 0 ? a.grid : num_cus;
    if (grid > a.N) grid = a.N;
    if (grid < 1) grid = 1;
    const int rmax = (a.N + grid - 1) / grid;
    size_t need = 64 + (size_t)((rmax + 3) & ~3) * 4 + (size_t)rmax * kWaves * 4;
    // More than half of the CU's LDS keeps one workgroup per CU, so the
    // grid spreads over every CU instead of doubling up on some.
    size_t lds = need > 84 * 1024 ? need : 84 * 1024;
    int per_cu = 0;
    hipError_t e = hipOccupancyMaxActiveBlocksPerMultiprocessor(
        &per_cu, reinterpret_cast<const void *>(in->fn), kTrainBlock, lds);
    if (e != hipSuccess) return e;
    if (per_cu < 1 || grid > per_cu * num_cus) return hipErrorCooperativeLaunchTooLarge;
    plan->grid = grid;
    plan->block = kTrainBlock;
    plan->variant = 0;
    plan->kslots = in->k;
    plan->lds_bytes = lds;
    return hipSuccess;
}

hipError_t launch_train(const TrainArgs &a, const TrainPlan &plan, hipStream_t s) {
    const Instance *in = pick(a.ld / 4);
    if (!in || in->k != plan.kslots) return hipErrorInvalidValue;
    TrainArgs args = a;
    args.grid = plan.grid;
    void *params[] = {&args};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(in->fn),
                                      dim3(plan.grid), dim3(plan.block), params,
                                      (unsigned)plan.lds_bytes, s);
}

}  // namespace som
