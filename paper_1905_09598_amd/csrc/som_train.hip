// Persistent online-SOM training kernel for gfx950 (MI355X).
//
// One cooperative launch runs every step of a som_train call (paper Sec. 6C
// runs three kernels and a host round trip per sample; here the per-sample
// loop never leaves the device).  Each workgroup owns a fixed, contiguous
// range of prototype rows for the whole launch, so a row is only ever read
// and written by one workgroup (and so by one XCD and its L2).  The rows
// live either in device memory, swept every step (variant "stream"), or in
// the workgroup's LDS for the whole launch, loaded at the start and written
// back at the end (variant "lds", when the slice fits).
//
// Step s of the call (global step t = step0 + s) with BMU c_s known:
//   1. h_u = lr(t) 2^(-g(u, c_s) * log2(e) / (2 sigma(t)^2)) for the owned
//      rows (Eq. (1) with a Gaussian kernel; lr(t) and the exponent scale
//      come from a per-step table built in fp64 before the launch);
//   2. one sweep over the owned rows that applies Eq. (1),
//      w <- fma(h, x_s, fma(-h, w, w)), and in the same pass accumulates
//      the squared distance of the updated row to the next sample x_{s+1};
//   3. the workgroup's (distance, unit) minimum goes to a grid exchange and
//      every workgroup reads all minima, so each learns c_{s+1} on its own.
// A distance-only sweep before step 0 gives c_0.  Sample rows are loaded two
// steps ahead so their latency hides behind the sweep and the exchange.
//
// The grid exchange uses one 64-bit slot per workgroup and parity,
// dist_bits << 32 | tag << 24 | unit, written and polled with relaxed
// device-scope atomics only (no fences, so no cache write-back or
// invalidation).  The minimum over slots with the current tag is the
// minimum over (distance, unit): squared distances are non-negative, so their
// IEEE bits order like the values, and equal distances fall to the lowest
// unit.  Slots alternate by step parity, so a fast workgroup can publish step
// e+1 while a slow one still reads step e.  Every wait is bounded in time and
// also ends when any workgroup has flagged an error.
#include "som_internal.h"

#include <math.h>

namespace som {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kWaves = kTrainBlock / 64;
constexpr int32_t kStatusTimeout = 5;  // SOM_E_TIMEOUT
constexpr int kHeader = 64;            // LDS bytes for the broadcast words

// Sums over the 64 lanes of a wave, for U values at once, returned to every
// lane.  Within each row of 16 lanes a butterfly of DPP moves (quad swaps,
// half-row and row mirrors) leaves the row's sum in all of its lanes,
// bit-identical because every pairwise add is commutative; the four row sums
// are then read out and added in a fixed order.  The U chains run in
// lockstep so their DPP hazards overlap.
template <int CTRL>
__device__ inline int dpp_move(int v) {
    return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xf, 0xf, false);
}
template <int CTRL>
__device__ inline float dpp_pair(float v) {
    return v + __int_as_float(dpp_move<CTRL>(__float_as_int(v)));
}
__device__ inline float lane_f(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
template <int U>
__device__ inline void wave_sums(float (&v)[U]) {
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_pair<0xB1>(v[u]);   // quad_perm [1,0,3,2]
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_pair<0x4E>(v[u]);   // quad_perm [2,3,0,1]
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_pair<0x141>(v[u]);  // row_half_mirror
#pragma unroll
    for (int u = 0; u < U; ++u) v[u] = dpp_pair<0x140>(v[u]);  // row_mirror
#pragma unroll
    for (int u = 0; u < U; ++u)
        v[u] = (lane_f(v[u], 0) + lane_f(v[u], 16)) + (lane_f(v[u], 32) + lane_f(v[u], 48));
}

__device__ inline unsigned long long u64_min(unsigned long long a, unsigned long long b) {
    return a < b ? a : b;
}

template <int CTRL>
__device__ inline unsigned long long dpp_min_u64(unsigned long long v) {
    const unsigned lo = (unsigned)dpp_move<CTRL>((int)(unsigned)(v & 0xffffffffu));
    const unsigned hi = (unsigned)dpp_move<CTRL>((int)(unsigned)(v >> 32));
    return u64_min(v, ((unsigned long long)hi << 32) | lo);
}

__device__ inline unsigned long long lane_u64(unsigned long long v, int l) {
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(v & 0xffffffffu), l);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(v >> 32), l);
    return ((unsigned long long)hi << 32) | lo;
}

// Minimum over the 64 lanes of a wave (same DPP pattern), to every lane.
__device__ inline unsigned long long wave_min_u64(unsigned long long v) {
    v = dpp_min_u64<0xB1>(v);
    v = dpp_min_u64<0x4E>(v);
    v = dpp_min_u64<0x141>(v);
    v = dpp_min_u64<0x140>(v);
    return u64_min(u64_min(lane_u64(v, 0), lane_u64(v, 16)),
                   u64_min(lane_u64(v, 32), lane_u64(v, 48)));
}

// Lane layout.  A workgroup's 256 threads form P = 256 / L groups of L
// lanes; group g sweeps rows g, g + P, g + 2P, ... of the workgroup's slice
// and lane j of a group holds the 16-byte columns j, j + L, ..., j + (K-1) L
// of its rows (and of the sample rows).  With L = 64 a wave owns whole rows,
// so a row's distance needs one wave-level reduction and nothing else; with
// L = 256 every wave holds a quarter of every row (long rows) and the four
// partial sums meet in LDS.
// Sample row i into the lane's slots; columns past d (row padding) are 0.
template <int K, int L>
__device__ inline void load_sample(f4 (&x)[K], const TrainArgs &a, int64_t i) {
    const int li = threadIdx.x % L;
    if (a.x_vec4) {
        const f4 *xr = reinterpret_cast<const f4 *>(a.X + i * a.d);
        const int xd4 = a.d >> 2;  // d % 4 == 0 on this path
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const int q = li + L * k;
            x[k] = (q < xd4) ? xr[q] : f4{0.f, 0.f, 0.f, 0.f};
        }
    } else {
        const float *xr = a.X + i * a.d;
#pragma unroll
        for (int k = 0; k < K; ++k) {
            const int j = 4 * (li + L * k);
            f4 v;
            v.x = (j + 0 < a.d) ? xr[j + 0] : 0.f;
            v.y = (j + 1 < a.d) ? xr[j + 1] : 0.f;
            v.z = (j + 2 < a.d) ? xr[j + 2] : 0.f;
            v.w = (j + 3 < a.d) ? xr[j + 3] : 0.f;
            x[k] = v;
        }
    }
}

// Per-step inputs (sample index, schedule entry) are fetched 64 steps at a
// time: lane l of a window holds the entry of step base + l, loaded with one
// vector load, and a step's entry is read out with readlane.  Vector loads
// keep these fetches off the scalar-memory counter that LDS operations
// share, so waiting for LDS never waits for them.  The next window is
// loaded while the current one is in use.
__device__ inline int fetch_entry(const TrainArgs &a, int64_t s, int) {
    int i = s < a.nsteps ? a.order[s] : 0;
    return (i >= 0 && (int64_t)i < a.n) ? i : 0;  // range-checked before launch
}
__device__ inline float2 fetch_entry(const TrainArgs &a, int64_t s, float2) {
    return s < a.nsteps ? a.sched[s] : make_float2(0.f, 0.f);
}

template <typename T>
struct StepWindow {
    int64_t base;
    T cur, next;

    __device__ void init(const TrainArgs &a, int64_t b) {
        base = b;
        cur = fetch_entry(a, b + (threadIdx.x & 63), T());
        next = fetch_entry(a, b + 64 + (threadIdx.x & 63), T());
    }
    // Entry of step s, for non-decreasing s >= base.
    __device__ T get(const TrainArgs &a, int64_t s) {
        if (s >= base + 64) {
            base += 64;
            cur = next;
            next = fetch_entry(a, base + 64 + (threadIdx.x & 63), T());
        }
        return lane_value((int)(s - base));
    }
    __device__ T lane_value(int l) const;
};

template <>
__device__ inline int StepWindow<int>::lane_value(int l) const {
    return __builtin_amdgcn_readlane(cur, l);
}
template <>
__device__ inline float2 StepWindow<float2>::lane_value(int l) const {
    return make_float2(__int_as_float(__builtin_amdgcn_readlane(__float_as_int(cur.x), l)),
                       __int_as_float(__builtin_amdgcn_readlane(__float_as_int(cur.y), l)));
}

__device__ inline unsigned long long row_key(float D, int u) {
    return ((unsigned long long)__float_as_uint(D) << 32) | (unsigned)u;
}

// One pass over the workgroup's R rows, each L * K float4 long (the row
// pitch is padded to exactly the lanes' slots, padding zero), from `rows`.
// UPD applies Eq. (1) with row r's factor (lane r of hl when R <= 64, else
// hs[r]).  DIST accumulates |xb - w|^2 of the updated rows: with L = 64 the
// wave's best (distance, unit) key over its rows is returned; with L = 256
// the wave's partial sum of row r goes to part[r * 4 + wave].
template <int K, int U, int L, bool UPD, bool DIST>
__device__ inline unsigned long long sweep(f4 *__restrict__ rows, int r0, int R,
                                           const f4 (&xa)[K], const f4 (&xb)[K], float hl,
                                           const float *hs, float *part) {
    constexpr int P = kTrainBlock / L;
    constexpr int P4 = L * K;  // float4 per row
    const int tid = threadIdx.x, g = tid / L, li = tid % L, lane = tid & 63;
    const int wave = tid >> 6;
    unsigned long long best = ~0ull;
    for (int rb = g; rb < R; rb += P * U) {
        f4 w[U][K];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = rb + u * P;
            if (r < R) {
                const f4 *row = rows + (size_t)r * P4 + li;
#pragma unroll
                for (int k = 0; k < K; ++k) w[u][k] = row[L * k];
            }
        }
        float acc[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = rb + u * P;
            acc[u] = 0.f;
            if (r < R) {
                f4 *row = rows + (size_t)r * P4 + li;
                float h = 0.f;
                if (UPD) h = (R <= 64) ? lane_f(hl, r) : hs[r];
#pragma unroll
                for (int k = 0; k < K; ++k) {
                    f4 v = w[u][k];
                    if (UPD) {
                        v.x = fmaf(h, xa[k].x, fmaf(-h, v.x, v.x));
                        v.y = fmaf(h, xa[k].y, fmaf(-h, v.y, v.y));
                        v.z = fmaf(h, xa[k].z, fmaf(-h, v.z, v.z));
                        v.w = fmaf(h, xa[k].w, fmaf(-h, v.w, v.w));
                        row[L * k] = v;
                    }
                    if (DIST) {
                        const f4 df = xb[k] - v;
                        acc[u] = fmaf(df.x, df.x, acc[u]);
                        acc[u] = fmaf(df.y, df.y, acc[u]);
                        acc[u] = fmaf(df.z, df.z, acc[u]);
                        acc[u] = fmaf(df.w, df.w, acc[u]);
                    }
                }
            }
        }
        if (DIST) {
            wave_sums<U>(acc);
            if (L == 64) {
#pragma unroll
                for (int u = 0; u < U; ++u)
                    if (rb + u * P < R) best = u64_min(best, row_key(acc[u], r0 + rb + u * P));
            } else if (lane == 0) {
#pragma unroll
                for (int u = 0; u < U; ++u)
                    if (rb + u * P < R) part[(rb + u * P) * kWaves + wave] = acc[u];
            }
        }
    }
    return best;
}

struct Bcast {
    unsigned long long key;
    int abort;
    int pad;
    unsigned long long wave_best[kWaves];
};

// Wave 0, after the sweep's barrier: the workgroup's best (distance, unit).
template <int L>
__device__ inline unsigned long long workgroup_best(int r0, int R, const float *part,
                                                    const Bcast *bc) {
    const int lane = threadIdx.x & 63;
    unsigned long long best = ~0ull;
    if (L == 64) {
        if (lane < kWaves) best = bc->wave_best[lane];
    } else {
        for (int r = lane; r < R; r += 64) {
            float D = part[r * kWaves + 0];
#pragma unroll
            for (int w = 1; w < kWaves; ++w) D += part[r * kWaves + w];
            best = u64_min(best, row_key(D, r0 + r));
        }
    }
    return wave_min_u64(best);
}

// Wave 0 only: publish the workgroup's best key to grid exchange number e,
// then take the minimum over every workgroup's slot into bc->key (bc->abort
// set if the wait was given up).
__device__ inline void exchange_wave0(const TrainArgs &a, int64_t e,
                                      unsigned long long best, Bcast *bc) {
    const int lane = threadIdx.x & 63, G = a.grid;
    if (G == 1) {
        if (lane == 0) { bc->key = best; bc->abort = 0; }
        return;
    }
    const unsigned tag = 0x80u | (unsigned)((e >> 1) & 0x7f);
    unsigned long long *slots = a.slots + (e & 1) * (int64_t)G;
    if (lane == 0) {
        const unsigned long long v = (best & 0xffffffff00000000ull) |
                                     ((unsigned long long)tag << kUnitBits) |
                                     (best & (unsigned long long)kMaxUnits);
        __hip_atomic_store(slots + blockIdx.x, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    }
    unsigned long long m = ~0ull;
    int abort = 0;
    for (int i = lane; i < G && !abort; i += 64) {
        const uint64_t t0 = __builtin_amdgcn_s_memrealtime();
        unsigned spins = 0;
        for (;;) {
            const unsigned long long v =
                __hip_atomic_load(slots + i, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
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
                    __hip_atomic_store(&a.state->status, kStatusTimeout, __ATOMIC_RELAXED,
                                       __HIP_MEMORY_SCOPE_AGENT);
                    abort = 1;
                    break;
                }
            }
        }
    }
    m = wave_min_u64(m);
    const unsigned long long any_abort = __ballot(abort);
    if (lane == 0) { bc->key = m; bc->abort = any_abort != 0; }
}

// Neighbourhood factor of owned row r given BMU c: lr * 2^(-g * c2) with g
// the squared lattice distance.  pos[r] holds (row, column, row parity) of
// unit r0 + r.  RECT: g = dr^2 + dc^2.  HEX: odd rows shifted by 1/2 and rows
// sqrt(3)/2 apart, so g = 3/4 dr^2 + (dc + (parity difference) / 2)^2, exact
// in fp32 for the map sizes the library accepts.
__device__ inline float neighbour_h(const TrainArgs &a, float4 p, float cr, float cc,
                                    float cpar, float lr, float c2) {
    const float dr = p.x - cr;
    float dx = p.y - cc, g;
    if (a.topology == 1) {
        dx += 0.5f * (p.z - cpar);
        g = 0.75f * dr * dr + dx * dx;
    } else {
        g = dr * dr + dx * dx;
    }
    return lr * exp2f(-g * c2);
}

template <int K, int U, int L, bool LDSW>
__global__ __launch_bounds__(kTrainBlock, 1) void train_kernel(TrainArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int G = a.grid, b = blockIdx.x, tid = threadIdx.x, wave = tid >> 6, lane = tid & 63;
    const int r0 = (int)(((int64_t)b * a.N) / G);
    const int r1 = (int)(((int64_t)(b + 1) * a.N) / G);
    const int R = r1 - r0;
    const int Rp = (R + 3) & ~3;
    Bcast *bc = reinterpret_cast<Bcast *>(smem);
    float *hs = reinterpret_cast<float *>(smem + kHeader);
    float *part = hs + Rp;
    float4 *pos = reinterpret_cast<float4 *>(part + (int64_t)Rp * kWaves);
    f4 *lw = reinterpret_cast<f4 *>(pos + Rp);

    if (a.state->order_bad) return;  // same value for every workgroup
    if (a.nsteps <= 0) return;

    for (int r = tid; r < R; r += kTrainBlock) {
        const int u = r0 + r, ur = u / a.cols, uc = u - ur * a.cols;
        pos[r] = make_float4((float)ur, (float)uc, (float)(ur & 1), 0.f);
    }
    const int64_t ld4 = a.ld / 4;
    f4 *gw = reinterpret_cast<f4 *>(a.W) + (int64_t)r0 * ld4;
    f4 *rows = gw;
    if (LDSW) {
        for (int64_t e = tid; e < (int64_t)R * ld4; e += kTrainBlock) lw[e] = gw[e];
        rows = lw;
    }

    f4 xa[K], xb[K], xc[K];
#pragma unroll
    for (int k = 0; k < K; ++k) xa[k] = f4{0.f, 0.f, 0.f, 0.f};
    StepWindow<int> ow;      // sample indices, read two steps ahead
    StepWindow<float2> sw;   // schedule entries
    ow.init(a, 0);
    sw.init(a, 0);

    // Prologue: distance-only sweep against the first sample gives c_0.
    load_sample<K, L>(xb, a, ow.get(a, 0));
    load_sample<K, L>(xc, a, a.nsteps > 1 ? ow.get(a, 1) : 0);
    __syncthreads();
    float4 mypos = make_float4(0.f, 0.f, 0.f, 0.f);  // lane l: row l's position
    if (lane < R) mypos = pos[lane];
    unsigned long long wb = sweep<K, U, L, false, true>(rows, r0, R, xa, xb, 0.f, hs, part);
    if (L == 64 && lane == 0) bc->wave_best[wave] = wb;
    __syncthreads();
    if (wave == 0) exchange_wave0(a, 0, workgroup_best<L>(r0, R, part, bc), bc);
    __syncthreads();
    if (bc->abort) return;
    int c = (int)(bc->key & (unsigned long long)kMaxUnits);

    for (int64_t s = 0; s < a.nsteps; ++s) {
        if (b == 0 && tid == 0 && a.bmu_trace) a.bmu_trace[s] = c;
        // rotate the sample pipeline: xa = x_s, xb = x_{s+1}, xc <- x_{s+2}
#pragma unroll
        for (int k = 0; k < K; ++k) { xa[k] = xb[k]; xb[k] = xc[k]; }
        const bool has_next = s + 1 < a.nsteps;
        if (s + 2 < a.nsteps) load_sample<K, L>(xc, a, ow.get(a, s + 2));
        const float2 cur = sw.get(a, s);

        const int cr = c / a.cols, ccol = c - cr * a.cols;
        const float fcr = (float)cr, fcc = (float)ccol, fcp = (float)(cr & 1);
        float hl = 0.f;
        if (R <= 64) {
            if (lane < R) hl = neighbour_h(a, mypos, fcr, fcc, fcp, cur.x, cur.y);
        } else {
            for (int r = tid; r < R; r += kTrainBlock)
                hs[r] = neighbour_h(a, pos[r], fcr, fcc, fcp, cur.x, cur.y);
            __syncthreads();
        }

        if (has_next) {
            wb = sweep<K, U, L, true, true>(rows, r0, R, xa, xb, hl, hs, part);
            if (L == 64 && lane == 0) bc->wave_best[wave] = wb;
            __syncthreads();
            if (wave == 0) exchange_wave0(a, s + 1, workgroup_best<L>(r0, R, part, bc), bc);
            __syncthreads();
            if (bc->abort) return;
            c = (int)(bc->key & (unsigned long long)kMaxUnits);
        } else {
            sweep<K, U, L, true, false>(rows, r0, R, xa, xb, hl, hs, part);
        }
    }
    if (LDSW) {
        __syncthreads();
        for (int64_t e = tid; e < (int64_t)R * ld4; e += kTrainBlock) gw[e] = lw[e];
    }
}

// Rows in flight per group: enough 16-byte loads outstanding per lane for
// the streamed variant, enough independent reductions for the LDS one.
template <int K>
constexpr int stream_unroll() {
    return K <= 2 ? 8 : (K <= 4 ? 4 : (K <= 8 ? 2 : 1));
}
template <int K>
constexpr int lds_unroll() {
    return K <= 2 ? 4 : (K <= 8 ? 2 : 1);
}

typedef void (*TrainKernel)(TrainArgs);

struct Instance {
    int lanes, k;
    TrainKernel stream, lds;
};

template <int L, int K>
constexpr Instance instance() {
    return Instance{L, K, train_kernel<K, stream_unroll<K>(), L, false>,
                    train_kernel<K, lds_unroll<K>(), L, true>};
}

// Rows up to 512 float4 (d <= 2048) use wave-owned rows; longer rows span
// the workgroup.
const Instance kInstances[] = {
    instance<64, 1>(),   instance<64, 2>(),   instance<64, 3>(),   instance<64, 4>(),
    instance<64, 5>(),   instance<64, 6>(),   instance<64, 8>(),   instance<256, 3>(),
    instance<256, 4>(),  instance<256, 5>(),  instance<256, 6>(),  instance<256, 8>(),
    instance<256, 10>(), instance<256, 12>(), instance<256, 16>(),
};

const Instance *pick(int64_t ld4) {
    for (const Instance &in : kInstances)
        if ((int64_t)in.k * in.lanes >= ld4) return &in;
    return nullptr;
}

size_t lds_bytes_for(int rmax, int64_t ld4, bool ldsw) {
    const size_t rp = (size_t)((rmax + 3) & ~3);
    size_t b = kHeader + rp * 4 + rp * kWaves * 4 + rp * 16;
    if (ldsw) b += (size_t)rmax * (size_t)ld4 * 16;
    return b;
}

// Estimated microseconds per step (model fitted to MI355X measurements of
// the exchange and of LDS / memory sweeps); only ranks launch shapes.
double exchange_us(int g) { return g <= 1 ? 0.2 : 0.6 + 0.3 * log2((double)g); }

}  // namespace

int64_t train_row_pitch(int32_t d) {
    const Instance *in = pick(((int64_t)d + 3) / 4);
    return in ? 4 * (int64_t)in->lanes * in->k : 0;
}

hipError_t plan_train(const TrainArgs &a, int num_cus, TrainPlan *plan) {
    const int64_t ld4 = a.ld / 4;
    const Instance *in = pick(ld4);
    if (!in || (int64_t)in->lanes * in->k != ld4) return hipErrorInvalidValue;
    int max_lds = 0;
    hipError_t e = hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, 0);
    if (e != hipSuccess) return e;
    const int max_grid = a.N < num_cus ? a.N : num_cus;
    const double row_bytes = 2.0 * 16.0 * (double)ld4;  // read + write per row per step

    int grid = 0, variant = 0;
    if (a.grid > 0) {
        grid = a.grid < a.N ? a.grid : a.N;
        const int rmax = (a.N + grid - 1) / grid;
        variant = (a.variant != 0 && lds_bytes_for(rmax, ld4, true) <= (size_t)max_lds) ? 1 : 0;
        if (a.variant == 1 && variant == 0) return hipErrorInvalidValue;
    } else {
        // streamed sweep over the whole chip: about 30 GB/s per CU of memory
        // traffic (measured at MALL-resident sizes) plus the exchange
        double best = 1e300;
        {
            const int g = max_grid;
            const int rmax = (a.N + g - 1) / g;
            best = exchange_us(g) + rmax * row_bytes / 30e3 + 0.5;
            grid = g;
            variant = 0;
        }
        if (a.variant != 2) {
            // LDS-resident slices: ~300 GB/s of LDS traffic per CU
            for (int g = 1; g <= max_grid; g *= 2) {
                const int gg = g;
                const int rmax = (a.N + gg - 1) / gg;
                if (lds_bytes_for(rmax, ld4, true) > (size_t)max_lds) continue;
                const double t = exchange_us(gg) + rmax * row_bytes / 300e3 + 0.3;
                if (t < best) { best = t; grid = gg; variant = 1; }
            }
            if (variant == 1) {
                // a non-power-of-two grid up to the CU count may fit better
                const int g = max_grid;
                const int rmax = (a.N + g - 1) / g;
                if (lds_bytes_for(rmax, ld4, true) <= (size_t)max_lds) {
                    const double t = exchange_us(g) + rmax * row_bytes / 300e3 + 0.3;
                    if (t < best) { best = t; grid = g; }
                }
            }
        }
    }
    if (grid < 1) grid = 1;
    const int rmax = (a.N + grid - 1) / grid;
    size_t lds = lds_bytes_for(rmax, ld4, variant == 1);
    if (lds > (size_t)max_lds) return hipErrorInvalidValue;
    // More than half of the CU's LDS keeps one workgroup per CU, so the
    // grid spreads over every CU instead of doubling up on some.
    if (lds < 84 * 1024) lds = 84 * 1024;
    TrainKernel fn = variant ? in->lds : in->stream;
    int per_cu = 0;
    e = hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, reinterpret_cast<const void *>(fn),
                                                     kTrainBlock, lds);
    if (e != hipSuccess) return e;
    if (per_cu < 1 || grid > per_cu * num_cus) return hipErrorCooperativeLaunchTooLarge;
    plan->grid = grid;
    plan->block = kTrainBlock;
    plan->variant = variant;
    plan->kslots = in->k;
    plan->lds_bytes = lds;
    return hipSuccess;
}

hipError_t launch_train(const TrainArgs &a, const TrainPlan &plan, hipStream_t s) {
    const Instance *in = pick(a.ld / 4);
    if (!in || in->k != plan.kslots || (int64_t)in->lanes * in->k != a.ld / 4)
        return hipErrorInvalidValue;
    TrainArgs args = a;
    args.grid = plan.grid;
    TrainKernel fn = plan.variant ? in->lds : in->stream;
    void *params[] = {&args};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(fn), dim3(plan.grid),
                                      dim3(plan.block), params, (unsigned)plan.lds_bytes, s);
}

}  // namespace som
