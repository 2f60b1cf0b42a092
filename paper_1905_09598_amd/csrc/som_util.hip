// Small helper kernels: prototype initialisation, per-call preparation of
// the training kernel (exchange slots, order check, schedule table), the
// non-finite scan of training data, row squared norms.
#include "som_internal.h"

namespace som {
namespace {

// SplitMix64 (Steele, Lea and Flood, OOPSLA 2014), counter form: the i-th
// output of the generator seeded with `seed`.
__device__ inline uint64_t splitmix64_at(uint64_t seed, uint64_t i) {
    uint64_t z = seed + (i + 1u) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    return z ^ (z >> 31);
}

// W[u][j] = top 24 bits of output u * d + j, times 2^-24; padding = 0.
__global__ void init_uniform_kernel(float *W, int64_t ld, int32_t N, int32_t d,
                                    uint64_t seed) {
    const int64_t total = (int64_t)N * ld;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t u = e / ld, j = e - u * ld;
        float v = 0.f;
        if (j < d) {
            const uint64_t r = splitmix64_at(seed, (uint64_t)(u * d + j));
            v = (float)(r >> 40) * (1.0f / 16777216.0f);
        }
        W[e] = v;
    }
}

// Zero the exchange words a grid of `grid` workgroups uses (every replica,
// both parities) and the order flag.
__global__ void reset_train_kernel(unsigned long long *slots, int64_t per_replica,
                                   DevState *state) {
    const int64_t total = kSlotReplicas * per_replica;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t rep = i / per_replica, off = i - rep * per_replica;
        slots[rep * kSlotReplicaStride + off] = 0ull;
    }
    if (blockIdx.x == 0 && threadIdx.x == 0) state->order_bad = 0;
}

__device__ inline double decay_at(double a, double b, int kind, double p) {
    if (a == b) return a;
    // p = 0 gives a and p = 1 gives b exactly
    if (kind == 0) return (1.0 - p) * a + p * b;
    return pow(a, 1.0 - p) * pow(b, p);
}

// Per local step s: range-check order[s]; sched[s] = (lr(t), log2(e) / (2
// sigma(t)^2)) at global step t = step0 + s, p = t / (T - 1) (p = 0 when
// T = 1).  sigma = 0 gives the largest finite scale (a delta at the BMU),
// sigma = +inf gives 0 (h = lr everywhere).
__global__ void prepare_train_kernel(const int32_t *order, int64_t nsteps, int64_t n,
                                     int64_t step0, int64_t total, double lr0, double lr1,
                                     int lr_kind, double s0, double s1, int s_kind,
                                     float2 *sched, DevState *state) {
    const int64_t s = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    if (s >= nsteps) return;
    const int32_t v = order[s];
    if (v < 0 || (int64_t)v >= n) {
        atomicOr(&state->order_bad, 1);
        atomicCAS(&state->status, 0, 7);  // SOM_E_BAD_ORDER unless an error is pending
    }
    const int64_t t = step0 + s;
    const double p = total > 1 ? (double)t / (double)(total - 1) : 0.0;
    const double lr = decay_at(lr0, lr1, lr_kind, p);
    const double sg = decay_at(s0, s1, s_kind, p);
    double c2;
    if (sg == 0.0) {
        c2 = 3.4028234663852886e38;  // FLT_MAX
    } else if (isinf(sg)) {
        c2 = 0.0;
    } else {
        c2 = 1.4426950408889634 / (2.0 * sg * sg);  // log2(e) / (2 sigma^2)
        if (c2 > 3.4028234663852886e38) c2 = 3.4028234663852886e38;
    }
    sched[s] = make_float2((float)lr, (float)c2);
}

// Raise the call's input flag (which stops the training kernels before any
// update) and the sticky status, SOM_E_NONFINITE unless an error is pending,
// when any of the `count` floats at x is a NaN or an infinity (all exponent
// bits set).  One read of x: 16-byte loads, four in flight per thread.
__global__ void scan_finite_kernel(const float *x, int64_t count, DevState *state) {
    constexpr unsigned kExp = 0x7f800000u;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    const int64_t t = blockIdx.x * (int64_t)blockDim.x + threadIdx.x;
    const unsigned *xu = reinterpret_cast<const unsigned *>(x);
    bool bad = false;
    int64_t tail = 0;  // first element the vector loop leaves to the scalar one
    if (reinterpret_cast<uintptr_t>(x) % 16 == 0) {
        const uint4 *x4 = reinterpret_cast<const uint4 *>(x);
        const int64_t n4 = count / 4;
        const auto nonfinite4 = [&](const uint4 v) {
            return ((v.x & kExp) == kExp) | ((v.y & kExp) == kExp) | ((v.z & kExp) == kExp) |
                   ((v.w & kExp) == kExp);
        };
        int64_t i = t;
        for (; i + 3 * stride < n4; i += 4 * stride) {
            const uint4 a = x4[i], b = x4[i + stride], c = x4[i + 2 * stride],
                        d = x4[i + 3 * stride];
            bad |= nonfinite4(a) | nonfinite4(b) | nonfinite4(c) | nonfinite4(d);
        }
        for (; i < n4; i += stride) bad |= nonfinite4(x4[i]);
        tail = n4 * 4;
    }
    for (int64_t i = tail + t; i < count; i += stride) bad |= (xu[i] & kExp) == kExp;
    if (__ballot(bad) != 0 && (threadIdx.x & 63) == 0) {
        atomicOr(&state->order_bad, 1);
        atomicCAS(&state->status, 0, 8);  // SOM_E_NONFINITE unless an error is pending
    }
}

// out[u] = sum_j W[u][j]^2 (fp32, fixed order): `tpr` threads per row (64,
// 128 or 256; 256 / tpr rows per workgroup), 16-byte loads, four in flight.
__global__ __launch_bounds__(256) void row_sqnorm_kernel(const float *W, int64_t ld, int32_t N,
                                                         float *out, int tpr) {
    __shared__ float part[4];
    const int rsub = threadIdx.x / tpr, t = threadIdx.x - rsub * tpr;
    const int64_t row = (int64_t)blockIdx.x * (256 / tpr) + rsub;
    float acc = 0.f;
    if (row < N) {
        const float4 *w = reinterpret_cast<const float4 *>(W + row * ld);
        const int64_t n4 = ld / 4;
#pragma unroll 4
        for (int64_t j = t; j < n4; j += tpr) {
            const float4 v = w[j];
            acc = fmaf(v.x, v.x, acc);
            acc = fmaf(v.y, v.y, acc);
            acc = fmaf(v.z, v.z, acc);
            acc = fmaf(v.w, v.w, acc);
        }
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if ((threadIdx.x & 63) == 0) part[threadIdx.x >> 6] = acc;
    __syncthreads();
    if (t == 0 && row < N) {
        const int w0 = threadIdx.x >> 6, nw = tpr / 64;
        float s = part[w0];
        for (int k = 1; k < nw; ++k) s += part[w0 + k];
        out[row] = s;
    }
}

__global__ void pad_rows_kernel(const float *X, int64_t n, int32_t d, float *out, int64_t xld) {
    const int64_t total = n * xld;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t i = e / xld, c = e - i * xld;
        out[e] = c < d ? X[i * d + c] : 0.f;
    }
}

}  // namespace

hipError_t launch_init_uniform(float *W, int64_t ld, int32_t N, int32_t d,
                               uint64_t seed, hipStream_t s) {
    const int64_t total = (int64_t)N * ld;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    if (blocks < 1) blocks = 1;
    init_uniform_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(W, ld, N, d, seed);
    return hipGetLastError();
}

hipError_t launch_prepare_train(const TrainArgs &a, float2 *sched, hipStream_t s) {
    if (a.grid < 1 || a.grid > kMaxTrainGrid || a.slot_spread < 1 ||
        a.slot_spread > kMaxSlotSpread)
        return hipErrorInvalidValue;
    const int64_t per_replica = 2LL * a.grid * a.slot_spread;
    reset_train_kernel<<<dim3(16), dim3(256), 0, s>>>(a.slots, per_replica, a.state);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t blocks = (a.nsteps + 255) / 256;
    prepare_train_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(
        a.order, a.nsteps, a.n, a.step0, a.total_steps, a.lr0, a.lr1, a.lr_decay, a.sigma0,
        a.sigma1, a.sigma_decay, sched, a.state);
    return hipGetLastError();
}

hipError_t launch_scan_finite(const float *x, int64_t count, DevState *state,
                              hipStream_t s) {
    if (count <= 0) return hipSuccess;
    int64_t blocks = (count / 4 + 255) / 256;
    if (blocks > 4096) blocks = 4096;
    if (blocks < 1) blocks = 1;
    scan_finite_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(x, count, state);
    return hipGetLastError();
}

hipError_t launch_row_sqnorm(const float *W, int64_t ld, int32_t N, float *out,
                             hipStream_t s) {
    const int64_t n4 = ld / 4;
    const int tpr = n4 > 512 ? 256 : n4 > 128 ? 128 : 64;
    const int64_t blocks = ((int64_t)N + 256 / tpr - 1) / (256 / tpr);
    row_sqnorm_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(W, ld, N, out, tpr);
    return hipGetLastError();
}

hipError_t launch_pad_rows(const float *X, int64_t n, int32_t d, float *out, int64_t xld,
                           hipStream_t s) {
    const int64_t total = n * xld;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    pad_rows_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(X, n, d, out, xld);
    return hipGetLastError();
}

}  // namespace som
