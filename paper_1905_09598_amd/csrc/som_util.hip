// Small helper kernels: prototype initialisation, per-call preparation of
// the training kernel's exchange slots and order check, row squared norms.
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

// One workgroup: zero the exchange slots and set state->order_bad to
// whether any order entry lies outside [0, n) (also raising the sticky
// status).  Runs before every training launch on the same stream.
constexpr int kPrepBlock = 1024;
__global__ __launch_bounds__(kPrepBlock) void prepare_train_kernel(
    const int32_t *order, int64_t nsteps, int64_t n, unsigned long long *slots,
    int32_t nslots, DevState *state) {
    for (int i = threadIdx.x; i < nslots; i += kPrepBlock) slots[i] = 0ull;
    int bad = 0;
    for (int64_t k = threadIdx.x; k < nsteps; k += kPrepBlock) {
        const int32_t v = order[k];
        bad |= (v < 0 || (int64_t)v >= n);
    }
    bad = __syncthreads_or(bad);
    if (threadIdx.x == 0) {
        state->order_bad = bad;
        if (bad) state->status = 7;  // SOM_E_BAD_ORDER
    }
}

// out[u] = sum_j W[u][j]^2, one wave per row (fp32, fixed order).
__global__ void row_sqnorm_kernel(const float *W, int64_t ld, int32_t N, float *out) {
    const int lane = threadIdx.x & 63;
    const int64_t row = blockIdx.x * (int64_t)(blockDim.x / 64) + (threadIdx.x >> 6);
    if (row >= N) return;
    const float *w = W + row * ld;
    float acc = 0.f;
    for (int64_t j = lane; j < ld; j += 64) acc = fmaf(w[j], w[j], acc);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
    if (lane == 0) out[row] = acc;
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

hipError_t launch_prepare_train(const int32_t *order, int64_t nsteps, int64_t n,
                                unsigned long long *slots, int32_t nslots,
                                DevState *state, hipStream_t s) {
    prepare_train_kernel<<<dim3(1), dim3(kPrepBlock), 0, s>>>(order, nsteps, n, slots,
                                                              nslots, state);
    return hipGetLastError();
}

hipError_t launch_row_sqnorm(const float *W, int64_t ld, int32_t N, float *out,
                             hipStream_t s) {
    const int waves = 4;
    const int64_t blocks = (N + waves - 1) / waves;
    row_sqnorm_kernel<<<dim3((unsigned)blocks), dim3(64 * waves), 0, s>>>(W, ld, N, out);
    return hipGetLastError();
}

}  // namespace som
