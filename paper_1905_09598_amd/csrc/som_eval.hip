// Batched best-matching-unit assignment and map quality (QE, TE).
//
// After training, every document is assigned to its BMU (paper Sec. 8A) and
// the map is scored by its quantization error (Sec. 6D, Sec. 8B).  Over all
// n samples this is a dense contraction: ranking units by
//     |x - w|^2 = |x|^2 - 2 x.w + |w|^2
// only needs s(x, w) = |w|^2 - 2 x.w, and X W^T is an (n x d) by (d x N)
// matrix product, computed here on the fp32 matrix cores
// (v_mfma_f32_16x16x4_f32) without ever materialising the n x N matrix: each
// workgroup keeps, per sample, the kCand units of smallest s among its group
// of units (when there are few samples, the units are split into groups
// searched by separate workgroups, so that the grid still fills the chip).
// A second kernel re-ranks the groups' candidates by direct fp32 distances
// sum (x_j - w_j)^2, which fixes the BMU, the second BMU and the BMU's
// squared distance.
#include "som_internal.h"

#include <math.h>

#include <mutex>

namespace som {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

// Candidate kernel tiling: a workgroup owns kBM samples and walks all units
// in tiles of kBN, staging kBK-wide slices of X and W in LDS.  Its 4 waves
// form a 2 x 2 grid: 32 samples x 64 units each, i.e. 2 x 4 MFMA tiles of
// 16 x 16.
constexpr int kBM = 64;
constexpr int kBN = 128;
constexpr int kBK = 64;
constexpr int kPad = 4;
constexpr int kLdsStride = kBK + kPad;  // floats per staged row
constexpr int kEvalBlock = 256;

struct Cand {
    float s;
    int u;
};

__device__ inline bool better(float sa, int ua, float sb, int ub) {
    return sa < sb || (sa == sb && (unsigned)ua < (unsigned)ub);
}

// Insert (s, u) into an ascending top-kCand list (u = -1 marks empty slots,
// whose score is +inf).
__device__ inline void insert_top(float (&ts)[kCand], int (&tu)[kCand], float s, int u) {
    if (!better(s, u, ts[kCand - 1], tu[kCand - 1])) return;
    ts[kCand - 1] = s;
    tu[kCand - 1] = u;
#pragma unroll
    for (int i = kCand - 1; i > 0; --i) {
        if (better(ts[i], tu[i], ts[i - 1], tu[i - 1])) {
            float t = ts[i]; ts[i] = ts[i - 1]; ts[i - 1] = t;
            int v = tu[i]; tu[i] = tu[i - 1]; tu[i - 1] = v;
        }
    }
}

// Two workgroups per compute unit (the register budget that allows, and the
// planner's grid, assume it).
__global__ __launch_bounds__(kEvalBlock, 2) void bmu_candidates_kernel(EvalArgs a) {
    __shared__ __align__(16) float xs[kBM * kLdsStride];
    __shared__ __align__(16) float ws[kBN * kLdsStride];
    __shared__ float wn[kBN];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wsamp = wave & 1, wunit = wave >> 1;
    const int64_t s0 = (int64_t)blockIdx.x * kBM;
    const int grp = blockIdx.y;
    const int u_begin = grp * a.group_units;
    const int u_end = u_begin + a.group_units < a.N ? u_begin + a.group_units : a.N;
    const int lrow = lane & 15, lk = (lane >> 4) * 4;

    float ts[2][kCand];
    int tu[2][kCand];
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int c = 0; c < kCand; ++c) { ts[j][c] = INFINITY; tu[j][c] = -1; }

    for (int u0 = u_begin; u0 < u_end; u0 += kBN) {
        f4 acc[4][2];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

        __syncthreads();
        if (tid < kBN) wn[tid] = (u0 + tid < u_end) ? a.wnorm[u0 + tid] : 0.f;

        // The next kBK-wide slices of X and W are loaded into registers
        // before the current ones are multiplied, so their memory latency
        // overlaps the MFMAs.  The loads are unconditional (addresses clamped
        // into the operands); what lies outside them is zeroed as the slices
        // go to LDS, after the multiply: a select on a value in flight would
        // make the compiler wait for the load on the spot.
        constexpr int kXPer = (kBM * kBK / 4) / kEvalBlock;  // float4 per thread
        constexpr int kWPer = (kBN * kBK / 4) / kEvalBlock;
        f4 xv[kXPer], wv[kWPer];
        const auto fetch = [&](int k0) {
#pragma unroll
            for (int i = 0; i < kXPer; ++i) {
                const int idx = tid + i * kEvalBlock;
                const int r = idx / (kBK / 4), c4 = idx % (kBK / 4);
                const int64_t smp = s0 + r < a.n ? s0 + r : a.n - 1;
                const float *xr = a.X + smp * a.d;
                const int64_t col = k0 + 4 * c4;
                if (a.x_vec4) {
                    xv[i] = *reinterpret_cast<const f4 *>(xr + (col < a.d ? col : a.d - 4));
                } else {
#pragma unroll
                    for (int e = 0; e < 4; ++e) xv[i][e] = xr[col + e < a.d ? col + e : a.d - 1];
                }
            }
#pragma unroll
            for (int i = 0; i < kWPer; ++i) {
                const int idx = tid + i * kEvalBlock;
                const int r = idx / (kBK / 4), c4 = idx % (kBK / 4);
                const int64_t unit = u0 + r < u_end ? u0 + r : u_end - 1;
                const int64_t col = k0 + 4 * c4;
                wv[i] = *reinterpret_cast<const f4 *>(a.W + unit * a.ld +
                                                      (col < a.ld ? col : a.ld - 4));
            }
        };
        const auto stage = [&](int k0) {
#pragma unroll
            for (int i = 0; i < kXPer; ++i) {
                const int idx = tid + i * kEvalBlock;
                const int r = idx / (kBK / 4), c4 = idx % (kBK / 4);
                const int64_t col = k0 + 4 * c4;
                f4 v = xv[i];
                const bool row_ok = s0 + r < a.n;
#pragma unroll
                for (int e = 0; e < 4; ++e) v[e] = (row_ok && col + e < a.d) ? v[e] : 0.f;
                *reinterpret_cast<f4 *>(&xs[r * kLdsStride + 4 * c4]) = v;
            }
#pragma unroll
            for (int i = 0; i < kWPer; ++i) {
                const int idx = tid + i * kEvalBlock;
                const int r = idx / (kBK / 4), c4 = idx % (kBK / 4);
                const int64_t col = k0 + 4 * c4;
                const f4 zero = {0.f, 0.f, 0.f, 0.f};
                *reinterpret_cast<f4 *>(&ws[r * kLdsStride + 4 * c4]) =
                    (u0 + r < u_end && col < a.ld) ? wv[i] : zero;
            }
        };
        fetch(0);
        for (int k0 = 0; k0 < a.ld; k0 += kBK) {
            __syncthreads();
            stage(k0);
            __syncthreads();
            if (k0 + kBK < a.ld) fetch(k0 + kBK);

#pragma unroll
            for (int kq = 0; kq < kBK; kq += 16) {
                // Lane l supplies k = kq + 4 * (l / 16) + kk at sub-step kk for
                // both operands, so one 16-byte LDS read feeds four MFMAs.
                f4 af[4], bf[2];
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    af[i] = *reinterpret_cast<const f4 *>(
                        &ws[(wunit * 64 + i * 16 + lrow) * kLdsStride + kq + lk]);
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    bf[j] = *reinterpret_cast<const f4 *>(
                        &xs[(wsamp * 32 + j * 16 + lrow) * kLdsStride + kq + lk]);
#pragma unroll
                for (int kk = 0; kk < 4; ++kk)
#pragma unroll
                    for (int i = 0; i < 4; ++i)
#pragma unroll
                        for (int j = 0; j < 2; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                af[i][kk], bf[j][kk], acc[i][j], 0, 0, 0);
            }
        }

        // acc[i][j][v] = x.w for unit u0 + wunit*64 + i*16 + 4*(lane/16) + v
        // and sample s0 + wsamp*32 + j*16 + lane%16.
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int v = 0; v < 4; ++v) {
                const int ul = wunit * 64 + i * 16 + (lane >> 4) * 4 + v;
                const int u = u0 + ul;
                if (u < u_end) {
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        insert_top(ts[j], tu[j], wn[ul] - 2.f * acc[i][j][v], u);
                }
            }
    }

    // Merge the 8 partial lists of each sample (2 unit-waves x 4 lane groups).
    __syncthreads();
    Cand *pool = reinterpret_cast<Cand *>(ws);  // kBM * 8 * kCand entries
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int sl = wsamp * 32 + j * 16 + lrow;
        const int src = wunit * 4 + (lane >> 4);
#pragma unroll
        for (int c = 0; c < kCand; ++c)
            pool[(sl * 8 + src) * kCand + c] = Cand{ts[j][c], tu[j][c]};
    }
    __syncthreads();
    if (tid < kBM && s0 + tid < a.n) {
        float ms[kCand];
        int mu[kCand];
#pragma unroll
        for (int c = 0; c < kCand; ++c) { ms[c] = INFINITY; mu[c] = -1; }
        for (int e = 0; e < 8 * kCand; ++e) {
            const Cand cd = pool[tid * 8 * kCand + e];
            if (cd.u >= 0) insert_top(ms, mu, cd.s, cd.u);
        }
#pragma unroll
        for (int c = 0; c < kCand; ++c)
            a.cand[((s0 + tid) * a.ugroups + grp) * kCand + c] = mu[c];
    }
}

// One wave per sample: exact fp32 distances to the candidates, then the
// best and second best by (distance, unit).
constexpr int kRerankWaves = 4;
__global__ __launch_bounds__(64 * kRerankWaves) void bmu_rerank_kernel(EvalArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t i = (int64_t)blockIdx.x * kRerankWaves + (threadIdx.x >> 6);
    if (i >= a.n) return;
    const float *x = a.X + i * a.d;
    float bd = INFINITY, sd = INFINITY;
    int bu = -1, su = -1;
    const int nc = a.ugroups * kCand;
    for (int c = 0; c < nc; ++c) {
        const int u = a.cand[i * nc + c];
        if (u < 0) continue;  // same for the whole wave
        const float *w = a.W + (int64_t)u * a.ld;
        float acc = 0.f;
        for (int64_t j = lane; j < a.d; j += 64) {
            const float df = x[j] - w[j];
            acc = fmaf(df, df, acc);
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) acc += __shfl_xor(acc, o, 64);
        if (better(acc, u, bd, bu)) {
            sd = bd; su = bu;
            bd = acc; bu = u;
        } else if (better(acc, u, sd, su)) {
            sd = acc; su = u;
        }
    }
    if (lane == 0) {
        a.idx1[i] = bu;
        if (a.idx2) a.idx2[i] = su;
        if (a.d1) a.d1[i] = bd;
    }
}

// One workgroup sums sqrt(d1) and the count of non-adjacent (idx1, idx2)
// pairs in fp64, with a fixed thread-to-sample map and reduction tree.
constexpr int kReduceBlock = 1024;
__global__ __launch_bounds__(kReduceBlock) void qe_te_reduce_kernel(
    const int32_t *idx1, const int32_t *idx2, const float *d1, int64_t n,
    int32_t cols, int32_t topology, double *out2) {
    __shared__ double rq[kReduceBlock / 64], rt[kReduceBlock / 64];
    double q = 0.0, t = 0.0;
    for (int64_t i = threadIdx.x; i < n; i += kReduceBlock) {
        q += sqrt((double)d1[i]);
        const int b = idx2[i];
        if (b >= 0 && sqrt(lattice_sq(idx1[i], b, cols, topology)) > 1.0 + 1e-9) t += 1.0;
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        q += __shfl_xor(q, o, 64);
        t += __shfl_xor(t, o, 64);
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) { rq[wave] = q; rt[wave] = t; }
    __syncthreads();
    if (threadIdx.x == 0) {
        double sq = 0.0, st = 0.0;
        for (int w = 0; w < kReduceBlock / 64; ++w) { sq += rq[w]; st += rt[w]; }
        out2[0] = sq;
        out2[1] = st;
    }
}

}  // namespace

// Scratch of the evaluation entry point that allocates nothing
// (som_bmu2_noalloc): one fixed array per device, held from the code
// object's load until the process ends.  Host code never passes the array's
// name to a kernel: it is a host-side stand-in, not a device address; the
// address each device holds it at comes from hipGetSymbolAddress below.
static __device__ __align__(256) unsigned char scratch[kNoAllocScratchBytes];

hipError_t noalloc_scratch(void **ptr) {
    constexpr int kMaxDevices = 64;
    static std::mutex mu;
    static void *addr[kMaxDevices] = {};
    int dev = -1;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    if (dev < 0 || dev >= kMaxDevices) return hipErrorInvalidDevice;
    std::lock_guard<std::mutex> lock(mu);
    if (!addr[dev]) {
        void *p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        if (!p) return hipErrorInvalidSymbol;
        addr[dev] = p;
    }
    *ptr = addr[dev];
    return hipSuccess;
}

void plan_bmu_candidates(EvalArgs *a) {
    const int64_t tiles = (a->n + kBM - 1) / kBM;
    const int64_t unit_tiles = (a->N + kBN - 1) / kBN;
    // aim at two workgroups per compute unit
    int64_t g = (512 + tiles - 1) / tiles;
    if (g > unit_tiles) g = unit_tiles;
    if (g < 1) g = 1;
    const int64_t tiles_per_group = (unit_tiles + g - 1) / g;
    a->group_units = (int32_t)(tiles_per_group * kBN);
    a->ugroups = (int32_t)((a->N + a->group_units - 1) / a->group_units);
}

hipError_t launch_bmu_candidates(const EvalArgs &a, hipStream_t s) {
    const int64_t blocks = (a.n + kBM - 1) / kBM;
    if (a.ugroups < 1 || a.group_units % kBN != 0 ||
        (int64_t)a.ugroups * a.group_units < a.N)
        return hipErrorInvalidValue;
    bmu_candidates_kernel<<<dim3((unsigned)blocks, (unsigned)a.ugroups), dim3(kEvalBlock), 0, s>>>(
        a);
    return hipGetLastError();
}

hipError_t launch_bmu_rerank(const EvalArgs &a, hipStream_t s) {
    const int64_t blocks = (a.n + kRerankWaves - 1) / kRerankWaves;
    bmu_rerank_kernel<<<dim3((unsigned)blocks), dim3(64 * kRerankWaves), 0, s>>>(a);
    return hipGetLastError();
}

hipError_t launch_qe_te_reduce(const int32_t *idx1, const int32_t *idx2,
                               const float *d1, int64_t n, int32_t cols,
                               int32_t topology, double *out2, hipStream_t s) {
    qe_te_reduce_kernel<<<dim3(1), dim3(kReduceBlock), 0, s>>>(idx1, idx2, d1, n, cols,
                                                              topology, out2);
    return hipGetLastError();
}

}  // namespace som
