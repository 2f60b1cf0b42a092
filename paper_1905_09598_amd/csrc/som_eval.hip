// Batched best-matching-unit assignment and map quality (QE, TE).
//
// After training, every document is assigned to its BMU (paper Sec. 8A) and
// the map is scored by its quantization error (Sec. 6D, Sec. 8B).  Over all
// n samples this is a dense contraction: ranking units by
//     |x - w|^2 = |x|^2 - 2 x.w + |w|^2
// only needs s(x, w) = |w|^2 - 2 x.w, and X W^T is an (n x d) by (d x N)
// matrix product, computed here on the fp32 matrix cores
// (v_mfma_f32_16x16x4_f32) in tiles of kBM samples by kBN units.  Two ways
// of spreading the tiles over the chip, chosen per call by the number of
// rounds of workgroups each needs (plan_bmu_candidates):
//   * fused: a workgroup walks a group of unit tiles over the whole of d and
//     keeps, per sample, the kCand (score, unit) pairs of smallest s among
//     its units, without ever materialising the n x N matrix;
//   * split: when there are too few tiles to fill the chip, d is cut into
//     `splits` ranges and each workgroup writes the partial products of one
//     tile over one range (n x N floats per range).
// A last kernel, one wave per sample, takes the sample's kCand best units by
// score (merging the fused search's pairs, or summing the sample's partial
// products in range order) and re-ranks them by direct fp32 distances
// sum (x_j - w_j)^2, which fixes the BMU, the second BMU and the BMU's
// squared distance.
#include "som_internal.h"

#include <math.h>

#include <mutex>

namespace som {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

// Candidate kernel tiling: a workgroup owns kBM samples and kBN units and
// walks d in kBK-wide slices of X and W staged in LDS.  Its 4 waves form a
// 2 x 2 grid: 32 samples x 64 units each, i.e. 2 x 4 MFMA tiles of 16 x 16.
constexpr int kBM = 64;
constexpr int kBN = 128;
constexpr int kBK = 64;
constexpr int kPad = 4;
constexpr int kLdsStride = kBK + kPad;  // floats per staged row
constexpr int kEvalBlock = 256;

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

struct EvalSmem {
    float xs[kBM * kLdsStride];
    float ws[kBN * kLdsStride];
    float wn[kBN];
};

// acc[i][j] = x.w over columns [k_begin, k_end) for the 16 x 16 MFMA tile
// (i, j) of this wave: units u0 + wunit*64 + i*16 + 4*(lane/16) + v (v the
// f4 component) and samples s0 + wsamp*32 + j*16 + lane%16.  k_begin is a
// multiple of kBK; columns past d are zero.
// With kFull false (a unit tile that reaches past N) a wave multiplies only
// its 16-unit MFMA tiles that hold units below u_end.
template <bool kFull>
__device__ inline void tile_products(const EvalArgs &a, int64_t s0, int u0, int u_end,
                                     int k_begin, int k_end, EvalSmem &sm, f4 (&acc)[4][2]) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wsamp = wave & 1, wunit = wave >> 1;
    const int lrow = lane & 15, lk = (lane >> 4) * 4;
    int live = 4;  // MFMA unit tiles of this wave that hold units
    if (!kFull) {
        const int rest = u_end - (u0 + wunit * 64);
        live = rest <= 0 ? 0 : (rest >= 64 ? 4 : (rest + 15) / 16);
        live = __builtin_amdgcn_readfirstlane(live);
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 2; ++j) acc[i][j] = f4{0.f, 0.f, 0.f, 0.f};

    // The next kBK-wide slices of X and W are loaded into registers before
    // the current ones are multiplied, so their memory latency overlaps the
    // MFMAs.  The loads are unconditional (addresses clamped into the
    // operands); what lies outside them is zeroed as the slices go to LDS,
    // after the multiply: a select on a value in flight would make the
    // compiler wait for the load on the spot.
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
            *reinterpret_cast<f4 *>(&sm.xs[r * kLdsStride + 4 * c4]) = v;
        }
#pragma unroll
        for (int i = 0; i < kWPer; ++i) {
            const int idx = tid + i * kEvalBlock;
            const int r = idx / (kBK / 4), c4 = idx % (kBK / 4);
            const int64_t col = k0 + 4 * c4;
            const f4 zero = {0.f, 0.f, 0.f, 0.f};
            *reinterpret_cast<f4 *>(&sm.ws[r * kLdsStride + 4 * c4]) =
                (u0 + r < u_end && col < a.ld) ? wv[i] : zero;
        }
    };
    fetch(k_begin);
    for (int k0 = k_begin; k0 < k_end; k0 += kBK) {
        __syncthreads();
        stage(k0);
        __syncthreads();
        if (k0 + kBK < k_end) fetch(k0 + kBK);

#pragma unroll
        for (int kq = 0; kq < kBK; kq += 16) {
            // Lane l supplies k = kq + 4 * (l / 16) + kk at sub-step kk for
            // both operands, so one 16-byte LDS read feeds four MFMAs.
            f4 af[4], bf[2];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                if (kFull || i < live)
                    af[i] = *reinterpret_cast<const f4 *>(
                        &sm.ws[(wunit * 64 + i * 16 + lrow) * kLdsStride + kq + lk]);
#pragma unroll
            for (int j = 0; j < 2; ++j)
                bf[j] = *reinterpret_cast<const f4 *>(
                    &sm.xs[(wsamp * 32 + j * 16 + lrow) * kLdsStride + kq + lk]);
#pragma unroll
            for (int kk = 0; kk < 4; ++kk)
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    if (kFull || i < live)
#pragma unroll
                        for (int j = 0; j < 2; ++j)
                            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(
                                af[i][kk], bf[j][kk], acc[i][j], 0, 0, 0);
        }
    }
}

// Fold the scores s = |w|^2 - 2 x.w of one unit tile (products in acc,
// norms of units u0 .. in wn) into this thread's per-sample top lists.
__device__ inline void tile_insert(const f4 (&acc)[4][2], int u0, int u_end, const float *wn,
                                   float (&ts)[2][kCand], int (&tu)[2][kCand]) {
    const int lane = threadIdx.x & 63, wunit = (threadIdx.x >> 6) >> 1;
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

// Merge the 8 partial lists of each of the tile's samples (2 unit-waves x 4
// lane groups) and write its kCand (score, unit) pairs as group `grp`.
__device__ inline void write_candidates(const EvalArgs &a, int64_t s0, int grp,
                                        const float (&ts)[2][kCand], const int (&tu)[2][kCand],
                                        EvalSmem &sm) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wsamp = wave & 1, wunit = wave >> 1, lrow = lane & 15;
    __syncthreads();
    float *ps = sm.ws;                                       // kBM * 8 * kCand scores
    int *pu = reinterpret_cast<int *>(sm.ws) + kBM * 8 * kCand;  // and units
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int sl = wsamp * 32 + j * 16 + lrow;
        const int src = wunit * 4 + (lane >> 4);
#pragma unroll
        for (int c = 0; c < kCand; ++c) {
            ps[(sl * 8 + src) * kCand + c] = ts[j][c];
            pu[(sl * 8 + src) * kCand + c] = tu[j][c];
        }
    }
    __syncthreads();
    if (tid < kBM && s0 + tid < a.n) {
        float ms[kCand];
        int mu[kCand];
#pragma unroll
        for (int c = 0; c < kCand; ++c) { ms[c] = INFINITY; mu[c] = -1; }
        for (int e = 0; e < 8 * kCand; ++e) {
            const int u = pu[tid * 8 * kCand + e];
            if (u >= 0) insert_top(ms, mu, ps[tid * 8 * kCand + e], u);
        }
        int2 *out = reinterpret_cast<int2 *>(a.cand) + ((s0 + tid) * a.ugroups + grp) * kCand;
#pragma unroll
        for (int c = 0; c < kCand; ++c) out[c] = make_int2(__float_as_int(ms[c]), mu[c]);
    }
}

__device__ inline void empty_lists(float (&ts)[2][kCand], int (&tu)[2][kCand]) {
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int c = 0; c < kCand; ++c) { ts[j][c] = INFINITY; tu[j][c] = -1; }
}

// Fused form: sample tile blockIdx.x, unit group blockIdx.y (group_units
// units, walked tile by tile over all of d).  Two workgroups per compute
// unit (the register budget that allows, and the planner, assume it).
__global__ __launch_bounds__(kEvalBlock, 2) void bmu_candidates_kernel(EvalArgs a) {
    __shared__ __align__(16) EvalSmem sm;
    const int64_t s0 = (int64_t)blockIdx.x * kBM;
    const int grp = blockIdx.y;
    const int u_begin = grp * a.group_units;
    const int u_end = u_begin + a.group_units < a.N ? u_begin + a.group_units : a.N;
    float ts[2][kCand];
    int tu[2][kCand];
    empty_lists(ts, tu);
    for (int u0 = u_begin; u0 < u_end; u0 += kBN) {
        f4 acc[4][2];
        if (u0 + kBN <= u_end)
            tile_products<true>(a, s0, u0, u_end, 0, a.d, sm, acc);
        else
            tile_products<false>(a, s0, u0, u_end, 0, a.d, sm, acc);
        __syncthreads();
        if (threadIdx.x < kBN) sm.wn[threadIdx.x] = (u0 + threadIdx.x < u_end) ? a.wnorm[u0 + threadIdx.x] : 0.f;
        __syncthreads();
        tile_insert(acc, u0, u_end, sm.wn, ts, tu);
    }
    write_candidates(a, s0, grp, ts, tu, sm);
}

// Split form: the products of sample tile blockIdx.x with unit tile
// blockIdx.y over columns [z * split_len, (z + 1) * split_len) of d,
// z = blockIdx.z, stored sample-major: part[(z n + i) Np + u] for sample i
// and unit u, Np = tiles_u * kBN (each lane's four consecutive units in one
// 16-byte store).  The re-rank sums a sample's ranges in order.
__global__ __launch_bounds__(kEvalBlock, 2) void bmu_partial_kernel(EvalArgs a) {
    __shared__ __align__(16) EvalSmem sm;
    const int64_t s0 = (int64_t)blockIdx.x * kBM;
    const int u0 = blockIdx.y * kBN;
    const int u_end = u0 + kBN < a.N ? u0 + kBN : a.N;
    const int z = blockIdx.z;
    const int k_begin = z * a.split_len;
    const int k_end = k_begin + a.split_len < a.d ? k_begin + a.split_len : a.d;
    f4 acc[4][2];
    if (u0 + kBN <= u_end)
        tile_products<true>(a, s0, u0, u_end, k_begin, k_end, sm, acc);
    else
        tile_products<false>(a, s0, u0, u_end, k_begin, k_end, sm, acc);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int wsamp = wave & 1, wunit = wave >> 1;
    const int64_t np = (int64_t)a.tiles_u * kBN;
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int64_t smp = s0 + wsamp * 32 + j * 16 + (lane & 15);
        if (smp >= a.n) continue;
        f4 *row = reinterpret_cast<f4 *>(a.part + ((int64_t)z * a.n + smp) * np +
                                         u0 + wunit * 64 + (lane >> 4) * 4);
#pragma unroll
        for (int i = 0; i < 4; ++i) row[i * 4] = acc[i][j];
    }
}

// Unsigned key ordered like (score, unit): the score's bits mapped so that
// unsigned order is numeric order (NaN last), then the unit.
__device__ inline unsigned long long cand_key(float s, int u) {
    uint32_t b = __float_as_uint(s);
    b = (s != s) ? 0xffffffffu : ((b & 0x80000000u) ? ~b : (b | 0x80000000u));
    return ((unsigned long long)b << 32) | (uint32_t)u;
}

__device__ inline unsigned long long wave_min_u64(unsigned long long k) {
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) {
        const unsigned long long v = __shfl_xor(k, o, 64);
        k = v < k ? v : k;
    }
    return k;
}

// One wave per sample.  Its candidates: the kCand best by (score, unit)
// among the ugroups * kCand pairs of the fused search, or, when d was
// split, among all units, from the sample's rows of partial products
// (summed in range order).  Their exact fp32 distances (one pass over x and
// the kCand rows) then give the best and second best by (distance, unit).
constexpr int kRerankWaves = 4;
__global__ __launch_bounds__(64 * kRerankWaves) void bmu_rerank_kernel(EvalArgs a) {
    const int lane = threadIdx.x & 63;
    const int64_t i = (int64_t)blockIdx.x * kRerankWaves + (threadIdx.x >> 6);
    if (i >= a.n) return;
    float ls[kCand];
    int lu[kCand];
#pragma unroll
    for (int c = 0; c < kCand; ++c) { ls[c] = INFINITY; lu[c] = -1; }
    if (a.splits > 1) {
        // each lane's best units among 4 q .. 4 q + 3, q = lane, lane + 64, ...
        const int64_t np = (int64_t)a.tiles_u * kBN;
        const int nq = (a.N + 3) / 4;
        const f4 *row = reinterpret_cast<const f4 *>(a.part + i * np);
        const int64_t zstride = (int64_t)a.n * np / 4;
        // (the norms are read as float4: the array holds roundup(N, 4) floats)
        const f4 *wn4 = reinterpret_cast<const f4 *>(a.wnorm);
        for (int q0 = 0; q0 < nq; q0 += 64 * 4) {
            f4 dot[4], wn[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int q = q0 + lane + 64 * k;
                dot[k] = f4{0.f, 0.f, 0.f, 0.f};
                wn[k] = q < nq ? wn4[q] : f4{0.f, 0.f, 0.f, 0.f};
            }
            for (int z = 0; z < a.splits; ++z) {
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    const int q = q0 + lane + 64 * k;
                    if (q < nq) {
                        const f4 v = row[z * zstride + q];
                        dot[k] = z == 0 ? v : dot[k] + v;
                    }
                }
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int q = q0 + lane + 64 * k;
#pragma unroll
                for (int e = 0; e < 4; ++e) {
                    const int u = 4 * q + e;
                    if (q < nq && u < a.N) insert_top(ls, lu, wn[k][e] - 2.f * dot[k][e], u);
                }
            }
        }
    } else {
        const int nc = a.ugroups * kCand;
        const int2 *cp = reinterpret_cast<const int2 *>(a.cand) + i * nc;
        for (int e = lane; e < nc; e += 64) {
            const int2 p = cp[e];
            if (p.y >= 0) insert_top(ls, lu, __int_as_float(p.x), p.y);
        }
    }
    // kCand rounds of a wave-wide minimum over the lanes' list heads
    int cu[kCand];
#pragma unroll
    for (int c = 0; c < kCand; ++c) {
        const unsigned long long mine = lu[0] >= 0 ? cand_key(ls[0], lu[0]) : ~0ull;
        const unsigned long long win = wave_min_u64(mine);
        cu[c] = win == ~0ull ? -1 : (int)(uint32_t)win;
        if (mine == win && win != ~0ull) {
#pragma unroll
            for (int q = 0; q < kCand - 1; ++q) { ls[q] = ls[q + 1]; lu[q] = lu[q + 1]; }
            ls[kCand - 1] = INFINITY;
            lu[kCand - 1] = -1;
        }
    }
    // exact distances to the kCand units in one pass over x
    float acc[kCand];
    const float *wr[kCand];
#pragma unroll
    for (int c = 0; c < kCand; ++c) {
        acc[c] = 0.f;
        wr[c] = a.W + (int64_t)(cu[c] >= 0 ? cu[c] : 0) * a.ld;
    }
    const float *x = a.X + i * a.d;
    int64_t j0 = 0;
    if (a.x_vec4) {
        const int64_t d4 = a.d / 4;
        for (int64_t j = lane; j < d4; j += 64) {
            const f4 xv = reinterpret_cast<const f4 *>(x)[j];
#pragma unroll
            for (int c = 0; c < kCand; ++c) {
                const f4 df = xv - reinterpret_cast<const f4 *>(wr[c])[j];
                acc[c] = fmaf(df[0], df[0], acc[c]);
                acc[c] = fmaf(df[1], df[1], acc[c]);
                acc[c] = fmaf(df[2], df[2], acc[c]);
                acc[c] = fmaf(df[3], df[3], acc[c]);
            }
        }
        j0 = d4 * 4;
    }
    for (int64_t j = j0 + lane; j < a.d; j += 64) {
        const float xj = x[j];
#pragma unroll
        for (int c = 0; c < kCand; ++c) {
            const float df = xj - wr[c][j];
            acc[c] = fmaf(df, df, acc[c]);
        }
    }
#pragma unroll
    for (int c = 0; c < kCand; ++c)
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) acc[c] += __shfl_xor(acc[c], o, 64);
    float bd = INFINITY, sd = INFINITY;
    int bu = -1, su = -1;
#pragma unroll
    for (int c = 0; c < kCand; ++c) {
        const int u = cu[c];
        if (u < 0) continue;
        if (better(acc[c], u, bd, bu)) {
            sd = bd; su = bu;
            bd = acc[c]; bu = u;
        } else if (better(acc[c], u, sd, su)) {
            sd = acc[c]; su = u;
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

// Cost of a plan in units of one kBK-wide slice of one tile on a
// workgroup (about 4.3 us with two workgroups per compute unit, measured on
// MI355X), for `slots` co-resident workgroups.  Workgroups run in rounds;
// each costs its slices plus a fixed start and finish.
namespace {
constexpr double kWgFixed = 0.6;      // first loads, candidate merge, stores
constexpr double kPairCost = 2e-6;    // per (score, unit) pair the re-rank merges

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
}  // namespace

bool plan_bmu_candidates(EvalArgs *a, int num_cus, uint64_t max_scratch_bytes) {
    const int64_t slots = 2 * (int64_t)(num_cus > 0 ? num_cus : 1);
    const int64_t tiles_s = ceil_div(a->n, kBM);
    const int64_t tiles_u = ceil_div(a->N, kBN);
    const int64_t slices = ceil_div(a->d, kBK);
    double best = 1e300;
    a->tiles_s = (int32_t)tiles_s;
    a->tiles_u = (int32_t)tiles_u;
    // fused: g groups of tpg unit tiles, one workgroup per (sample tile, group)
    for (int64_t tpg = tiles_u; tpg >= 1; --tpg) {
        const int64_t g = ceil_div(tiles_u, tpg);
        const uint64_t cand = (uint64_t)a->n * g * kCand * 8;
        if (cand > max_scratch_bytes) break;  // more groups only grow the lists
        const double cost = ceil_div(tiles_s * g, slots) * ((double)tpg * slices + kWgFixed) +
                            (double)a->n * g * kCand * kPairCost;
        if (cost < best) {
            best = cost;
            a->splits = 1;
            a->split_len = a->d;
            a->ugroups = (int32_t)g;
            a->group_units = (int32_t)(tpg * kBN);
        }
    }
    // split: every (sample tile, unit tile, range of d) a workgroup
    for (int64_t S = 2; S <= 16 && S <= slices; ++S) {
        const int64_t chunk = ceil_div(slices, S);
        const int64_t Se = ceil_div(slices, chunk);
        if (Se != S) continue;
        const uint64_t part = (uint64_t)Se * a->n * tiles_u * kBN * 4;
        if (part > max_scratch_bytes) continue;
        // the partial products go out and come back at about 5 TB/s
        const double traffic = 2.0 * (double)part / 5e12 / 4.3e-6;
        const double cost = ceil_div(tiles_s * tiles_u * Se, slots) * ((double)chunk + kWgFixed) +
                            traffic;
        if (cost < best) {
            best = cost;
            a->splits = (int32_t)Se;
            a->split_len = (int32_t)(chunk * kBK);
            a->ugroups = 0;
            a->group_units = 0;
        }
    }
    return best < 1e300;
}

int64_t bmu_cand_ints(const EvalArgs &a) {
    return a.splits > 1 ? 0 : a.n * (int64_t)a.ugroups * kCand * 2;
}

int64_t bmu_part_floats(const EvalArgs &a) {
    return a.splits > 1 ? (int64_t)a.splits * a.n * a.tiles_u * kBN : 0;
}

hipError_t launch_bmu_candidates(const EvalArgs &a, hipStream_t s) {
    if (a.tiles_s != ceil_div(a.n, kBM) || a.tiles_u != ceil_div(a.N, kBN))
        return hipErrorInvalidValue;
    if (a.splits <= 1) {
        if (a.ugroups < 1 || a.group_units % kBN != 0 ||
            (int64_t)a.ugroups * a.group_units < a.N || !a.cand)
            return hipErrorInvalidValue;
        bmu_candidates_kernel<<<dim3((unsigned)a.tiles_s, (unsigned)a.ugroups), dim3(kEvalBlock),
                                0, s>>>(a);
        return hipGetLastError();
    }
    if (!a.part || a.split_len % kBK != 0 ||
        (int64_t)a.splits * a.split_len < a.d || (int64_t)(a.splits - 1) * a.split_len >= a.d)
        return hipErrorInvalidValue;
    bmu_partial_kernel<<<dim3((unsigned)a.tiles_s, (unsigned)a.tiles_u, (unsigned)a.splits),
                         dim3(kEvalBlock), 0, s>>>(a);
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
