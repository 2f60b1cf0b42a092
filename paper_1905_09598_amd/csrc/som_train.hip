// Persistent online-SOM training kernel for gfx950 (MI355X).
//
// One cooperative launch runs every step of a som_train call (paper Sec. 6C
// runs three kernels and a host round trip per sample; here the per-sample
// loop never leaves the device).  Each workgroup owns a fixed, contiguous
// range of prototype rows for the whole launch, so a row is only ever read
// and written by one workgroup (and so by one XCD and its L2).  The rows
// live either in device memory (variant "stream") or in the workgroup's LDS
// for the whole launch, loaded at the start and written back at the end
// (variant "lds", when the slice fits).
//
// Blocked sweeps.  Eq. (1) applied for steps k = 0..M-1 of a block keeps
// every prototype an affine combination of its value W at the block start
// and the block's samples x_0..x_{M-1}:
//     W^(k) = beta_k W + sum_{j<k} gamma_kj x_j,   beta_k + sum_j gamma_kj = 1,
// with beta_{k+1} = (1 - h_k) beta_k, gamma_{k+1,j} = (1 - h_k) gamma_kj and
// gamma_{k+1,k} = h_k, h_k the unit's neighbourhood factor at step k.  So
//     x_k - W^(k) = e_k - sum_{j<k} gamma_kj e_j,   e_j = x_j - W,
// and the squared distance that picks step k's BMU is
//     D_k = E_kk - 2 sum_j gamma_kj E_jk + sum_ij gamma_ki gamma_kj E_ij
// with E the Gram matrix of the e_j, per unit.  One sweep over the owned rows
// therefore (a) applies a whole block's updates at once,
// w <- beta w + sum_j gamma_j x_j, and (b) accumulates the Gram matrix of the
// next block's samples against the updated rows.  Between sweeps the M BMUs
// of a block come from these per-unit scalars alone.  This is Eq. (1)
// step by step in exact arithmetic, with one pass over the prototypes per M
// samples; the first distance of each block is the plain direct-difference
// squared distance E_00.
//
// Per step the workgroup's (distance, unit) minimum goes to a grid exchange:
// one 64-bit slot per workgroup and parity, dist_bits << 32 | tag << 24 |
// unit, written and polled with relaxed device-scope atomics only (no fences,
// so no cache write-back or invalidation).  The slot array is replicated once
// per XCD and each workgroup polls its XCD's copy, which cuts the number of
// pollers per cache line eightfold; slots are spread over cache lines.  The minimum over slots with the
// current tag is the minimum over (distance, unit): squared distances are
// non-negative, so their IEEE bits order like the values, and equal distances
// fall to the lowest unit.  Slots alternate by step parity, so a fast
// workgroup can publish step e+1 while a slow one still reads step e.  Every
// wait is bounded in time and also ends when any workgroup has flagged an
// error.
#include "som_device.h"

namespace som {
namespace {

using namespace dev;

constexpr int kHeader = 64;  // LDS bytes for the broadcast words

// Lane layout.  A workgroup's 256 threads form P = 256 / L groups of L
// lanes; group g sweeps rows g, g + P, g + 2P, ... of the workgroup's slice,
// and lane j of a group holds the 16-byte columns j, j + L, ..., j + (K-1) L
// of its rows and of the samples.  The row pitch is padded with zeros to
// exactly L * K columns, so the sweep has no column bounds.

// Load the M samples of the block starting at call step s_begin (steps past
// the end load sample 0; their coefficients stay zero).
template <int K, int L, int M>
__device__ inline void load_block(f4 (&x)[M][K], const TrainArgs &a, int64_t s_begin,
                                  StepWindow<int> &ow) {
#pragma unroll
    for (int j = 0; j < M; ++j) {
        const int64_t s = s_begin + j;
        const int i = (s < a.nsteps) ? ow.get(a, s) : 0;
        load_sample<K, L>(x[j], a, i);
    }
}

// One pass over R rows.  UPD applies the block's updates from coef[r] =
// (beta, gamma_0..gamma_{M-1}); GRAM accumulates the Gram matrix of
// e_j = xg_j - w over the (updated) row into E[r] (or, with more than one
// wave per row, the wave's partials into part[(r * T + t) * WPR + w]).
// Callers sweeping a part of the rows pass coef, E and part advanced to its
// first row.
template <int K, int L, int M, int U, bool LDSW, bool UPD, bool GRAM>
__device__ inline void sweep(f4 *rows_p, int R, const f4 (&xu)[M][K], const f4 (&xg)[M][K],
                             const float *coef, float *E, float *part) {
    if (R <= 0) return;
    row_t<LDSW> *__restrict__ rows = rows_as<LDSW>(rows_p);
    constexpr int P = kTrainBlock / L;
    constexpr int P4 = L * K;
    constexpr int T = M * (M + 1) / 2;
    constexpr int WPR = L / 64;
    const int tid = threadIdx.x, g = tid / L, li = tid % L, lane = tid & 63, wig = li >> 6;
    for (int rb = g; rb < R; rb += P * U) {
        f4 w[U][K];
        // unconditional loads (clamped row, unused past R): see load_f4_or_zero
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = rb + u * P < R ? rb + u * P : R - 1;
            const row_t<LDSW> *row = rows + (size_t)r * P4 + li;
#pragma unroll
            for (int k = 0; k < K; ++k) w[u][k] = row[L * k];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int r = rb + u * P;
            if (r >= R) continue;
            row_t<LDSW> *row = rows + (size_t)r * P4 + li;
            float beta = 1.f, gam[M];
#pragma unroll
            for (int j = 0; j < M; ++j) gam[j] = 0.f;
            if (UPD) {
                beta = coef[r * (M + 1)];
#pragma unroll
                for (int j = 0; j < M; ++j) gam[j] = coef[r * (M + 1) + 1 + j];
            }
            float acc[T];
#pragma unroll
            for (int t = 0; t < T; ++t) acc[t] = 0.f;
#pragma unroll
            for (int k = 0; k < K; ++k) {
                f4 v = w[u][k];
                if (UPD) {
                    v = v * beta;
#pragma unroll
                    for (int j = 0; j < M; ++j) {
                        v.x = fmaf(gam[j], xu[j][k].x, v.x);
                        v.y = fmaf(gam[j], xu[j][k].y, v.y);
                        v.z = fmaf(gam[j], xu[j][k].z, v.z);
                        v.w = fmaf(gam[j], xu[j][k].w, v.w);
                    }
                    row[L * k] = v;
                }
                if (GRAM) {
                    f4 e[M];
#pragma unroll
                    for (int j = 0; j < M; ++j) e[j] = xg[j][k] - v;
#pragma unroll
                    for (int j = 0; j < M; ++j)
#pragma unroll
                        for (int i = 0; i <= j; ++i) {
                            float t = acc[tri(i, j)];
                            t = fmaf(e[i].x, e[j].x, t);
                            t = fmaf(e[i].y, e[j].y, t);
                            t = fmaf(e[i].z, e[j].z, t);
                            t = fmaf(e[i].w, e[j].w, t);
                            acc[tri(i, j)] = t;
                        }
                }
            }
            if (GRAM) {
                constexpr int NT = (T + 3) / 4;
                float tot[NT];
                wave_sums_rows<T>(acc, tot);
                if ((lane & 15) == 0) {
                    // lane 16 q writes the sums its row holds
                    const int q = lane >> 4;
#pragma unroll
                    for (int j = 0; j < NT; ++j) {
                        const int t = 4 * j + 2 * (q & 1) + (q >> 1);  // sum_row(t) == q
                        if (t < T) {
                            if (WPR == 1) E[r * T + t] = tot[j];
                            else part[(r * T + t) * WPR + wig] = tot[j];
                        }
                    }
                }
            }
        }
    }
}

// A pass over the workgroup's R rows: rows [0, RL) in LDS and, in the
// streamed variant (LDSW false), rows [RL, R) in memory at gs.
template <int K, int L, int M, int U, bool LDSW, bool UPD, bool GRAM>
__device__ inline void sweep_rows(f4 *lw, int RL, f4 *gs, int R, const f4 (&xu)[M][K],
                                  const f4 (&xg)[M][K], const float *coef, float *E,
                                  float *part) {
    constexpr int T = M * (M + 1) / 2;
    constexpr int WPR = L / 64;
    sweep<K, L, M, U, true, UPD, GRAM>(lw, RL, xu, xg, coef, E, part);
    if constexpr (!LDSW)
        sweep<K, L, M, U, false, UPD, GRAM>(gs, R - RL, xu, xg, coef + (size_t)RL * (M + 1),
                                            E + (size_t)RL * T, part + (size_t)RL * T * WPR);
}

// Wave 0 only: the BMUs of the block's mb steps, s0 .. s0 + mb - 1, from the
// Gram matrices E of the owned rows (LDS), leaving each row's update
// coefficients (beta, gamma_0..) in coef.  Returns false if an exchange
// was given up.
template <int L, int M>
__device__ inline bool block_bmus(const TrainArgs &a, int64_t s0, int mb, int r0, int R,
                                  float *E, const float *part, float *coef, const float4 *pos,
                                  StepWindow<float2> &sw) {
    constexpr int T = M * (M + 1) / 2;
    constexpr int WPR = L / 64;
    // Polls in flight per exchange.  One-wave workgroups hold their sample
    // blocks across the exchange, and one poll at a time keeps those in
    // registers.
    constexpr int kPolls = L == 64 ? 1 : 4;
    PollRegs<kPolls> pr{};  // exchange poll registers, held between this block's exchanges
    const int lane = threadIdx.x & 63;
    const float inv_cols = 1.f / (float)a.cols;
    if (WPR > 1) {
        for (int idx = lane; idx < R * T; idx += 64) {
            float v = part[idx * WPR];
#pragma unroll
            for (int w = 1; w < WPR; ++w) v += part[idx * WPR + w];
            E[idx] = v;
        }
    }
    if (R <= 64) {
        // Lane r keeps row r's Gram matrix and coefficients in registers.
        float Er[T], gam[M], beta;
        float4 p = make_float4(0.f, 0.f, 0.f, 0.f);
#pragma unroll
        for (int t = 0; t < T; ++t) Er[t] = lane < R ? E[lane * T + t] : 0.f;
        if (lane < R) p = pos[lane];
        const bool ok = block_steps<M, kPolls>(a, s0, mb, r0, R, Er, p, inv_cols, sw, beta, gam, pr);
        if (lane < R) {
            coef[lane * (M + 1)] = beta;
#pragma unroll
            for (int j = 0; j < M; ++j) coef[lane * (M + 1) + 1 + j] = gam[j];
        }
        return ok;
    }
    for (int r = lane; r < R; r += 64) {
        coef[r * (M + 1)] = 1.f;
#pragma unroll
        for (int j = 0; j < M; ++j) coef[r * (M + 1) + 1 + j] = 0.f;
    }
#pragma unroll
    for (int k = 0; k < M; ++k) {
        if (k >= mb) break;
        const int64_t s = s0 + k;
        unsigned long long best = ~0ull;
        for (int r = lane; r < R; r += 64) {
            const float *Er = E + r * T;
            const float *gr = coef + r * (M + 1) + 1;
            float lin = 0.f, quad = 0.f;
#pragma unroll
            for (int j = 0; j < k; ++j) {
                float inner = 0.f;
#pragma unroll
                for (int i = 0; i < k; ++i) inner = fmaf(gr[i], Er[tri_any(i, j)], inner);
                lin = fmaf(gr[j], Er[tri(j, k)], lin);
                quad = fmaf(gr[j], inner, quad);
            }
            const float D = fmaf(-2.f, lin, Er[tri(k, k)]) + quad;
            best = u64_min(best, row_key(D, r0 + r));
        }
        best = wave_min_key(best, false);
        const int c = exchange<kPolls>(a, s, best, pr);
        if (c < 0) return false;
        if (blockIdx.x == 0 && lane == 0 && a.bmu_trace) a.bmu_trace[s] = c;
        const float2 sc = sw.get(a, s);
        int cr, ccol;
        unit_rc(c, a.cols, inv_cols, cr, ccol);
        const float fcr = (float)cr, fcc = (float)ccol, fcp = (float)(cr & 1);
        for (int r = lane; r < R; r += 64) {
            const float h = neighbour_h(a, pos[r], fcr, fcc, fcp, sc.x, sc.y);
            const float om = 1.f - h;
            float *cf = coef + r * (M + 1);
            cf[0] *= om;
#pragma unroll
            for (int j = 0; j < k; ++j) cf[1 + j] *= om;
            cf[1 + k] = h;
        }
    }
    return true;
}

struct Layout {
    int Rp;
    float *E, *part, *coef;
    float4 *pos;
    f4 *lw;
};

template <int K, int L, int M>
__device__ inline Layout layout(unsigned char *smem, int R) {
    constexpr int T = M * (M + 1) / 2;
    constexpr int WPR = L / 64;
    Layout l;
    l.Rp = (R + 3) & ~3;
    unsigned char *p = smem + kHeader;
    l.E = reinterpret_cast<float *>(p);
    p += (size_t)l.Rp * T * 4;
    l.part = reinterpret_cast<float *>(p);
    if (WPR > 1) p += (size_t)l.Rp * T * WPR * 4;
    l.coef = reinterpret_cast<float *>(p);
    p += (size_t)l.Rp * (M + 1) * 4;
    p = reinterpret_cast<unsigned char *>((reinterpret_cast<uintptr_t>(p) + 15) & ~(uintptr_t)15);
    l.pos = reinterpret_cast<float4 *>(p);
    p += (size_t)l.Rp * 16;
    l.lw = reinterpret_cast<f4 *>(p);
    return l;
}

// One block: its BMUs (wave 0), then one sweep that applies the block's
// updates with samples xu and accumulates the next block's Gram matrices
// with samples xg, then the samples of the block after next go into xu.
template <int K, int L, int M, int U, bool LDSW>
__device__ inline bool run_block(const TrainArgs &a, int64_t blk, int64_t nblocks, int r0,
                                 int R, int RL, f4 *gs, const Layout &l, f4 (&xu)[M][K],
                                 const f4 (&xg)[M][K], StepWindow<int> &ow,
                                 StepWindow<float2> &sw, Bcast *bc) {
    const int wave = threadIdx.x >> 6;
    const int64_t s0 = blk * M;
    const int mb = (int)((a.nsteps - s0) < M ? (a.nsteps - s0) : M);
    if (wave == 0) {
        const bool ok = block_bmus<L, M>(a, s0, mb, r0, R, l.E, l.part, l.coef, l.pos, sw);
        if ((threadIdx.x & 63) == 0) bc->abort = ok ? 0 : 1;
    }
    __syncthreads();
    if (bc->abort) return false;
    if (blk + 1 < nblocks)
        sweep_rows<K, L, M, U, LDSW, true, true>(l.lw, RL, gs, R, xu, xg, l.coef, l.E, l.part);
    else
        sweep_rows<K, L, M, U, LDSW, true, false>(l.lw, RL, gs, R, xu, xg, l.coef, l.E, l.part);
    if (blk + 2 < nblocks) load_block<K, L, M>(xu, a, (blk + 2) * M, ow);
    __syncthreads();
    return true;
}

template <int K, int L, int M, int U, bool LDSW>
__global__ __launch_bounds__(kTrainBlock, 1) void train_kernel(TrainArgs a) {
    extern __shared__ __align__(16) unsigned char smem[];
    const int G = a.grid, b = blockIdx.x, tid = threadIdx.x;
    const int r0 = (int)(((int64_t)b * a.N) / G);
    const int r1 = (int)(((int64_t)(b + 1) * a.N) / G);
    const int R = r1 - r0;
    constexpr int P4 = L * K;
    Bcast *bc = reinterpret_cast<Bcast *>(smem);
    const Layout l = layout<K, L, M>(smem, R);

    if (a.state->order_bad) return;  // same value for every workgroup
    if (a.nsteps <= 0) return;

    for (int r = tid; r < R; r += kTrainBlock) {
        const int u = r0 + r, ur = u / a.cols, uc = u - ur * a.cols;
        l.pos[r] = make_float4((float)ur, (float)uc, (float)(ur & 1), 0.f);
    }
    f4 *gw = reinterpret_cast<f4 *>(a.W) + (int64_t)r0 * P4;
    // Rows [0, RL) live in LDS for the whole launch; the streamed variant
    // keeps as many as its LDS holds (planner) and streams the rest.
    const int RL = LDSW ? R : (a.lds_rows < R ? (a.lds_rows > 0 ? a.lds_rows : 0) : R);
    for (int e = tid; e < RL * P4; e += kTrainBlock) l.lw[e] = gw[e];
    f4 *gs = gw + (int64_t)RL * P4;  // first streamed row

    StepWindow<int> ow;      // sample indices
    StepWindow<float2> sw;   // schedule entries (wave 0)
    ow.init(a, 0);
    sw.init(a, 0);
    const int64_t nblocks = (a.nsteps + M - 1) / M;
    f4 xA[M][K], xB[M][K];
    load_block<K, L, M>(xA, a, 0, ow);
    if (nblocks > 1) load_block<K, L, M>(xB, a, M, ow);
    __syncthreads();
    // Gram matrices of block 0 against the initial prototypes.
    sweep_rows<K, L, M, U, LDSW, false, true>(l.lw, RL, gs, R, xA, xA, l.coef, l.E, l.part);
    __syncthreads();

    for (int64_t blk = 0; blk < nblocks; blk += 2) {
        if (!run_block<K, L, M, U, LDSW>(a, blk, nblocks, r0, R, RL, gs, l, xA, xB, ow, sw, bc))
            return;
        if (blk + 1 < nblocks &&
            !run_block<K, L, M, U, LDSW>(a, blk + 1, nblocks, r0, R, RL, gs, l, xB, xA, ow, sw,
                                         bc))
            return;
    }
    for (int e = tid; e < RL * P4; e += kTrainBlock) gw[e] = l.lw[e];
}

typedef void (*TrainKernel)(TrainArgs);

struct Instance {
    int lanes, k, m;
    TrainKernel stream, lds;
};

template <int L, int K, int M, int U>
constexpr Instance instance() {
    return Instance{L, K, M, train_kernel<K, L, M, U, false>, train_kernel<K, L, M, U, true>};
}

// Row pitch L * K float4 (d up to 4 L K floats) and block length M, sized so
// the two blocks of samples (2 M K float4 per lane) stay in registers, the
// longer rows' ones partly in the accumulation registers.  A longer block
// reads and writes the streamed rows once for more steps (measured on
// MI355X with 256 workgroups: 6.0k floats 4.96 -> 4.60 us per step from
// M = 2 to 4, 8.0k 10.2 -> 7.7, 10k 13.7 -> 10.5 from M = 2 to 3, 12k and
// 16k 28.8 -> 16.6 and 41.6 -> 23.1 from M = 1 to 2).  Per row length
// (lanes x k) the first instance is preferred; later ones of the same row
// length (shorter blocks, less LDS per owned row) serve maps whose
// workgroups own too many rows for the first.
const Instance kInstances[] = {
    instance<64, 1, 8, 1>(),   instance<64, 1, 4, 1>(),   instance<64, 1, 2, 1>(),
    instance<64, 2, 8, 1>(),   instance<64, 4, 4, 1>(),
    instance<128, 4, 4, 2>(),  instance<256, 3, 4, 1>(),  instance<256, 4, 4, 1>(),
    instance<256, 5, 3, 1>(),  instance<256, 6, 4, 1>(),  instance<256, 6, 2, 1>(),
    instance<256, 8, 4, 1>(),  instance<256, 8, 2, 1>(),  instance<256, 10, 3, 1>(),
    instance<256, 10, 2, 1>(), instance<256, 12, 2, 1>(), instance<256, 12, 1, 1>(),
    instance<256, 16, 2, 1>(), instance<256, 16, 1, 1>(),
};

const Instance *pick(int64_t ld4) {
    for (const Instance &in : kInstances)
        if ((int64_t)in.k * in.lanes >= ld4) return &in;
    return nullptr;
}

size_t lds_bytes_for(const Instance &in, int rmax, bool ldsw) {
    const size_t rp = (size_t)((rmax + 3) & ~3);
    const size_t T = (size_t)in.m * (in.m + 1) / 2, wpr = in.lanes / 64;
    size_t b = kHeader + rp * T * 4 + (wpr > 1 ? rp * T * wpr * 4 : 0) + rp * (in.m + 1) * 4;
    b = (b + 15) & ~(size_t)15;
    b += rp * 16;
    if (ldsw) b += (size_t)rmax * in.lanes * in.k * 16;
    return b;
}

// Estimated microseconds per step, from MI355X measurements; only ranks
// launch shapes.  Exchange latency by grid size (replicated, spread slots).
double exchange_us_impl(int g) {
    static const double gs[] = {1, 8, 32, 64, 128, 256, 1024};
    static const double us[] = {0.1, 1.1, 1.3, 1.35, 1.7, 2.5, 6.0};
    if (g <= 1) return us[0];
    for (int i = 1; i < 7; ++i)
        if (g <= gs[i]) {
            const double f = (log2((double)g) - log2(gs[i - 1])) / (log2(gs[i]) - log2(gs[i - 1]));
            return us[i - 1] + f * (us[i] - us[i - 1]);
        }
    return us[6];
}

// Sweep time per step: VALU issue of the rows of one lane group (4 cycles
// per wave64 instruction at 2.4 GHz) and, for the streamed rows (all but
// the rl kept in LDS), memory traffic at about 30 GB/s per CU; both spread
// over the block's M steps.
double sweep_us(const Instance &in, int rmax, bool ldsw, int rl) {
    const double P = 256.0 / in.lanes, M = in.m, T = M * (M + 1) / 2;
    const double rows = ceil(rmax / P);
    const double instr_per_row = in.k * (4 * M + 4 * T + 4 * (M + 1)) + 12 * T + 20;
    const double valu = rows * instr_per_row * 4 / 2400.0;
    const double mem = ldsw ? 0.0 : (rmax - rl) * 2.0 * 16.0 * in.lanes * in.k / 30e3;
    return (valu > mem ? valu : mem) / M + 1.0 / M;
}

}  // namespace

int64_t train_row_pitch(int32_t d) {
    const Instance *in = pick(((int64_t)d + 3) / 4);
    return in ? 4 * (int64_t)in->lanes * in->k : 0;
}

hipError_t plan_train(const TrainArgs &a, int num_cus, TrainPlan *plan) {
    const int64_t ld4 = a.ld / 4;
    int max_lds = 0;
    hipError_t e = hipDeviceGetAttribute(&max_lds, hipDeviceAttributeMaxSharedMemoryPerBlock, 0);
    if (e != hipSuccess) return e;
    const int max_grid = a.N < num_cus ? a.N : num_cus;
    // first instance of this row length whose per-row state fits in LDS at
    // the largest grid (or the requested one), of the requested block
    // length when the build has one that fits
    const Instance *in = nullptr;
    {
        const int g = a.grid > 0 ? (a.grid < a.N ? a.grid : a.N) : max_grid;
        const int rmax = (a.N + g - 1) / g;
        for (int pass = a.block_m > 0 ? 0 : 1; pass < 2 && !in; ++pass)
            for (const Instance &c : kInstances)
                if ((int64_t)c.lanes * c.k == ld4 && (pass == 1 || c.m == a.block_m) &&
                    lds_bytes_for(c, rmax, false) <= (size_t)max_lds) {
                    in = &c;
                    break;
                }
    }
    if (!in) return hipErrorInvalidValue;

    // The streamed variant keeps as many leading rows per workgroup in LDS
    // as fit beside its per-row state (or a.lds_rows when set).
    const int64_t row_bytes = (int64_t)in->lanes * in->k * 16;
    auto lds_rows_for = [&](int rmax) {
        const int64_t base = (int64_t)lds_bytes_for(*in, rmax, false);
        int64_t rl = base < max_lds ? ((int64_t)max_lds - base) / row_bytes : 0;
        if (rl > rmax) rl = rmax;
        if (a.lds_rows >= 0 && a.lds_rows < rl) rl = a.lds_rows;
        return (int)rl;
    };
    int grid = 0, variant = 0;
    if (a.grid > 0) {
        grid = a.grid < a.N ? a.grid : a.N;
        const int rmax = (a.N + grid - 1) / grid;
        variant = (a.variant != 2 && lds_bytes_for(*in, rmax, true) <= (size_t)max_lds) ? 1 : 0;
        if (a.variant == 1 && variant == 0) return hipErrorInvalidValue;
    } else {
        double best = 1e300;
        for (int v = 1; v >= 0; --v) {  // LDS first: it wins ties
            if ((v == 0 && a.variant == 1) || (v == 1 && a.variant == 2)) continue;
            for (int g = 1;; g = g * 2 > max_grid && g < max_grid ? max_grid : g * 2) {
                const int rmax = (a.N + g - 1) / g;
                if (v == 0 || lds_bytes_for(*in, rmax, true) <= (size_t)max_lds) {
                    const double t = exchange_us_impl(g) +
                                     sweep_us(*in, rmax, v == 1, v == 1 ? rmax : lds_rows_for(rmax)) +
                                     0.3;
                    if (t < best) { best = t; grid = g; variant = v; }
                }
                if (g >= max_grid) break;
            }
        }
    }
    if (grid < 1) grid = 1;
    const int rmax = (a.N + grid - 1) / grid;
    const int lds_rows = variant == 1 ? 0 : lds_rows_for(rmax);
    size_t lds = lds_bytes_for(*in, rmax, variant == 1) + (size_t)lds_rows * row_bytes;
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
    if (grid > kMaxTrainGrid) return hipErrorCooperativeLaunchTooLarge;
    // The pipelined kernel, which overlaps the pass over the prototypes with
    // the exchanges, is used wherever its shape limits allow (measured faster
    // on every such workload); variant 5 keeps this kernel, 3 / 4 require the
    // pipelined one.
    if (a.variant == 0 || a.variant == 3 || a.variant == 4) {
        TrainPlan pp;
        TrainArgs ap = a;
        ap.variant = a.variant >= 3 ? a.variant - 2 : 0;
        const double tp = plan_train_pipe(ap, num_cus, max_lds, &pp);
        if (tp < 1e300) {
            *plan = pp;
            return hipSuccess;
        }
        if (a.variant >= 3) return hipErrorInvalidValue;
    }
    plan->grid = grid;
    // Measured on MI355X.  One-poll exchanges (one-wave workgroups): one
    // slot per 128-byte line is fastest up to 64 workgroups, 32-byte spacing
    // beyond.  Multi-poll exchanges: packed slots (fewer lines per poll).
    plan->slot_spread = in->lanes == 64 ? (grid <= 64 ? 16 : 4) : 1;
    plan->block = kTrainBlock;
    plan->variant = variant;
    plan->kslots = in->k;
    plan->block_m = in->m;
    plan->lds_rows = lds_rows;
    plan->lds_bytes = lds;
    return hipSuccess;
}

hipError_t launch_train(const TrainArgs &a, const TrainPlan &plan, hipStream_t s) {
    if (plan.absent < 0 || plan.absent >= plan.grid) return hipErrorInvalidValue;
    if (plan.variant >= 2) return launch_train_pipe(a, plan, s);
    const Instance *in = nullptr;
    for (const Instance &c : kInstances)
        if ((int64_t)c.lanes * c.k == a.ld / 4 && c.m == plan.block_m) {
            in = &c;
            break;
        }
    if (!in || in->k != plan.kslots) return hipErrorInvalidValue;
    TrainArgs args = a;
    args.grid = plan.grid;
    args.slot_spread = plan.slot_spread;
    args.lds_rows = plan.variant ? 0 : plan.lds_rows;
    TrainKernel fn = plan.variant ? in->lds : in->stream;
    void *params[] = {&args};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(fn),
                                      dim3(plan.grid - plan.absent), dim3(plan.block), params,
                                      (unsigned)plan.lds_bytes, s);
}

}  // namespace som
