// Pipelined online-SOM training kernel for gfx950 (MI355X): the pass over
// the prototypes runs concurrently with the grid exchanges.
//
// The training of som_train.hip alternates two phases per block of M steps:
// wave 0 finds the block's M BMUs (M grid exchanges), then every wave sweeps
// the prototypes once.  Here wave 3 (the controller) runs the exchanges of
// block b while waves 0-2 (the sweepers) already sweep for block b + 1, so a
// step costs about one exchange instead of one exchange plus a share of the
// sweep.  What makes this possible is that block b + 1's Gram matrices need
// block b's coefficients only through scalars:
//
//   F_b      prototype at the start of block b (materialised in memory/LDS),
//   z        a centring vector, the first sample of block b,
//   f        = F_b - z,   A_i = x_{b,i} - z,   B_j = x_{b+1,j} - z,
//   F_{b+1}  = beta F_b + sum_i gamma_i x_{b,i}   (beta + sum_i gamma_i = 1)
//   e_j      = x_{b+1,j} - F_{b+1} = B_j - beta f - sum_i gamma_i A_i
//   E_{b+1}[j,l] = e_j . e_l
//            = B_j.B_l - P_j - P_l + Q,
//   P_j      = beta f.B_j + sum_i gamma_i A_i.B_j,
//   Q        = beta^2 f.f + 2 beta sum_i gamma_i f.A_i + sum_ik gamma_i gamma_k A_i.A_k.
//
// Per unit the sweep of block b needs only F_b and the samples: it
// materialises F_b from F_{b-1} with block b-1's coefficients (known when
// block b starts) and accumulates f.f, f.A_i and f.B_j.  The sample-sample
// products A.A, A.B and B.B are the same for every unit and come from a
// prepass over the blocks.  The controller then forms E_{b+1} from these
// scalars and block b's coefficients.  Centring on a sample keeps every term
// at the scale of sample-to-prototype distances.
//
// Samples live in an LDS ring of four blocks: the sweep of block b reads
// blocks b-1 (to materialise), b and b+1 (for the products) and fills block
// b+2.  Everything else (exchange, schedule table, neighbourhood, windows)
// is shared with the other training kernel (som_device.h).
#include "som_device.h"

namespace som {
namespace {

using namespace dev;

constexpr int kSweepers = 3;      // waves 0..2 sweep
constexpr int kController = 3;    // wave 3 runs the exchanges
constexpr int kPipeHeader = 64;
constexpr int kStageMax = 16;     // staged sample float4 per sweeper lane

template <int M>
constexpr int dots_stride() { return M * (M + 1) + M * M; }  // AA (T), AB (M*M), BB (T)

// ---------------------------------------------------------------- prepass
// Per block b: z = x_{b,0}; A_i = x_{b,i} - z; B_j = x_{b+1,j} - z (samples
// past the last step are sample 0, as in the training kernel).  Writes
// out[b] = (A_i.A_k for i <= k, A_i.B_j row-major in i, B_j.B_l for j <= l).
template <int M>
__global__ __launch_bounds__(256) void block_dots_kernel(TrainArgs a, float *out,
                                                         int64_t nblocks) {
    constexpr int T = M * (M + 1) / 2;
    constexpr int ND = dots_stride<M>();
    __shared__ float red[4][ND];
    const int64_t b = blockIdx.x;
    if (b >= nblocks) return;
    const float *xa[M], *xb[M];
#pragma unroll
    for (int j = 0; j < M; ++j) {
        const int64_t sa = b * M + j, sb = (b + 1) * M + j;
        int ia = sa < a.nsteps ? a.order[sa] : 0, ib = sb < a.nsteps ? a.order[sb] : 0;
        ia = (ia >= 0 && (int64_t)ia < a.n) ? ia : 0;
        ib = (ib >= 0 && (int64_t)ib < a.n) ? ib : 0;
        xa[j] = a.X + (int64_t)ia * a.d;
        xb[j] = a.X + (int64_t)ib * a.d;
    }
    float acc[ND];
#pragma unroll
    for (int t = 0; t < ND; ++t) acc[t] = 0.f;
    for (int c = threadIdx.x; c < a.d; c += 256) {
        const float z = xa[0][c];
        float A[M], B[M];
#pragma unroll
        for (int j = 0; j < M; ++j) {
            A[j] = xa[j][c] - z;
            B[j] = xb[j][c] - z;
        }
#pragma unroll
        for (int k = 0; k < M; ++k)
#pragma unroll
            for (int i = 0; i <= k; ++i) {
                acc[tri(i, k)] = fmaf(A[i], A[k], acc[tri(i, k)]);
                acc[T + M * M + tri(i, k)] = fmaf(B[i], B[k], acc[T + M * M + tri(i, k)]);
            }
#pragma unroll
        for (int i = 0; i < M; ++i)
#pragma unroll
            for (int j = 0; j < M; ++j) acc[T + i * M + j] = fmaf(A[i], B[j], acc[T + i * M + j]);
    }
    wave_sums<ND>(acc);
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0)
#pragma unroll
        for (int t = 0; t < ND; ++t) red[wave][t] = acc[t];
    __syncthreads();
    if (threadIdx.x < ND) {
        const int t = threadIdx.x;
        out[b * ND + t] = (red[0][t] + red[1][t]) + (red[2][t] + red[3][t]);
    }
}

// ---------------------------------------------------------------- sweepers
struct PipeLayout {
    int Rp, P4;
    f4 *xs;        // 4 slots x M samples x P4 float4
    float *dots;   // 2 parities x Rp x 2M
    float *coef;   // 2 parities x Rp x (M + 1)
    float4 *pos;   // Rp
    f4 *lw;        // R x P4 (LDS variant)
};

template <int M>
__device__ inline PipeLayout pipe_layout(unsigned char *smem, int R, int P4) {
    PipeLayout l;
    l.Rp = (R + 3) & ~3;
    l.P4 = P4;
    unsigned char *p = smem + kPipeHeader;
    l.xs = reinterpret_cast<f4 *>(p);
    p += (size_t)4 * M * P4 * 16;
    l.dots = reinterpret_cast<float *>(p);
    p += (size_t)2 * l.Rp * 2 * M * 4;
    l.coef = reinterpret_cast<float *>(p);
    p += (size_t)2 * l.Rp * (M + 1) * 4;
    p = reinterpret_cast<unsigned char *>((reinterpret_cast<uintptr_t>(p) + 15) & ~(uintptr_t)15);
    l.pos = reinterpret_cast<float4 *>(p);
    p += (size_t)l.Rp * 16;
    l.lw = reinterpret_cast<f4 *>(p);
    return l;
}

__device__ inline int sample_index(const TrainArgs &a, int64_t s, StepWindow<int> &ow) {
    return s < a.nsteps ? ow.get(a, s) : 0;
}

// Sweepers: load block blk's M samples into registers (issue only).
template <int M>
__device__ inline void stage_block(const TrainArgs &a, int64_t blk, int P4, StepWindow<int> &ow,
                                   f4 (&st)[kStageMax]) {
    int idx[M];
#pragma unroll
    for (int j = 0; j < M; ++j) idx[j] = sample_index(a, blk * M + j, ow);
    const int tid = threadIdx.x;
    const int xd4 = a.d >> 2;
#pragma unroll
    for (int e = 0; e < kStageMax; ++e) {
        const int flat = tid + kSweepers * 64 * e;
        f4 v = {0.f, 0.f, 0.f, 0.f};
        if (flat < M * P4) {
            const int j = flat / P4, q = flat - j * P4;
            int i = idx[0];
#pragma unroll
            for (int jj = 1; jj < M; ++jj) i = (j == jj) ? idx[jj] : i;
            if (a.x_vec4) {
                if (q < xd4) v = reinterpret_cast<const f4 *>(a.X + (int64_t)i * a.d)[q];
            } else {
                const float *xr = a.X + (int64_t)i * a.d;
                const int c = 4 * q;
                v.x = c + 0 < a.d ? xr[c + 0] : 0.f;
                v.y = c + 1 < a.d ? xr[c + 1] : 0.f;
                v.z = c + 2 < a.d ? xr[c + 2] : 0.f;
                v.w = c + 3 < a.d ? xr[c + 3] : 0.f;
            }
        }
        st[e] = v;
    }
}

template <int M>
__device__ inline void commit_block(f4 *slot, int P4, const f4 (&st)[kStageMax]) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int e = 0; e < kStageMax; ++e) {
        const int flat = tid + kSweepers * 64 * e;
        if (flat < M * P4) slot[flat] = st[e];
    }
}

// Operands of one item of a sweep: one row's float4 column slice q.
template <int M, bool MAT, bool ADOT, bool BDOT>
struct SweepItem {
    f4 w, z;
    f4 xp[MAT ? M : 1];
    f4 A[(ADOT && M > 1) ? M - 1 : 1];
    f4 B[BDOT ? M : 1];
};

template <int M, bool MAT, bool ADOT, bool BDOT, typename RowT>
__device__ inline void load_item(SweepItem<M, MAT, ADOT, BDOT> &it, const RowT *row, int q, int P4,
                                 const f4 *xp, const f4 *xc, const f4 *xn) {
    it.w = row[q];
    if (MAT) {
#pragma unroll
        for (int i = 0; i < M; ++i) it.xp[i] = xp[i * P4 + q];
    }
    if (ADOT || BDOT) it.z = xc[q];
    if (ADOT) {
#pragma unroll
        for (int i = 1; i < M; ++i) it.A[i - 1] = xc[i * P4 + q];
    }
    if (BDOT) {
#pragma unroll
        for (int j = 0; j < M; ++j) it.B[j] = xn[j * P4 + q];
    }
}

__device__ inline float dot4(f4 a, f4 b, float acc) {
    return fmaf(a.x, b.x, fmaf(a.y, b.y, fmaf(a.z, b.z, fmaf(a.w, b.w, acc))));
}

// One pass of the sweepers over the workgroup's rows (row r by sweeper wave
// r mod 3, 64 float4 columns per item).  MAT materialises w <- beta w +
// sum_i gamma_i xp_i from coef_prev; then with z = xc_0 and f = w - z it
// accumulates f.f, f.(xc_i - z) for i >= 1 (ADOT) and f.(xn_j - z) (BDOT)
// into dots[r * 2M + ...].  The operands of the next item are loaded before
// the current one is used, two register sets in turn.
template <int M, bool LDSW, bool MAT, bool ADOT, bool BDOT>
__device__ inline void pipe_sweep(f4 *rows_p, int R, int P4, const f4 *xp, const f4 *xc,
                                  const f4 *xn, const float *coef_prev, float *dots) {
    row_t<LDSW> *rows = rows_as<LDSW>(rows_p);
    constexpr int ND = 2 * M;
    constexpr bool DOTS = ADOT || BDOT;
    typedef SweepItem<M, MAT, ADOT, BDOT> Item;
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (wave >= R) return;
    const int KK = P4 >> 6;
    const int n = ((R - 1 - wave) / kSweepers + 1) * KK;
    int r = wave, k = 0;    // item in use
    int rl = wave, kl = 0;  // next item to load
    float beta = 1.f, gam[M], acc[ND];
#pragma unroll
    for (int t = 0; t < ND; ++t) acc[t] = 0.f;
    auto load_coef = [&](int rr) {
        if (MAT) {
            beta = coef_prev[rr * (M + 1)];
#pragma unroll
            for (int i = 0; i < M; ++i) gam[i] = coef_prev[rr * (M + 1) + 1 + i];
        }
    };
    auto issue = [&](Item &it) {
        load_item<M, MAT, ADOT, BDOT>(it, rows + (size_t)rl * P4, lane + 64 * kl, P4, xp, xc, xn);
        if (++kl == KK) {
            kl = 0;
            rl += kSweepers;
        }
    };
    auto use = [&](Item &it) {
        f4 w = it.w;
        if (MAT) {
            w = w * beta;
#pragma unroll
            for (int i = 0; i < M; ++i) {
                w.x = fmaf(gam[i], it.xp[i].x, w.x);
                w.y = fmaf(gam[i], it.xp[i].y, w.y);
                w.z = fmaf(gam[i], it.xp[i].z, w.z);
                w.w = fmaf(gam[i], it.xp[i].w, w.w);
            }
            rows[(size_t)r * P4 + lane + 64 * k] = w;
        }
        if (DOTS) {
            const f4 f = w - it.z;
            acc[0] = dot4(f, f, acc[0]);
            if (ADOT) {
#pragma unroll
                for (int i = 1; i < M; ++i) acc[i] = dot4(f, it.A[i - 1] - it.z, acc[i]);
            }
            if (BDOT) {
#pragma unroll
                for (int j = 0; j < M; ++j) acc[M + j] = dot4(f, it.B[j] - it.z, acc[M + j]);
            }
        }
        if (++k == KK) {
            if (DOTS) {
                wave_sums<ND>(acc);
                if (lane == 0)
#pragma unroll
                    for (int t = 0; t < ND; ++t) dots[r * ND + t] = acc[t];
#pragma unroll
                for (int t = 0; t < ND; ++t) acc[t] = 0.f;
            }
            k = 0;
            r += kSweepers;
            if (r < R) load_coef(r);
        }
    };
    load_coef(r);
    Item ia, ib;
    issue(ia);
    for (int i = 0; i < n; i += 2) {
        if (i + 1 < n) issue(ib);
        use(ia);
        if (i + 1 >= n) break;
        if (i + 2 < n) issue(ia);
        use(ib);
    }
}

// ---------------------------------------------------------------- controller
// Controller lane r (< R): Gram matrix E of the block starting at call step
// s0 from the sweep's products of row r (dots: f.f, f.A_1.., f.B_0..), the
// previous block's coefficients (beta, gam) and the block's sample products
// (sd: AA, AB, BB of the previous block; for the first block BB = its own AA).
template <int M>
__device__ inline void gram_from_dots(const float *d, float beta, const float (&gam)[M],
                                      const float (&AA)[M * (M + 1) / 2], const float (&AB)[M * M],
                                      const float (&BB)[M * (M + 1) / 2],
                                      float (&E)[M * (M + 1) / 2]) {
    float fA[M], fB[M], P[M];
    const float ff = d[0];
    fA[0] = 0.f;
#pragma unroll
    for (int i = 1; i < M; ++i) fA[i] = d[i];
#pragma unroll
    for (int j = 0; j < M; ++j) fB[j] = d[M + j];
#pragma unroll
    for (int j = 0; j < M; ++j) {
        float p = beta * fB[j];
#pragma unroll
        for (int i = 0; i < M; ++i) p = fmaf(gam[i], AB[i * M + j], p);
        P[j] = p;
    }
    float lin = 0.f, quad = 0.f;
#pragma unroll
    for (int i = 0; i < M; ++i) {
        float inner = 0.f;
#pragma unroll
        for (int k = 0; k < M; ++k) inner = fmaf(gam[k], AA[tri_any(i, k)], inner);
        lin = fmaf(gam[i], fA[i], lin);
        quad = fmaf(gam[i], inner, quad);
    }
    const float Q = fmaf(beta * beta, ff, fmaf(2.f * beta, lin, quad));
#pragma unroll
    for (int l = 0; l < M; ++l)
#pragma unroll
        for (int j = 0; j <= l; ++j) E[tri(j, l)] = BB[tri(j, l)] - P[j] - P[l] + Q;
}

// Read the sample products of block blk (lane t < ND holds entry t).
template <int M>
__device__ inline float load_sd(const float *sdots, int64_t blk, int64_t nblocks) {
    constexpr int ND = dots_stride<M>();
    const int lane = threadIdx.x & 63;
    return (lane < ND && blk < nblocks) ? sdots[blk * ND + lane] : 0.f;
}

template <int M>
__device__ inline void unpack_sd(float v, float (&AA)[M * (M + 1) / 2], float (&AB)[M * M],
                                 float (&BB)[M * (M + 1) / 2]) {
    constexpr int T = M * (M + 1) / 2;
#pragma unroll
    for (int t = 0; t < T; ++t) AA[t] = lane_f(v, t);
#pragma unroll
    for (int t = 0; t < M * M; ++t) AB[t] = lane_f(v, T + t);
#pragma unroll
    for (int t = 0; t < T; ++t) BB[t] = lane_f(v, T + M * M + t);
}

template <int M, bool LDSW>
__global__ __launch_bounds__(256, 1) void train_pipe_kernel(TrainArgs a) {
    constexpr int T = M * (M + 1) / 2;
    constexpr int ND = 2 * M;
    extern __shared__ __align__(16) unsigned char smem[];
    const int G = a.grid, b = blockIdx.x, tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int r0 = (int)(((int64_t)b * a.N) / G);
    const int r1 = (int)(((int64_t)(b + 1) * a.N) / G);
    const int R = r1 - r0;  // <= 64 (planner)
    const int P4 = (int)(a.ld / 4);
    const float inv_cols = 1.f / (float)a.cols;
    Bcast *bc = reinterpret_cast<Bcast *>(smem);
    const PipeLayout l = pipe_layout<M>(smem, R, P4);

    if (a.state->order_bad) return;  // same value for every workgroup
    if (a.nsteps <= 0) return;

    for (int r = tid; r < R; r += 256) {
        const int u = r0 + r, ur = u / a.cols, uc = u - ur * a.cols;
        l.pos[r] = make_float4((float)ur, (float)uc, (float)(ur & 1), 0.f);
    }
    if (tid == 0) bc->abort = 0;
    f4 *gw = reinterpret_cast<f4 *>(a.W) + (int64_t)r0 * P4;
    f4 *rows = gw;
    if (LDSW) {
        for (int e = tid; e < R * P4; e += 256) l.lw[e] = gw[e];
        rows = l.lw;
    }
    const int64_t nb = (a.nsteps + M - 1) / M;
    StepWindow<int> ow;
    StepWindow<float2> sw;
    ow.init(a, 0);
    sw.init(a, 0);
    f4 st[kStageMax];
    if (wave < kSweepers) {
        stage_block<M>(a, 0, P4, ow, st);
        commit_block<M>(l.xs, P4, st);
        if (nb > 1) {
            stage_block<M>(a, 1, P4, ow, st);
            commit_block<M>(l.xs + (size_t)1 * M * P4, P4, st);
        }
    }
    __syncthreads();
    // Products of the initial prototypes with block 0 (centred on its first
    // sample), parity 1.
    if (wave < kSweepers)
        pipe_sweep<M, LDSW, false, false, true>(rows, R, P4, l.xs, l.xs, l.xs, l.coef,
                                          l.dots + (size_t)l.Rp * ND);
    __syncthreads();

    // controller state (lane r = row r)
    float beta_prev = 1.f, gam_prev[M];
#pragma unroll
    for (int j = 0; j < M; ++j) gam_prev[j] = 0.f;
    float4 p = make_float4(0.f, 0.f, 0.f, 0.f);
    float sd = 0.f;
    if (wave == kController) {
        if (lane < R) p = l.pos[lane];
        sd = load_sd<M>(a.block_dots, 0, nb);
    }

    for (int64_t blk = 0; blk < nb; ++blk) {
        const int par = (int)(blk & 1);
        if (wave == kController) {
            float AA[T], AB[M * M], BB[T], E[T];
            unpack_sd<M>(sd, AA, AB, BB);
            if (blk == 0) {
#pragma unroll
                for (int t = 0; t < T; ++t) BB[t] = AA[t];
            }
            const float *d = l.dots + ((size_t)(par ^ 1) * l.Rp + (lane < R ? lane : 0)) * ND;
            gram_from_dots<M>(d, beta_prev, gam_prev, AA, AB, BB, E);
            const float sd_next = (blk + 1 < nb) ? load_sd<M>(a.block_dots, blk, nb) : 0.f;
            const int64_t s0 = blk * M;
            const int mb = (int)((a.nsteps - s0) < M ? (a.nsteps - s0) : M);
            float beta, gam[M];
            const bool ok = block_steps<M>(a, s0, mb, r0, R, E, p, inv_cols, sw, beta, gam);
            if (lane < R) {
                float *cf = l.coef + ((size_t)par * l.Rp + lane) * (M + 1);
                cf[0] = beta;
#pragma unroll
                for (int j = 0; j < M; ++j) cf[1 + j] = gam[j];
            }
            beta_prev = beta;
#pragma unroll
            for (int j = 0; j < M; ++j) gam_prev[j] = gam[j];
            sd = sd_next;
            if (!ok && lane == 0) bc->abort = 1;
        } else {
            const bool stage = blk + 2 < nb;
            if (stage) stage_block<M>(a, blk + 2, P4, ow, st);
            const f4 *xp = l.xs + (size_t)((blk + 3) & 3) * M * P4;
            const f4 *xc = l.xs + (size_t)(blk & 3) * M * P4;
            const f4 *xn = l.xs + (size_t)((blk + 1) & 3) * M * P4;
            const float *cp = l.coef + (size_t)(par ^ 1) * l.Rp * (M + 1);
            float *dd = l.dots + (size_t)par * l.Rp * ND;
            const bool has_next = blk + 1 < nb;
            if (blk == 0) {
                if (has_next) pipe_sweep<M, LDSW, false, true, true>(rows, R, P4, xp, xc, xn, cp, dd);
            } else if (has_next) {
                pipe_sweep<M, LDSW, true, true, true>(rows, R, P4, xp, xc, xn, cp, dd);
            } else {
                pipe_sweep<M, LDSW, true, false, false>(rows, R, P4, xp, xc, xn, cp, dd);
            }
            if (stage) commit_block<M>(l.xs + (size_t)((blk + 2) & 3) * M * P4, P4, st);
        }
        __syncthreads();
        if (bc->abort) return;
    }
    // apply the last block's updates
    if (wave < kSweepers)
        pipe_sweep<M, LDSW, true, false, false>(rows, R, P4, l.xs + (size_t)((nb - 1) & 3) * M * P4,
                                          l.xs, l.xs, l.coef + (size_t)((nb - 1) & 1) * l.Rp * (M + 1),
                                          l.dots);
    if (LDSW) {
        __syncthreads();
        for (int e = tid; e < R * P4; e += 256) gw[e] = l.lw[e];
    }
}

typedef void (*PipeKernel)(TrainArgs);
typedef void (*DotsKernel)(TrainArgs, float *, int64_t);

struct PipeInstance {
    int m;
    PipeKernel stream, lds;
    DotsKernel dots;
};

template <int M>
constexpr PipeInstance pipe_instance() {
    return PipeInstance{M, train_pipe_kernel<M, false>, train_pipe_kernel<M, true>,
                        block_dots_kernel<M>};
}

const PipeInstance kPipe[] = {pipe_instance<1>(), pipe_instance<2>(), pipe_instance<4>()};

const PipeInstance *pipe_for(int m) {
    for (const PipeInstance &p : kPipe)
        if (p.m == m) return &p;
    return nullptr;
}

size_t pipe_lds_bytes(int m, int rmax, int64_t P4, bool ldsw) {
    const size_t rp = (size_t)((rmax + 3) & ~3);
    size_t b = kPipeHeader + (size_t)4 * m * P4 * 16 + 2 * rp * 2 * m * 4 + 2 * rp * (m + 1) * 4;
    b = (b + 15) & ~(size_t)15;
    b += rp * 16;
    if (ldsw) b += (size_t)rmax * P4 * 16;
    return b;
}

}  // namespace

double plan_train_pipe(const TrainArgs &a, int num_cus, int max_lds, TrainPlan *plan,
                       double (*exchange_us)(int)) {
    const int64_t P4 = a.ld / 4;
    if (P4 % 64 != 0) return 1e300;
    const int max_grid = a.N < num_cus ? a.N : num_cus;
    double best = 1e300;
    for (const PipeInstance &pi : kPipe) {
        if ((int64_t)pi.m * P4 > (int64_t)kSweepers * 64 * kStageMax) continue;
        for (int v = 0; v < 2; ++v) {
            const bool ldsw = v == 1;
            if ((a.variant == 1 && !ldsw) || (a.variant == 2 && ldsw)) continue;
            for (int g = 1;; g = (g * 2 > max_grid && g < max_grid) ? max_grid : g * 2) {
                const int gg = a.grid > 0 ? (a.grid < a.N ? a.grid : a.N) : g;
                const int rmax = (a.N + gg - 1) / gg;
                if (rmax <= 64 && pipe_lds_bytes(pi.m, rmax, P4, ldsw) <= (size_t)max_lds) {
                    // controller: exchange + per-step scalar work; sweepers:
                    // LDS traffic of one pass per block (3M + 2 float4 per slot)
                    // or memory traffic of the streamed rows, per step.
                    const double rows = ceil(rmax / (double)kSweepers) * kSweepers;
                    const double lds_b = rows * P4 * 16.0 * (3 * pi.m + (ldsw ? 2 : 0));
                    const double lds_us = lds_b / 300e3;
                    const double mem_us = ldsw ? 0.0 : rmax * P4 * 32.0 / 30e3;
                    const double sweep = (lds_us > mem_us ? lds_us : mem_us) / pi.m;
                    const double ctl = exchange_us(gg) + 0.4;
                    const double t = (sweep > ctl ? sweep : ctl) + 0.4 / pi.m;
                    if (t < best) {
                        best = t;
                        plan->grid = gg;
                        plan->variant = ldsw ? 3 : 2;
                        plan->pipe_m = pi.m;
                    }
                }
                if (a.grid > 0 || g >= max_grid) break;
            }
        }
    }
    if (best < 1e300) {
        plan->lds_bytes = pipe_lds_bytes(plan->pipe_m, (a.N + plan->grid - 1) / plan->grid, P4,
                                          plan->variant == 3);
        if (plan->lds_bytes < 84 * 1024) plan->lds_bytes = 84 * 1024;
        plan->block = 256;
        plan->slot_spread = plan->grid <= 64 ? 16 : 4;
        const PipeInstance *pi = pipe_for(plan->pipe_m);
        PipeKernel fn = plan->variant == 3 ? pi->lds : pi->stream;
        int per_cu = 0;
        if (hipOccupancyMaxActiveBlocksPerMultiprocessor(
                &per_cu, reinterpret_cast<const void *>(fn), 256, plan->lds_bytes) != hipSuccess ||
            per_cu < 1 || plan->grid > per_cu * num_cus || plan->grid > kMaxTrainGrid)
            return 1e300;
    }
    return best;
}

int64_t pipe_block_dots_floats(int m, int64_t nsteps) {
    const int64_t nb = (nsteps + m - 1) / m;
    return nb * (m * (m + 1) + m * m);
}

hipError_t launch_train_pipe(const TrainArgs &a, const TrainPlan &plan, hipStream_t s) {
    const PipeInstance *pi = pipe_for(plan.pipe_m);
    if (!pi || !a.block_dots) return hipErrorInvalidValue;
    TrainArgs args = a;
    args.grid = plan.grid;
    args.slot_spread = plan.slot_spread;
    const int64_t nb = (a.nsteps + pi->m - 1) / pi->m;
    pi->dots<<<dim3((unsigned)nb), dim3(256), 0, s>>>(args, args.block_dots, nb);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    PipeKernel fn = plan.variant == 3 ? pi->lds : pi->stream;
    void *params[] = {&args};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(fn), dim3(plan.grid),
                                      dim3(256), params, (unsigned)plan.lds_bytes, s);
}

}  // namespace som
