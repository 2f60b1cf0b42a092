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
// The sweepers split the columns, not the rows: sweeper s owns the 64-column
// float4 slices s, s + 3, s + 6, ... of every row and keeps its slices of the
// samples of blocks b - 1, b and b + 1 in registers, so a row visit reads
// and writes only the row itself.  Each sweeper reduces its partial dot
// products over its lanes and the controller adds the three partials.  Rows
// are loaded a few rows ahead of their use.  The next block's samples are
// loaded at the end of a sweep, while the sweepers wait for the controller.
// The samples stay raw (centred per use, as the prepass does), so that a
// unit rate with a zero radius still copies a sample bit-exactly.
//
// The kernel template lives in this header because its instances are split
// over two translation units: som_train_pipe.hip holds the LDS-resident ones
// and the planner, som_train_pipe_stream.hip the streamed ones, which are
// compiled without the structurizer option of the former (see build.py).
#pragma once

#include "som_device.h"

namespace som {
namespace {  // each translation unit emits only the instances it uses


using namespace dev;

// Waves 0 .. NS-1 sweep and wave NS runs the exchanges.  NS = 3 puts each
// wave on a SIMD of its own; NS = 4 (the streamed kernels of long
// sweeps) puts every SIMD to sweeping and the controller beside sweeper 0.
constexpr int kSweepers = 3;
constexpr int kPipeHeader = 64;

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
        xa[j] = a.X + (int64_t)ia * a.xld;
        xb[j] = a.X + (int64_t)ib * a.xld;
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
    for (int t = threadIdx.x; t < ND; t += 256)
        out[b * ND + t] = (red[0][t] + red[1][t]) + (red[2][t] + red[3][t]);
}

// ---------------------------------------------------------------- layout
struct PipeLayout {
    int Rp;
    float *dots;   // 2 parities x Rp rows x 3 sweepers x 2M
    float *coef;   // 2 parities x Rp x (M + 1)
    float4 *pos;   // Rp
    f4 *dummy;     // column-walk sweep: 3 sweepers x 64 float4 that its
                   // discarded LDS row writes land in
    f4 *lw;        // R x P4 (LDS variant)
};

// The column-walk sweep's discarded-write area, in float4.
constexpr int kPipeDummy = kSweepers * 64;

template <int M, int NS = kSweepers>
__device__ inline PipeLayout pipe_layout(unsigned char *smem, int R, bool cols) {
    PipeLayout l;
    l.Rp = (R + 3) & ~3;
    unsigned char *p = smem + kPipeHeader;
    l.dots = reinterpret_cast<float *>(p);
    p += (size_t)2 * l.Rp * NS * 2 * M * 4;
    l.coef = reinterpret_cast<float *>(p);
    p += (size_t)2 * l.Rp * (M + 1) * 4;
    p = reinterpret_cast<unsigned char *>((reinterpret_cast<uintptr_t>(p) + 15) & ~(uintptr_t)15);
    l.pos = reinterpret_cast<float4 *>(p);
    p += (size_t)l.Rp * 16;
    l.dummy = reinterpret_cast<f4 *>(p);
    if (cols) p += (size_t)kPipeDummy * 16;
    l.lw = reinterpret_cast<f4 *>(p);
    return l;
}

// ---------------------------------------------------------------- sweepers
// Sweeper slices: wave s owns slices s + NS t, t < nw (nw <= KS).
template <int NS = kSweepers>
__device__ inline int sweeper_slices(int nsl) {
    const int s = threadIdx.x >> 6;
    return nsl > s ? (nsl - s + NS - 1) / NS : 0;
}

// This wave's slices of the M samples of block blk (steps past the end load
// sample 0; columns past d, and slices t >= nw, are zero).
template <int M, int KS, int NS = kSweepers>
__device__ inline void load_samples(f4 (&x)[M][KS], const TrainArgs &a, int64_t blk,
                                    StepWindow<int> &ow) {
    const int lane = threadIdx.x & 63, s = threadIdx.x >> 6;
#pragma unroll
    for (int j = 0; j < M; ++j) {
        const int64_t st = blk * M + j;
        const int i = st < a.nsteps ? ow.get(a, st) : 0;
#pragma unroll
        for (int t = 0; t < KS; ++t) x[j][t] = sample_f4(a, i, 64 * (s + NS * t) + lane);
    }
}

__device__ inline float dot4(f4 a, f4 b, float acc) {
    return fmaf(a.x, b.x, fmaf(a.y, b.y, fmaf(a.z, b.z, fmaf(a.w, b.w, acc))));
}

// One pass of a sweeper over the workgroup's R rows, on its slices.  MAT
// materialises w <- beta w + sum_i gamma_i xp_i from coef_prev; then with
// z = xc_0 and f = w - z it accumulates f.f, f.(xc_i - z) for i >= 1 (ADOT)
// and f.(xn_j - z) (BDOT), the last two as f.x - f.z of sums over the wave,
// into dots[(r * 3 + sweeper) * 2M + ...] (written by lane 63).  Rows (and their
// coefficients) are loaded D rows ahead, into a ring of registers indexed
// statically.  Callers sweeping a part of the rows pass coef_prev and dots
// advanced to its first row.
template <int M, int KS, int D, bool LDSW, bool MAT, bool ADOT, bool BDOT, int NS = kSweepers>
__device__ inline void pipe_sweep(f4 *rows_p, int R, int P4, int nw, const f4 (&xp)[M][KS],
                                  const f4 (&xc)[M][KS], const f4 (&xn)[M][KS],
                                  const float *coef_prev, float *dots) {
    if (R <= 0) return;
    constexpr int ND = 2 * M;
    constexpr bool DOTS = ADOT || BDOT;
    constexpr int NA = ND + 1;  // f.f, f.x_i, f.xn_j and f.z (last)
    [[maybe_unused]] row_t<LDSW> *rows = rows_as<LDSW>(rows_p);
    // (the sweeper index as a scalar: derived from the thread index, the
    // compiler could not prove it uniform, and the buffer resource and its
    // offsets below would go through per-lane loops)
    const int lane = threadIdx.x & 63, s = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    // Streamed rows go through a buffer resource over the R rows: a slice
    // past the sweeper's share gets an offset beyond its end, so that its
    // load returns zeros and its store is dropped, with no select or branch
    // (either would make the compiler wait for the row loads in flight).
    // (unused by the LDS variant)
    const uint64_t rbase = reinterpret_cast<uintptr_t>(rows_p);
    f4 *rows_u = reinterpret_cast<f4 *>(
        ((uint64_t)(uint32_t)__builtin_amdgcn_readfirstlane((int)(rbase >> 32)) << 32) |
        (uint32_t)__builtin_amdgcn_readfirstlane((int)(uint32_t)rbase));
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        rows_u, (short)0, __builtin_amdgcn_readfirstlane(LDSW ? 0 : R * P4 * 16), 0x00020000);
    constexpr int kOutside = 1 << 30;  // bytes, beyond any sweep's rows
    const auto slice_off = [&](int r, int t) {
        return t < nw ? (r * P4 + 64 * (s + NS * t) + lane) * 16 : kOutside;
    };
    f4 ring[D][KS];
    float cring[D][M + 1];
    // Loads are unconditional (clamped row and column, unused when out of
    // range) so that a burst of them is waited for once.  In LDS, slices past
    // the sweeper's share are zeroed where they are used, not here: a select
    // on a value as it is loaded makes the compiler wait for the load on the
    // spot, which would cancel the rows' prefetch.
    auto issue = [&](int r, f4 (&dst)[KS], float (&cdst)[M + 1]) {
        const int rr = r < R ? r : R - 1;
#pragma unroll
        for (int t = 0; t < KS; ++t) {
            if constexpr (LDSW) {
                const int q = 64 * (s + NS * t) + lane;
                dst[t] = rows[(size_t)rr * P4 + (q < P4 ? q : P4 - 1)];
            } else {
                dst[t] = __builtin_bit_cast(
                    f4, __builtin_amdgcn_raw_buffer_load_b128(rs, slice_off(rr, t), 0, 0));
            }
        }
        if (MAT) {
#pragma unroll
            for (int i = 0; i <= M; ++i) cdst[i] = coef_prev[rr * (M + 1) + i];
        }
    };
#pragma unroll
    for (int u = 0; u < D; ++u) issue(u, ring[u], cring[u]);
    for (int rb = 0; rb < R; rb += D) {
#pragma unroll
        for (int u = 0; u < D; ++u) {
            const int r = rb + u;
            if (r < R) {
                float acc[NA];
#pragma unroll
                for (int t = 0; t < NA; ++t) acc[t] = 0.f;
                // slices t >= nw hold zeros in w and in the samples
#pragma unroll
                for (int t = 0; t < KS; ++t) {
                    {
                        const f4 zero = {0.f, 0.f, 0.f, 0.f};
                        f4 w = (!LDSW || t < nw) ? ring[u][t] : zero;
                        if (MAT) {
                            w = w * cring[u][0];
#pragma unroll
                            for (int i = 0; i < M; ++i) {
                                const float g = cring[u][1 + i];
                                w.x = fmaf(g, xp[i][t].x, w.x);
                                w.y = fmaf(g, xp[i][t].y, w.y);
                                w.z = fmaf(g, xp[i][t].z, w.z);
                                w.w = fmaf(g, xp[i][t].w, w.w);
                            }
                            if constexpr (LDSW) {
                                if (t < nw) rows[(size_t)r * P4 + 64 * (s + NS * t) + lane] = w;
                            } else {
                                __builtin_amdgcn_raw_buffer_store_b128(
                                    __builtin_bit_cast(u32x4, w), rs, slice_off(r, t), 0, 0);
                            }
                        }
                        if (DOTS) {
                            // f.(x - z) as f.x - f.z after the lane sums:
                            // the centring costs one dot per row instead of
                            // a subtraction per sample and column
                            const f4 z = xc[0][t];
                            const f4 f = w - z;
                            acc[0] = dot4(f, f, acc[0]);
                            acc[ND] = dot4(f, z, acc[ND]);
                            if (ADOT) {
#pragma unroll
                                for (int i = 1; i < M; ++i) acc[i] = dot4(f, xc[i][t], acc[i]);
                            }
                            if (BDOT) {
#pragma unroll
                                for (int j = 0; j < M; ++j)
                                    acc[M + j] = dot4(f, xn[j][t], acc[M + j]);
                            }
                        }
                    }
                }
                issue(r + D, ring[u], cring[u]);
                if (DOTS) {
                    constexpr int NT = (NA + 3) / 4;
                    float tot[NT];
                    wave_sums_rows<NA>(acc, tot);
                    const float fz = lane_f(tot[ND / 4], 16 * sum_row(ND));
                    if ((lane & 15) == 0) {
                        // lane 16 q writes the values its row holds
                        float *dr = dots + (r * NS + s) * ND;
                        const int q = lane >> 4;
#pragma unroll
                        for (int j = 0; j < NT; ++j) {
                            const int t = 4 * j + 2 * (q & 1) + (q >> 1);  // sum_row(t) == q
                            const bool used = t == 0 || (t < M ? ADOT : BDOT);
                            if (t < ND) dr[t] = t == 0 ? tot[j] : (used ? tot[j] - fz : 0.f);
                        }
                    }
                }
            }
        }
    }
}

// A sweep over the workgroup's R rows: rows [0, RL) from LDS (loaded two
// ahead) and, in the streamed variant (LDSW false), rows [RL, R) from
// memory at gs (loaded four ahead on three sweepers, two ahead on four:
// four sweepers on 5-step blocks have no registers left for deeper loads).
template <int M, int KS, bool LDSW, bool MAT, bool ADOT, bool BDOT, int NS = kSweepers>
__device__ inline void sweep_rows(f4 *lw, int RL, f4 *gs, int R, int P4, int nw,
                                  const f4 (&xp)[M][KS], const f4 (&xc)[M][KS],
                                  const f4 (&xn)[M][KS], const float *coef_prev, float *dots) {
    constexpr int ND = 2 * M;
    constexpr int AHEAD = NS == 4 ? 2 : 4;
    pipe_sweep<M, KS, 2, true, MAT, ADOT, BDOT, NS>(lw, RL, P4, nw, xp, xc, xn, coef_prev, dots);
    if constexpr (!LDSW)
        pipe_sweep<M, KS, AHEAD, false, MAT, ADOT, BDOT, NS>(gs, R - RL, P4, nw, xp, xc, xn,
                                                         coef_prev + (size_t)RL * (M + 1),
                                                         dots + (size_t)RL * NS * ND);
}

// ---------------------------------------------------------------- long rows
// Sample indices of the M steps of block blk (steps past the end: sample 0).
template <int M>
__device__ inline void block_indices(int (&idx)[M], const TrainArgs &a, int64_t blk,
                                     StepWindow<int> &ow) {
#pragma unroll
    for (int j = 0; j < M; ++j) {
        const int64_t st = blk * M + j;
        idx[j] = st < a.nsteps ? ow.get(a, st) : 0;
    }
}

// The same pass as sweep_rows, for rows too long for three blocks of sample
// slices to stay in registers: the sweeper walks its slices and, for each,
// every row of the workgroup; the samples' rows must be as long as the
// prototypes' (xld = ld, zero past d).  A slice of the 3 M samples (the previous
// block's for the update, the current block's for the centring and the
// current products, the next block's for the next products) is loaded from
// memory once per slice and reused for all rows; the samples are read by
// every workgroup, so they come from L2.  The products of each row
// accumulate in registers across the slices (RMAX rows at most) and are
// reduced over the lanes once, at the end.  Rows [0, RL) (RL <= RLMAX) live
// in LDS, the others stream from memory at gs; the next slice's rows and
// samples are loaded while the current one is computed.  Arguments as
// sweep_rows; ip, ic, inx are the sample indices of the previous, current
// and next block; dummy is this sweeper's 64-float4 area for the LDS writes
// of streamed rows.  This call walks the window of rows [R0, R0 + RMAX) of
// the workgroup's R (sweep_cols_split below walks all of them in windows);
// LDS rows must lie in a window with R0 = 0.
template <int M, int RMAX, int RLMAX, bool MAT, bool ADOT, bool BDOT, int R0 = 0>
__device__ inline void sweep_cols(const TrainArgs &a, f4 *lw_p, int RL, f4 *gs, int R, int P4,
                                  int nw, const int (&ip)[M], const int (&ic)[M],
                                  const int (&inx)[M], const float *coef_prev, float *dots,
                                  f4 *dummy_p) {
    constexpr int ND = 2 * M;
    constexpr bool DOTS = ADOT || BDOT;
    constexpr int NA = ND + 1;  // f.f, f.x_i, f.xn_j and f.z (last)
    // The sweeper index and its slice count as scalars: left as functions
    // of the thread index they would make the slice loop divergent, and
    // every row offset with it.
    const int s = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    nw = __builtin_amdgcn_readfirstlane(nw);
    static_assert(R0 == 0 || RLMAX == 0, "LDS rows lie in the first window");
    if (R <= R0 || nw <= 0) return;
    row_t<true> *lw = rows_as<true>(lw_p);
    row_t<true> *dummy = rows_as<true>(dummy_p);
    const int lane = threadIdx.x & 63;
    const int RS = R - RL;  // streamed rows
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        gs, (short)0, RS > 0 ? RS * P4 * 16 : 0, 0x00020000);
    constexpr int kOutside = 1 << 30;  // bytes, beyond any sweep's rows
    // Streamed row R0 + r's byte offset (a scalar per row): LDS rows and
    // rows past R read zeros and drop their stores.
    int soff[RMAX];
#pragma unroll
    for (int r = 0; r < RMAX; ++r) {
        const int rg = R0 + r;
        soff[r] = __builtin_amdgcn_readfirstlane((rg >= RL && rg < R) ? (rg - RL) * P4 * 16
                                                                      : kOutside);
    }
    const auto row_off = [&](int r) { return soff[r]; };
    float acc[RMAX][NA];
#pragma unroll
    for (int r = 0; r < RMAX; ++r)
#pragma unroll
        for (int t = 0; t < NA; ++t) acc[r][t] = 0.f;
    // The rows' update coefficients, as wave-uniform scalars for the whole
    // pass: read from LDS per row and slice, each read's wait would also
    // wait for the LDS rows in flight, and held in vector registers they
    // take RMAX (M + 1) of them per lane, which kept blocks longer than 4
    // steps from fitting beside the double-buffered slices.  (What does not
    // fit in scalar registers the compiler keeps in lanes of a few vector
    // registers, one read-lane per use.)
    float cf[RMAX][M + 1];
    if (MAT) {
#pragma unroll
        for (int r = 0; r < RMAX; ++r)
#pragma unroll
            for (int i = 0; i <= M; ++i)
                cf[r][i] = __builtin_bit_cast(
                    float, __builtin_amdgcn_readfirstlane(__builtin_bit_cast(
                               int, coef_prev[(R0 + r < R ? R0 + r : 0) * (M + 1) + i])));
    }
    const float *xprev[M], *xcur[M], *xnext[M];
#pragma unroll
    for (int i = 0; i < M; ++i) {
        xprev[i] = a.X + (int64_t)ip[i] * a.xld;
        xcur[i] = a.X + (int64_t)ic[i] * a.xld;
        xnext[i] = a.X + (int64_t)inx[i] * a.xld;
    }
    const auto slice_col = [&](int t) {
        const int tc = t < nw ? t : nw - 1;  // clamped: its values go unused
        return 64 * (s + kSweepers * tc) + lane;
    };
    // One slice's rows and samples.  The next slice's are all loaded at the
    // start of the current one, ahead of its stores: the wait for a slice's
    // loads then finds them issued a whole slice earlier (the memory counter
    // is waited on in issue order, stores included).  Loads are
    // unconditional: a select or branch on a value as it is loaded would
    // make the compiler wait for it on the spot.
    struct Slice {
        f4 g[RMAX];   // streamed rows
        f4 l[RLMAX > 0 ? RLMAX : 1];  // LDS rows
        f4 x[3][M];   // samples: previous, current, next block
    };
    // (a 32-bit unsigned byte offset from a scalar row base: one address
    // register per slice for all the samples)
    const auto at = [](const float *row, unsigned off) {
        return *(gf4 *)((const __attribute__((address_space(1))) char *)row + off);
    };
    const auto load = [&](int q, Slice &sl) {
#pragma unroll
        for (int r = 0; r < RMAX; ++r)
            sl.g[r] = __builtin_bit_cast(
                f4, __builtin_amdgcn_raw_buffer_load_b128(rs, q * 16, row_off(r), 0));
        // (with no LDS rows this reads the slack after the layout, unused)
        const int ql = RL > 0 ? q : lane;
#pragma unroll
        for (int r = 0; r < RLMAX; ++r) sl.l[r] = lw[(size_t)(r < RL ? r : 0) * P4 + ql];
        const unsigned off = (unsigned)q * 16u;
#pragma unroll
        for (int i = 0; i < M; ++i) {
            if (MAT) sl.x[0][i] = at(xprev[i], off);
            if (DOTS && (i == 0 || ADOT)) sl.x[1][i] = at(xcur[i], off);
            if (BDOT) sl.x[2][i] = at(xnext[i], off);
        }
    };
    const auto work = [&](int t, Slice &sl) {
        const int q = 64 * (s + kSweepers * t) + lane;
        // Every row slot is computed, also past R (those read zeros and
        // store nothing, and their sums are never read): a branch per row
        // would merge the memory counters' state at each join, and the
        // compiler would then wait for every load in flight.
        // Streamed rows first and the LDS rows last: the memory counter's
        // wait at the next slice then finds the last streamed store a few
        // rows old.
#pragma unroll
        for (int rr = 0; rr < RMAX; ++rr) {
            const int r = RMAX - 1 - rr;
            f4 w = (r < RLMAX && r < RL) ? sl.l[r < RLMAX ? r : 0] : sl.g[r];
            if (MAT) {
                w = w * cf[r][0];
#pragma unroll
                for (int i = 0; i < M; ++i) {
                    const float g = cf[r][1 + i];
                    w.x = fmaf(g, sl.x[0][i].x, w.x);
                    w.y = fmaf(g, sl.x[0][i].y, w.y);
                    w.z = fmaf(g, sl.x[0][i].z, w.z);
                    w.w = fmaf(g, sl.x[0][i].w, w.w);
                }
                if (r < RLMAX) {
                    row_t<true> *dst = r < RL ? lw + (size_t)r * P4 + q : dummy + 64 * s + lane;
                    *dst = w;
                }
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, w), rs, q * 16,
                                                       row_off(r), 0);
            }
            if (DOTS) {
                const f4 z = sl.x[1][0];
                const f4 f = w - z;
                acc[r][0] = dot4(f, f, acc[r][0]);
                acc[r][ND] = dot4(f, z, acc[r][ND]);
                if (ADOT) {
#pragma unroll
                    for (int i = 1; i < M; ++i) acc[r][i] = dot4(f, sl.x[1][i], acc[r][i]);
                }
                if (BDOT) {
#pragma unroll
                    for (int j = 0; j < M; ++j) acc[r][M + j] = dot4(f, sl.x[2][j], acc[r][M + j]);
                }
            }
        }
    };
    // Two slices per iteration, so that each buffer keeps its registers; an
    // odd last slice is peeled.
    Slice A, B;
    load(slice_col(0), A);
    int t = 0;
    for (; t + 2 <= nw; t += 2) {
        load(slice_col(t + 1), B);
        work(t, A);
        load(slice_col(t + 2), A);
        work(t + 1, B);
    }
    if (t < nw) work(t, A);
    if (DOTS) {
        constexpr int NT = (NA + 3) / 4;
#pragma unroll
        for (int r = 0; r < RMAX; ++r) {
            if (R0 + r < R) {
                float tot[NT];
                wave_sums_rows<NA>(acc[r], tot);
                const float fz = lane_f(tot[ND / 4], 16 * sum_row(ND));
                if ((lane & 15) == 0) {
                    float *dr = dots + ((R0 + r) * kSweepers + s) * ND;
                    const int qq = lane >> 4;
#pragma unroll
                    for (int j = 0; j < NT; ++j) {
                        const int t = 4 * j + 2 * (qq & 1) + (qq >> 1);  // sum_row(t) == qq
                        const bool used = t == 0 || (t < M ? ADOT : BDOT);
                        if (t < ND) dr[t] = t == 0 ? tot[j] : (used ? tot[j] - fz : 0.f);
                    }
                }
            }
        }
    }
}

// The column walk over all of a workgroup's rows in two windows, the first
// holding the LDS rows: each window keeps only its rows' running products
// and coefficients live, so the registers they free hold longer blocks'
// samples instead.  Every row's products sum over the slices in the same
// order as in a single pass; the samples' slices are read once per window
// (from L2).
template <int M, int RMAX, int RLMAX, bool MAT, bool ADOT, bool BDOT>
__device__ inline void sweep_cols_split(const TrainArgs &a, f4 *lw_p, int RL, f4 *gs, int R,
                                        int P4, int nw, const int (&ip)[M], const int (&ic)[M],
                                        const int (&inx)[M], const float *coef_prev, float *dots,
                                        f4 *dummy_p) {
    constexpr int H = (RMAX + 1) / 2;
    static_assert(RLMAX <= H, "the LDS rows lie in the first window");
    sweep_cols<M, H, RLMAX, MAT, ADOT, BDOT, 0>(a, lw_p, RL, gs, R, P4, nw, ip, ic, inx,
                                                coef_prev, dots, dummy_p);
    sweep_cols<M, RMAX - H, 0, MAT, ADOT, BDOT, H>(a, lw_p, RL, gs, R, P4, nw, ip, ic, inx,
                                                   coef_prev, dots, dummy_p);
}

// ---------------------------------------------------------------- controller
// Controller lane r (< R): Gram matrix E of the next block from the sweep's
// products of row r (d: f.f, f.A_1.., f.B_0.., summed over the sweepers),
// the previous block's coefficients (beta, gam) and the block's sample
// products (AA, AB, BB of the previous block; for the first block BB = its
// own AA).
template <int M>
__device__ inline void gram_from_dots(const float (&d)[2 * M], float beta, const float (&gam)[M],
                                      const float (&AA)[M * (M + 1) / 2], const float (&AB)[M * M],
                                      const float (&BB)[M * (M + 1) / 2],
                                      float (&E)[M * (M + 1) / 2]) {
    float P[M];
    const float ff = d[0];
#pragma unroll
    for (int j = 0; j < M; ++j) {
        float p = beta * d[M + j];
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
        if (i > 0) lin = fmaf(gam[i], d[i], lin);
        quad = fmaf(gam[i], inner, quad);
    }
    const float Q = fmaf(beta * beta, ff, fmaf(2.f * beta, lin, quad));
#pragma unroll
    for (int l = 0; l < M; ++l)
#pragma unroll
        for (int j = 0; j <= l; ++j) E[tri(j, l)] = BB[tri(j, l)] - P[j] - P[l] + Q;
}

// The sample products of block blk, spread over the lanes: entry t is held
// by lane t % 64 of word t / 64.
template <int M>
struct SampleDots {
    static constexpr int N = dots_stride<M>();
    static constexpr int W = (N + 63) / 64;
    float v[W];
    // Block blk < the number of blocks.  Lanes past the N entries load the
    // last one again and are never read: no select on a loaded value, which
    // would wait for the load right away.
    __device__ void load(const float *sdots, int64_t blk) {
        const int lane = threadIdx.x & 63;
#pragma unroll
        for (int w = 0; w < W; ++w) {
            const int t = 64 * w + lane;
            v[w] = sdots[blk * N + (t < N ? t : N - 1)];
        }
    }
    __device__ float at(int t) const { return lane_f(v[t / 64], t % 64); }
};

// RMAX > 0: rows too long for sample registers, swept by sweep_cols (rows
// streamed, at most RMAX per workgroup, the first RL <= kColsLdsRows of them
// in LDS); KS is then unused.
constexpr int kColsLdsRows = 4;

template <int M, int KS, bool LDSW, int RMAX = 0, int NS = kSweepers>
__global__ __launch_bounds__(64 * (NS + 1), 1) void train_pipe_kernel(TrainArgs a) {
    static_assert(RMAX == 0 || NS == kSweepers, "the column-walk sweep runs three sweepers");
    constexpr int kBlock = 64 * (NS + 1);
    constexpr int kController = NS;
    constexpr int T = M * (M + 1) / 2;
    constexpr int ND = 2 * M;
    extern __shared__ __align__(16) unsigned char smem[];
    const int G = a.grid, b = blockIdx.x, tid = threadIdx.x;
    const int wave = tid >> 6, lane = tid & 63;
    const int r0 = (int)(((int64_t)b * a.N) / G);
    const int r1 = (int)(((int64_t)(b + 1) * a.N) / G);
    const int R = r1 - r0;  // 1 <= R <= 64 (planner)
    const int P4 = (int)(a.ld / 4);
    const int nw = sweeper_slices<NS>(P4 / 64);  // <= KS (planner) unless RMAX > 0
    const float inv_cols = 1.f / (float)a.cols;
    // Polls in flight per exchange: the LDS-resident kernels keep four; the
    // streamed ones one, where more polling traffic slows the row streams.
    constexpr int kPolls = LDSW ? 4 : 1;
    Bcast *bc = reinterpret_cast<Bcast *>(smem);
    const PipeLayout l = pipe_layout<M, NS>(smem, R, RMAX > 0);

    if (a.state->order_bad) return;  // same value for every workgroup
    if (a.nsteps <= 0) return;

    for (int r = tid; r < R; r += kBlock) {
        const int u = r0 + r, ur = u / a.cols, uc = u - ur * a.cols;
        l.pos[r] = make_float4((float)ur, (float)uc, (float)(ur & 1), 0.f);
    }
    if (tid == 0) bc->abort = 0;
    f4 *gw = reinterpret_cast<f4 *>(a.W) + (int64_t)r0 * P4;
    // Rows [0, RL) live in LDS for the whole launch; the streamed variant
    // keeps as many as its LDS holds (planner) and streams the rest.
    int RL = LDSW ? R : (a.lds_rows < R ? (a.lds_rows > 0 ? a.lds_rows : 0) : R);
    if (RMAX > 0 && RL > kColsLdsRows) RL = kColsLdsRows;
    if (RL > 0) {
        row_t<true> *lw = rows_as<true>(l.lw);
        const row_t<false> *g = rows_as<false>(gw);
        for (int e = tid; e < RL * P4; e += kBlock) lw[e] = g[e];
    }
    f4 *gs = gw + (int64_t)RL * P4;  // first streamed row
    const int64_t nb = (a.nsteps + M - 1) / M;
    __syncthreads();
    // The controller and the sweepers run separate loops over the blocks that
    // meet at one barrier per block (and one before the first), so that each
    // keeps only its own state in registers.
    if (wave == kController) {
        StepWindow<float2> sw;
        sw.init(a, 0);
        float beta_prev = 1.f, gam_prev[M];
#pragma unroll
        for (int j = 0; j < M; ++j) gam_prev[j] = 0.f;
        const float4 p = lane < R ? l.pos[lane] : make_float4(0.f, 0.f, 0.f, 0.f);
        SampleDots<M> sd;
        sd.load(a.block_dots, 0);
        PollRegs<kPolls> pr{};  // exchange poll registers, held across blocks
        // The sample products of the coming block, spread over the lanes in
        // sd when loaded and read out into AA, AB, BB one block ahead: by the
        // end of a block the loads have long landed (the block's exchange
        // polls, issued after them, have been waited for), while reading them
        // at the top of the block waited for every memory operation in flight.
        float AA[T], AB[M * M], BB[T];
#pragma unroll
        for (int t = 0; t < T; ++t) AA[t] = sd.at(t);
#pragma unroll
        for (int t = 0; t < M * M; ++t) AB[t] = sd.at(T + t);
#pragma unroll
        for (int t = 0; t < T; ++t) BB[t] = AA[t];  // block 0: B = A
        __syncthreads();  // the sweepers' products of the initial prototypes
        for (int64_t blk = 0; blk < nb; ++blk) {
            const int par = (int)(blk & 1);
            float E[T], d[ND];
            const float *dr =
                l.dots + ((size_t)(par ^ 1) * l.Rp + (lane < R ? lane : 0)) * NS * ND;
#pragma unroll
            for (int t = 0; t < ND; ++t) {
                if constexpr (NS == 4)
                    d[t] = (dr[t] + dr[ND + t]) + (dr[2 * ND + t] + dr[3 * ND + t]);
                else
                    d[t] = (dr[t] + dr[ND + t]) + dr[2 * ND + t];
            }
            if (blk == 0) {
                // the initial prototypes' products with block 0 itself:
                // f.B_j = f.A_j (B_0 = A_0 = 0)
                d[M] = 0.f;
#pragma unroll
                for (int j = 1; j < M; ++j) d[M + j] = d[j];
            }
            gram_from_dots<M>(d, beta_prev, gam_prev, AA, AB, BB, E);
            if (blk + 1 < nb) sd.load(a.block_dots, blk);
            const int64_t s0 = blk * M;
            const int mb = (int)((a.nsteps - s0) < M ? (a.nsteps - s0) : M);
            float beta, gam[M];
            const bool ok = block_steps<M, kPolls>(a, s0, mb, r0, R, E, p, inv_cols, sw, beta, gam, pr);
            if (lane < R) {
                float *cf = l.coef + ((size_t)par * l.Rp + lane) * (M + 1);
                cf[0] = beta;
#pragma unroll
                for (int j = 0; j < M; ++j) cf[1 + j] = gam[j];
            }
            beta_prev = beta;
#pragma unroll
            for (int j = 0; j < M; ++j) gam_prev[j] = gam[j];
            if (blk + 1 < nb) {
#pragma unroll
                for (int t = 0; t < T; ++t) AA[t] = sd.at(t);
#pragma unroll
                for (int t = 0; t < M * M; ++t) AB[t] = sd.at(T + t);
#pragma unroll
                for (int t = 0; t < T; ++t) BB[t] = sd.at(T + M * M + t);
            }
            if (!ok && lane == 0) bc->abort = 1;
            __syncthreads();
            if (!ok) return;  // the sweepers read it from bc->abort
        }
    } else if constexpr (RMAX > 0) {
        // Long rows: the same block loop as below, with the samples' indices
        // in place of their slices (sweep_cols loads the slices).
        StepWindow<int> own;
        own.init(a, 0);
        int ip[M], ic[M], inx[M];
        block_indices<M>(ic, a, 0, own);
#pragma unroll
        for (int j = 0; j < M; ++j) inx[j] = ip[j] = ic[j];
        if (nb > 1) block_indices<M>(inx, a, 1, own);
        f4 *dm = l.dummy;
        sweep_cols_split<M, RMAX, kColsLdsRows, false, true, false>(
            a, l.lw, RL, gs, R, P4, nw, ic, ic, ic, l.coef, l.dots + (size_t)l.Rp * kSweepers * ND,
            dm);
        __syncthreads();
        for (int64_t blk = 0; blk < nb; ++blk) {
            const int par = (int)(blk & 1);
            const float *cp = l.coef + (size_t)(par ^ 1) * l.Rp * (M + 1);
            float *dd = l.dots + (size_t)par * l.Rp * kSweepers * ND;
            const bool has_next = blk + 1 < nb;
            if (blk == 0) {
                if (has_next)
                    sweep_cols_split<M, RMAX, kColsLdsRows, false, true, true>(
                        a, l.lw, RL, gs, R, P4, nw, ip, ic, inx, cp, dd, dm);
            } else if (has_next) {
                sweep_cols_split<M, RMAX, kColsLdsRows, true, true, true>(
                    a, l.lw, RL, gs, R, P4, nw, ip, ic, inx, cp, dd, dm);
            } else {
                sweep_cols_split<M, RMAX, kColsLdsRows, true, false, false>(
                    a, l.lw, RL, gs, R, P4, nw, ip, ic, inx, cp, dd, dm);
            }
#pragma unroll
            for (int j = 0; j < M; ++j) {
                ip[j] = ic[j];
                ic[j] = inx[j];
            }
            if (blk + 2 < nb) block_indices<M>(inx, a, blk + 2, own);
            __syncthreads();
            if (bc->abort) return;
        }
        // apply the last block's updates
        sweep_cols_split<M, RMAX, kColsLdsRows, true, false, false>(
            a, l.lw, RL, gs, R, P4, nw, ip, ic, inx,
            l.coef + (size_t)((nb - 1) & 1) * l.Rp * (M + 1), l.dots, dm);
    } else {
        StepWindow<int> own;
        own.init(a, 0);
        // Slices of the samples of the previous, current and next block.
        f4 xp[M][KS], xc[M][KS], xn[M][KS];
        load_samples<M, KS, NS>(xc, a, 0, own);
        if (nb > 1) load_samples<M, KS, NS>(xn, a, 1, own);
        // Products of the initial prototypes with block 0 (centred on its
        // first sample): f.f and f.(x_{0,i} - z), parity 1.
        sweep_rows<M, KS, LDSW, false, true, false, NS>(l.lw, RL, gs, R, P4, nw, xc, xc, xc, l.coef,
                                                     l.dots + (size_t)l.Rp * NS * ND);
        __syncthreads();
        for (int64_t blk = 0; blk < nb; ++blk) {
            const int par = (int)(blk & 1);
            const float *cp = l.coef + (size_t)(par ^ 1) * l.Rp * (M + 1);
            float *dd = l.dots + (size_t)par * l.Rp * NS * ND;
            const bool has_next = blk + 1 < nb;
            if (blk == 0) {
                if (has_next)
                    sweep_rows<M, KS, LDSW, false, true, true, NS>(l.lw, RL, gs, R, P4, nw, xp, xc, xn,
                                                                   cp, dd);
            } else if (has_next) {
                sweep_rows<M, KS, LDSW, true, true, true, NS>(l.lw, RL, gs, R, P4, nw, xp, xc, xn, cp,
                                                              dd);
            } else {
                sweep_rows<M, KS, LDSW, true, false, false, NS>(l.lw, RL, gs, R, P4, nw, xp, xc, xn,
                                                                cp, dd);
            }
#pragma unroll
            for (int j = 0; j < M; ++j)
#pragma unroll
                for (int t = 0; t < KS; ++t) {
                    xp[j][t] = xc[j][t];
                    xc[j][t] = xn[j][t];
                }
            if (blk + 2 < nb) load_samples<M, KS, NS>(xn, a, blk + 2, own);
            __syncthreads();
            if (bc->abort) return;
        }
        // apply the last block's updates
        sweep_rows<M, KS, LDSW, true, false, false, NS>(
            l.lw, RL, gs, R, P4, nw, xp, xc, xn, l.coef + (size_t)((nb - 1) & 1) * l.Rp * (M + 1),
            l.dots);
    }
    if (RL > 0) {
        __syncthreads();
        const row_t<true> *lw = rows_as<true>(l.lw);
        row_t<false> *g = rows_as<false>(gw);
        for (int e = tid; e < RL * P4; e += kBlock) g[e] = lw[e];
    }
}
}  // namespace

typedef void (*PipeKernel)(TrainArgs);

// The streamed-prototype kernel for block length m, kslots ks and ns
// sweepers, or null when there is none (defined in som_train_pipe_stream.hip).
PipeKernel pipe_stream_kernel(int m, int ks, int ns);
// The long-row (column-walk) kernel for block length m and at most rmax
// rows per workgroup, or null (som_train_pipe_stream.hip).
PipeKernel pipe_cols_kernel(int m, int rmax);

}  // namespace som
