// Sparse-input online training: the per-step method of the dense kernels
// (Eq. (1); BMU = smallest squared Euclidean distance, lowest index on
// ties) for samples given as CSR rows, at a cost per step that grows with
// the sample's non-zeros instead of with d.
//
// Lazy scale.  Prototype u is held as w_u = S_u v_u.  A step with factor h
// moves w_u to (1 - h) w_u + h x, which is S' = (1 - h) S together with
// v += (h / S') x: only v's entries at the sample's non-zero features
// change.  Distances use D = |x|^2 - 2 S (x . v) + |w|^2 with |w|^2 carried
// in w-space, |w'|^2 = (1-h)^2 |w|^2 + 2h(1-h) (x . w) + h^2 |x|^2, all in
// fp64.  v is fp64, so S may fall to 2^-900 before a unit's column is
// rescaled (v <- S' v, S' <- 1, then the step's sparse add with h / 1);
// h = 1 (1 - h = 0) takes the same path and leaves w = x exactly at the
// sample's features and 0 elsewhere.
//
// Layout.  V is feature-major, V[j * ldv + u], and lane l of workgroup b
// owns unit 64 b + l for the whole launch.  A step reads and writes, per
// non-zero, one contiguous run of 64 fp64 values per workgroup, and every
// access to a unit's column comes from that unit's lane, so program order
// is the only ordering the kernel relies on.
//
// Two waves per workgroup.  Wave 1 only polls the grid exchange: it waits
// for every workgroup's key of step s, leaves the BMU in LDS and meets
// wave 0 at one barrier per step.  Its memory counter then holds nothing
// but its own polls, so wave 0's gathers stay in flight across the
// exchange instead of being waited for by it.  Wave 0, on step s:
//   with step s-1's BMU: its factor h, S', the rescale if needed, and
//     x_s . v^(s-1) = (sum of step s's gathers, loaded two steps earlier)
//     + c_{s-2} x_{s-2} . x_s + c_{s-1} x_{s-1} . x_s, where c_t = h_t / S'_t
//     is step t's coefficient on x in v-space; then step s's key, published;
//   the sum of step s+1's gathers (loaded a step earlier);
//   stores of step s-1 at its features, from its corrected gathers (LDS);
//   step s's corrected gathers, G_s + c_{s-2} x_{s-2} + c_{s-1} x_{s-1} at
//     its features (the products only where the samples share a feature),
//     into LDS;
//   gathers of step s+2 (after the stores of step s-1 in program order).
#include "som_device.h"

namespace som {
namespace {
using namespace dev;

constexpr double kScaleLo = 0x1p-900;
constexpr double kScaleHi = 0x1p+64;

__device__ inline double readlane_d(double v, int l) {
    const long long b = __double_as_longlong(v);
    const unsigned lo = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)b, l);
    const unsigned hi = (unsigned)__builtin_amdgcn_readlane((int)(unsigned)(b >> 32), l);
    return __longlong_as_double((long long)(((unsigned long long)hi << 32) | lo));
}

// ---------------------------------------------------------------- CSR check

__global__ void csr_reset_kernel(DevState *state) {
    state->csr_bad = 0;
    state->csr_max_len = 0;
}

// Row i is entries [indptr[i], indptr[i+1]) of (indices, values); a row is
// well formed when 0 <= indptr[i] <= indptr[i+1] <= nnz and its indices
// increase strictly within [0, d).
__global__ __launch_bounds__(256) void csr_check_kernel(const int64_t *indptr,
                                                        const int32_t *indices, int64_t n,
                                                        int64_t nnz, int32_t d, DevState *state) {
    int longest = 0, bad = 0;
    for (int64_t i = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; i < n;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int64_t p0 = indptr[i], p1 = indptr[i + 1];
        if (p0 < 0 || p1 < p0 || p1 > nnz) {
            bad = 1;
            continue;
        }
        int prev = -1;
        for (int64_t k = p0; k < p1; ++k) {
            const int j = indices[k];
            if (j <= prev || j >= d) {
                bad = 1;
                break;
            }
            prev = j;
        }
        const int64_t len = p1 - p0;
        longest = max(longest, (int)min(len, (int64_t)INT32_MAX));
    }
    for (int o = 32; o > 0; o >>= 1) {
        longest = max(longest, __shfl_xor(longest, o));
        bad |= __shfl_xor(bad, o);
    }
    if ((threadIdx.x & 63) == 0) {
        if (bad) atomicOr(&state->csr_bad, 1);
        atomicMax(&state->csr_max_len, longest);
    }
}

// ---------------------------------------------------------- per-step entries

// Value of sample row r at feature j (0 if absent): binary search.
__device__ inline float csr_at(const int64_t *indptr, const int32_t *indices,
                               const float *values, int64_t r, int j) {
    const int64_t b0 = indptr[r], b1 = indptr[r + 1];
    int64_t lo = b0, hi = b1;
    while (lo < hi) {
        const int64_t mid = (lo + hi) >> 1;
        if (indices[mid] < j)
            lo = mid + 1;
        else
            hi = mid;
    }
    return (lo < b1 && indices[lo] == j) ? values[lo] : 0.f;
}

// One wave per step s of the call, and one more for a padding step: lane
// q < K holds entry q of sample order[s] (rows no longer than K): the byte offset of its feature's row of
// V (row d past the row's end), its value (0 past the end) and the values
// of the samples of steps s-1 and s-2 at that feature (0 where absent and
// before the call's first step).  sst[s] gets the products of the sample
// with itself and with those two samples (fp64), the mask of entries
// shared with either and the step's schedule entry (lr = 0 for padding).
template <int K>
__global__ __launch_bounds__(256) void sparse_steps_kernel(TrainArgs a, SparseArgs sp,
                                                           const int64_t *indptr,
                                                           const int32_t *indices,
                                                           const float *values) {
    const int q = threadIdx.x & 63;
    const int64_t s = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (s > a.nsteps) return;
    // step nsteps is padding only: it stands for the steps past the last
    const int64_t i = fetch_entry(a, s, 0);
    const int64_t p0 = indptr[i], len = s < a.nsteps ? indptr[i + 1] - p0 : 0;
    int j = a.d;
    float v = 0.f, pv1 = 0.f, pv2 = 0.f;
    if (q < len) {
        j = indices[p0 + q];
        v = values[p0 + q];
        if (s > 0) pv1 = csr_at(indptr, indices, values, fetch_entry(a, s - 1, 0), j);
        if (s > 1) pv2 = csr_at(indptr, indices, values, fetch_entry(a, s - 2, 0), j);
    }
    const uint64_t both = __ballot(pv1 != 0.f || pv2 != 0.f);
    double xx = (double)v * v, x1 = (double)v * pv1, x2 = (double)v * pv2;
    for (int o = 32; o > 0; o >>= 1) {
        xx += __shfl_xor(xx, o);
        x1 += __shfl_xor(x1, o);
        x2 += __shfl_xor(x2, o);
    }
    if (q < K) {
        sp.soff[s * K + q] = (uint32_t)((uint64_t)j * (uint64_t)sp.ldv * sizeof(double));
        sp.sval[s * K + q] = v;
        sp.spv1[s * K + q] = pv1;
        sp.spv2[s * K + q] = pv2;  // fp64: no conversion between load and use
    }
    if (q == 0) {
        const float2 sc = s < a.nsteps ? a.sched[s] : make_float2(0.f, 0.f);
        sp.sst[s] = {xx, x1, x2, both, sc.x, sc.y};
    }
}

// ----------------------------------------------------------- enter / leave

// V[j][u] = W[u][j] for u < N, j < d; 0 for padding units and row d.
// Workgroup (x, y) transposes the 64 x 64 tile of features 64x.. and units
// 64y.. through LDS.
__global__ __launch_bounds__(256) void sparse_enter_kernel(const float *W, int64_t ld, int32_t N,
                                                           int32_t d, double *V, int64_t ldv) {
    __shared__ float tile[64][65];
    const int64_t j0 = (int64_t)blockIdx.x * 64, u0 = (int64_t)blockIdx.y * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int r = ty; r < 64; r += 4) {
        const int64_t u = u0 + r, j = j0 + tx;
        tile[r][tx] = (u < N && j < d) ? W[u * ld + j] : 0.f;
    }
    __syncthreads();
    for (int r = ty; r < 64; r += 4) {
        const int64_t j = j0 + r, u = u0 + tx;
        if (j <= d) V[j * ldv + u] = (double)tile[tx][r];
    }
}

// S[u] = 1 and WW[u] = |w_u|^2 (fp64; 0 for padding units): one wave per unit.
__global__ __launch_bounds__(256) void sparse_norms_kernel(const float *W, int64_t ld, int32_t N,
                                                           int32_t d, double *S, double *WW,
                                                           int64_t ldv) {
    const int lane = threadIdx.x & 63;
    const int64_t u = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (u >= ldv) return;
    double acc = 0.0;
    if (u < N)
        for (int64_t j = lane; j < d; j += 64) {
            const double w = W[u * ld + j];
            acc += w * w;
        }
    for (int o = 32; o > 0; o >>= 1) acc += __shfl_xor(acc, o);
    if (lane == 0) {
        S[u] = 1.0;
        WW[u] = acc;
    }
}

// W[u][j] = fp32(S[u] V[j][u]) for u < N, j < d (tiles as sparse_enter).
__global__ __launch_bounds__(256) void sparse_leave_kernel(float *W, int64_t ld, int32_t N,
                                                           int32_t d, const double *V,
                                                           int64_t ldv, const double *S) {
    __shared__ float tile[64][65];
    const int64_t j0 = (int64_t)blockIdx.x * 64, u0 = (int64_t)blockIdx.y * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int r = ty; r < 64; r += 4) {
        const int64_t j = j0 + r, u = u0 + tx;
        tile[r][tx] = (j < d && u < N) ? (float)(S[u] * V[j * ldv + u]) : 0.f;
    }
    __syncthreads();
    for (int r = ty; r < 64; r += 4) {
        const int64_t u = u0 + r, j = j0 + tx;
        if (u < N && j < d) W[u * ld + j] = tile[tx][r];
    }
}

// ------------------------------------------------------------ training

// Entry q of one step's padded non-zeros, held by lane q, and word q of the
// step's scalars (lanes below kSparseStepWords).
struct Entries {
    uint32_t off;
    double vl, pv1, pv2;
    uint32_t word;
};

// Entries of step s; past the call's last step those of the padding step
// (the scratch row, value 0, lr 0), so the steps that round the loop up to
// a multiple of four read and write nothing but the scratch row.  The index
// is clamped before the loads, and no value is selected or copied after
// them: either would wait for the load.
template <int K>
__device__ inline Entries load_entries(const TrainArgs &a, const SparseArgs &sp, int64_t s) {
    const int lane = threadIdx.x & 63;
    const int64_t t = s < a.nsteps ? s : a.nsteps;
    const int64_t e = t * K + min(lane, K - 1);
    const uint32_t *w = reinterpret_cast<const uint32_t *>(sp.sst + t);
    return {sp.soff[e], sp.sval[e], sp.spv1[e], sp.spv2[e],
            w[min(lane, kSparseStepWords - 1)]};
}

__device__ inline uint32_t word_at(const Entries &e, int l) {
    return (uint32_t)__builtin_amdgcn_readlane((int)e.word, l);
}

// The step's scalars, read out of its entries.
__device__ inline SparseStep step_scalars(const Entries &e) {
    auto dbl = [&](int l) {
        return __longlong_as_double((long long)(((uint64_t)word_at(e, l + 1) << 32) | word_at(e, l)));
    };
    SparseStep st;
    st.xx = dbl(0);
    st.xd1 = dbl(2);
    st.xd2 = dbl(4);
    st.both = ((uint64_t)word_at(e, 7) << 32) | word_at(e, 6);
    st.lr = __uint_as_float(word_at(e, 8));
    st.c2 = __uint_as_float(word_at(e, 9));
    return st;
}

// LDS shared by the two waves of a workgroup.
template <int K>
struct SparseShared {
    double cur[2][K][64];  // wave 0: corrected gathers of a step, by parity
    int bmu[2];            // wave 1 -> wave 0: BMU of the step, by parity
    int abort;
};

// Raw buffer access to this workgroup's columns of V: the row's byte
// offset goes in the scalar offset and the lane's column in the vector
// offset, so a step's addresses cost no vector arithmetic.
__device__ inline double buf_load(__amdgpu_buffer_rsrc_t r, int voff, uint32_t soff) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b64(r, voff, (int)soff, 0);
    return __builtin_bit_cast(double, v);
}
__device__ inline void buf_store(__amdgpu_buffer_rsrc_t r, int voff, uint32_t soff, double x) {
    typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));
    __builtin_amdgcn_raw_buffer_store_b64(__builtin_bit_cast(u32x2, x), r, voff, (int)soff, 0);
}

template <int K>
struct SparseLane {
    const TrainArgs &a;
    const SparseArgs &sp;
    SparseShared<K> &sh;
    __amdgpu_buffer_rsrc_t rv;  // V from this workgroup's first column
    int u0, u, lane;
    bool active;
    float4 p;
    float inv_cols;
    double S, WW;       // scale and |w|^2 of the lane's unit
    double c1, c2;      // coefficients on x in v-space of the last two steps
    double dpre;        // sum of the next step's gathers times its values
    double xx, xw;      // |x|^2 and x . w of the step last keyed
    // Entries of four consecutive steps; step s uses slot s % 4, so the
    // slots rotate by index, not by register copies (a copy of a value
    // still being loaded would wait for the load).
    Entries E[4];
    double G0[K], G1[K];  // raw gathers of two steps (by parity)
    double g0, g1;        // factors still to apply to them (rescales)

    __device__ SparseLane(const TrainArgs &a_, const SparseArgs &sp_, SparseShared<K> &sh_)
        : a(a_), sp(sp_), sh(sh_) {}

    // v <- F v over the lane's whole column (rows 0..d).
    __device__ void rescale(double F) {
        const int64_t rows = (int64_t)a.d + 1, ldv = sp.ldv;
        double *col = sp.V + u;
        int64_t j = 0;
        for (; j + 8 <= rows; j += 8) {
            double t[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) t[k] = col[(j + k) * ldv];
#pragma unroll
            for (int k = 0; k < 8; ++k) col[(j + k) * ldv] = t[k] * F;
        }
        for (; j < rows; ++j) col[j * ldv] *= F;
    }

    __device__ void gather(double (&G)[K], const Entries &e) {
#pragma unroll
        for (int q = 0; q < K; ++q)
            G[q] = buf_load(rv, lane * 8, (uint32_t)__builtin_amdgcn_readlane((int)e.off, q));
    }

    __device__ double dot_pre(const double (&G)[K], const Entries &e) const {
        double t = 0.0;
#pragma unroll
        for (int q = 0; q < K; ++q) t = fma(readlane_d(e.vl, q), G[q], t);
        return t;
    }

    // Stores of the step whose entries are e, from cur[b], coefficient c;
    // LDS is read eight entries at a time ahead of the stores.
    __device__ void store(const Entries &e, int b, double c) {
#pragma unroll
        for (int q0 = 0; q0 < K; q0 += 8) {
            double t[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) t[k] = sh.cur[b][q0 + k][lane];
#pragma unroll
            for (int k = 0; k < 8; ++k)
                buf_store(rv, lane * 8, (uint32_t)__builtin_amdgcn_readlane((int)e.off, q0 + k),
                          fma(c, readlane_d(e.vl, q0 + k), t[k]));
        }
    }

    __device__ unsigned long long key_of(double D) const {
        return wave_argmin_key(active ? dist_order_bits((float)D) : 0xffffffffu, u0);
    }

    // Step s-1's update from its BMU c and scalars prev, up to step s's
    // distance (from its scalars st): the factor h, S' = (1 - h) S, the
    // rescale if S' leaves its range, |w|^2 and x_s . w.  No division: with
    // F = S', x_s . w = F (dpre + c_{s-2} x_{s-2}.x_s) + h x_{s-1}.x_s.  Sets
    // hF = (h, F) for coefficients(); ga and gb are the pending factors of
    // step s's and step s+1's gathers, cb the LDS buffer of step s-1's.
    __device__ double finish(int c, const SparseStep &prev, double &ga, double &gb, int cb,
                             const SparseStep &st, double2 &hF) {
        int cr, cc;
        unit_rc(c, a.cols, inv_cols, cr, cc);
        const float h =
            active ? neighbour_h(a, p, (float)cr, (float)cc, (float)(cr & 1), prev.lr, prev.c2)
                   : 0.f;
        const double hd = h, om = 1.0 - hd;
        double F = om * S;
        const double xw_s = fma(F, fma(c1, st.xd2, dpre), hd * st.xd1);
        WW = fma(om * om, WW, hd * fma(2.0 * om, xw, hd * xx));
        const bool out = active && !(fabs(F) >= kScaleLo && fabs(F) <= kScaleHi);
        if (__ballot(out) != 0) {
            if (!active) F = 1.0;
            rescale(F);
#pragma unroll
            for (int q = 0; q < K; ++q) sh.cur[cb][q][lane] *= F;
            // gathers still in flight are scaled where they are used
            ga *= F;
            gb *= F;
            c1 *= F;
            hF = make_double2(hd, 1.0);
            S = 1.0;
        } else {
            hF = make_double2(hd, F);
            S = F;
        }
        xw = xw_s;
        xx = st.xx;
        return fma(-2.0, xw_s, xx) + WW;
    }

    // After the key is out: step s-1's coefficient on x in v-space.
    __device__ void coefficients(double2 hF) {
        c2 = c1;
        c1 = hF.x / hF.y;
    }

    // One step of wave 0; returns false once the exchange gave up.
    template <int P>
    __device__ bool step(int64_t s, double (&Ga)[K], double &ga, double (&Gb)[K], double &gb) {
        const Entries &ep = E[(P + 3) & 3], &ec = E[P], &en = E[(P + 1) & 3],
                      &enn = E[(P + 2) & 3];
        constexpr int bc = P & 1, bp = bc ^ 1;  // LDS buffers of steps s and s-1
        // step s's gathers are Ga (loaded two steps ago), step s+1's Gb
        const SparseStep st = step_scalars(ec);
        double D;
        double2 hF = make_double2(0.0, 1.0);
        if (s == 0) {
            xw = S * dpre;
            xx = st.xx;
            D = fma(-2.0, xw, xx) + WW;
        } else {
            __syncthreads();   // step s-1's BMU from wave 1
            if (sh.abort) return false;
            D = finish(sh.bmu[(s - 1) & 1], step_scalars(ep), ga, gb, bp, st, hF);
        }
        const unsigned long long key = key_of(D);
        if (a.grid == 1) {
            if (lane == 0) sh.bmu[s & 1] = (int)(key & (unsigned long long)kMaxUnits);
        } else {
            exchange_publish(a, s, key);
        }
        if (s > 0) coefficients(hF);
        // step s's corrected gathers into LDS (before this step's stores, so
        // waiting for its gathers never waits for them)
#pragma unroll
        for (int q = 0; q < K; ++q) sh.cur[bc][q][lane] = Ga[q] * ga;
        // the updates of steps s-1 and s-2 at the features shared with them
        for (uint64_t m = st.both; m != 0; m &= m - 1) {
            const int q = __builtin_ctzll(m);
            const double v = sh.cur[bc][q][lane];
            sh.cur[bc][q][lane] = fma(c2, readlane_d(ec.pv2, q), fma(c1, readlane_d(ec.pv1, q), v));
        }
        dpre = gb * dot_pre(Gb, en);
        store(ep, bp, c1);
        gather(Ga, enn);
        ga = 1.0;
        E[(P + 3) & 3] = load_entries<K>(a, sp, s + 3);
        return true;
    }
};

// Wave 1: the BMU of every step over the grid into LDS (with one
// workgroup wave 0 leaves it there itself), one barrier per step.
__device__ inline void sparse_exchange_wave(const TrainArgs &a, int *bmu, int *abort,
                                            int64_t nsteps4) {
    const int lane = threadIdx.x & 63;
    PollRegs<1> no_regs;  // one poll at a time: none left in flight
    for (int64_t s = 0; s < nsteps4; ++s) {
        if (a.grid > 1) {
            const int c = exchange_wait<1>(a, s, 0ull, [] {}, no_regs);
            if (lane == 0) {
                if (c < 0)
                    *abort = 1;
                else
                    bmu[s & 1] = c;
            }
        }
        __syncthreads();
        if (*abort) return;
        if (blockIdx.x == 0 && lane == 0 && a.bmu_trace && s < a.nsteps)
            a.bmu_trace[s] = bmu[s & 1];
    }
}

// One persistent cooperative launch over the call's steps; workgroup b owns
// units 64 b .. 64 b + 63 (wave 0 lane l: unit 64 b + l) and wave 1 runs its
// exchange.  The step loop runs to a multiple of four steps; the extra
// steps have lr = 0 and touch only the scratch row.
template <int K>
__global__ __launch_bounds__(128) void sparse_train_kernel(TrainArgs a, SparseArgs sp) {
    __shared__ SparseShared<K> sh;
    if (a.state->order_bad) return;  // same value for every workgroup
    const int64_t T4 = (a.nsteps + 3) & ~(int64_t)3;
    if (threadIdx.x == 0) sh.abort = 0;
    __syncthreads();
    if (threadIdx.x >= 64) {
        sparse_exchange_wave(a, sh.bmu, &sh.abort, T4);
        return;
    }
    SparseLane<K> L(a, sp, sh);
    L.lane = threadIdx.x & 63;
    L.u0 = blockIdx.x * 64;
    L.u = L.u0 + L.lane;
    L.rv = __builtin_amdgcn_make_buffer_rsrc(sp.V + L.u0, (short)0, 0x7fffffff, 0x00020000);
    L.active = L.u < a.N;
    L.inv_cols = 1.f / (float)a.cols;
    int ur, uc;
    unit_rc(L.active ? L.u : 0, a.cols, L.inv_cols, ur, uc);
    L.p = make_float4((float)ur, (float)uc, (float)(ur & 1), 0.f);
    L.S = sp.S[L.u];
    L.WW = sp.WW[L.u];
    L.c1 = 0.0;
    L.c2 = 0.0;
    // "Step -1" stores zeros into the scratch row.
    L.E[3] = {(uint32_t)((uint64_t)a.d * (uint64_t)sp.ldv * sizeof(double)), 0.0, 0.0, 0.0, 0u};
    L.E[0] = load_entries<K>(a, sp, 0);
    L.E[1] = load_entries<K>(a, sp, 1);
    L.E[2] = load_entries<K>(a, sp, 2);
#pragma unroll
    for (int q = 0; q < K; ++q) {
        sh.cur[0][q][L.lane] = 0.0;
        sh.cur[1][q][L.lane] = 0.0;
    }
    L.gather(L.G0, L.E[0]);
    L.gather(L.G1, L.E[1]);
    L.g0 = 1.0;
    L.g1 = 1.0;
    L.dpre = L.dot_pre(L.G0, L.E[0]);
    for (int64_t s = 0; s < T4; s += 4) {
        if (!L.template step<0>(s, L.G0, L.g0, L.G1, L.g1)) return;
        if (!L.template step<1>(s + 1, L.G1, L.g1, L.G0, L.g0)) return;
        if (!L.template step<2>(s + 2, L.G0, L.g0, L.G1, L.g1)) return;
        if (!L.template step<3>(s + 3, L.G1, L.g1, L.G0, L.g0)) return;
    }
    // the last step's update and stores
    __syncthreads();
    if (sh.abort) return;
    const SparseStep none = {0.0, 0.0, 0.0, 0ull, 0.f, 0.f};
    double2 hF;
    (void)L.finish(sh.bmu[(T4 - 1) & 1], step_scalars(L.E[3]), L.g0, L.g1, 1, none, hF);
    L.coefficients(hF);
    L.store(L.E[3], 1, L.c1);
    sp.S[L.u] = L.S;
    sp.WW[L.u] = L.WW;
}

template <int K>
hipError_t launch_sparse_train_k(const TrainArgs &a, const SparseArgs &sp, hipStream_t s) {
    TrainArgs aa = a;
    SparseArgs ss = sp;
    void *args[] = {&aa, &ss};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(&sparse_train_kernel<K>),
                                      dim3(a.grid), dim3(128), args, 0, s);
}

template <int K>
hipError_t launch_sparse_steps_k(const TrainArgs &a, const SparseArgs &sp, const int64_t *indptr,
                                 const int32_t *indices, const float *values, hipStream_t s) {
    const int64_t blocks = (a.nsteps + 1 + 3) / 4;
    sparse_steps_kernel<K><<<dim3((unsigned)blocks), dim3(256), 0, s>>>(a, sp, indptr, indices,
                                                                         values);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_csr_check(const int64_t *indptr, const int32_t *indices, int64_t n,
                            int64_t nnz, int32_t d, DevState *state, hipStream_t s) {
    csr_reset_kernel<<<1, 1, 0, s>>>(state);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t blocks = (n + 255) / 256 < 2048 ? (n + 255) / 256 : 2048;
    csr_check_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(indptr, indices, n, nnz, d,
                                                                 state);
    return hipGetLastError();
}

hipError_t launch_sparse_steps(const TrainArgs &a, const SparseArgs &sp, const int64_t *indptr,
                               const int32_t *indices, const float *values, hipStream_t s) {
    switch (sp.K) {
        case 16: return launch_sparse_steps_k<16>(a, sp, indptr, indices, values, s);
        case 32: return launch_sparse_steps_k<32>(a, sp, indptr, indices, values, s);
        case 64: return launch_sparse_steps_k<64>(a, sp, indptr, indices, values, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_sparse_enter(const TrainArgs &a, const SparseArgs &sp, hipStream_t s) {
    const dim3 grid((unsigned)(((int64_t)a.d + 1 + 63) / 64), (unsigned)(sp.ldv / 64));
    sparse_enter_kernel<<<grid, dim3(256), 0, s>>>(a.W, a.ld, a.N, a.d, sp.V, sp.ldv);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    sparse_norms_kernel<<<dim3((unsigned)(sp.ldv / 4)), dim3(256), 0, s>>>(a.W, a.ld, a.N, a.d,
                                                                           sp.S, sp.WW, sp.ldv);
    return hipGetLastError();
}

hipError_t launch_sparse_leave(const TrainArgs &a, const SparseArgs &sp, hipStream_t s) {
    const dim3 grid((unsigned)(((int64_t)a.d + 63) / 64), (unsigned)((a.N + 63) / 64));
    sparse_leave_kernel<<<grid, dim3(256), 0, s>>>(a.W, a.ld, a.N, a.d, sp.V, sp.ldv, sp.S);
    return hipGetLastError();
}

hipError_t launch_train_sparse(const TrainArgs &a, const SparseArgs &sp, hipStream_t s) {
    if (a.grid < 1 || (int64_t)a.grid * 64 != sp.ldv || a.grid > kSparseMaxGrid)
        return hipErrorInvalidValue;
    switch (sp.K) {
        case 16: return launch_sparse_train_k<16>(a, sp, s);
        case 32: return launch_sparse_train_k<32>(a, sp, s);
        case 64: return launch_sparse_train_k<64>(a, sp, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace som
