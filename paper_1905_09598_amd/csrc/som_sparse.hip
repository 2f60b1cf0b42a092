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
// Step s, after its key is published to the grid exchange:
//   (A) store step s-1's update at its features, from its corrected
//       gathered values (kept in LDS, one slot per lane and entry);
//   (B) correct step s's gathered values (read before step s-1's stores)
//       by step s-1's update at the features the two samples share, using
//       the previous sample's value at each of step s's features, into LDS;
//   (C) gather step s+1's features (these loads follow every store so far
//       in program order);
//   then wait for the exchange and compute h, S', and
//   x_{s+1} . v^(s) = (sum over step s+1's gathers) + (h / S') x_s . x_{s+1},
//   which gives step s+1's distance.  Only that sum sits between the
//   exchange and the next key; (A)-(C) overlap the exchange.
#include "som_device.h"

namespace som {
namespace {
using namespace dev;

constexpr double kScaleLo = 0x1p-900;
constexpr double kScaleHi = 0x1p+64;

__device__ inline float readlane_f(float v, int l) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(v), l));
}
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

// One wave per step s of the call: lane q < K holds entry q of sample
// order[s] (rows no longer than K): its feature (d past the row's end), its
// value (0 past the end) and the value of step s-1's sample at that feature
// (0 where that sample has none, and at s = 0), found by binary search in
// the previous row.  sxs[s] = (|x_s|^2, x_{s-1} . x_s) in fp64.
template <int K>
__global__ __launch_bounds__(256) void sparse_steps_kernel(TrainArgs a, SparseArgs sp,
                                                           const int64_t *indptr,
                                                           const int32_t *indices,
                                                           const float *values) {
    const int q = threadIdx.x & 63;
    const int64_t s = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (s >= a.nsteps) return;
    const int64_t i = fetch_entry(a, s, 0);
    const int64_t p0 = indptr[i], len = indptr[i + 1] - p0;
    int j = a.d;
    float v = 0.f, pv = 0.f;
    if (q < len) {
        j = indices[p0 + q];
        v = values[p0 + q];
        if (s > 0) {
            const int64_t ip = fetch_entry(a, s - 1, 0);
            const int64_t b0 = indptr[ip], b1 = indptr[ip + 1];
            int64_t lo = b0, hi = b1;
            while (lo < hi) {
                const int64_t mid = (lo + hi) >> 1;
                if (indices[mid] < j)
                    lo = mid + 1;
                else
                    hi = mid;
            }
            if (lo < b1 && indices[lo] == j) pv = values[lo];
        }
    }
    double xx = (double)v * v, xd = (double)v * pv;
    for (int o = 32; o > 0; o >>= 1) {
        xx += __shfl_xor(xx, o);
        xd += __shfl_xor(xd, o);
    }
    if (q < K) {
        sp.sidx[s * K + q] = j;
        sp.sval[s * K + q] = v;
        sp.spv[s * K + q] = pv;
    }
    if (q == 0) sp.sxs[s] = make_double2(xx, xd);
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

// Entry q of one step's padded non-zeros, held by lane q.
struct Entries {
    int ix;
    float vl, pv;
};

// Entries of step s; past the call's last step, padding only (feature d,
// value 0), so the steps that round the loop up to a multiple of four
// read and write nothing but the scratch row.
template <int K>
__device__ inline Entries load_entries(const TrainArgs &a, const SparseArgs &sp, int64_t s) {
    const int q = min((int)(threadIdx.x & 63), K - 1);
    const int64_t e = (s < a.nsteps ? s : 0) * K + q;
    const Entries v = {sp.sidx[e], sp.sval[e], sp.spv[e]};
    const Entries pad = {a.d, 0.f, 0.f};
    return s < a.nsteps ? v : pad;
}

// (|x_s|^2, x_{s-1} . x_s) of step s, 64 steps per window: lane l holds
// step base + l, the next window is loaded while this one is in use; 0
// past the call's last step.
struct XsWindow {
    int64_t base;
    double2 cur, next;

    __device__ static double2 fetch(const TrainArgs &a, const SparseArgs &sp, int64_t s) {
        const double2 v = sp.sxs[s < a.nsteps ? s : 0];
        return s < a.nsteps ? v : make_double2(0.0, 0.0);
    }
    __device__ void init(const TrainArgs &a, const SparseArgs &sp) {
        base = 0;
        cur = fetch(a, sp, threadIdx.x & 63);
        next = fetch(a, sp, 64 + (threadIdx.x & 63));
    }
    // non-decreasing s >= base
    __device__ double2 get(const TrainArgs &a, const SparseArgs &sp, int64_t s) {
        if (s >= base + 64) {
            base += 64;
            cur = next;
            next = fetch(a, sp, base + 64 + (threadIdx.x & 63));
        }
        const int l = (int)(s - base);
        return make_double2(readlane_d(cur.x, l), readlane_d(cur.y, l));
    }
};

template <int K>
struct SparseLane {
    const TrainArgs &a;
    const SparseArgs &sp;
    double (*cur)[64];  // LDS [K][64]: lane l's corrected gathers of one step
    int u0, u, lane;
    bool active;
    float4 p;
    float inv_cols;
    double S, WW;   // scale and |w|^2 of the lane's unit
    double dot;     // x_s . v (v before step s)
    double xx;      // |x_s|^2
    double coef;    // step s-1's coefficient on x in v-space
    // Entries of four consecutive steps; step s uses slot s % 4, so the
    // slots rotate by index, not by register copies (a copy of a value
    // still being loaded would wait for the load).
    Entries E[4];
    StepWindow<float2> sw;
    XsWindow xw;
    double R[K];    // raw gathers of the next step

    __device__ SparseLane(const TrainArgs &a_, const SparseArgs &sp_, double (*cur_)[64])
        : a(a_), sp(sp_), cur(cur_) {}

    __device__ double *at(int j) const { return sp.V + (int64_t)j * sp.ldv + u; }

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

    // Stores of the step whose entries are ep, from cur.
    __device__ void store_prev(const Entries &ep) {
#pragma unroll
        for (int q = 0; q < K; ++q)
            *at(__builtin_amdgcn_readlane(ep.ix, q)) =
                fma(coef, (double)readlane_f(ep.vl, q), cur[q][lane]);
    }

    template <int P>
    __device__ bool step(int64_t s) {
        const Entries &ep = E[(P + 3) & 3], &ec = E[P], &en = E[(P + 1) & 3];
        const double xw_ = S * dot;
        const double D = fma(-2.0, xw_, xx) + WW;
        const unsigned long long key =
            wave_argmin_key(active ? dist_order_bits((float)D) : 0xffffffffu, u0);
        exchange_publish(a, s, key);
        store_prev(ep);
#pragma unroll
        for (int q = 0; q < K; ++q) cur[q][lane] = fma(coef, (double)readlane_f(ec.pv, q), R[q]);
#pragma unroll
        for (int q = 0; q < K; ++q) R[q] = *at(__builtin_amdgcn_readlane(en.ix, q));
        const float2 sc = sw.get(a, s);
        const double2 xs_n = xw.get(a, sp, s + 1);

        const int c = exchange_wait(a, s, key);
        if (c < 0) return false;
        if (blockIdx.x == 0 && lane == 0 && a.bmu_trace && s < a.nsteps) a.bmu_trace[s] = c;
        int cr, cc;
        unit_rc(c, a.cols, inv_cols, cr, cc);
        const float h =
            active ? neighbour_h(a, p, (float)cr, (float)cc, (float)(cr & 1), sc.x, sc.y) : 0.f;
        const double hd = h, om = 1.0 - hd;
        double F = om * S;
        double dpre = 0.0;
#pragma unroll
        for (int q = 0; q < K; ++q) dpre = fma((double)readlane_f(en.vl, q), R[q], dpre);
        const bool out = active && !(fabs(F) >= kScaleLo && fabs(F) <= kScaleHi);
        if (__ballot(out) != 0) {
            if (!active) F = 1.0;
            rescale(F);
#pragma unroll
            for (int q = 0; q < K; ++q) {
                cur[q][lane] *= F;
                R[q] *= F;
            }
            dpre *= F;
            S = 1.0;
            coef = hd;
        } else {
            S = F;
            coef = hd / F;
        }
        WW = fma(om * om, WW, hd * fma(2.0 * om, xw_, hd * xx));
        dot = fma(coef, xs_n.y, dpre);
        xx = xs_n.x;
        E[(P + 3) & 3] = load_entries<K>(a, sp, s + 3);
        return true;
    }
};

// One persistent cooperative launch over the call's steps; workgroup b (one
// wave) owns units 64 b .. 64 b + 63.  The step loop runs to a multiple of
// four steps; the extra steps have lr = 0 and touch only the scratch row.
template <int K>
__global__ __launch_bounds__(64) void sparse_train_kernel(TrainArgs a, SparseArgs sp) {
    __shared__ double cur[K][64];
    if (a.state->order_bad) return;  // same value for every workgroup
    SparseLane<K> L(a, sp, cur);
    L.lane = threadIdx.x & 63;
    L.u0 = blockIdx.x * 64;
    L.u = L.u0 + L.lane;
    L.active = L.u < a.N;
    L.inv_cols = 1.f / (float)a.cols;
    int ur, uc;
    unit_rc(L.active ? L.u : 0, a.cols, L.inv_cols, ur, uc);
    L.p = make_float4((float)ur, (float)uc, (float)(ur & 1), 0.f);
    L.S = sp.S[L.u];
    L.WW = sp.WW[L.u];
    L.coef = 0.0;
    L.sw.init(a, 0);
    L.xw.init(a, sp);
    // "Step -1" stores zeros into the scratch row.
    L.E[3] = {a.d, 0.f, 0.f};
    L.E[0] = load_entries<K>(a, sp, 0);
    L.E[1] = load_entries<K>(a, sp, 1);
    L.E[2] = load_entries<K>(a, sp, 2);
    double dot = 0.0;
#pragma unroll
    for (int q = 0; q < K; ++q) {
        cur[q][L.lane] = 0.0;
        L.R[q] = *L.at(__builtin_amdgcn_readlane(L.E[0].ix, q));
        dot = fma((double)readlane_f(L.E[0].vl, q), L.R[q], dot);
    }
    L.dot = dot;
    L.xx = L.xw.get(a, sp, 0).x;
    for (int64_t s = 0; s < a.nsteps; s += 4) {
        if (!L.template step<0>(s)) return;
        if (!L.template step<1>(s + 1)) return;
        if (!L.template step<2>(s + 2)) return;
        if (!L.template step<3>(s + 3)) return;
    }
    L.store_prev(L.E[3]);
    sp.S[L.u] = L.S;
    sp.WW[L.u] = L.WW;
}

template <int K>
hipError_t launch_sparse_train_k(const TrainArgs &a, const SparseArgs &sp, hipStream_t s) {
    TrainArgs aa = a;
    SparseArgs ss = sp;
    void *args[] = {&aa, &ss};
    return hipLaunchCooperativeKernel(reinterpret_cast<const void *>(&sparse_train_kernel<K>),
                                      dim3(a.grid), dim3(64), args, 0, s);
}

template <int K>
hipError_t launch_sparse_steps_k(const TrainArgs &a, const SparseArgs &sp, const int64_t *indptr,
                                 const int32_t *indices, const float *values, hipStream_t s) {
    const int64_t blocks = (a.nsteps + 3) / 4;
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
