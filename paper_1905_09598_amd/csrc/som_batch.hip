// Batch-map training: Kohonen's batch rule, the SOM variant that Sec. 4
// attributes to earlier GPU SOMs ([25], [26]), beside the paper's online
// rule.  One epoch assigns every sample to its BMU (the batched MFMA BMU of
// som_eval.hip) and then sets
//     w_u = sum_c h(u, c) S_c / sum_c h(u, c) n_c,
// S_c and n_c being the sum and the number of the samples whose BMU is c,
// h the Gaussian of Eq. (1) without the learning rate.  A unit whose
// denominator is 0 keeps its prototype.
//
// The lattice Gaussian factors over the two lattice axes: with a = 1 (RECT)
// or 3/4 (HEX, the square of its row pitch sqrt(3)/2) and the column offset
// o = (parity(u) - parity(c)) / 2 of HEX's shifted odd rows (0 for RECT),
//     h(u, c) = exp(-a dr^2 / (2 sigma^2)) exp(-(dc + o)^2 / (2 sigma^2)),
// so the N x N product is a blur along the columns (one table per offset)
// followed by a blur along the rows, O(N d (rows + cols)) instead of
// O(N^2 d).  Everything after the BMU is fp64; the count n_c rides along
// as column d of S.
#include "som_internal.h"

#include <math.h>

#include <algorithm>

namespace som {
namespace {

constexpr int kUnitsPerWG = 64;   // batch_sums_kernel: units per workgroup
constexpr int kColsPerWG = 256;   // ... and columns (one per thread)

// S[u][j] (u < N, j <= d, row pitch dp) = sum of X[i][j] over the samples
// i with BMU u, in increasing i; S[u][d] = their number.  Workgroup (x, y)
// owns units 64 x .. and columns 256 y ..: it walks the BMU list 256 at a
// time, compacts the samples that fall in its units and adds their rows
// into fp64 accumulators in LDS (one column per thread).
__global__ __launch_bounds__(256) void batch_sums_kernel(const int32_t *bmu, const float *X,
                                                         int64_t n, int32_t d, int32_t N,
                                                         double *S, int64_t dp) {
    __shared__ double acc[kUnitsPerWG][kColsPerWG];
    __shared__ int hit_i[256];
    __shared__ int hit_u[256];
    __shared__ int wave_count[4];
    const int t = threadIdx.x, lane = t & 63, wave = t >> 6;
    const int u0 = blockIdx.x * kUnitsPerWG;
    const int64_t j = (int64_t)blockIdx.y * kColsPerWG + t;
    for (int r = 0; r < kUnitsPerWG; ++r) acc[r][t] = 0.0;
    for (int64_t i0 = 0; i0 < n; i0 += 256) {
        const int64_t i = i0 + t;
        const int c = i < n ? bmu[i] - u0 : -1;
        const bool mine = c >= 0 && c < kUnitsPerWG;
        const unsigned long long m = __ballot(mine);
        const int before = __builtin_popcountll(m & ((1ull << lane) - 1ull));
        if (lane == 0) wave_count[wave] = __builtin_popcountll(m);
        __syncthreads();
        int base = 0, total = 0;
        for (int w = 0; w < 4; ++w) {
            if (w < wave) base += wave_count[w];
            total += wave_count[w];
        }
        if (mine) {
            hit_i[base + before] = (int)(i - i0);
            hit_u[base + before] = c;
        }
        __syncthreads();
        for (int k = 0; k < total; ++k) {  // in increasing sample index
            const int64_t s = i0 + hit_i[k];
            const double v = j < d ? (double)X[s * d + j] : (j == d ? 1.0 : 0.0);
            acc[hit_u[k]][t] += v;
        }
        __syncthreads();
    }
    if (j < dp)
        for (int r = 0; r < kUnitsPerWG && u0 + r < N; ++r) S[(int64_t)(u0 + r) * dp + j] = acc[r][t];
}

// Factor tables of the lattice Gaussian at radius sigma:
//   Hr[ru][rc]     = exp(-a (ru - rc)^2 / (2 sigma^2)),
//   Hc[o][cu][cc]  = exp(-(cu - cc + off_o)^2 / (2 sigma^2)), off = 0, +1/2, -1/2
// (a = 1 and one offset for RECT; a = 3/4 and three for HEX); sigma = 0
// gives the Kronecker delta, sigma = inf all ones.
__global__ void batch_tables_kernel(int32_t rows, int32_t cols, int32_t topology, double sigma,
                                    double *Hr, double *Hc) {
    const int64_t nr = (int64_t)rows * rows, nc = (int64_t)cols * cols;
    const int planes = topology == 1 ? 3 : 1;
    const double a = topology == 1 ? 0.75 : 1.0;
    const double off[3] = {0.0, 0.5, -0.5};
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < nr + planes * nc;
         e += (int64_t)gridDim.x * blockDim.x) {
        double g;
        if (e < nr) {
            const double dr = (double)(e / rows) - (double)(e % rows);
            g = a * dr * dr;
        } else {
            const int64_t k = e - nr, o = k / nc, q = k % nc;
            const double dx = (double)(q / cols) - (double)(q % cols) + off[o];
            g = dx * dx;
        }
        double h;
        if (sigma == 0.0)
            h = g == 0.0 ? 1.0 : 0.0;
        else if (isinf(sigma))
            h = 1.0;
        else
            h = exp(-g / (2.0 * sigma * sigma));
        if (e < nr)
            Hr[e] = h;
        else
            Hc[e - nr] = h;
    }
}

// Column blur: T[o][r][cu][j] = sum_cc Hc[o][cu][cc] S[r][cc][j].  Workgroup
// (x, y, z): lattice row r = x / ceil(cols/64) with output columns
// 64 (x % ceil(cols/64)) .., columns 64 y .. of j, offset plane z.  Thread
// t: j = t % 64, outputs cu = cu0 + t / 64 + 4 k (k < 16).  S and Hc are
// staged through LDS 32 lattice columns at a time.
__global__ __launch_bounds__(256) void batch_col_pass_kernel(const double *S, const double *Hc,
                                                             double *T, int32_t rows,
                                                             int32_t cols, int64_t dp) {
    __shared__ double ls[32][64];
    __shared__ double lh[64][33];
    const int t = threadIdx.x, jl = t & 63, g = t >> 6;
    const int cblocks = (cols + 63) / 64;
    const int r = blockIdx.x / cblocks, cu0 = (blockIdx.x % cblocks) * 64;
    const int64_t j = (int64_t)blockIdx.y * 64 + jl;
    const int o = blockIdx.z;
    const double *hc = Hc + (int64_t)o * cols * cols;
    double acc[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) acc[k] = 0.0;
    for (int cc0 = 0; cc0 < cols; cc0 += 32) {
        for (int e = t; e < 32 * 64; e += 256) {
            const int cc = cc0 + e / 64;
            const int64_t jj = (int64_t)blockIdx.y * 64 + (e % 64);
            ls[e / 64][e % 64] =
                (cc < cols && jj < dp) ? S[((int64_t)r * cols + cc) * dp + jj] : 0.0;
        }
        for (int e = t; e < 64 * 32; e += 256) {
            const int cu = cu0 + e / 32, cc = cc0 + e % 32;
            lh[e / 32][e % 32] = (cu < cols && cc < cols) ? hc[(int64_t)cu * cols + cc] : 0.0;
        }
        __syncthreads();
        for (int c = 0; c < 32; ++c) {
            const double s = ls[c][jl];
#pragma unroll
            for (int k = 0; k < 16; ++k) acc[k] = fma(lh[g + 4 * k][c], s, acc[k]);
        }
        __syncthreads();
    }
    if (j < dp)
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            const int cu = cu0 + g + 4 * k;
            if (cu < cols)
                T[(((int64_t)o * rows + r) * cols + cu) * dp + j] = acc[k];
        }
}

// Row blur: O[ru][cu][j] = sum_rc Hr[ru][rc] T[o(ru, rc)][rc][cu][j], where
// the HEX offset plane o follows the rows' parities (0 equal, 1 for an odd
// ru over an even rc, 2 the other way).  Workgroup (x, y): lattice column
// cu = x / ceil(rows/64) with output rows 64 (x % ceil(rows/64)) .., columns
// 64 y .. of j.  Thread t: j = t % 64, outputs ru = ru0 + t / 64 + 4 k; the
// parity of ru is the same for all of a thread's k.
__global__ __launch_bounds__(256) void batch_row_pass_kernel(const double *T, const double *Hr,
                                                             double *O, int32_t rows,
                                                             int32_t cols, int32_t planes,
                                                             int64_t dp) {
    __shared__ double lt[3][32][64];
    __shared__ double lh[64][33];
    const int t = threadIdx.x, jl = t & 63, g = t >> 6;
    const int rblocks = (rows + 63) / 64;
    const int cu = blockIdx.x / rblocks, ru0 = (blockIdx.x % rblocks) * 64;
    const int64_t j = (int64_t)blockIdx.y * 64 + jl;
    const int pu = (ru0 + g) & 1;
    double acc[16];
#pragma unroll
    for (int k = 0; k < 16; ++k) acc[k] = 0.0;
    for (int rc0 = 0; rc0 < rows; rc0 += 32) {
        for (int e = t; e < planes * 32 * 64; e += 256) {
            const int o = e / (32 * 64), q = e % (32 * 64);
            const int rc = rc0 + q / 64;
            const int64_t jj = (int64_t)blockIdx.y * 64 + (q % 64);
            lt[o][q / 64][q % 64] =
                (rc < rows && jj < dp) ? T[(((int64_t)o * rows + rc) * cols + cu) * dp + jj] : 0.0;
        }
        for (int e = t; e < 64 * 32; e += 256) {
            const int ru = ru0 + e / 32, rc = rc0 + e % 32;
            lh[e / 32][e % 32] = (ru < rows && rc < rows) ? Hr[(int64_t)ru * rows + rc] : 0.0;
        }
        __syncthreads();
        for (int c = 0; c < 32; ++c) {
            const int pc = (rc0 + c) & 1;
            const int o = planes == 1 ? 0 : (pu == pc ? 0 : (pu ? 1 : 2));
            const double v = lt[o][c][jl];
#pragma unroll
            for (int k = 0; k < 16; ++k) acc[k] = fma(lh[g + 4 * k][c], v, acc[k]);
        }
        __syncthreads();
    }
    if (j < dp)
#pragma unroll
        for (int k = 0; k < 16; ++k) {
            const int ru = ru0 + g + 4 * k;
            if (ru < rows) O[((int64_t)ru * cols + cu) * dp + j] = acc[k];
        }
}

// W[u][j] = fp32(O[u][j] / O[u][d]) where the denominator is positive.
__global__ void batch_finish_kernel(const double *O, float *W, int64_t ld, int32_t N, int32_t d,
                                    int64_t dp) {
    const int64_t total = (int64_t)N * d;
    for (int64_t e = blockIdx.x * (int64_t)blockDim.x + threadIdx.x; e < total;
         e += (int64_t)gridDim.x * blockDim.x) {
        const int64_t u = e / d, j = e - u * d;
        const double den = O[u * dp + d];
        if (den > 0.0) W[u * ld + j] = (float)(O[u * dp + j] / den);
    }
}

}  // namespace

size_t batch_work_doubles(int32_t rows, int32_t cols, int32_t d, int32_t topology) {
    const int64_t N = (int64_t)rows * cols, dp = (int64_t)d + 1;
    const int planes = topology == 1 ? 3 : 1;
    return (size_t)(N * dp * (2 + planes) + (int64_t)rows * rows + (int64_t)planes * cols * cols);
}

hipError_t launch_batch_epoch(const BatchArgs &b, hipStream_t s) {
    const int64_t N = (int64_t)b.rows * b.cols, dp = (int64_t)b.d + 1;
    const int planes = b.topology == 1 ? 3 : 1;
    if (b.rows < 1 || b.cols < 1 || (dp + 63) / 64 > 65535) return hipErrorInvalidValue;
    double *S = b.work, *T = S + N * dp, *O = T + planes * N * dp;
    double *Hr = O + N * dp, *Hc = Hr + (int64_t)b.rows * b.rows;
    batch_sums_kernel<<<dim3((unsigned)((N + kUnitsPerWG - 1) / kUnitsPerWG),
                          (unsigned)((dp + kColsPerWG - 1) / kColsPerWG)),
                        dim3(256), 0, s>>>(b.bmu, b.X, b.n, b.d, (int32_t)N, S, dp);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
    const int64_t tab = (int64_t)b.rows * b.rows + (int64_t)planes * b.cols * b.cols;
    batch_tables_kernel<<<dim3((unsigned)std::min<int64_t>((tab + 255) / 256, 4096)), dim3(256), 0,
                          s>>>(b.rows, b.cols, b.topology, b.sigma, Hr, Hc);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    batch_col_pass_kernel<<<dim3((unsigned)(b.rows * ((b.cols + 63) / 64)), (unsigned)((dp + 63) / 64),
                              (unsigned)planes),
                         dim3(256), 0, s>>>(S, Hc, T, b.rows, b.cols, dp);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    batch_row_pass_kernel<<<dim3((unsigned)(b.cols * ((b.rows + 63) / 64)), (unsigned)((dp + 63) / 64)),
                         dim3(256), 0, s>>>(T, Hr, O, b.rows, b.cols, planes, dp);
    if ((e = hipGetLastError()) != hipSuccess) return e;
    batch_finish_kernel<<<dim3((unsigned)std::min<int64_t>((N * b.d + 255) / 256, 65536)), dim3(256),
                          0, s>>>(O, b.W, b.ld, (int32_t)N, b.d, dp);
    return hipGetLastError();
}

}  // namespace som
