// Principal components of the data and the linear initialisation of a map
// (paper Sec. 6D, Fig. 2): the prototypes start as a regular grid in the
// plane through the data mean spanned by the two largest principal
// components, and the map size follows from the two largest variances.
//
// On the device:
//   1. column means (fp64 partial sums over row chunks, summed in a fixed
//      order);
//   2. the covariance C = (1/n) sum_i (x_i - mu)(x_i - mu)^T on the fp32
//      matrix cores (v_mfma_f32_16x16x4_f32), one 64 x 64 tile per
//      workgroup, upper tiles only, mirrored on the store;
//   3. subspace iteration with kPcaBlock vectors: Y = C V, then in one
//      workgroup the Rayleigh-Ritz step (H = V^T Y, Jacobi eigen-pairs of H,
//      V <- V Q, Y <- Y Q), the residuals |y_a - theta_a v_a| of the top two
//      Ritz pairs, and modified Gram-Schmidt on Y for the next V;
//   4. the grid itself.
#include "som_internal.h"

#include <math.h>

namespace som {
namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kMeanChunks = 64;
constexpr int kCovTile = 64;
constexpr int kCovK = 32;
constexpr int kCovPitch = kCovTile + 4;
constexpr int kMatvecRows = 32;     // rows of C per workgroup (8 per wave)
constexpr int kMatvecChunk = 1024;  // columns of V staged in LDS at a time
constexpr int kOrthThreads = 1024;

__global__ __launch_bounds__(256) void col_partial_kernel(const float *X, int64_t n, int32_t d,
                                                          double *part) {
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int chunk = blockIdx.y;
    if (j >= d) return;
    const int64_t r0 = n * chunk / kMeanChunks, r1 = n * (chunk + 1) / kMeanChunks;
    double s = 0.0;
    for (int64_t i = r0; i < r1; ++i) s += (double)X[i * d + j];
    part[(int64_t)chunk * d + j] = s;
}

__global__ __launch_bounds__(256) void col_mean_kernel(const double *part, int64_t n, int32_t d,
                                                       float *mean) {
    const int64_t j = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (j >= d) return;
    double s = 0.0;
    for (int c = 0; c < kMeanChunks; ++c) s += part[(int64_t)c * d + j];
    mean[j] = (float)(s / (double)n);
}

// Upper tile t of the nt x nt tile grid, row-major over ti <= tj.
__device__ inline void upper_tile(int t, int nt, int &ti, int &tj) {
    int i = 0, left = t;
    while (left >= nt - i) {
        left -= nt - i;
        ++i;
    }
    ti = i;
    tj = i + left;
}

__global__ __launch_bounds__(256) void covariance_kernel(const float *X, int64_t n, int32_t d,
                                                         const float *mean, float *C) {
    __shared__ float As[kCovK][kCovPitch];
    __shared__ float Bs[kCovK][kCovPitch];
    const int nt = (d + kCovTile - 1) / kCovTile;
    int ti, tj;
    upper_tile(blockIdx.x, nt, ti, tj);
    const int i0 = ti * kCovTile, j0 = tj * kCovTile;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = (wave & 1) * 32, wn = (wave >> 1) * 32;
    const int l16 = lane & 15, lk = lane >> 4;
    f4 acc[2][2];
#pragma unroll
    for (int a = 0; a < 2; ++a)
#pragma unroll
        for (int b = 0; b < 2; ++b) acc[a][b] = f4{0.f, 0.f, 0.f, 0.f};
    // staging: 32 rows x 64 columns per operand, 8 floats per thread
    const int sc = tid & 63, sr = tid >> 6;  // column, first row (stride 4)
    // out-of-range columns and rows are loaded clamped and zeroed by a select
    const bool ci = i0 + sc < d, cj = j0 + sc < d;
    const int64_t ii = ci ? i0 + sc : d - 1, jj = cj ? j0 + sc : d - 1;
    const float mi = mean[ii], mj = mean[jj];
    for (int64_t k0 = 0; k0 < n; k0 += kCovK) {
        __syncthreads();
#pragma unroll
        for (int rr = 0; rr < kCovK / 4; ++rr) {
            const int r = sr + 4 * rr;
            const int64_t k = k0 + r;
            const bool in = k < n;
            const int64_t kk = in ? k : n - 1;
            const float va = X[kk * d + ii] - mi, vb = X[kk * d + jj] - mj;
            As[r][sc] = (in && ci) ? va : 0.f;
            Bs[r][sc] = (in && cj) ? vb : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int ks = 0; ks < kCovK; ks += 4) {
            float a[2], b[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                a[u] = As[ks + lk][wm + 16 * u + l16];
                b[u] = Bs[ks + lk][wn + 16 * u + l16];
            }
#pragma unroll
            for (int u = 0; u < 2; ++u)
#pragma unroll
                for (int v = 0; v < 2; ++v)
                    acc[u][v] = __builtin_amdgcn_mfma_f32_16x16x4f32(a[u], b[v], acc[u][v], 0, 0, 0);
        }
    }
    // acc[u][v][e]: row i0 + wm + 16u + 4 lk + e, column j0 + wn + 16v + l16
    const float inv_n = (float)(1.0 / (double)n);
#pragma unroll
    for (int u = 0; u < 2; ++u)
#pragma unroll
        for (int v = 0; v < 2; ++v)
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                const int i = i0 + wm + 16 * u + 4 * lk + e, j = j0 + wn + 16 * v + l16;
                if (i < d && j < d) {
                    const float c = acc[u][v][e] * inv_n;
                    C[(int64_t)i * d + j] = c;
                    if (ti != tj) C[(int64_t)j * d + i] = c;
                }
            }
}

// Y = C V for kMatvecRows rows of C per workgroup (V, Y: d x kPcaBlock,
// column-major).
__global__ __launch_bounds__(256) void matvec_kernel(const float *C, int32_t d, const float *V,
                                                     float *Y) {
    constexpr int P = kPcaBlock;
    constexpr int RW = kMatvecRows / 4;  // rows per wave
    __shared__ float vs[kMatvecChunk * P];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int64_t r0 = (int64_t)blockIdx.x * kMatvecRows + wave * RW;
    float acc[RW][P];
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
        for (int a = 0; a < P; ++a) acc[r][a] = 0.f;
    for (int c0 = 0; c0 < d; c0 += kMatvecChunk) {
        const int cn = d - c0 < kMatvecChunk ? d - c0 : kMatvecChunk;
        __syncthreads();
        for (int e = tid; e < cn * P; e += 256) {
            const int j = e / P, a = e - j * P;
            vs[e] = V[(int64_t)a * d + c0 + j];
        }
        __syncthreads();
        for (int j = lane; j < cn; j += 64) {
            float vv[P];
#pragma unroll
            for (int a = 0; a < P; ++a) vv[a] = vs[j * P + a];
#pragma unroll
            for (int r = 0; r < RW; ++r) {
                const int64_t row = r0 + r < d ? r0 + r : d - 1;  // clamped; unused past d
                const float c = C[row * d + c0 + j];
#pragma unroll
                for (int a = 0; a < P; ++a) acc[r][a] = fmaf(c, vv[a], acc[r][a]);
            }
        }
    }
#pragma unroll
    for (int r = 0; r < RW; ++r)
#pragma unroll
        for (int a = 0; a < P; ++a) {
            float s = acc[r][a];
#pragma unroll
            for (int o = 32; o >= 1; o >>= 1) s += __shfl_xor(s, o, 64);
            acc[r][a] = s;
        }
    if (lane == 0)
#pragma unroll
        for (int r = 0; r < RW; ++r) {
            const int64_t row = r0 + r;
            if (row < d)
#pragma unroll
                for (int a = 0; a < P; ++a) Y[(int64_t)a * d + row] = acc[r][a];
        }
}

// Sum over the workgroup of one value per thread, in double, fixed order.
__device__ inline double block_sum(double v, double *red) {
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
    __syncthreads();
    if (lane == 0) red[wave] = v;
    __syncthreads();
    double s = 0.0;
    for (int w = 0; w < kOrthThreads / 64; ++w) s += red[w];
    return s;
}

// Jacobi eigen-decomposition of the symmetric P x P matrix H (row-major,
// one thread): H <- diag, Q <- eigenvectors (columns).
__device__ void jacobi_eigen(double (&H)[kPcaBlock][kPcaBlock], double (&Q)[kPcaBlock][kPcaBlock]) {
    constexpr int P = kPcaBlock;
    for (int i = 0; i < P; ++i)
        for (int j = 0; j < P; ++j) Q[i][j] = i == j ? 1.0 : 0.0;
    for (int sweep = 0; sweep < 60; ++sweep) {
        double off = 0.0;
        for (int i = 0; i < P; ++i)
            for (int j = i + 1; j < P; ++j) off += H[i][j] * H[i][j];
        if (off < 1e-30) break;
        for (int p = 0; p < P; ++p)
            for (int q = p + 1; q < P; ++q) {
                if (H[p][q] == 0.0) continue;
                const double theta = (H[q][q] - H[p][p]) / (2.0 * H[p][q]);
                const double t = (theta >= 0 ? 1.0 : -1.0) /
                                 (fabs(theta) + sqrt(theta * theta + 1.0));
                const double c = 1.0 / sqrt(t * t + 1.0), s = t * c;
                for (int k = 0; k < P; ++k) {
                    const double hkp = H[k][p], hkq = H[k][q];
                    H[k][p] = c * hkp - s * hkq;
                    H[k][q] = s * hkp + c * hkq;
                }
                for (int k = 0; k < P; ++k) {
                    const double hpk = H[p][k], hqk = H[q][k];
                    H[p][k] = c * hpk - s * hqk;
                    H[q][k] = s * hpk + c * hqk;
                }
                for (int k = 0; k < P; ++k) {
                    const double qkp = Q[k][p], qkq = Q[k][q];
                    Q[k][p] = c * qkp - s * qkq;
                    Q[k][q] = s * qkp + c * qkq;
                }
            }
    }
}

// One workgroup: Rayleigh-Ritz on (V, Y = C V), residuals of the two
// largest Ritz pairs, then V <- orthonormal basis of the rotated Y.
// stats: theta_0, theta_1, residual_0, residual_1.  With ritz_only the Ritz
// vectors stay in V (the final step).
__global__ __launch_bounds__(kOrthThreads) void ritz_orth_kernel(float *V, float *Y, int32_t d,
                                                                 double *stats, int ritz_only) {
    constexpr int P = kPcaBlock;
    __shared__ double red[kOrthThreads / 64];
    __shared__ double Hs[P][P], Qs[P][P], theta[2];
    __shared__ int order[P];
    const int tid = threadIdx.x;
    // H = V^T Y (symmetrised)
    for (int a = 0; a < P; ++a)
        for (int b = a; b < P; ++b) {
            double s = 0.0;
            for (int64_t j = tid; j < d; j += kOrthThreads)
                s += (double)V[(int64_t)a * d + j] * (double)Y[(int64_t)b * d + j];
            s = block_sum(s, red);
            double s2 = 0.0;
            for (int64_t j = tid; j < d; j += kOrthThreads)
                s2 += (double)V[(int64_t)b * d + j] * (double)Y[(int64_t)a * d + j];
            s2 = block_sum(s2, red);
            if (tid == 0) Hs[a][b] = Hs[b][a] = 0.5 * (s + s2);
        }
    __syncthreads();
    if (tid == 0) {
        double H[P][P], Q[P][P];
        for (int i = 0; i < P; ++i)
            for (int j = 0; j < P; ++j) H[i][j] = Hs[i][j];
        jacobi_eigen(H, Q);
        // Ritz values in descending order
        for (int i = 0; i < P; ++i) order[i] = i;
        for (int i = 0; i < P; ++i)
            for (int j = i + 1; j < P; ++j)
                if (H[order[j]][order[j]] > H[order[i]][order[i]]) {
                    const int t = order[i];
                    order[i] = order[j];
                    order[j] = t;
                }
        for (int i = 0; i < P; ++i)
            for (int j = 0; j < P; ++j) Qs[i][j] = Q[i][order[j]];
        theta[0] = H[order[0]][order[0]];
        theta[1] = H[order[1]][order[1]];
        stats[0] = theta[0];
        stats[1] = theta[1];
    }
    __syncthreads();
    // V <- V Q, Y <- Y Q (columns in descending Ritz order)
    for (int64_t j = tid; j < d; j += kOrthThreads) {
        float v[P], y[P];
        for (int a = 0; a < P; ++a) {
            v[a] = V[(int64_t)a * d + j];
            y[a] = Y[(int64_t)a * d + j];
        }
        for (int b = 0; b < P; ++b) {
            double sv = 0.0, sy = 0.0;
            for (int a = 0; a < P; ++a) {
                sv += (double)v[a] * Qs[a][b];
                sy += (double)y[a] * Qs[a][b];
            }
            V[(int64_t)b * d + j] = (float)sv;
            Y[(int64_t)b * d + j] = (float)sy;
        }
    }
    __syncthreads();
    // residuals of the two largest Ritz pairs
    for (int a = 0; a < 2; ++a) {
        const double th = theta[a];
        double s = 0.0;
        for (int64_t j = tid; j < d; j += kOrthThreads) {
            const double r = (double)Y[(int64_t)a * d + j] - th * (double)V[(int64_t)a * d + j];
            s += r * r;
        }
        s = block_sum(s, red);
        if (tid == 0) stats[2 + a] = sqrt(s);
    }
    if (ritz_only) return;
    // next basis: modified Gram-Schmidt on Y
    for (int a = 0; a < P; ++a) {
        for (int b = 0; b < a; ++b) {
            double s = 0.0;
            for (int64_t j = tid; j < d; j += kOrthThreads)
                s += (double)Y[(int64_t)a * d + j] * (double)V[(int64_t)b * d + j];
            s = block_sum(s, red);
            for (int64_t j = tid; j < d; j += kOrthThreads)
                Y[(int64_t)a * d + j] -= (float)s * V[(int64_t)b * d + j];
            __syncthreads();
        }
        double s = 0.0;
        for (int64_t j = tid; j < d; j += kOrthThreads) {
            const double y = Y[(int64_t)a * d + j];
            s += y * y;
        }
        s = block_sum(s, red);
        const double inv = s > 0.0 ? 1.0 / sqrt(s) : 0.0;
        for (int64_t j = tid; j < d; j += kOrthThreads)
            V[(int64_t)a * d + j] = (float)(Y[(int64_t)a * d + j] * inv);
        __syncthreads();
    }
}

// Starting basis: SplitMix64 values in [-1/2, 1/2), orthonormalised by the
// first ritz_orth_kernel call (with Y = V and the Rayleigh-Ritz step acting
// on the identity).
__global__ void start_basis_kernel(float *V, int64_t count, uint64_t seed) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= count) return;
    uint64_t z = seed + (uint64_t)(i + 1) * 0x9E3779B97F4A7C15ull;
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ull;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBull;
    z ^= z >> 31;
    V[i] = (float)((double)(z >> 40) * (1.0 / 16777216.0) - 0.5);
}

// Sign convention: the component of largest magnitude (lowest index on
// ties) of each of the two vectors is made positive.
__global__ __launch_bounds__(kOrthThreads) void sign_fix_kernel(float *V, int32_t d) {
    __shared__ unsigned long long best[kOrthThreads / 64];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    for (int a = 0; a < 2; ++a) {
        unsigned long long k = ~0ull;  // (~|v| bits, index): the minimum is the largest |v|
        for (int64_t j = tid; j < d; j += kOrthThreads) {
            const unsigned mag = __float_as_uint(fabsf(V[(int64_t)a * d + j]));
            const unsigned long long key = ((unsigned long long)(~mag) << 32) | (unsigned)j;
            k = key < k ? key : k;
        }
#pragma unroll
        for (int o = 32; o >= 1; o >>= 1) {
            const unsigned long long other = __shfl_xor(k, o, 64);
            k = other < k ? other : k;
        }
        __syncthreads();
        if (lane == 0) best[wave] = k;
        __syncthreads();
        unsigned long long m = best[0];
        for (int w = 1; w < kOrthThreads / 64; ++w) m = best[w] < m ? best[w] : m;
        const int j = (int)(unsigned)(m & 0xffffffffull);
        const bool flip = V[(int64_t)a * d + j] < 0.f;
        __syncthreads();
        if (flip)
            for (int64_t i = tid; i < d; i += kOrthThreads) V[(int64_t)a * d + i] = -V[(int64_t)a * d + i];
        __syncthreads();
    }
}

__global__ void linear_init_kernel(float *W, int64_t ld, int32_t rows, int32_t cols, int32_t d,
                                   const float *mean, const float *v1, const float *v2, float s1,
                                   float s2) {
    const int64_t e = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t total = (int64_t)rows * cols * ld;
    if (e >= total) return;
    const int64_t u = e / ld, j = e - u * ld;
    if (j >= d) {
        W[e] = 0.f;
        return;
    }
    const int r = (int)(u / cols), c = (int)(u - (int64_t)r * cols);
    const float a = cols > 1 ? (float)(2.0 * c / (cols - 1) - 1.0) : 0.f;
    const float b = rows > 1 ? (float)(2.0 * r / (rows - 1) - 1.0) : 0.f;
    W[e] = fmaf(b * s2, v2[j], fmaf(a * s1, v1[j], mean[j]));
}

}  // namespace

// Work buffer: C (d x d), V and Y (d x kPcaBlock each), then the fp64
// column partials (kMeanChunks x d) at an even float offset.
static size_t pca_part_offset(int32_t d) {
    const size_t dd = (size_t)d;
    return (dd * dd + 2 * dd * kPcaBlock + 1) & ~(size_t)1;
}

size_t pca_work_floats(int32_t d) {
    return pca_part_offset(d) + 2 * (size_t)d * kMeanChunks;
}

hipError_t pca_top2(const float *X, int64_t n, int32_t d, float *work, float *mean, double *stats,
                    int max_iters, double tol, hipStream_t s, double *lambda, int *iters) {
    float *C = work;
    float *V = C + (size_t)d * d;
    float *Y = V + (size_t)d * kPcaBlock;
    double *part = reinterpret_cast<double *>(work + pca_part_offset(d));
    const unsigned col_blocks = (unsigned)((d + 255) / 256);
    col_partial_kernel<<<dim3(col_blocks, kMeanChunks), dim3(256), 0, s>>>(X, n, d, part);
    col_mean_kernel<<<dim3(col_blocks), dim3(256), 0, s>>>(part, n, d, mean);
    const int nt = (d + kCovTile - 1) / kCovTile;
    covariance_kernel<<<dim3((unsigned)(nt * (nt + 1) / 2)), dim3(256), 0, s>>>(X, n, d, mean, C);
    const int64_t vcount = (int64_t)d * kPcaBlock;
    start_basis_kernel<<<dim3((unsigned)((vcount + 255) / 256)), dim3(256), 0, s>>>(
        V, vcount, 0x5043412d494e4954ull);
    hipError_t e = hipMemcpyAsync(Y, V, (size_t)vcount * sizeof(float), hipMemcpyDeviceToDevice, s);
    if (e != hipSuccess) return e;
    ritz_orth_kernel<<<dim3(1), dim3(kOrthThreads), 0, s>>>(V, Y, d, stats, 0);
    const unsigned mv_blocks = (unsigned)((d + kMatvecRows - 1) / kMatvecRows);
    double h[4] = {0, 0, 0, 0};
    int it = 0;
    for (;;) {
        matvec_kernel<<<dim3(mv_blocks), dim3(256), 0, s>>>(C, d, V, Y);
        ++it;
        const bool check = (it % 8) == 0 || it >= max_iters;
        ritz_orth_kernel<<<dim3(1), dim3(kOrthThreads), 0, s>>>(V, Y, d, stats, 0);
        if ((e = hipGetLastError()) != hipSuccess) return e;
        if (!check) continue;
        e = hipMemcpyAsync(h, stats, sizeof(h), hipMemcpyDeviceToHost, s);
        if (e == hipSuccess) e = hipStreamSynchronize(s);
        if (e != hipSuccess) return e;
        const double scale = h[0] > 0.0 ? h[0] : 1.0;
        if ((h[2] <= tol * scale && h[3] <= tol * scale) || it >= max_iters) break;
    }
    // final Rayleigh-Ritz pair in V (columns 0, 1), signs fixed
    matvec_kernel<<<dim3(mv_blocks), dim3(256), 0, s>>>(C, d, V, Y);
    ritz_orth_kernel<<<dim3(1), dim3(kOrthThreads), 0, s>>>(V, Y, d, stats, 1);
    sign_fix_kernel<<<dim3(1), dim3(kOrthThreads), 0, s>>>(V, d);
    e = hipMemcpyAsync(h, stats, sizeof(h), hipMemcpyDeviceToHost, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return e;
    lambda[0] = h[0] > 0.0 ? h[0] : 0.0;
    lambda[1] = h[1] > 0.0 ? h[1] : 0.0;
    if (iters) *iters = it;
    return hipGetLastError();
}

const float *pca_vectors(const float *work, int32_t d) { return work + (size_t)d * d; }

hipError_t launch_linear_init(float *W, int64_t ld, int32_t rows, int32_t cols, int32_t d,
                              const float *mean, const float *v1, const float *v2, double lambda1,
                              double lambda2, hipStream_t s) {
    const int64_t total = (int64_t)rows * cols * ld;
    linear_init_kernel<<<dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s>>>(
        W, ld, rows, cols, d, mean, v1, v2, (float)sqrt(lambda1), (float)sqrt(lambda2));
    return hipGetLastError();
}

}  // namespace som
