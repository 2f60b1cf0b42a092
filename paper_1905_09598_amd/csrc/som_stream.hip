// In-place stream over one device buffer: the memory reference against
// which the training kernels' measured traffic is judged.  Not a step of
// the method.
//
// Workgroup b of G owns the contiguous 16-byte words [b n4 / G, (b+1) n4 / G)
// of the buffer, as a training workgroup owns a contiguous range of
// prototype rows, and rewrites each of them `passes` times in one launch
// (read, scale by `a`, write back in place), four words per thread in
// flight.  No workgroup touches another's words, so the passes need no
// barrier and the launch has no gaps between them.
#include "som_internal.h"

namespace som {
namespace {

constexpr int kStreamBlock = 256;
constexpr int kStreamUnroll = 4;

__global__ __launch_bounds__(kStreamBlock) void stream_inplace_kernel(float4 *buf, int64_t n4,
                                                                      int32_t passes, float a) {
    const int64_t G = gridDim.x, b = blockIdx.x;
    const int64_t lo = n4 * b / G, hi = n4 * (b + 1) / G;
    constexpr int64_t step = (int64_t)kStreamBlock * kStreamUnroll;
    for (int32_t p = 0; p < passes; ++p) {
        int64_t i = lo + threadIdx.x;
        for (; i + (kStreamUnroll - 1) * kStreamBlock < hi; i += step) {
            float4 v[kStreamUnroll];
#pragma unroll
            for (int k = 0; k < kStreamUnroll; ++k) v[k] = buf[i + k * kStreamBlock];
#pragma unroll
            for (int k = 0; k < kStreamUnroll; ++k) {
                v[k].x *= a;
                v[k].y *= a;
                v[k].z *= a;
                v[k].w *= a;
                buf[i + k * kStreamBlock] = v[k];
            }
        }
        for (; i < hi; i += kStreamBlock) {
            float4 v = buf[i];
            v.x *= a;
            v.y *= a;
            v.z *= a;
            v.w *= a;
            buf[i] = v;
        }
    }
}

}  // namespace

hipError_t launch_stream_inplace(float *buf, int64_t bytes, int32_t passes, int32_t grid,
                                 float a, hipStream_t s) {
    stream_inplace_kernel<<<dim3((unsigned)grid), dim3(kStreamBlock), 0, s>>>(
        reinterpret_cast<float4 *>(buf), bytes / 16, passes, a);
    return hipGetLastError();
}

}  // namespace som
