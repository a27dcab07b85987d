// Elementwise helpers used between the convolutions of a layer stack (ReLU,
// 2x2 max-pool).  They are not part of the convolution.
#include "internal.h"

namespace ilpm {
namespace {

__global__ __launch_bounds__(256) void relu_kernel(float *x, int64_t n)
{
    int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t step = (int64_t)gridDim.x * 256;
    for (; i < n; i += step) {
        const float v = x[i];
        x[i] = v > 0.f ? v : 0.f;
    }
}

__global__ __launch_bounds__(256) void maxpool2x2_kernel(const float *__restrict__ in, int c, int h, int w,
                                                         float *__restrict__ out, int relu)
{
    const int ho = h / 2, wo = w / 2;
    const int64_t total = (int64_t)c * ho * wo;
    int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int64_t step = (int64_t)gridDim.x * 256;
    for (; i < total; i += step) {
        const int j = (int)(i % wo);
        const int r = (int)((i / wo) % ho);
        const int ch = (int)(i / ((int64_t)wo * ho));
        const float *p = in + ((size_t)ch * h + 2 * r) * w + 2 * j;
        float m = p[0];
        m = p[1] > m ? p[1] : m;
        m = p[w] > m ? p[w] : m;
        m = p[w + 1] > m ? p[w + 1] : m;
        out[i] = relu && m < 0.f ? 0.f : m;
    }
}

int grid_for(int64_t n)
{
    int64_t b = (n + 255) / 256;
    if (b < 1) b = 1;
    if (b > 65536) b = 65536;
    return (int)b;
}

}  // namespace

hipError_t launch_relu(float *x, int64_t n, hipStream_t stream)
{
    if (n == 0) return hipSuccess;
    hipLaunchKernelGGL(relu_kernel, dim3(grid_for(n)), dim3(256), 0, stream, x, n);
    return hipGetLastError();
}

hipError_t launch_maxpool2x2(const float *in, int c, int h, int w, float *out, hipStream_t stream, bool relu)
{
    const int64_t total = (int64_t)c * (h / 2) * (w / 2);
    if (total == 0) return hipSuccess;
    hipLaunchKernelGGL(maxpool2x2_kernel, dim3(grid_for(total)), dim3(256), 0, stream, in, c, h, w, out,
                       relu ? 1 : 0);
    return hipGetLastError();
}

}  // namespace ilpm
