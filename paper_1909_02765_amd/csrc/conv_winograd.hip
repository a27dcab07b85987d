// Winograd F(2x2, 3x3) convolution -- a comparison path, not the ILP-M
// method.  The paper measures ILP-M against Winograd (Sections 3 and 5);
// this file rebuilds that competitor for the 3x3 / stride-1 layers so the two
// can be timed on the same GPU.
//
// For each 2x2 output tile and each input channel, the 4x4 input patch d and
// the 3x3 filter g are transformed, multiplied elementwise and transformed
// back (the minimal filtering algorithm of Lavin and Gray, 2016):
//
//   U = G g G^T,  V = B^T d B,  Y = A^T (sum over channels of U (.) V) A
//
//   G   = [1 0 0; 1/2 1/2 1/2; 1/2 -1/2 1/2; 0 0 1]
//   B^T = [1 0 -1 0; 0 1 1 0; 0 -1 1 0; 0 1 0 -1]
//   A^T = [1 1 1 0; 0 1 -1 -1]
//
// The channel sum for each of the 16 (xi, nu) positions is a matrix product
// M_b = U_b V_b (U_b: C_out x C_in, V_b: C_in x tiles), done as one batched
// library GEMM (rocBLAS, loaded at run time from the copy the process already
// has).  Per 2x2 outputs that is 16 products per channel instead of 36.
#include <dlfcn.h>

#include <mutex>

#include <rocblas/rocblas.h>

#include "internal.h"

namespace ilpm {
namespace {

// U[b][co][ci], b = 4*xi + nu, from w[co][ci][3][3].
__global__ __launch_bounds__(256) void winograd_filter(const float *__restrict__ w, float *__restrict__ u, int c_in,
                                                       int c_out)
{
    const int64_t n = (int64_t)c_out * c_in;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const float *g = w + i * 9;
    float gg[4][3];  // G g
#pragma unroll
    for (int c = 0; c < 3; ++c) {
        const float g0 = g[c], g1 = g[3 + c], g2 = g[6 + c];
        gg[0][c] = g0;
        gg[1][c] = 0.5f * (g0 + g1 + g2);
        gg[2][c] = 0.5f * (g0 - g1 + g2);
        gg[3][c] = g2;
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const float a0 = gg[r][0], a1 = gg[r][1], a2 = gg[r][2];
        const float row[4] = {a0, 0.5f * (a0 + a1 + a2), 0.5f * (a0 - a1 + a2), a2};
#pragma unroll
        for (int c = 0; c < 4; ++c) u[(int64_t)(4 * r + c) * n + i] = row[c];
    }
}

// V[b][ci][t] for tile t = ty * tiles_w + tx (input patch at rows 2*ty - pad,
// columns 2*tx - pad; zero outside the image).
__global__ __launch_bounds__(256) void winograd_input(const float *__restrict__ x, float *__restrict__ v, int c_in,
                                                      int h, int w, int pad, int tiles_h, int tiles_w)
{
    const int64_t tiles = (int64_t)tiles_h * tiles_w;
    const int64_t n = (int64_t)c_in * tiles;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const int ci = (int)(i / tiles);
    const int t = (int)(i - (int64_t)ci * tiles);
    const int ty = t / tiles_w, tx = t - ty * tiles_w;
    const int y0 = 2 * ty - pad, x0 = 2 * tx - pad;
    const float *xp = x + (int64_t)ci * h * w;
    float d[4][4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            const int yy = y0 + r, xx = x0 + c;
            d[r][c] = (yy >= 0 && yy < h && xx >= 0 && xx < w) ? xp[(int64_t)yy * w + xx] : 0.f;
        }
    float e[4][4];  // B^T d
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        e[0][c] = d[0][c] - d[2][c];
        e[1][c] = d[1][c] + d[2][c];
        e[2][c] = d[2][c] - d[1][c];
        e[3][c] = d[1][c] - d[3][c];
    }
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const float row[4] = {e[r][0] - e[r][2], e[r][1] + e[r][2], e[r][2] - e[r][1], e[r][1] - e[r][3]};
#pragma unroll
        for (int c = 0; c < 4; ++c) v[(int64_t)(4 * r + c) * n + i] = row[c];
    }
}

// out[co][2*ty + i][2*tx + j] = (A^T M A)[i][j] + bias[co], M[b] = m[b][co][t].
__global__ __launch_bounds__(256) void winograd_output(const float *__restrict__ m, const float *__restrict__ bias,
                                                       float *__restrict__ out, int c_out, int h_out, int w_out,
                                                       int tiles_h, int tiles_w)
{
    const int64_t tiles = (int64_t)tiles_h * tiles_w;
    const int64_t n = (int64_t)c_out * tiles;
    const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= n) return;
    const int co = (int)(i / tiles);
    const int t = (int)(i - (int64_t)co * tiles);
    const int ty = t / tiles_w, tx = t - ty * tiles_w;
    float mm[4][4];
#pragma unroll
    for (int r = 0; r < 4; ++r)
#pragma unroll
        for (int c = 0; c < 4; ++c) mm[r][c] = m[(int64_t)(4 * r + c) * n + i];
    float e[2][4];  // A^T M
#pragma unroll
    for (int c = 0; c < 4; ++c) {
        e[0][c] = mm[0][c] + mm[1][c] + mm[2][c];
        e[1][c] = mm[1][c] - mm[2][c] - mm[3][c];
    }
    const float b = bias ? bias[co] : 0.f;
    float *o = out + (int64_t)co * h_out * w_out;
#pragma unroll
    for (int r = 0; r < 2; ++r) {
        const float y0 = e[r][0] + e[r][1] + e[r][2];
        const float y1 = e[r][1] - e[r][2] - e[r][3];
        const int oy = 2 * ty + r, ox = 2 * tx;
        if (oy < h_out) {
            if (ox < w_out) o[(int64_t)oy * w_out + ox] = y0 + b;
            if (ox + 1 < w_out) o[(int64_t)oy * w_out + ox + 1] = y1 + b;
        }
    }
}

// ---- rocBLAS, resolved at run time ----
struct Blas {
    decltype(&rocblas_create_handle) create = nullptr;
    decltype(&rocblas_set_stream) set_stream = nullptr;
    decltype(&rocblas_set_atomics_mode) set_atomics = nullptr;
    decltype(&rocblas_sgemm_strided_batched) sgemm = nullptr;
    rocblas_handle handle[64] = {};
    bool tried = false, ok = false;
};
Blas g_blas;
std::mutex g_blas_mu;

bool blas_load()
{
    if (g_blas.tried) return g_blas.ok;
    g_blas.tried = true;
    // Prefer the rocBLAS this process already mapped (torch's); else load one.
    void *lib = dlopen("librocblas.so.5", RTLD_NOW | RTLD_NOLOAD);
    if (!lib) lib = dlopen("librocblas.so.5", RTLD_NOW | RTLD_LOCAL);
    if (!lib) return false;
    g_blas.create = reinterpret_cast<decltype(g_blas.create)>(dlsym(lib, "rocblas_create_handle"));
    g_blas.set_stream = reinterpret_cast<decltype(g_blas.set_stream)>(dlsym(lib, "rocblas_set_stream"));
    g_blas.set_atomics = reinterpret_cast<decltype(g_blas.set_atomics)>(dlsym(lib, "rocblas_set_atomics_mode"));
    g_blas.sgemm = reinterpret_cast<decltype(g_blas.sgemm)>(dlsym(lib, "rocblas_sgemm_strided_batched"));
    g_blas.ok = g_blas.create && g_blas.set_stream && g_blas.set_atomics && g_blas.sgemm;
    return g_blas.ok;
}

}  // namespace

int64_t winograd_tiles(const ConvShape &s) { return (int64_t)ceil_div(s.h_out, 2) * ceil_div(s.w_out, 2); }

size_t winograd_workspace_bytes(const ConvShape &s)
{
    const int64_t t = winograd_tiles(s);
    return sizeof(float) * (size_t)(16 * (int64_t)s.c_in * t + 16 * (int64_t)s.c_out * t);
}

hipError_t winograd_filter_launch(const float *w, int c_in, int c_out, float *u, hipStream_t stream)
{
    const int64_t n = (int64_t)c_out * c_in;
    hipLaunchKernelGGL(winograd_filter, dim3((unsigned)((n + 255) / 256)), dim3(256), 0, stream, w, u, c_in, c_out);
    return hipGetLastError();
}

// 0 on success, else an ILPM_ERR_* (rocBLAS missing or failing: ILPM_ERR_UNSUPPORTED / ILPM_ERR_HIP).
int winograd_launch(const ConvShape &s, const float *x, const float *u, const float *bias, float *out,
                    void *workspace, int dev, hipStream_t stream, hipError_t *err)
{
    *err = hipSuccess;
    std::lock_guard<std::mutex> lk(g_blas_mu);
    if (!blas_load()) return ILPM_ERR_UNSUPPORTED;
    rocblas_handle &h = g_blas.handle[dev];
    if (!h) {
        if (g_blas.create(&h) != rocblas_status_success) {
            h = nullptr;
            return ILPM_ERR_HIP;
        }
        g_blas.set_atomics(h, rocblas_atomics_not_allowed);  // a fixed summation order
    }
    if (g_blas.set_stream(h, stream) != rocblas_status_success) return ILPM_ERR_HIP;
    const int tiles_h = ceil_div(s.h_out, 2), tiles_w = ceil_div(s.w_out, 2);
    const int64_t t = (int64_t)tiles_h * tiles_w;
    float *v = static_cast<float *>(workspace);
    float *m = v + 16 * (int64_t)s.c_in * t;
    const int64_t nin = (int64_t)s.c_in * t;
    hipLaunchKernelGGL(winograd_input, dim3((unsigned)((nin + 255) / 256)), dim3(256), 0, stream, x, v, s.c_in, s.h,
                       s.w, s.pad, tiles_h, tiles_w);
    if ((*err = hipGetLastError()) != hipSuccess) return ILPM_ERR_HIP;
    // Row-major M_b (C_out x T) = U_b (C_out x C_in) V_b (C_in x T), i.e.
    // column-major M_b^T (T x C_out) = V_b^T (T x C_in) U_b^T (C_in x C_out).
    const float one = 1.f, zero = 0.f;
    if (g_blas.sgemm(h, rocblas_operation_none, rocblas_operation_none, (rocblas_int)t, s.c_out, s.c_in, &one, v,
                     (rocblas_int)t, nin, u, s.c_in, (rocblas_stride)s.c_out * s.c_in, &zero, m, (rocblas_int)t,
                     (rocblas_stride)s.c_out * t, 16) != rocblas_status_success)
        return ILPM_ERR_HIP;
    const int64_t nout = (int64_t)s.c_out * t;
    hipLaunchKernelGGL(winograd_output, dim3((unsigned)((nout + 255) / 256)), dim3(256), 0, stream, m, bias, out,
                       s.c_out, s.h_out, s.w_out, tiles_h, tiles_w);
    if ((*err = hipGetLastError()) != hipSuccess) return ILPM_ERR_HIP;
    return ILPM_OK;
}

}  // namespace ilpm
