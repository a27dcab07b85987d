// Direct convolution on the vector ALUs (any filter size and stride).
//
// The ILP-M idea (Section 4, Algorithm 2) is to stage an input-channel tile in
// LDS with one barrier, then run a barrier-free inner loop in which one weight
// is applied to a whole register tile of outputs, taps (r, s) outermost.  On
// CDNA the natural way to get "one weight, many FMAs" without the paper's
// uncoalesced stores is the transpose of its mapping: lanes sit on output
// pixels (so NCHW stores coalesce along W) and each thread keeps a block of
// output channels in registers; the weight of each (channel, tap) is the same
// for the whole wavefront and comes from LDS as a broadcast read, so the
// inner loop is one LDS pixel read per block of FMAs.
//
// Variant 0: 8 x 32 output pixels x 16 output channels per 256-thread
//            workgroup; halo tile and weight slice of a chunk of input
//            channels staged in LDS.
// Variant 1: no LDS, one thread per output element reading global memory;
//            the fallback for shapes whose halo does not fit LDS.
#include "internal.h"

namespace ilpm {
namespace {

constexpr int kTileH = 8;
constexpr int kTileW = 32;
constexpr int kCoGroup = 16;
constexpr int kThreads = 256;
constexpr int kLdsFloats = 16384;  // 64 KiB

struct DirectArgs {
    int c_in, h, w, c_out, k, stride, pad, h_out, w_out;
    int halo_h, halo_w, chunk, tiles_w;
    int relu;  // store max(., 0)
};

__global__ __launch_bounds__(kThreads) void conv_direct_lds(const float *__restrict__ x,
                                                            const float *__restrict__ wt,
                                                            const float *__restrict__ bias,
                                                            float *__restrict__ out, DirectArgs a)
{
    extern __shared__ float lds[];
    const int kk = a.k * a.k;
    const int plane = a.halo_h * a.halo_w;
    float *xl = lds;                          // [chunk][halo_h][halo_w]
    float *wl = lds + ((a.chunk * plane + 3) & ~3);  // [chunk * kk][kCoGroup], 16-byte aligned

    const int tw_i = blockIdx.x % a.tiles_w;
    const int th_i = blockIdx.x / a.tiles_w;
    const int co0 = blockIdx.y * kCoGroup;
    const int oh0 = th_i * kTileH, ow0 = tw_i * kTileW;
    const int ih0 = oh0 * a.stride - a.pad, iw0 = ow0 * a.stride - a.pad;
    const int tid = threadIdx.x;
    const int ty = tid / kTileW, tx = tid % kTileW;

    float acc[kCoGroup];
#pragma unroll
    for (int j = 0; j < kCoGroup; ++j) acc[j] = 0.f;

    for (int ci0 = 0; ci0 < a.c_in; ci0 += a.chunk) {
        const int cc = min(a.chunk, a.c_in - ci0);
        // Stage the zero-padded halo of cc input channels (thread <-> pixel).
        const int xe = cc * plane;
        for (int e = tid; e < xe; e += kThreads) {
            const int c = e / plane;
            const int rem = e - c * plane;
            const int r = rem / a.halo_w;
            const int col = rem - r * a.halo_w;
            const int ih = ih0 + r, iw = iw0 + col;
            float v = 0.f;
            if (ih >= 0 && ih < a.h && iw >= 0 && iw < a.w)
                v = x[((size_t)(ci0 + c) * a.h + ih) * a.w + iw];
            xl[e] = v;
        }
        // Stage the weight slice as [channel, tap][output channel].
        const int row = cc * kk;
        const int we = kCoGroup * row;
        for (int e = tid; e < we; e += kThreads) {
            const int j = e / row;
            const int q = e - j * row;
            const int co = co0 + j;
            float v = 0.f;
            if (co < a.c_out) v = wt[((size_t)co * a.c_in + ci0) * kk + q];
            wl[q * kCoGroup + j] = v;
        }
        __syncthreads();
        for (int c = 0; c < cc; ++c) {
            const float *xc = xl + c * plane + (ty * a.stride) * a.halo_w + tx * a.stride;
            const float *wc = wl + c * kk * kCoGroup;
            for (int kh = 0; kh < a.k; ++kh) {
                for (int kw = 0; kw < a.k; ++kw) {
                    const float xv = xc[kh * a.halo_w + kw];
                    const float4 *wp = reinterpret_cast<const float4 *>(wc + (kh * a.k + kw) * kCoGroup);
#pragma unroll
                    for (int j4 = 0; j4 < kCoGroup / 4; ++j4) {
                        const float4 wv = wp[j4];
                        acc[4 * j4 + 0] = fmaf(wv.x, xv, acc[4 * j4 + 0]);
                        acc[4 * j4 + 1] = fmaf(wv.y, xv, acc[4 * j4 + 1]);
                        acc[4 * j4 + 2] = fmaf(wv.z, xv, acc[4 * j4 + 2]);
                        acc[4 * j4 + 3] = fmaf(wv.w, xv, acc[4 * j4 + 3]);
                    }
                }
            }
        }
        __syncthreads();
    }

    const int oh = oh0 + ty, ow = ow0 + tx;
    if (oh < a.h_out && ow < a.w_out) {
#pragma unroll
        for (int j = 0; j < kCoGroup; ++j) {
            const int co = co0 + j;
            if (co < a.c_out) {
                const float b = bias ? bias[co] : 0.f;
                const float v = acc[j] + b;
                out[((size_t)co * a.h_out + oh) * a.w_out + ow] = a.relu && v < 0.f ? 0.f : v;
            }
        }
    }
}

__global__ __launch_bounds__(kThreads) void conv_direct_global(const float *__restrict__ x,
                                                               const float *__restrict__ wt,
                                                               const float *__restrict__ bias,
                                                               float *__restrict__ out, DirectArgs a)
{
    const int64_t total = (int64_t)a.c_out * a.h_out * a.w_out;
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i >= total) return;
    const int ow = (int)(i % a.w_out);
    const int oh = (int)((i / a.w_out) % a.h_out);
    const int co = (int)(i / ((int64_t)a.w_out * a.h_out));
    float acc = 0.f;
    for (int ci = 0; ci < a.c_in; ++ci) {
        for (int kh = 0; kh < a.k; ++kh) {
            const int ih = oh * a.stride - a.pad + kh;
            if (ih < 0 || ih >= a.h) continue;
            for (int kw = 0; kw < a.k; ++kw) {
                const int iw = ow * a.stride - a.pad + kw;
                if (iw < 0 || iw >= a.w) continue;
                acc = fmaf(wt[(((size_t)co * a.c_in + ci) * a.k + kh) * a.k + kw],
                           x[((size_t)ci * a.h + ih) * a.w + iw], acc);
            }
        }
    }
    const float v = acc + (bias ? bias[co] : 0.f);
    out[i] = a.relu && v < 0.f ? 0.f : v;
}

DirectArgs make_args(const ConvShape &s)
{
    DirectArgs a;
    a.c_in = s.c_in; a.h = s.h; a.w = s.w; a.c_out = s.c_out; a.k = s.k;
    a.stride = s.stride; a.pad = s.pad; a.h_out = s.h_out; a.w_out = s.w_out;
    a.halo_h = (kTileH - 1) * s.stride + s.k;
    a.halo_w = (kTileW - 1) * s.stride + s.k;
    a.chunk = 1;
    a.tiles_w = ceil_div(s.w_out, kTileW);
    return a;
}

// Input channels per LDS stage for variant 0, 0 if even one does not fit.
int lds_chunk(const ConvShape &s)
{
    const DirectArgs a = make_args(s);
    const long per_channel = (long)a.halo_h * a.halo_w + (long)s.k * s.k * kCoGroup;
    if (per_channel + 3 > kLdsFloats) return 0;
    long c = (kLdsFloats - 3) / per_channel;
    if (c > 16) c = 16;
    if (c > s.c_in) c = s.c_in;
    return (int)c;
}

}  // namespace

int direct_num_variants() { return 2; }

const char *direct_variant_name(int v)
{
    if (v == 0) return "direct_lds_t8x32_co16";
    if (v == 1) return "direct_global";
    return nullptr;
}

bool direct_variant_info(int v, int *k, int *stride, int *tile_h, int *tile_w, int *co_tile)
{
    if (v < 0 || v >= 2) return false;
    *k = 0;
    *stride = 0;
    *tile_h = v == 0 ? kTileH : 1;
    *tile_w = v == 0 ? kTileW : 1;
    *co_tile = v == 0 ? kCoGroup : 1;
    return true;
}

bool direct_make_plan(const ConvShape &s, int variant, ilpm_plan *p)
{
    ilpm_plan q = {};
    q.path = ILPM_PATH_DIRECT;
    q.variant = variant;
    q.splits = 1;
    q.h_out = s.h_out;
    q.w_out = s.w_out;
    q.block = kThreads;
    q.workspace_bytes = 0;
    if (variant == 0) {
        const int cc = lds_chunk(s);
        if (cc == 0) return false;
        const DirectArgs a = make_args(s);
        q.tile_h = kTileH;
        q.tile_w = kTileW;
        q.co_tile = kCoGroup;
        q.ci_chunk = cc;
        const long tiles = (long)ceil_div(s.h_out, kTileH) * ceil_div(s.w_out, kTileW);
        const long groups = ceil_div(s.c_out, kCoGroup);
        if (tiles > 0x7fffffffL || groups > 65535) return false;
        q.grid = (int)(tiles * groups);
        const long halo = ((long)cc * a.halo_h * a.halo_w + 3) & ~3L;
        q.lds_bytes = (int)(sizeof(float) * (halo + (long)cc * s.k * s.k * kCoGroup));
    } else if (variant == 1) {
        const int64_t total = (int64_t)s.c_out * s.h_out * s.w_out;
        const int64_t blocks = (total + kThreads - 1) / kThreads;
        if (blocks > 0x7fffffffLL) return false;
        q.tile_h = 1;
        q.tile_w = 1;
        q.co_tile = 1;
        q.ci_chunk = 0;
        q.grid = (int)blocks;
        q.lds_bytes = 0;
    } else {
        return false;
    }
    *p = q;
    return true;
}

hipError_t direct_launch(const ilpm_plan &p, const ConvShape &s, const float *x, const float *w,
                         const float *bias, float *out, hipStream_t stream, bool relu)
{
    DirectArgs a = make_args(s);
    a.relu = relu ? 1 : 0;
    if (p.variant == 0) {
        a.chunk = p.ci_chunk;
        const int tiles = ceil_div(s.h_out, kTileH) * ceil_div(s.w_out, kTileW);
        dim3 grid(tiles, ceil_div(s.c_out, kCoGroup));
        hipLaunchKernelGGL(conv_direct_lds, grid, dim3(kThreads), p.lds_bytes, stream, x, w, bias, out, a);
    } else {
        hipLaunchKernelGGL(conv_direct_global, dim3(p.grid), dim3(kThreads), 0, stream, x, w, bias, out, a);
    }
    return hipGetLastError();
}

}  // namespace ilpm
