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
// Variants 2..: low-channel layers (C_in*K*K at most 28 or 64), see
//            conv_direct_mfma below.
#include "internal.h"

namespace ilpm {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) void *lds_ptr_t;

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

// ---- Low-channel layers on the matrix cores ----
//
// When C_in*K*K is small (the network's first layer: 3 input channels, 27
// products per output) the whole contraction is one short run of matrix
// instructions, and the layer's time is its output write (VGG-16's first
// layer writes 12.85 MB and reads 0.6 MB).  What matters is that stores start
// early and keep streaming, so the work is cut into many small independent
// wave tiles -- no LDS, no barrier, several waves per SIMD -- each of which
// gathers its own inputs, runs its matrix instructions and stores its
// results straight from the accumulators.
//
// A wave owns 16*MB output channels x 16*NPB consecutive output pixels (in
// the row-major order of the output plane, so a block may span two rows).
// The contraction index is k = (ci*K + kh)*K + kw, i.e. an OIHW weight row
// read as it is; step s of the v_mfma_f32_16x16x4_f32 chain covers k = 4s..
// 4s+3, lane (g, l) supplying A = w[co0 + 16m + l][4s + g] (loaded once) and
// B = the input tap of k = 4s + g for pixel 16n + l of the tile, gathered
// with buffer loads whose offset is pushed past the range for padding taps
// and for k >= C_in*K*K (a buffer load out of range returns 0).
//
// Divisions by sizes fixed at launch are multiply-shifts with multipliers
// from the host: k / d = (k * ceil(2^16 / d)) >> 16, exact for k < 64 and
// d <= 64 (the error k*(ceil(2^16/d) - 2^16/d)/2^16 < 2^-10 stays below the
// 1/d gap to the next integer), and p / W_out = mulhi(p, ceil(2^32 / W_out)),
// exact while p * W_out < 2^32 (checked when the plan is made) -- for W_out
// >= 2; the multiplier for W_out = 1 would be 2^32, so that case is p itself.
struct LowcArgs {
    int c_in, h, w, c_out, k, stride, pad, h_out, w_out;
    int kt;          // C_in*K*K
    int units;       // wave tiles
    int co_groups;   // output-channel groups of 16*MB
    int relu;
    unsigned m_kk, m_k;  // ceil(2^16 / (K*K)), ceil(2^16 / K)
    unsigned m_w;        // ceil(2^32 / W_out) for W_out >= 2 (unused for W_out = 1)
};

__device__ __forceinline__ __amdgpu_buffer_rsrc_t lowc_rsrc(const float *base, unsigned bytes)
{
    const uint64_t b = reinterpret_cast<uint64_t>(base);
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)b);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(b >> 32));
    float *q = reinterpret_cast<float *>(((uint64_t)hi << 32) | lo);
    return __builtin_amdgcn_make_buffer_rsrc(q, (short)0, (int)__builtin_amdgcn_readfirstlane(bytes), 0x00020000);
}

template <int MB, int NPB, int STEPS>
__global__ __launch_bounds__(256) void conv_direct_mfma(const float *__restrict__ x, const float *__restrict__ wt,
                                                        const float *__restrict__ bias, float *__restrict__ out,
                                                        LowcArgs a)
{
    constexpr unsigned kFar = 0x80000000u;  // past every descriptor's range
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int g = lane >> 4, l = lane & 15;
    // Workgroups are dealt to the 8 XCDs round-robin; give each XCD a
    // contiguous run of tiles so that neighbouring pixels (shared input rows)
    // meet in one L2.
    const int nwg = (int)gridDim.x;
    const int xcd = (int)blockIdx.x % 8, slot = (int)blockIdx.x / 8;
    const int per = nwg / 8, extra = nwg % 8;
    const int lin = xcd * per + min(xcd, extra) + slot;
    const int unit = lin * 4 + wave;
    if (unit >= a.units) return;  // whole waves only; the kernel has no barrier
    const int cg = unit % a.co_groups;
    const int pg = unit / a.co_groups;
    const int co0 = cg * 16 * MB;
    const int plane = a.h_out * a.w_out;

    const __amdgpu_buffer_rsrc_t rw = lowc_rsrc(wt, (unsigned)a.c_out * a.kt * 4u);
    const __amdgpu_buffer_rsrc_t rx = lowc_rsrc(x, (unsigned)a.c_in * a.h * a.w * 4u);
    const __amdgpu_buffer_rsrc_t ro = lowc_rsrc(out, (unsigned)a.c_out * plane * 4u);

    // Input pixel of each of this lane's blocks: top-left tap (ih0, iw0).
    int ih0[NPB], iw0[NPB];
    bool pix_ok[NPB];
#pragma unroll
    for (int n = 0; n < NPB; ++n) {
        const int p = (pg * NPB + n) * 16 + l;
        const int oh = a.w_out == 1 ? p : (int)__umulhi((unsigned)p, a.m_w), ow = p - oh * a.w_out;
        pix_ok[n] = p < plane;
        ih0[n] = oh * a.stride - a.pad;
        iw0[n] = ow * a.stride - a.pad;
    }
    // B gathers, all issued before the first matrix instruction.
    float bv[STEPS][NPB];
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
        const int k = 4 * s + g;
        const int ci = (int)(((unsigned)k * a.m_kk) >> 16), t = k - ci * a.k * a.k;
        const int kh = (int)(((unsigned)t * a.m_k) >> 16), kw = t - kh * a.k;
#pragma unroll
        for (int n = 0; n < NPB; ++n) {
            const int ih = ih0[n] + kh, iw = iw0[n] + kw;
            const bool ok = k < a.kt && pix_ok[n] && (unsigned)ih < (unsigned)a.h && (unsigned)iw < (unsigned)a.w;
            const unsigned off = ok ? (unsigned)((ci * a.h + ih) * a.w + iw) * 4u : kFar;
            bv[s][n] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rx, (int)off, 0, 0));
        }
    }
    // A: this lane's weights, w[co0 + 16m + l][4s + g].
    float av[MB][STEPS];
#pragma unroll
    for (int m = 0; m < MB; ++m) {
        const int co = co0 + 16 * m + l;
#pragma unroll
        for (int s = 0; s < STEPS; ++s) {
            const int k = 4 * s + g;
            const unsigned off = (co < a.c_out && k < a.kt) ? (unsigned)(co * a.kt + k) * 4u : kFar;
            av[m][s] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rw, (int)off, 0, 0));
        }
    }
    // Accumulators start from the bias: register r of block (m, n) is output
    // channel co0 + 16m + 4g + r at pixel 16n + l.
    floatx4 acc[MB][NPB];
#pragma unroll
    for (int m = 0; m < MB; ++m) {
        float b4[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int co = co0 + 16 * m + 4 * g + r;
            b4[r] = (bias != nullptr && co < a.c_out) ? bias[co] : 0.f;
        }
#pragma unroll
        for (int n = 0; n < NPB; ++n) acc[m][n] = floatx4{b4[0], b4[1], b4[2], b4[3]};
    }
#pragma unroll
    for (int s = 0; s < STEPS; ++s)
#pragma unroll
        for (int n = 0; n < NPB; ++n)
#pragma unroll
            for (int m = 0; m < MB; ++m)
                acc[m][n] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[m][s], bv[s][n], acc[m][n], 0, 0, 0);
    // Stores: lanes along pixels (16 consecutive pixels of one channel per
    // lane group); channels past C_out and pixels past the plane go out of
    // range and are dropped.
#pragma unroll
    for (int m = 0; m < MB; ++m) {
        const int co = co0 + 16 * m + 4 * g;
#pragma unroll
        for (int n = 0; n < NPB; ++n) {
            const int p = (pg * NPB + n) * 16 + l;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const bool ok = pix_ok[n] && co + r < a.c_out;
                const unsigned off = ok ? (unsigned)((co + r) * plane + p) * 4u : kFar;
                float v = acc[m][n][r];
                if (a.relu && v < 0.f) v = 0.f;
                __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), ro, (int)off, 0, 0);
            }
        }
    }
}

struct LowcVariant {
    const char *name;
    int mb, npb, steps;
    void (*launch)(dim3, hipStream_t, const float *, const float *, const float *, float *, const LowcArgs &);
};

template <int MB, int NPB, int STEPS>
void lowc_launch(dim3 grid, hipStream_t st, const float *x, const float *w, const float *b, float *o,
                 const LowcArgs &a)
{
    hipLaunchKernelGGL((conv_direct_mfma<MB, NPB, STEPS>), grid, dim3(256), 0, st, x, w, b, o, a);
}

const LowcVariant kLowc[] = {
    {"direct_mfma_k28_co16_px16", 1, 1, 7, &lowc_launch<1, 1, 7>},
    {"direct_mfma_k28_co64_px32", 4, 2, 7, &lowc_launch<4, 2, 7>},
    {"direct_mfma_k64_co16_px32", 1, 2, 16, &lowc_launch<1, 2, 16>},
};
constexpr int kNumLowc = sizeof(kLowc) / sizeof(kLowc[0]);
constexpr int kFirstLowc = 2;  // direct variants 0 and 1 are the VALU kernels

// ---- Low-channel layers, whole row segments per workgroup ----
//
// The same contraction as conv_direct_mfma -- k = 4s + g, accumulators
// starting from the bias, step s = 0, 1, ... in order -- so the two give the
// same bits; cut differently.  A workgroup takes one segment of 16*NB*PW
// consecutive pixels of one output row, for a group of 16*CW output channels
// (waves (pw, cw): wave pw's NB blocks of 16 pixels, channels 16*cw..), and
// first copies the C_in*K input rows that segment reads into LDS by buffer
// DMA (zeros for padding rows and columns), then reads every B operand from
// there.  Its stores cover whole pieces of 16 consecutive pixels of a row, so
// where the row length is a multiple of 16 floats each lane group writes one
// aligned 64-byte piece.  (On MI355X a write-only kernel storing VGG-16's
// first-layer output, 12.85 MB, in such pieces ran at 3.8 us per launch, as
// fast as a linear copy; in the 14-pixel pieces of 14x14 tiles, 5.7 us.)
// Each pair of blocks is stored once its matrix instructions are issued, so
// the stores stream behind the matrix work.
//
// The weights and bias come in by the same DMA: a channel group's weights
// are 16*CW*C_in*K*K consecutive words of the OIHW tensor, copied whole in
// 16-byte lanes (4-byte lanes where C_out*C_in*K*K is not a multiple of 4,
// so that no lane's access crosses the end of the tensor), and each lane
// reads its A operands from LDS after the barrier.  (Loaded per lane from
// the tensor instead -- lane (g, l) reading w[co0 + l][4s + g], 16 lanes at
// a stride of C_in*K*K words -- every workgroup sent ~400 cache-line
// requests for the same few lines at kernel start; on MI355X, for VGG-16's
// first layer, the DMA form ran 0.6 us per launch faster.)
//
// LDS: row r = ci*K + kh holds input row oy*S - pad + kh from column ax0
// on at r*lwp; row C_in*K is all zeros and serves the contraction slots
// k >= C_in*K*K.  Where W is a multiple of 4 and the input 16-byte aligned,
// ax0 = ix0 rounded down to a multiple of 4 and each row is copied in
// 16-byte lanes (lwp = 256 * ceil((lw + 3) / 256): one DMA of 256 words per
// wave and chunk), so that a lane's four columns lie all inside the input
// row or all in its padding; else ax0 = ix0 and 4-byte lanes (one DMA of 64
// words per chunk; lwp = 64 * ceil(lw / 64), or the 16-byte layout's pitch
// where the plan allotted it).  For VGG-16's first layer the 16-byte rows
// halve the input DMAs (9 instead of 18 per workgroup).  The group's weights follow at
// (C_in*K + 1)*lwp (wregion = 256 * ceil(16*CW*C_in*K*K / 256) words, whole
// 16-byte DMAs), then its 16*CW biases (64 words, one DMA).
struct RowsArgs {
    int c_in, h, w, c_out, k, stride, pad, h_out, w_out;
    int kt;         // C_in*K*K
    int segs;       // segments per output row
    int co_groups;  // output-channel groups of 16*CW
    int lw, lwp, chunks;
    int chunks16;   // 256-word chunks per row in the 16-byte layout (0: the plan has no such layout)
    int x16;        // 1: input rows by 16-byte DMA lanes (chunks16 > 0, input 16-byte aligned)
    int wregion;    // LDS words of the weight area
    int w16;        // 1: weights by 16-byte DMA lanes (C_out*kt a multiple of 4)
    int relu;
    unsigned m_kk, m_k;  // ceil(2^16 / (K*K)), ceil(2^16 / K)
};

// SK = 1: instantiated for stride 1 (B operand offsets fold into the LDS
// reads' immediates); SK = 0: any stride.
template <int NB, int PW, int CW, int STEPS, int POL, int SK>
__global__ __launch_bounds__(256) void conv_direct_rows(const float *__restrict__ x, const float *__restrict__ wt,
                                                        const float *__restrict__ bias, float *__restrict__ out,
                                                        RowsArgs a)
{
    extern __shared__ float xl[];
    constexpr unsigned kFar = 0x80000000u;  // past every descriptor's range
    constexpr int kNI = 2;                  // blocks whose matrix chains are interleaved
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int g = lane >> 4, l = lane & 15;
    // Contiguous runs of units per XCD (workgroup i runs on XCD i mod 8), so
    // that neighbouring rows -- which read the same input rows -- meet in one
    // L2.  Unit order: channel group fastest, then segment, then row.
    const int nwg = (int)gridDim.x;
    const int xcd = (int)blockIdx.x % 8, slot = (int)blockIdx.x / 8;
    const int per = nwg / 8, extra = nwg % 8;
    const int lin = xcd * per + min(xcd, extra) + slot;
    const int cgi = lin % a.co_groups;
    const int rest = lin / a.co_groups;
    const int seg = rest % a.segs;
    const int oy = rest / a.segs;
    const int px0 = seg * 16 * NB * PW;
    const int ix0 = px0 * a.stride - a.pad, iy0 = oy * a.stride - a.pad;
    const int rows = a.c_in * a.k;

    const __amdgpu_buffer_rsrc_t rx = lowc_rsrc(x, (unsigned)a.c_in * a.h * a.w * 4u);
    const __amdgpu_buffer_rsrc_t rw = lowc_rsrc(wt, (unsigned)a.c_out * a.kt * 4u);
    const __amdgpu_buffer_rsrc_t rb = lowc_rsrc(bias, bias != nullptr ? (unsigned)a.c_out * 4u : 0u);
    const __amdgpu_buffer_rsrc_t ro = lowc_rsrc(out, (unsigned)a.c_out * a.h_out * a.w_out * 4u);

    const int pw = wave % PW, cw = wave / PW;
    const bool active = wave < PW * CW;
    const int cg0 = cgi * CW * 16;  // the group's first channel
    const int co0 = cg0 + cw * 16;
    float *const wl = xl + (rows + 1) * a.lwp;
    float *const bl = wl + a.wregion;
    // The group's weights and biases into LDS (channels past C_out read as
    // zeros: their offsets lie past the descriptors' ranges).
    {
        const unsigned wbase = (unsigned)cg0 * (unsigned)a.kt;
        const int nw = 16 * CW * a.kt;
        if (a.w16) {
            for (int q = wave; 256 * q < nw; q += 4) {
                const int j = 256 * q + 4 * lane;
                const unsigned off = j < nw ? (wbase + (unsigned)j) * 4u : kFar;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr_t)(wl + 256 * q), 16, (int)off, 0, 0, 0);
            }
        } else {
            for (int q = wave; 64 * q < nw; q += 4) {
                const int j = 64 * q + lane;
                const unsigned off = j < nw ? (wbase + (unsigned)j) * 4u : kFar;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_ptr_t)(wl + 64 * q), 4, (int)off, 0, 0, 0);
            }
        }
        if (wave == 3) {
            const unsigned off = lane < 16 * CW ? (unsigned)(cg0 + lane) * 4u : kFar;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(rb, (lds_ptr_t)bl, 4, (int)off, 0, 0, 0);
        }
    }
    // Input rows into LDS: wave w issues chunks w, w + 4, ... of the
    // rows * chunks list (chunk i of row r = input columns ax0 + 64i .. in
    // 4-byte lanes, ax0 + 256i .. in 16-byte lanes).  (r, i) and
    // r = (ci, kh) advance by counting, without divisions.
    const int ax0 = a.x16 ? (ix0 & ~3) : ix0;
    const int shift = ix0 - ax0;  // LDS column of input column ix0
    {
        const int nch = a.x16 ? a.chunks16 : a.chunks;
        int r = 0, i = wave, ci = 0, kh = 0;
        auto settle = [&]() {
            while (i >= nch) {
                i -= nch;
                ++r;
                if (++kh == a.k) {
                    kh = 0;
                    ++ci;
                }
            }
        };
        settle();
        if (a.x16) {
            while (r < rows) {
                const int iy = iy0 + kh;
                const int j = 256 * i + 4 * lane, cx = ax0 + j;
                const bool ok = j < a.lw + shift && (unsigned)iy < (unsigned)a.h && (unsigned)cx < (unsigned)a.w;
                const unsigned off = ok ? (unsigned)((ci * a.h + iy) * a.w + cx) * 4u : kFar;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_ptr_t)(xl + r * a.lwp + 256 * i), 16, (int)off, 0, 0,
                                                         0);
                i += 4;
                settle();
            }
        } else {
            while (r < rows) {
                const int iy = iy0 + kh;
                const int j = 64 * i + lane, ix = ix0 + j;
                const bool ok = j < a.lw && (unsigned)iy < (unsigned)a.h && (unsigned)ix < (unsigned)a.w;
                const unsigned off = ok ? (unsigned)((ci * a.h + iy) * a.w + ix) * 4u : kFar;
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_ptr_t)(xl + r * a.lwp + 64 * i), 4, (int)off, 0, 0,
                                                         0);
                i += 4;
                settle();
            }
        }
    }
    for (int j = tid; j < a.lwp; j += 256) xl[rows * a.lwp + j] = 0.f;

    // While the DMA is in flight: the LDS word that contraction slot
    // k = 4s + g reads for this lane's pixel of block 0 (slots past
    // C_in*K*K read the zero row), and the output offsets.
    const int stride = SK ? 1 : a.stride;
    const int pl = pw * NB * 16 + l;  // this lane's pixel of block 0, within the segment
    int tb[STEPS];
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
        const int k = 4 * s + g;
        const int ci = (int)(((unsigned)k * a.m_kk) >> 16), t = k - ci * a.k * a.k;
        const int kh = (int)(((unsigned)t * a.m_k) >> 16), kw = t - kh * a.k;
        tb[s] = (k < a.kt ? (ci * a.k + kh) * a.lwp + kw : rows * a.lwp) + shift + pl * stride;
    }
    const int plane = a.h_out * a.w_out;
    const unsigned obase = (unsigned)(co0 + 4 * g) * (unsigned)plane + (unsigned)(oy * a.w_out + px0 + pl);
    // Every pixel and channel of this wave's tile inside the output: stores
    // without per-lane checks, the channel row's offset in the scalar operand.
    const bool full = px0 + (pw + 1) * NB * 16 <= a.w_out && co0 + 16 <= a.c_out;

    __builtin_amdgcn_s_waitcnt(0);  // this wave's DMA has landed in LDS
    __syncthreads();
    if (!active) return;  // no barrier follows

    // A: this lane's weights w[co0 + l][4s + g] (read for every slot: the
    // word a slot past C_in*K*K would read lies inside the weight and bias
    // areas); the accumulators start at the bias.
    float av[STEPS];
#pragma unroll
    for (int s = 0; s < STEPS; ++s) {
        const int k = 4 * s + g;
        const float wv = wl[(cw * 16 + l) * a.kt + k];
        av[s] = k < a.kt ? wv : 0.f;
    }
    float b4[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) b4[r] = bl[cw * 16 + 4 * g + r];

#pragma unroll
    for (int n0 = 0; n0 < NB; n0 += kNI) {
        floatx4 acc[kNI];
#pragma unroll
        for (int u = 0; u < kNI; ++u) acc[u] = floatx4{b4[0], b4[1], b4[2], b4[3]};
#pragma unroll
        for (int s = 0; s < STEPS; ++s)
#pragma unroll
            for (int u = 0; u < kNI; ++u)
                if (n0 + u < NB) {
                    const float bv = xl[tb[s] + 16 * (n0 + u) * stride];
                    acc[u] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s], bv, acc[u], 0, 0, 0);
                }
        if (a.relu) {
#pragma unroll
            for (int u = 0; u < kNI; ++u)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    if (acc[u][r] < 0.f) acc[u][r] = 0.f;
        }
        if (full) {
#pragma unroll
            for (int u = 0; u < kNI; ++u)
                if (n0 + u < NB) {
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float v = acc[u][r];
                        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), ro,
                                                              (int)((obase + 16u * (n0 + u)) * 4u),
                                                              (int)((unsigned)(r * plane) * 4u), POL);
                    }
                }
        } else {
#pragma unroll
            for (int u = 0; u < kNI; ++u)
                if (n0 + u < NB) {
                    const bool pix_ok = px0 + pl + 16 * (n0 + u) < a.w_out;
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const bool ok = pix_ok && co0 + 4 * g + r < a.c_out;
                        const unsigned off = ok ? (obase + (unsigned)(r * plane + 16 * (n0 + u))) * 4u : kFar;
                        const float v = acc[u][r];
                        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), ro, (int)off, 0, POL);
                    }
                }
        }
    }
}

struct RowsVariant {
    const char *name;
    int nb, pw, cw;
    void (*launch)(dim3, int, hipStream_t, const float *, const float *, const float *, float *, const RowsArgs &);
};

template <int NB, int PW, int CW, int POL>
void rows_launch(dim3 grid, int lds, hipStream_t st, const float *x, const float *w, const float *b, float *o,
                 const RowsArgs &a)
{
    if (a.stride == 1)
        hipLaunchKernelGGL((conv_direct_rows<NB, PW, CW, 7, POL, 1>), grid, dim3(256), lds, st, x, w, b, o, a);
    else
        hipLaunchKernelGGL((conv_direct_rows<NB, PW, CW, 7, POL, 0>), grid, dim3(256), lds, st, x, w, b, o, a);
}

// Store policy SC1 (device scope): the output is written through each XCD's
// L2 to the level the XCDs share while the kernel runs, instead of being
// written back from the L2 caches when it ends; for VGG-16's first layer on
// MI355X that took 0.9 us off ~6.8 us per launch, and each row variant
// measured faster with it than with ordinary stores.
constexpr int kSc1 = 16;

const RowsVariant kRows[] = {
    {"direct_rows_k28_co64_px224_sc1", 14, 1, 4, &rows_launch<14, 1, 4, kSc1>},
    {"direct_rows_k28_co64_px112_sc1", 7, 1, 4, &rows_launch<7, 1, 4, kSc1>},
    {"direct_rows_k28_co64_px64_sc1", 4, 1, 4, &rows_launch<4, 1, 4, kSc1>},
    {"direct_rows_k28_co64_px32_sc1", 2, 1, 4, &rows_launch<2, 1, 4, kSc1>},
    {"direct_rows_k28_co32_px128_sc1", 4, 2, 2, &rows_launch<4, 2, 2, kSc1>},
    {"direct_rows_k28_co32_px32_sc1", 1, 2, 2, &rows_launch<1, 2, 2, kSc1>},
    {"direct_rows_k28_co16_px64_sc1", 1, 4, 1, &rows_launch<1, 4, 1, kSc1>},
    {"direct_rows_k28_co16_px32_sc1", 1, 2, 1, &rows_launch<1, 2, 1, kSc1>},
};
constexpr int kNumRows = sizeof(kRows) / sizeof(kRows[0]);
constexpr int kFirstRows = kFirstLowc + kNumLowc;
constexpr int kRowsLdsFloats = 16384;  // 64 KiB

RowsArgs rows_args(const ConvShape &s, const RowsVariant &d)
{
    RowsArgs a;
    a.c_in = s.c_in; a.h = s.h; a.w = s.w; a.c_out = s.c_out; a.k = s.k;
    a.stride = s.stride; a.pad = s.pad; a.h_out = s.h_out; a.w_out = s.w_out;
    a.kt = s.c_in * s.k * s.k;
    a.segs = ceil_div(s.w_out, 16 * d.nb * d.pw);
    a.co_groups = ceil_div(s.c_out, 16 * d.cw);
    a.lw = (16 * d.nb * d.pw - 1) * s.stride + s.k;
    a.chunks = ceil_div(a.lw, 64);
    a.lwp = 64 * a.chunks;
    a.chunks16 = 0;
    a.x16 = 0;
    a.wregion = 256 * ceil_div(16 * d.cw * a.kt, 256);
    a.w16 = ((int64_t)s.c_out * a.kt) % 4 == 0 ? 1 : 0;
    a.relu = 0;
    // The 16-byte row layout where W is a multiple of 4 and it fits in LDS.
    if (s.w % 4 == 0) {
        const int c16 = ceil_div(a.lw + 3, 256);
        if ((int64_t)(s.c_in * s.k + 1) * 256 * c16 + a.wregion + 64 <= kRowsLdsFloats) {
            a.chunks16 = c16;
            a.lwp = 256 * c16;
        }
    }
    a.m_kk = (65536u + (unsigned)(s.k * s.k) - 1) / (unsigned)(s.k * s.k);
    a.m_k = (65536u + (unsigned)s.k - 1) / (unsigned)s.k;
    return a;
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

int direct_num_variants() { return kFirstRows + kNumRows; }

const char *direct_variant_name(int v)
{
    if (v == 0) return "direct_lds_t8x32_co16";
    if (v == 1) return "direct_global";
    if (v >= kFirstLowc && v < kFirstLowc + kNumLowc) return kLowc[v - kFirstLowc].name;
    if (v >= kFirstRows && v < kFirstRows + kNumRows) return kRows[v - kFirstRows].name;
    return nullptr;
}

bool direct_variant_info(int v, int *k, int *stride, int *tile_h, int *tile_w, int *co_tile)
{
    if (v < 0 || v >= direct_num_variants()) return false;
    *k = 0;
    *stride = 0;
    if (v >= kFirstRows) {
        // A workgroup's tile: 16*NB*PW consecutive pixels of one output row.
        const RowsVariant &d = kRows[v - kFirstRows];
        *tile_h = 1;
        *tile_w = 16 * d.nb * d.pw;
        *co_tile = 16 * d.cw;
        return true;
    }
    if (v >= kFirstLowc) {
        // A wave's tile: 16*NPB consecutive pixels of the output plane.
        const LowcVariant &d = kLowc[v - kFirstLowc];
        *tile_h = 1;
        *tile_w = 16 * d.npb;
        *co_tile = 16 * d.mb;
        return true;
    }
    *tile_h = v == 0 ? kTileH : 1;
    *tile_w = v == 0 ? kTileW : 1;
    *co_tile = v == 0 ? kCoGroup : 1;
    return true;
}

bool direct_is_lowc(int v) { return v >= kFirstLowc && v < kFirstRows + kNumRows; }

int direct_lowc_max_kt(int v)
{
    if (v >= kFirstRows && v < kFirstRows + kNumRows) return 28;
    return direct_is_lowc(v) ? 4 * kLowc[v - kFirstLowc].steps : 0;
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
    } else if (variant >= kFirstLowc && variant < kFirstLowc + kNumLowc) {
        const LowcVariant &d = kLowc[variant - kFirstLowc];
        const int64_t kt = (int64_t)s.c_in * s.k * s.k;
        const int64_t plane = (int64_t)s.h_out * s.w_out;
        // The whole contraction in one run of matrix instructions; byte
        // offsets of 31 bits (input, weights) and 30 bits (output).
        if (kt > 4 * d.steps) return false;
        // p / W_out by multiply-shift (see LowcArgs): exact while p * W_out < 2^32.
        if ((plane + 16 * d.npb) * (int64_t)s.w_out >= (1LL << 32)) return false;
        if ((int64_t)s.c_in * s.h * s.w * 4 >= (1LL << 31) || (int64_t)s.c_out * kt * 4 >= (1LL << 31) ||
            (int64_t)s.c_out * plane * 4 >= (1LL << 30))
            return false;
        const int64_t co_groups = (s.c_out + 16 * d.mb - 1) / (16 * d.mb);
        const int64_t units = co_groups * ((plane + 16 * d.npb - 1) / (16 * d.npb));
        if (units > 0x7fffffffLL - 3) return false;
        q.tile_h = 1;
        q.tile_w = 16 * d.npb;
        q.co_tile = 16 * d.mb;
        q.ci_chunk = s.c_in;
        q.grid = (int)((units + 3) / 4);
        q.lds_bytes = 0;
    } else if (variant >= kFirstRows && variant < kFirstRows + kNumRows) {
        const RowsVariant &d = kRows[variant - kFirstRows];
        const int64_t kt = (int64_t)s.c_in * s.k * s.k;
        const int64_t plane = (int64_t)s.h_out * s.w_out;
        // The whole contraction in one run of 7 matrix steps; 31-bit byte
        // offsets; the input rows and the zero row within 64 KiB of LDS.
        if (kt > 28) return false;
        if ((int64_t)s.c_in * s.h * s.w * 4 >= (1LL << 31) || (int64_t)s.c_out * kt * 4 >= (1LL << 31) ||
            (int64_t)s.c_out * plane * 4 >= (1LL << 31))
            return false;
        const RowsArgs a = rows_args(s, d);
        const int64_t lds_floats = (int64_t)(s.c_in * s.k + 1) * a.lwp + a.wregion + 64;
        if (lds_floats > kRowsLdsFloats) return false;
        const int64_t units = (int64_t)s.h_out * a.segs * a.co_groups;
        if (units > 0x7fffffffLL) return false;
        q.tile_h = 1;
        q.tile_w = 16 * d.nb * d.pw;
        q.co_tile = 16 * d.cw;
        q.ci_chunk = s.c_in;
        q.grid = (int)units;
        q.lds_bytes = (int)(sizeof(float) * lds_floats);
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
    if (p.variant >= kFirstRows && p.variant < kFirstRows + kNumRows) {
        const RowsVariant &d = kRows[p.variant - kFirstRows];
        RowsArgs ra = rows_args(s, d);
        ra.relu = relu ? 1 : 0;
        ra.x16 = ra.chunks16 > 0 && (reinterpret_cast<uintptr_t>(x) & 15) == 0 ? 1 : 0;
        d.launch(dim3(p.grid), p.lds_bytes, stream, x, w, bias, out, ra);
        return hipGetLastError();
    }
    if (direct_is_lowc(p.variant)) {
        const LowcVariant &d = kLowc[p.variant - kFirstLowc];
        LowcArgs la;
        la.c_in = s.c_in; la.h = s.h; la.w = s.w; la.c_out = s.c_out; la.k = s.k;
        la.stride = s.stride; la.pad = s.pad; la.h_out = s.h_out; la.w_out = s.w_out;
        la.kt = s.c_in * s.k * s.k;
        la.co_groups = ceil_div(s.c_out, 16 * d.mb);
        la.units = la.co_groups * ceil_div(s.h_out * s.w_out, 16 * d.npb);
        la.relu = relu ? 1 : 0;
        la.m_kk = (65536u + (unsigned)(s.k * s.k) - 1) / (unsigned)(s.k * s.k);
        la.m_k = (65536u + (unsigned)s.k - 1) / (unsigned)s.k;
        la.m_w = s.w_out >= 2 ? (unsigned)(((1ull << 32) + (uint64_t)s.w_out - 1) / (uint64_t)s.w_out) : 0u;
        d.launch(dim3(p.grid), stream, x, w, bias, out, la);
        return hipGetLastError();
    }
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
