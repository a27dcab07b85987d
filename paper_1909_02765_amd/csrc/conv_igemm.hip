// Implicit-GEMM convolution on the fp32 matrix cores (v_mfma_f32_16x16x4_f32).
//
// The convolution is the product D = A * B with
//   A [C_out x C_in*K*K]  = the OIHW weights, read as they are,
//   B [C_in*K*K x pixels] = input patches, never materialised: every B element
//                           is read from a zero-padded input halo tile in LDS,
//   D [C_out x pixels]    = the NCHW output.
// This keeps the two properties the ILP-M paper argues for (Section 4): each
// input and weight element is fetched from global memory once per workgroup,
// staged collaboratively with one barrier per stage, and between barriers a
// wavefront runs a long barrier-free stream of independent multiply-adds (here
// matrix-core instructions, each 1024 MACs, with every operand reused by a
// whole row or column of accumulator blocks).
//
// Contraction order.  Within a stage of CC input channels the contraction
// index runs tap-major, channel-minor: MFMA step (t, c4) covers tap t and the
// four channels 4*c4 .. 4*c4+3, one channel per 16-lane group.  Any order of
// the sum is the same convolution; this one makes every LDS address a
// per-lane base plus a compile-time offset.
//
// Work split.  A workgroup owns TH x TW output pixels and COT = NWC*16*MA
// output channels.  Wave (wc, wp) owns 16*MA channels and NB blocks of 16
// pixels, so it keeps MA*NB 16x16 accumulator blocks.  Optional split of the
// input channels across `splits` workgroups (grid y): each writes its partial
// tile to the workspace and the last one to arrive (per-tile counter) sums the
// partials in split order, adds the bias and stores the tile, so the result
// does not depend on arrival order.
//
// LDS per stage (double buffered, one barrier per stage):
//   weights [COT][RS]   RS >= CC*K*K, row = one output channel's CC*K*K
//                       weights in OIHW order (a straight copy of global);
//                       RS = 2 mod 4 so the 16 rows one MFMA operand reads
//                       fall in distinct banks.
//   halo    [CC][PL]    plane = (TH-1)*S+K rows of (TW-1)*S+K pixels, planes
//                       padded to PL = 16 mod 32 words (stride 1) or odd
//                       (stride 2) so the four lane groups of a read spread
//                       over the banks.
#include <cmath>

#include "internal.h"

namespace ilpm {
namespace {

typedef float floatx4 __attribute__((ext_vector_type(4)));

constexpr int row_pad(int n)
{
    int r = n;
    while (r % 4 != 2) ++r;
    return r;
}

constexpr int plane_pad(int n, int s)
{
    int r = n;
    if (s % 2 == 1) {
        while (r % 32 != 16) ++r;
    } else {
        while (r % 2 != 1) ++r;
    }
    return r;
}

template <int KS_, int S_, int TH_, int TW_, int NWC_, int NWP_, int MA_, int CC_>
struct Cfg {
    static constexpr int KS = KS_, S = S_, TH = TH_, TW = TW_;
    static constexpr int NWC = NWC_, NWP = NWP_, MA = MA_, CC = CC_;
    static constexpr int NT = 64 * NWC * NWP;
    static constexpr int NPIX = TH * TW;
    static constexpr int NB = (NPIX + 16 * NWP - 1) / (16 * NWP);
    static constexpr int NPIXP = NWP * NB * 16;
    static constexpr int KK = KS * KS;
    static constexpr int HR = (TH - 1) * S + KS;
    static constexpr int HC = (TW - 1) * S + KS;
    static constexpr int PL = plane_pad(HR * HC, S);
    static constexpr int WROW = CC * KK;
    static constexpr int RS = row_pad(WROW);
    static constexpr int COT = NWC * 16 * MA;
    static constexpr int WSZ = COT * RS;
    static constexpr int XSZ = CC * PL;
    static constexpr int BUF = ((WSZ + XSZ + 3) / 4) * 4;
    static constexpr int XE = CC * HR * HC;
    static constexpr int XPT = (XE + NT - 1) / NT;
    static constexpr int WE = COT * WROW;
    static constexpr int WPT = (WE + NT - 1) / NT;
    static constexpr int LDS_BYTES = 2 * BUF * 4;
    static_assert(CC % 4 == 0, "a stage holds whole groups of 4 channels");
    static_assert(LDS_BYTES <= 65536, "LDS budget");
};

struct IgArgs {
    int c_in, h, w, c_out, pad, h_out, w_out;
    int tiles_w, co_tiles, nchunks, chunks_per_split, splits;
    size_t part_offset;  // floats from the workspace start to the partial sums
};

template <class C>
__device__ __forceinline__ void load_stage(const float *__restrict__ x, const float *__restrict__ w,
                                           const IgArgs &a, int ci0, int ih0, int iw0, int co0,
                                           float (&xr)[C::XPT], float (&wr)[C::WPT])
{
    const int tid = threadIdx.x;
#pragma unroll
    for (int j = 0; j < C::XPT; ++j) {
        const int e = tid + j * C::NT;
        float v = 0.f;
        if (e < C::XE) {
            const int c = e / (C::HR * C::HC);
            const int rem = e - c * (C::HR * C::HC);
            const int r = rem / C::HC;
            const int col = rem - r * C::HC;
            const int ci = ci0 + c, ih = ih0 + r, iw = iw0 + col;
            if (ci < a.c_in && ih >= 0 && ih < a.h && iw >= 0 && iw < a.w)
                v = x[((size_t)ci * a.h + ih) * a.w + iw];
        }
        xr[j] = v;
    }
#pragma unroll
    for (int j = 0; j < C::WPT; ++j) {
        const int e = tid + j * C::NT;
        float v = 0.f;
        if (e < C::WE) {
            const int row = e / C::WROW;
            const int q = e - row * C::WROW;
            const int co = co0 + row;
            const int ci = ci0 + q / C::KK;
            if (co < a.c_out && ci < a.c_in)
                v = w[((size_t)co * a.c_in + ci0) * C::KK + q];
        }
        wr[j] = v;
    }
}

template <class C>
__device__ __forceinline__ void store_stage(float *buf, const float (&xr)[C::XPT], const float (&wr)[C::WPT])
{
    const int tid = threadIdx.x;
    float *wl = buf;
    float *xl = buf + C::WSZ;
#pragma unroll
    for (int j = 0; j < C::XPT; ++j) {
        const int e = tid + j * C::NT;
        if (e < C::XE) {
            const int c = e / (C::HR * C::HC);
            const int rem = e - c * (C::HR * C::HC);
            xl[c * C::PL + rem] = xr[j];
        }
    }
#pragma unroll
    for (int j = 0; j < C::WPT; ++j) {
        const int e = tid + j * C::NT;
        if (e < C::WE) {
            const int row = e / C::WROW;
            const int q = e - row * C::WROW;
            wl[row * C::RS + q] = wr[j];
        }
    }
}

template <class C>
__global__ __launch_bounds__(C::NT) void conv_igemm(const float *__restrict__ x, const float *__restrict__ w,
                                                    const float *__restrict__ bias, float *__restrict__ out,
                                                    float *__restrict__ ws, IgArgs a)
{
    __shared__ __attribute__((aligned(16))) float lds[2 * C::BUF];
    __shared__ unsigned s_last;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wc = wave % C::NWC;
    const int wp = wave / C::NWC;
    const int g = lane >> 4;
    const int l16 = lane & 15;

    const int tile = blockIdx.x;
    const int co_t = tile % a.co_tiles;
    const int sp = tile / a.co_tiles;
    const int tw_i = sp % a.tiles_w;
    const int th_i = sp / a.tiles_w;
    const int split = blockIdx.y;
    const int co0 = co_t * C::COT;
    const int oh0 = th_i * C::TH, ow0 = tw_i * C::TW;
    const int ih0 = oh0 * C::S - a.pad, iw0 = ow0 * C::S - a.pad;
    const int c_begin = split * a.chunks_per_split;
    const int c_end = min(c_begin + a.chunks_per_split, a.nchunks);

    // Per-lane LDS bases of the two MFMA operands.
    const int a_base = (wc * 16 * C::MA + l16) * C::RS + g * C::KK;
    int b_base[C::NB];
#pragma unroll
    for (int nb = 0; nb < C::NB; ++nb) {
        int p = (wp * C::NB + nb) * 16 + l16;
        if (p >= C::NPIX) p = 0;  // padding lanes read a valid word; never stored
        b_base[nb] = g * C::PL + (p / C::TW) * C::S * C::HC + (p % C::TW) * C::S;
    }

    floatx4 acc[C::MA][C::NB];
#pragma unroll
    for (int m = 0; m < C::MA; ++m)
#pragma unroll
        for (int n = 0; n < C::NB; ++n) acc[m][n] = floatx4{0.f, 0.f, 0.f, 0.f};

    float xr[C::XPT], wr[C::WPT];
    if (c_begin < c_end) {
        load_stage<C>(x, w, a, c_begin * C::CC, ih0, iw0, co0, xr, wr);
        store_stage<C>(lds, xr, wr);
    }
    __syncthreads();

    for (int ch = c_begin; ch < c_end; ++ch) {
        const int it = ch - c_begin;
        const bool more = ch + 1 < c_end;
        if (more) load_stage<C>(x, w, a, (ch + 1) * C::CC, ih0, iw0, co0, xr, wr);

        const float *wl = lds + (it & 1) * C::BUF;
        const float *xl = wl + C::WSZ;
#pragma unroll
        for (int t = 0; t < C::KK; ++t) {
            const int kh = t / C::KS, kw = t % C::KS;
#pragma unroll
            for (int c4 = 0; c4 < C::CC / 4; ++c4) {
                float av[C::MA], bv[C::NB];
#pragma unroll
                for (int m = 0; m < C::MA; ++m) av[m] = wl[a_base + m * 16 * C::RS + c4 * 4 * C::KK + t];
#pragma unroll
                for (int n = 0; n < C::NB; ++n) bv[n] = xl[b_base[n] + c4 * 4 * C::PL + kh * C::HC + kw];
#pragma unroll
                for (int m = 0; m < C::MA; ++m)
#pragma unroll
                    for (int n = 0; n < C::NB; ++n)
                        acc[m][n] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[m], bv[n], acc[m][n], 0, 0, 0);
            }
        }
        if (more) store_stage<C>(lds + ((it + 1) & 1) * C::BUF, xr, wr);
        __syncthreads();
    }

    // Accumulator block (m, n), register r holds output channel
    // co0 + wc*16*MA + m*16 + 4*g + r at tile pixel (wp*NB + n)*16 + l16.
    if (a.splits == 1) {
#pragma unroll
        for (int m = 0; m < C::MA; ++m) {
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int co = co0 + wc * 16 * C::MA + m * 16 + 4 * g + r;
                const float b = (bias && co < a.c_out) ? bias[co] : 0.f;
#pragma unroll
                for (int n = 0; n < C::NB; ++n) {
                    const int p = (wp * C::NB + n) * 16 + l16;
                    const int oh = oh0 + p / C::TW, ow = ow0 + p % C::TW;
                    if (p < C::NPIX && co < a.c_out && oh < a.h_out && ow < a.w_out)
                        out[((size_t)co * a.h_out + oh) * a.w_out + ow] = acc[m][n][r] + b;
                }
            }
        }
        return;
    }

    // Split input channels: publish this partial tile, count arrivals.
    unsigned *counters = reinterpret_cast<unsigned *>(ws);
    float *part = ws + a.part_offset + (size_t)tile * a.splits * (C::COT * C::NPIXP);
    float *mine = part + (size_t)split * (C::COT * C::NPIXP);
#pragma unroll
    for (int m = 0; m < C::MA; ++m)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int col = wc * 16 * C::MA + m * 16 + 4 * g + r;
#pragma unroll
            for (int n = 0; n < C::NB; ++n)
                mine[col * C::NPIXP + (wp * C::NB + n) * 16 + l16] = acc[m][n][r];
        }
    __threadfence();
    __syncthreads();
    if (tid == 0) s_last = (atomicAdd(&counters[tile], 1u) == (unsigned)(a.splits - 1)) ? 1u : 0u;
    __syncthreads();
    if (!s_last) return;
    __threadfence();
    for (int e = tid; e < C::COT * C::NPIX; e += C::NT) {
        const int col = e / C::NPIX;
        const int p = e - col * C::NPIX;
        const int co = co0 + col;
        const int oh = oh0 + p / C::TW, ow = ow0 + p % C::TW;
        if (co < a.c_out && oh < a.h_out && ow < a.w_out) {
            float s = 0.f;
            for (int k = 0; k < a.splits; ++k) s += part[(size_t)k * (C::COT * C::NPIXP) + col * C::NPIXP + p];
            out[((size_t)co * a.h_out + oh) * a.w_out + ow] = s + (bias ? bias[co] : 0.f);
        }
    }
    if (tid == 0) counters[tile] = 0u;  // ready for the next call
}

struct Variant {
    const char *name;
    int ks, s, th, tw, nwc, nwp, ma, cc;
    int nt, npixp, cot, lds;
    void (*launch)(dim3 grid, hipStream_t st, const float *, const float *, const float *, float *, float *,
                   const IgArgs &);
};

template <class C>
void launch_cfg(dim3 grid, hipStream_t st, const float *x, const float *w, const float *b, float *o, float *ws,
                const IgArgs &a)
{
    hipLaunchKernelGGL(conv_igemm<C>, grid, dim3(C::NT), 0, st, x, w, b, o, ws, a);
}

template <class C>
constexpr Variant make_variant(const char *name)
{
    return Variant{name, C::KS, C::S, C::TH, C::TW, C::NWC, C::NWP, C::MA, C::CC,
                   C::NT, C::NPIXP, C::COT, C::LDS_BYTES, &launch_cfg<C>};
}

//                       KS S  TH  TW NWC NWP MA CC
using K3S1_T14_C64 = Cfg<3, 1, 14, 14, 4, 1, 1, 8>;
using K3S1_T7_C64 = Cfg<3, 1, 7, 7, 4, 1, 1, 8>;
using K3S1_T14_C128 = Cfg<3, 1, 14, 14, 4, 1, 2, 4>;
using K3S1_T8x32_C64 = Cfg<3, 1, 8, 32, 2, 2, 2, 4>;
using K3S2_T7_C64 = Cfg<3, 2, 7, 7, 4, 1, 1, 8>;
using K1S1_T7_C64 = Cfg<1, 1, 7, 7, 4, 1, 1, 16>;
using K1S1_T14_C64 = Cfg<1, 1, 14, 14, 4, 1, 1, 16>;
using K5S1_T7_C64 = Cfg<5, 1, 7, 7, 4, 1, 1, 4>;

const Variant kVariants[] = {
    make_variant<K3S1_T14_C64>("k3s1_t14x14_co64"),
    make_variant<K3S1_T7_C64>("k3s1_t7x7_co64"),
    make_variant<K3S1_T14_C128>("k3s1_t14x14_co128"),
    make_variant<K3S1_T8x32_C64>("k3s1_t8x32_co64"),
    make_variant<K3S2_T7_C64>("k3s2_t7x7_co64"),
    make_variant<K1S1_T7_C64>("k1s1_t7x7_co64"),
    make_variant<K1S1_T14_C64>("k1s1_t14x14_co64"),
    make_variant<K5S1_T7_C64>("k5s1_t7x7_co64"),
};
constexpr int kNumVariants = sizeof(kVariants) / sizeof(kVariants[0]);

constexpr int kCUs = 256;

size_t part_offset_floats() { return kCounterBytes / sizeof(float); }

}  // namespace

int igemm_num_variants() { return kNumVariants; }

bool igemm_variant_info(int v, int *k, int *stride, int *tile_h, int *tile_w, int *co_tile)
{
    if (v < 0 || v >= kNumVariants) return false;
    const Variant &d = kVariants[v];
    *k = d.ks;
    *stride = d.s;
    *tile_h = d.th;
    *tile_w = d.tw;
    *co_tile = d.cot;
    return true;
}

bool igemm_make_plan(const ConvShape &s, int variant, int splits, ilpm_plan *p)
{
    if (variant < 0 || variant >= kNumVariants) return false;
    const Variant &d = kVariants[variant];
    if (d.ks != s.k || d.s != s.stride) return false;
    const long tiles = (long)ceil_div(s.h_out, d.th) * ceil_div(s.w_out, d.tw) * ceil_div(s.c_out, d.cot);
    if (tiles > 0x7fffffffL) return false;
    const int nchunks = ceil_div(s.c_in, d.cc);
    if (splits <= 0) {
        // Enough workgroups to give every compute unit one, without splitting a
        // stage.
        splits = 1;
        if (tiles < kCUs) splits = (int)((kCUs + tiles - 1) / tiles);
        if (splits > nchunks) splits = nchunks;
    }
    if (splits > nchunks) return false;
    const int cps = ceil_div(nchunks, splits);
    splits = ceil_div(nchunks, cps);  // no empty split
    if (splits > 1 && tiles > kMaxTileCounters) return false;
    if (splits > 65535) return false;
    ilpm_plan q = {};
    q.path = ILPM_PATH_IGEMM;
    q.variant = variant;
    q.tile_h = d.th;
    q.tile_w = d.tw;
    q.co_tile = d.cot;
    q.ci_chunk = d.cc;
    q.splits = splits;
    q.grid = (int)tiles * splits;
    q.block = d.nt;
    q.lds_bytes = d.lds;
    q.h_out = s.h_out;
    q.w_out = s.w_out;
    q.workspace_bytes = splits > 1
                            ? kCounterBytes + sizeof(float) * (size_t)tiles * splits * d.cot * d.npixp
                            : 0;
    *p = q;
    return true;
}

double igemm_plan_cost(const ConvShape &s, const ilpm_plan &p)
{
    const Variant &d = kVariants[p.variant];
    const int nchunks = ceil_div(s.c_in, d.cc);
    const int cps = ceil_div(nchunks, p.splits);
    const int nb = d.npixp / (16 * d.nwp);
    // MFMA cycles of one wave for one stage: taps * channel groups * blocks * 32.
    const double stage = (double)d.ks * d.ks * (d.cc / 4) * d.ma * nb * 32.0;
    const double stage_overhead = 600.0;  // barrier, LDS stores, issue gaps
    double wg = cps * (stage + stage_overhead) + 3000.0;  // + first load and epilogue
    if (p.splits > 1) {
        // Partial tile out, and the reducer reads every partial back
        // (~13 bytes per cycle per compute unit of HBM bandwidth).
        const double bytes = 4.0 * d.cot * d.npixp;
        wg += bytes / 13.0 + bytes * p.splits / 13.0 / 2.0;
    }
    const long wgs = (long)p.grid;
    const double rounds = std::ceil((double)wgs / kCUs);
    return rounds * wg;
}

hipError_t igemm_launch(const ilpm_plan &p, const ConvShape &s, const float *x, const float *w,
                        const float *bias, float *out, void *workspace, hipStream_t stream)
{
    const Variant &d = kVariants[p.variant];
    IgArgs a;
    a.c_in = s.c_in;
    a.h = s.h;
    a.w = s.w;
    a.c_out = s.c_out;
    a.pad = s.pad;
    a.h_out = s.h_out;
    a.w_out = s.w_out;
    a.tiles_w = ceil_div(s.w_out, d.tw);
    a.co_tiles = ceil_div(s.c_out, d.cot);
    a.nchunks = ceil_div(s.c_in, d.cc);
    a.chunks_per_split = ceil_div(a.nchunks, p.splits);
    a.splits = p.splits;
    a.part_offset = part_offset_floats();
    const int tiles = p.grid / p.splits;
    d.launch(dim3(tiles, p.splits), stream, x, w, bias, out, static_cast<float *>(workspace), a);
    return hipGetLastError();
}

}  // namespace ilpm
