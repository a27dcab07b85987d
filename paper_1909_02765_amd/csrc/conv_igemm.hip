// Host side of the matrix-core (implicit-GEMM) family: the variant table,
// plans and their cost model, launches, and the kernels that sum split
// partial outputs and pack weights.  The kernel templates and the algorithm's
// description are in conv_igemm.h.
#include <atomic>
#include <vector>

#include "conv_igemm.h"

namespace ilpm {
namespace {

// out[i] = part[0][i] + part[1][i] + ... + part[splits-1][i] (then max(., 0)
// with relu), summed in that order; split 0's partial sums carry the bias.  Each thread owns V
// consecutive outputs (V = 4 when every split slice is 16-byte aligned) and
// issues the loads of up to kBatch slices before it adds any of them, so the
// latency of the partial sums (just written by the conv kernel, mostly still
// in the last-level cache) is paid once per batch rather than once per slice.
template <int V>
struct VecF;
template <>
struct VecF<1> {
    using T = float;
};
template <>
struct VecF<4> {
    using T = float4;
};

constexpr int kBatch = 16;

// Sum of the `splits` slices at element i of a T-typed view, in slice order.
template <class T>
__device__ __forceinline__ T sum_slices(const T *pv, int64_t stride, int64_t i, int splits)
{
    T s = pv[i];
    int k = 1;
    for (; k + kBatch <= splits; k += kBatch) {
        T v[kBatch];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) v[j] = pv[(size_t)(k + j) * stride + i];
#pragma unroll
        for (int j = 0; j < kBatch; ++j) s += v[j];
    }
    T v[kBatch];
#pragma unroll
    for (int j = 0; j < kBatch; ++j)
        if (k + j < splits) v[j] = pv[(size_t)(k + j) * stride + i];
#pragma unroll
    for (int j = 0; j < kBatch; ++j)
        if (k + j < splits) s += v[j];
    return s;
}

template <int V>
__global__ __launch_bounds__(128) void sum_splits(const float *__restrict__ part, float *__restrict__ out,
                                                  int splits, int64_t total, int relu)
{
    using T = typename VecF<V>::T;
    const int64_t nvec = total / V;
    const T *pv = reinterpret_cast<const T *>(part);
    const int64_t step = (int64_t)gridDim.x * 128;
    // Stores at device scope (the output is below 2^30 bytes).
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(out, (unsigned)total * 4u);
    for (int64_t i = (int64_t)blockIdx.x * 128 + threadIdx.x; i < nvec; i += step) {
        const T s = sum_slices<T>(pv, nvec, i, splits);
        const float *sv = reinterpret_cast<const float *>(&s);
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const float v = sv[e];
            const float r = relu && v < 0.f ? 0.f : v;
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, r), ro, (int)((i * V + e) * 4), 0,
                                                  kPolicyDeviceScope);
        }
    }
}

// The same sum for the four outputs of each 2x2 window, their maximum, then
// ReLU: out [c][h_out/2][w_out/2].  One thread per pooled output; its index
// is split into (channel, row, column) by multiply-and-shift division (a
// 64-bit divide is a long instruction sequence on the GPU, and three per
// output made this kernel compute-bound).  With an even w_out each window row
// is one aligned 8-byte pair (V2).  The values are those of the plain sum
// and maximum, in the same order.
template <bool V2>
__global__ __launch_bounds__(256) void sum_splits_pool(const float *__restrict__ part, float *__restrict__ out,
                                                       int splits, int c, int h_out, int w_out, FastDiv wp_d,
                                                       FastDiv hp_d, int relu)
{
    const unsigned hp = (unsigned)h_out / 2, wp = (unsigned)w_out / 2;
    const unsigned total = (unsigned)c * hp * wp;
    const int64_t slice = (int64_t)c * h_out * w_out;
    const unsigned step = gridDim.x * 256u;
    const __amdgpu_buffer_rsrc_t ro = make_rsrc(out, total * 4u);  // stores at device scope
    for (unsigned i = blockIdx.x * 256u + threadIdx.x; i < total; i += step) {
        const unsigned t = fast_div(i, wp_d);
        const unsigned j = i - t * wp;
        const unsigned ch = fast_div(t, hp_d);
        const unsigned r = t - ch * hp;
        const int64_t base = ((int64_t)ch * h_out + 2 * r) * w_out + 2 * j;
        float m, v;
        if constexpr (V2) {
            const float2 *p2 = reinterpret_cast<const float2 *>(part);
            const float2 top = sum_slices<float2>(p2, slice / 2, base / 2, splits);
            const float2 bot = sum_slices<float2>(p2, slice / 2, (base + w_out) / 2, splits);
            m = top.x;
            v = top.y;
            m = v > m ? v : m;
            v = bot.x;
            m = v > m ? v : m;
            v = bot.y;
            m = v > m ? v : m;
        } else {
            m = sum_slices<float>(part, slice, base, splits);
            v = sum_slices<float>(part, slice, base + 1, splits);
            m = v > m ? v : m;
            v = sum_slices<float>(part, slice, base + w_out, splits);
            m = v > m ? v : m;
            v = sum_slices<float>(part, slice, base + w_out + 1, splits);
            m = v > m ? v : m;
        }
        const float res = relu && m < 0.f ? 0.f : m;
        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, res), ro, (int)(i * 4u), 0,
                                              kPolicyDeviceScope);
    }
}

// The prepacked weight layout of a variant (see PackedWeights), one thread
// per packed float; channels past C_out or C_in become zeros.
struct PackGeom {
    int c_in, c_out, kk, cot, cc, nwc, nwk, ma, g4, nchunks;
    int c1;  // consecutive channels per lane (Cfg::C1)
};

__global__ __launch_bounds__(256) void pack_weights(const float *__restrict__ w, float *__restrict__ packed,
                                                    PackGeom g, int64_t total)
{
    const int epl = g.ma * g.g4 * g.kk;
    const int n4 = epl / 4;
    const int64_t step = (int64_t)gridDim.x * 256;
    for (int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x; idx < total; idx += step) {
        const int64_t block = idx / (64 * epl);
        const int within = (int)(idx - block * (64 * epl));
        int lane, e;
        if (within < n4 * 256) {
            lane = (within % 256) / 4;
            e = 4 * (within / 256) + within % 4;
        } else {
            const int r = within - n4 * 256;
            lane = r % 64;
            e = 4 * n4 + r / 64;
        }
        const int wc = (int)(block % g.nwc);
        const int64_t b1 = block / g.nwc;
        const int wk = (int)(b1 % g.nwk);
        const int64_t b2 = b1 / g.nwk;
        const int chunk = (int)(b2 % g.nchunks);
        const int co_t = (int)(b2 / g.nchunks);
        const int m = e / (g.g4 * g.kk), c4 = (e / g.kk) % g.g4, tap = e % g.kk;
        const int co = co_t * g.cot + wc * 16 * g.ma + 16 * m + (lane & 15);
        const int ci = g.c1 ? chunk * g.cc + g.g4 * (4 * wk + (lane >> 4)) + c4
                            : chunk * g.cc + 4 * wk + (lane >> 4) + 4 * g.nwk * c4;
        packed[idx] = (co < g.c_out && ci < g.c_in) ? w[((int64_t)co * g.c_in + ci) * g.kk + tap] : 0.f;
    }
}

// The whole variant table, its parts in order, assembled on first use.
const std::vector<const Variant *> &variant_table()
{
    static const std::vector<const Variant *> table = [] {
        int (*const parts[])(const Variant **) = {ig::variants_part0, ig::variants_part1, ig::variants_part2,
                                                  ig::variants_part3, ig::variants_part4, ig::variants_part5,
                                                  ig::variants_part6, ig::variants_part7, ig::variants_part8,
                                                  ig::variants_part9, ig::variants_part10};
        std::vector<const Variant *> t;
        for (auto part : parts) {
            const Variant *v = nullptr;
            const int n = part(&v);
            for (int i = 0; i < n; ++i) t.push_back(v + i);
        }
        return t;
    }();
    return table;
}

const Variant &variant_at(int v) { return *variant_table()[v]; }
int num_variants() { return (int)variant_table().size(); }

constexpr int kCUs = 256;

}  // namespace

int igemm_num_variants() { return num_variants(); }

const char *igemm_variant_name(int v) { return (v >= 0 && v < num_variants()) ? variant_at(v).name : nullptr; }

bool igemm_variant_info(int v, int *k, int *stride, int *tile_h, int *tile_w, int *co_tile)
{
    if (v < 0 || v >= num_variants()) return false;
    const Variant &d = variant_at(v);
    *k = d.ks;
    *stride = d.s;
    *tile_h = d.th;
    *tile_w = d.tw;
    *co_tile = d.cot;
    return true;
}

bool igemm_variant_pipeline(int v, int *ci_chunk, int *stages, int *buffers, int *flags)
{
    if (v < 0 || v >= num_variants()) return false;
    const Variant &d = variant_at(v);
    *ci_chunk = d.cc;
    *stages = d.stages;
    *buffers = d.nbuf;
    *flags = (d.wl ? ILPM_VARIANT_WEIGHTS_LDS : 0) | (d.pf ? ILPM_VARIANT_PROGRESSIVE_FIRST : 0) |
             (d.c1 ? ILPM_VARIANT_CONSECUTIVE_CHANNELS : 0);
    return true;
}

bool igemm_make_plan(const ConvShape &s, int variant, int splits, ilpm_plan *p)
{
    if (variant < 0 || variant >= num_variants()) return false;
    const Variant &d = variant_at(variant);
    if (d.ks != s.k || d.s != s.stride) return false;
    // Consecutive channels per lane: 16-byte weight loads that stay inside
    // the tensor only when C_in is a multiple of 4.
    if (d.c1 && s.c_in % 4 != 0) return false;
    // Load offsets are 31-bit byte offsets.
    if ((int64_t)s.c_in * s.h * s.w * 4 >= (1LL << 31)) return false;
    if ((int64_t)s.c_out * s.c_in * s.k * s.k * 4 >= (1LL << 31)) return false;
    if ((int64_t)s.c_out * s.h_out * s.w_out * 4 >= (1LL << 30)) return false;
    // ... and so are those of the prepacked weights (padded to whole tiles).
    if ((int64_t)ceil_div(s.c_out, d.cot) * d.cot * ceil_div(s.c_in, d.cc) * d.cc * s.k * s.k * 4 >= (1LL << 31))
        return false;
    // Spatial sizes below 2^23: the kernel's 24-bit multiplies are exact.
    if (s.h >= (1 << 23) || s.w >= (1 << 23) || s.h_out >= (1 << 23) || s.w_out >= (1 << 23)) return false;
    // A stage's channels (up to CC, past C_in too) stay within 31-bit offsets.
    if ((int64_t)(s.c_in > d.cc ? s.c_in : d.cc) * s.h * s.w * 4 >= (1LL << 31)) return false;
    const long tiles = (long)ceil_div(s.h_out, d.th) * ceil_div(s.w_out, d.tw) * ceil_div(s.c_out, d.cot);
    if (tiles > 0x7fffffffL) return false;
    const int nchunks = ceil_div(s.c_in, d.cc);
    if (splits <= 0) {
        // Enough workgroups to give every compute unit one.
        splits = 1;
        if (tiles < kCUs) splits = (int)((kCUs + tiles - 1) / tiles);
        if (splits > nchunks) splits = nchunks;
        if (d.stages > 0) splits = nchunks / d.stages;
        if (d.pf) splits = splits < nchunks / 2 ? splits : (nchunks / 2 > 0 ? nchunks / 2 : 1);
    }
    // A fixed-stage variant covers the input channels in whole splits of
    // exactly its stage count.
    if (d.stages > 0 && (nchunks % d.stages != 0 || splits * d.stages != nchunks)) return false;
    if (splits > nchunks) return false;
    const int cps = ceil_div(nchunks, splits);
    splits = ceil_div(nchunks, cps);  // no empty split
    // A progressive first stage is followed by at least one more.
    if (d.pf && (cps < 2 || nchunks - (splits - 1) * cps < 2)) return false;
    if (splits > 65535) return false;
    if ((int64_t)tiles * splits > 0x7fffffffL) return false;  // workgroup indices are divided as 31-bit values
    const size_t out_elems = (size_t)s.c_out * s.h_out * s.w_out;
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
    q.workspace_bytes = splits > 1 ? sizeof(float) * out_elems * splits : 0;
    *p = q;
    return true;
}

double igemm_plan_cost(const ConvShape &s, const ilpm_plan &p)
{
    const Variant &d = variant_at(p.variant);
    const int nchunks = ceil_div(s.c_in, d.cc);
    const int cps = ceil_div(nchunks, p.splits);
    const int nb = ceil_div(d.th * d.tw, 16 * d.nwp);
    // MFMA cycles of one SIMD for one stage: a workgroup's waves share the
    // compute unit's four SIMDs.
    const int waves = d.nwc * d.nwp * d.nwk;
    const double stage_wave = (double)d.ks * d.ks * (d.cc / 4 / d.nwk) * d.ma * nb * 32.0;
    const double stage_simd = stage_wave * waves / 4.0;
    const double stage_overhead = 700.0;
    double wg = cps * (stage_simd + stage_overhead) + 6000.0;
    if (d.nwk > 1) wg += 1500.0;
    const double rounds = std::ceil((double)p.grid / kCUs);
    double cycles = rounds * wg;
    if (p.splits > 1) {
        // Partial sums out and back in (~10 bytes per cycle per compute unit),
        // plus the second launch.
        const double bytes = 4.0 * s.c_out * s.h_out * s.w_out * (2.0 * p.splits + 1.0);
        cycles += bytes / (10.0 * kCUs) + 4000.0;
    }
    return cycles;
}

int64_t igemm_packed_floats(const ilpm_plan &p, int c_in, int c_out)
{
    const Variant &d = variant_at(p.variant);
    if (d.wl) return (int64_t)c_out * c_in * d.ks * d.ks;
    return (int64_t)ceil_div(c_out, d.cot) * ceil_div(c_in, d.cc) * d.cot * d.cc * d.ks * d.ks;
}

hipError_t igemm_pack(const ilpm_plan &p, int c_in, int c_out, const float *w, float *packed, hipStream_t stream)
{
    const Variant &d = variant_at(p.variant);
    if (d.wl)
        return hipMemcpyAsync(packed, w, sizeof(float) * (size_t)igemm_packed_floats(p, c_in, c_out),
                              hipMemcpyDeviceToDevice, stream);
    PackGeom g;
    g.c_in = c_in;
    g.c_out = c_out;
    g.kk = d.ks * d.ks;
    g.cot = d.cot;
    g.cc = d.cc;
    g.nwc = d.nwc;
    g.nwk = d.nwk;
    g.ma = d.ma;
    g.g4 = d.cc / 4 / d.nwk;
    g.nchunks = ceil_div(c_in, d.cc);
    g.c1 = d.c1 ? 1 : 0;
    const int64_t total = igemm_packed_floats(p, c_in, c_out);
    int64_t blocks = (total + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    hipLaunchKernelGGL(pack_weights, dim3((unsigned)blocks), dim3(256), 0, stream, w, packed, g, total);
    return hipGetLastError();
}

namespace {
std::atomic<int> g_split_sum_mode{ILPM_SPLIT_SUM_FUSED};
}

bool igemm_set_split_sum(int mode)
{
    if (mode != ILPM_SPLIT_SUM_FUSED && mode != ILPM_SPLIT_SUM_KERNEL) return false;
    g_split_sum_mode.store(mode, std::memory_order_relaxed);
    return true;
}

size_t igemm_workspace_bytes(const ilpm_plan &p, const ConvShape &s, int epilogue)
{
    const bool to_part = p.splits > 1 || (epilogue & ILPM_EPI_MAXPOOL2);
    return to_part ? sizeof(float) * (size_t)s.c_out * s.h_out * s.w_out * p.splits : 0;
}

hipError_t igemm_launch(const ilpm_plan &p, const ConvShape &s, const float *x, const float *w,
                        const float *bias, float *out, void *workspace, hipStream_t stream, bool packed,
                        int epilogue)
{
    const Variant &d = variant_at(p.variant);
    const bool pool = (epilogue & ILPM_EPI_MAXPOOL2) != 0;
    const bool relu = (epilogue & ILPM_EPI_RELU) != 0;
    IgArgs a;
    a.c_in = s.c_in;
    a.h = s.h;
    a.w = s.w;
    a.c_out = s.c_out;
    a.pad = s.pad;
    a.h_out = s.h_out;
    a.w_out = s.w_out;
    a.nchunks = ceil_div(s.c_in, d.cc);
    a.chunks_per_split = ceil_div(a.nchunks, p.splits);
    a.ntiles = make_fastdiv((unsigned)(p.grid / p.splits));
    a.co_tiles = make_fastdiv((unsigned)ceil_div(s.c_out, d.cot));
    a.tiles_w = make_fastdiv((unsigned)ceil_div(s.w_out, d.tw));
    a.sp_tiles = make_fastdiv((unsigned)(ceil_div(s.h_out, d.th) * ceil_div(s.w_out, d.tw)));
    // Each XCD runs a contiguous run of workgroups.  When the weights
    // outweigh the input, let the run share output-channel tiles (and so
    // weights) across spatial tiles; otherwise share spatial tiles (input).
    a.sp_fast = (int64_t)s.c_out * s.c_in * s.k * s.k > (int64_t)s.c_in * s.h * s.w ? 1 : 0;
    // A pooled epilogue of a one-split plan is done in the workgroup when the
    // variant allows it; otherwise the conv writes its full-size sums to the
    // workspace and sum_splits_pool pools them.
    a.pool_tile = (pool && p.splits == 1 && d.poolable) ? 1 : 0;
    a.to_part = (p.splits > 1 || (pool && !a.pool_tile)) ? 1 : 0;
    a.relu = relu ? 1 : 0;
    const int tiles = p.grid / p.splits;
    a.splits = p.splits;
    a.fuse = (p.splits > 1 && !pool && tiles <= kMaxFusedTiles &&
              ceil_div(d.cot * d.th * d.tw, d.nt) * p.splits <= kFuseMaxLoads &&
              g_split_sum_mode.load(std::memory_order_relaxed) == ILPM_SPLIT_SUM_FUSED)
                 ? 1
                 : 0;
    float *part = static_cast<float *>(workspace);
    d.launch(dim3(tiles * p.splits), stream, x, w, bias, out, part, a, packed);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess || !a.to_part || a.fuse) return e;
    if (pool) {
        // Pooled outputs number fewer than the output's, which are below 2^31.
        const int64_t total = (int64_t)s.c_out * (s.h_out / 2) * (s.w_out / 2);
        int64_t blocks = (total + 255) / 256;
        if (blocks > 8192) blocks = 8192;
        const FastDiv wp_d = make_fastdiv((unsigned)(s.w_out / 2)), hp_d = make_fastdiv((unsigned)(s.h_out / 2));
        if (s.w_out % 2 == 0)
            hipLaunchKernelGGL(sum_splits_pool<true>, dim3((unsigned)blocks), dim3(256), 0, stream, part, out, p.splits,
                               s.c_out, s.h_out, s.w_out, wp_d, hp_d, a.relu);
        else
            hipLaunchKernelGGL(sum_splits_pool<false>, dim3((unsigned)blocks), dim3(256), 0, stream, part, out,
                               p.splits, s.c_out, s.h_out, s.w_out, wp_d, hp_d, a.relu);
        return hipGetLastError();
    }
    const int64_t total = (int64_t)s.c_out * s.h_out * s.w_out;
    const bool vec4 = total % 4 == 0;
    const int64_t threads = vec4 ? total / 4 : total;
    int64_t blocks = (threads + 127) / 128;
    if (blocks > 8192) blocks = 8192;
    if (vec4)
        hipLaunchKernelGGL(sum_splits<4>, dim3((unsigned)blocks), dim3(128), 0, stream, part, out, p.splits, total,
                           a.relu);
    else
        hipLaunchKernelGGL(sum_splits<1>, dim3((unsigned)blocks), dim3(128), 0, stream, part, out, p.splits, total,
                           a.relu);
    return hipGetLastError();
}

}  // namespace ilpm
