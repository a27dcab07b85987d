// Microbenchmarks of the MI355X ceilings the convolution is measured against:
// fp32 matrix-core throughput (v_mfma_f32_16x16x4_f32), fp32 vector FMA
// throughput, HBM copy bandwidth and the cost of an empty launch.  Built into
// bench_peaks.so next to bench.py; used only by `bench.py --peaks`.
#include <hip/hip_runtime.h>
#include <stdint.h>

typedef float floatx4 __attribute__((ext_vector_type(4)));

// Every wave keeps 16 independent 16x16 accumulators busy for `iters` rounds.
// clk[2*blockIdx.x] / clk[2*blockIdx.x+1]: shader-clock and 100 MHz wall-clock
// ticks over the loop, read by thread 0.
__global__ __launch_bounds__(256) void peak_mfma_f32(float *out, uint64_t *clk, int iters)
{
    floatx4 acc[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) acc[j] = floatx4{0.f, 0.f, 0.f, 0.f};
    const float a = 1e-3f * (float)(threadIdx.x & 7);
    const float b = 1.0f + 1e-3f * (float)(threadIdx.x >> 6);
    const uint64_t c0 = clock64();
    const uint64_t w0 = wall_clock64();
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < 16; ++j) acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[j], 0, 0, 0);
    }
    const uint64_t c1 = clock64();
    const uint64_t w1 = wall_clock64();
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
    out[(size_t)blockIdx.x * 256 + threadIdx.x] = s;
    if (threadIdx.x == 0) {
        clk[2 * blockIdx.x] = c1 - c0;
        clk[2 * blockIdx.x + 1] = w1 - w0;
    }
}

// 16 independent fp32 FMA chains per lane.
__global__ __launch_bounds__(256) void peak_valu_fma(float *out, int iters)
{
    float x[16];
#pragma unroll
    for (int j = 0; j < 16; ++j) x[j] = 1e-3f * (float)(threadIdx.x + j);
    for (int i = 0; i < iters; ++i) {
#pragma unroll
        for (int j = 0; j < 16; ++j) x[j] = fmaf(x[j], 0.9999f, 1e-4f);
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 16; ++j) s += x[j];
    out[(size_t)blockIdx.x * 256 + threadIdx.x] = s;
}

__global__ __launch_bounds__(256) void copy_f4(const float4 *__restrict__ src, float4 *__restrict__ dst, size_t n)
{
    size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    const size_t step = (size_t)gridDim.x * 256;
    for (; i < n; i += step) dst[i] = src[i];
}

// Store-only bandwidth: 16 bytes per lane, consecutive lanes consecutive.
__global__ __launch_bounds__(256) void fill_f4(float4 *__restrict__ dst, size_t n, float v)
{
    size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    const size_t step = (size_t)gridDim.x * 256;
    for (; i < n; i += step) dst[i] = float4{v, v, v, v};
}

// Store-only bandwidth with the layout of a 16x16 matrix-core result written
// to NCHW: each store instruction puts 4 bytes per lane, lanes 16g..16g+15 on
// 16 consecutive floats of row (plane) 4*blk + g, i.e. four 64-byte segments
// `plane` floats apart; a wave writes 16 rows x 16 floats per tile, 4
// instructions.  dst holds rows x plane floats, rows a multiple of 16 and
// plane of 16.
__global__ __launch_bounds__(256) void fill_tiles(float *__restrict__ dst, int rows, int plane, float v)
{
    const int lane = threadIdx.x & 63, g = lane >> 4, l = lane & 15;
    const int tiles_p = plane / 16, tiles = (rows / 16) * tiles_p;
    for (int t = blockIdx.x * 4 + (threadIdx.x >> 6); t < tiles; t += gridDim.x * 4) {
        const int rb = t / tiles_p, pb = t - rb * tiles_p;
        float *o = dst + (size_t)(16 * rb + 4 * g) * plane + 16 * pb + l;
#pragma unroll
        for (int r = 0; r < 4; ++r) o[(size_t)r * plane] = v;
    }
}

// fill_tiles with a cache policy on every store (buffer store, policy bits
// as the store instruction takes them: 2 non-temporal, 16 SC1, 17 SC0+SC1).
template <int POL>
__global__ __launch_bounds__(256) void fill_tiles_pol(float *__restrict__ dst, int rows, int plane, float v)
{
    const int lane = threadIdx.x & 63, g = lane >> 4, l = lane & 15;
    const int tiles_p = plane / 16, tiles = (rows / 16) * tiles_p;
    const __amdgpu_buffer_rsrc_t ro =
        __builtin_amdgcn_make_buffer_rsrc(dst, (short)0, rows * plane * 4, 0x00020000);
    for (int t = blockIdx.x * 4 + (threadIdx.x >> 6); t < tiles; t += gridDim.x * 4) {
        const int rb = t / tiles_p, pb = t - rb * tiles_p;
        const int o = (16 * rb + 4 * g) * plane + 16 * pb + l;
#pragma unroll
        for (int r = 0; r < 4; ++r)
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(unsigned, v), ro, (o + r * plane) * 4, 0, POL);
    }
}

// LDS bank probe: one 64-thread workgroup reads LDS `iters` times, each lane
// at its own word address table[lane] (WIDTH dwords per lane: ds_read_b32,
// b64 or b128), so that SQ_LDS_BANK_CONFLICT / SQ_INSTS_LDS of the dispatch
// give the cost of that address pattern.  Addresses lie in [0, 16384 - WIDTH].
template <int WIDTH>
__global__ __launch_bounds__(64) void lds_probe(const int *__restrict__ table, float *__restrict__ out, int iters)
{
    __shared__ __attribute__((aligned(16))) float buf[16384];
    for (int i = threadIdx.x; i < 16384; i += 64) buf[i] = (float)i;
    __syncthreads();
    const unsigned addr = (unsigned)table[threadIdx.x] * 4u;
    float s = 0.f;
    for (int it = 0; it < iters; ++it) {
        if constexpr (WIDTH == 1) {
            float v;
            asm volatile("ds_read_b32 %0, %1\n s_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(addr) : "memory");
            s += v;
        } else if constexpr (WIDTH == 2) {
            float2 v;
            asm volatile("ds_read_b64 %0, %1\n s_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(addr) : "memory");
            s += v.x + v.y;
        } else {
            float4 v;
            asm volatile("ds_read_b128 %0, %1\n s_waitcnt lgkmcnt(0)" : "=v"(v) : "v"(addr) : "memory");
            s += v.x + v.y + v.z + v.w;
        }
    }
    out[threadIdx.x] = s;
}

__global__ void empty_kernel() {}

extern "C" {

int peak_mfma_launch(float *out, uint64_t *clk, int iters, int grid, hipStream_t s)
{
    hipLaunchKernelGGL(peak_mfma_f32, dim3(grid), dim3(256), 0, s, out, clk, iters);
    return (int)hipGetLastError();
}

int peak_valu_launch(float *out, int iters, int grid, hipStream_t s)
{
    hipLaunchKernelGGL(peak_valu_fma, dim3(grid), dim3(256), 0, s, out, iters);
    return (int)hipGetLastError();
}

// n16: number of 16-byte elements; src and dst 16-byte aligned, not overlapping.
int copy_launch(const void *src, void *dst, size_t n16, int grid, hipStream_t s)
{
    hipLaunchKernelGGL(copy_f4, dim3(grid), dim3(256), 0, s, (const float4 *)src, (float4 *)dst, n16);
    return (int)hipGetLastError();
}

// n16: number of 16-byte elements of dst (16-byte aligned).
int fill_launch(void *dst, size_t n16, int grid, hipStream_t s)
{
    hipLaunchKernelGGL(fill_f4, dim3(grid), dim3(256), 0, s, (float4 *)dst, n16, 1.0f);
    return (int)hipGetLastError();
}

// dst: rows x plane floats, rows and plane multiples of 16.
int fill_tiles_launch(void *dst, int rows, int plane, int grid, hipStream_t s)
{
    if (rows % 16 || plane % 16) return -1;
    hipLaunchKernelGGL(fill_tiles, dim3(grid), dim3(256), 0, s, (float *)dst, rows, plane, 1.0f);
    return (int)hipGetLastError();
}

// The same with store cache policy pol in {0, 2, 16, 17}; rows * plane * 4 < 2^31.
int fill_tiles_pol_launch(void *dst, int rows, int plane, int grid, int pol, hipStream_t s)
{
    if (rows % 16 || plane % 16 || (long long)rows * plane * 4 >= (1LL << 31)) return -1;
    float *d = (float *)dst;
    switch (pol) {
    case 0: hipLaunchKernelGGL(fill_tiles_pol<0>, dim3(grid), dim3(256), 0, s, d, rows, plane, 1.0f); break;
    case 2: hipLaunchKernelGGL(fill_tiles_pol<2>, dim3(grid), dim3(256), 0, s, d, rows, plane, 1.0f); break;
    case 16: hipLaunchKernelGGL(fill_tiles_pol<16>, dim3(grid), dim3(256), 0, s, d, rows, plane, 1.0f); break;
    case 17: hipLaunchKernelGGL(fill_tiles_pol<17>, dim3(grid), dim3(256), 0, s, d, rows, plane, 1.0f); break;
    default: return -1;
    }
    return (int)hipGetLastError();
}

// table: 64 word addresses in [0, 16384 - width], multiples of width; width 1, 2 or 4.
int lds_probe_launch(const int *table, float *out, int iters, int width, hipStream_t s)
{
    if (width == 1) hipLaunchKernelGGL(lds_probe<1>, dim3(1), dim3(64), 0, s, table, out, iters);
    else if (width == 2) hipLaunchKernelGGL(lds_probe<2>, dim3(1), dim3(64), 0, s, table, out, iters);
    else if (width == 4) hipLaunchKernelGGL(lds_probe<4>, dim3(1), dim3(64), 0, s, table, out, iters);
    else return -1;
    return (int)hipGetLastError();
}

int empty_launch(hipStream_t s)
{
    hipLaunchKernelGGL(empty_kernel, dim3(1), dim3(64), 0, s);
    return (int)hipGetLastError();
}

}  // extern "C"
