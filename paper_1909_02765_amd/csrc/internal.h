// Internal interfaces between the C-ABI layer (ilpm_api.hip) and the kernel
// families (conv_direct.hip, conv_igemm.hip, stack_ops.hip).
#pragma once

#include <hip/hip_runtime.h>

#include "ilpm.h"

namespace ilpm {

// One convolution call's geometry; h_out/w_out follow the output-size formula
// in ilpm.h.
struct ConvShape {
    int c_in, h, w, c_out, k, stride, pad, h_out, w_out;
};

// ---- direct (VALU) family ----
int direct_num_variants();
bool direct_variant_info(int v, int *k, int *stride, int *tile_h, int *tile_w, int *co_tile);
const char *direct_variant_name(int v);
bool direct_make_plan(const ConvShape &s, int variant, ilpm_plan *p);
// The low-channel matrix-core variants (the whole C_in*K*K contraction in one
// chain of matrix instructions) and the largest C_in*K*K each takes.
bool direct_is_lowc(int v);
int direct_lowc_max_kt(int v);
// relu: store max(conv + bias, 0).
hipError_t direct_launch(const ilpm_plan &p, const ConvShape &s, const float *x, const float *w,
                         const float *bias, float *out, hipStream_t stream, bool relu);

// ---- implicit-GEMM (fp32 MFMA) family ----
int igemm_num_variants();
bool igemm_variant_info(int v, int *k, int *stride, int *tile_h, int *tile_w, int *co_tile);
bool igemm_variant_pipeline(int v, int *ci_chunk, int *stages, int *buffers, int *flags);
const char *igemm_variant_name(int v);
// splits = 0 lets the family choose.
bool igemm_make_plan(const ConvShape &s, int variant, int splits, ilpm_plan *p);
// Modelled cost of a plan in SIMD cycles of the slowest compute unit, used to
// rank variants; lower is better.
double igemm_plan_cost(const ConvShape &s, const ilpm_plan &p);
// packed: w is in the variant's prepacked layout (igemm_pack) instead of OIHW.
// epilogue: ILPM_EPI_* bits.  With ILPM_EPI_MAXPOOL2, out is the pooled
// [C_out][H_out/2][W_out/2] tensor and the workspace holds every split's
// full-size partial sums (igemm_workspace_bytes).
hipError_t igemm_launch(const ilpm_plan &p, const ConvShape &s, const float *x, const float *w,
                        const float *bias, float *out, void *workspace, hipStream_t stream, bool packed,
                        int epilogue);
size_t igemm_workspace_bytes(const ilpm_plan &p, const ConvShape &s, int epilogue);
// ILPM_SPLIT_SUM_* for every later igemm_launch; false for another value.
bool igemm_set_split_sum(int mode);
// Floats of the prepacked weights of a variant for C_in, C_out (zero-padded
// to whole output-channel tiles and input-channel chunks).
int64_t igemm_packed_floats(const ilpm_plan &p, int c_in, int c_out);
hipError_t igemm_pack(const ilpm_plan &p, int c_in, int c_out, const float *w, float *packed, hipStream_t stream);

// ---- Winograd F(2x2, 3x3) comparison path (3x3, stride 1) ----
int64_t winograd_tiles(const ConvShape &s);
// V and M of the transformed problem (the filter transform U is the caller's).
size_t winograd_workspace_bytes(const ConvShape &s);
hipError_t winograd_filter_launch(const float *w, int c_in, int c_out, float *u, hipStream_t stream);
int winograd_launch(const ConvShape &s, const float *x, const float *u, const float *bias, float *out,
                    void *workspace, int dev, hipStream_t stream, hipError_t *err);

// ---- measured plan tables (tuned_plans*.inc) ----
// The plan the offline sweep found fastest for this exact shape, weight
// layout and epilogue (pooled: ReLU + 2x2 max-pool), if any.
bool tuned_plan(const ConvShape &s, ilpm_plan *p, bool prepacked, bool pooled);

// ---- helpers ----
hipError_t launch_relu(float *x, int64_t n, hipStream_t stream);
hipError_t launch_maxpool2x2(const float *in, int c, int h, int w, float *out, hipStream_t stream, bool relu);

inline int ceil_div(int a, int b) { return (a + b - 1) / b; }

}  // namespace ilpm
