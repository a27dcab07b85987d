/*
 * ilpm.h -- batch-1 2-D convolution forward pass on AMD MI355X (gfx950).
 *
 * The operation (ILP-M, Section 4 and Algorithm 2 of "ILP-M Conv: Optimize
 * Convolution Algorithm for Single-Image Convolution Neural Network Inference
 * on Mobile GPUs"): every output pixel of every output channel accumulates,
 * over all input channels and all K x K filter taps (r, s), the filter weight
 * times the input pixel at (y + r, x + s) -- a cross-correlation, no filter
 * flip.  The paper's algorithm is stride 1 with an implicit halo; this library
 * adds the standard stride s, symmetric zero padding p and an optional
 * per-output-channel bias:
 *
 *   H_out = floor((H + 2p - K) / s) + 1,  W_out = floor((W + 2p - K) / s) + 1
 *   out[co][oh][ow] = bias[co]
 *       + sum_{ci<C_in, kh<K, kw<K} w[co][ci][kh][kw] * x[ci][oh*s - p + kh][ow*s - p + kw]
 *   (x read as 0 outside [0,H) x [0,W)).
 *
 * Arithmetic is fp32 in, fp32 accumulate (fp32 FMA or fp32 MFMA), fp32 out.
 * The summation order is not the definition's; results agree with the exact
 * sum to within 1e-4 * (1 + S / (C_in*K*K)), S = sum of |products|.
 *
 * Conventions for every entry point:
 *   - Tensor pointers are DEVICE pointers to contiguous fp32 arrays, 4-byte
 *     aligned, on the current HIP device.  The caller owns (allocates and
 *     frees) them; the library keeps no tensor pointer after a call returns.
 *   - Work is only enqueued on `stream` (NULL = the default stream); no call
 *     synchronises the host.  A device-side fault shows up at the caller's
 *     next synchronisation.  The one exception to "only enqueued" is the
 *     library-owned workspace (see ilpm_conv2d_fwd): the first call that
 *     needs a larger one allocates it with hipMalloc.
 *   - Arguments are checked before anything is launched; on an error the
 *     call returns a negative status and writes nothing.
 *   - K in this library is the filter size; output channels are C_out.  (The
 *     paper's Algorithm 2 uses K for the output channels.)
 */
#ifndef ILPM_H
#define ILPM_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
enum {
    ILPM_OK = 0,
    ILPM_ERR_INVALID_ARG = -1, /* null pointer, dimension <= 0, stride <= 0, pad < 0,
                                  no output pixel, out overlapping an input, bad plan */
    ILPM_ERR_UNSUPPORTED = -2, /* a tensor above 2^31-1 elements */
    ILPM_ERR_WORKSPACE = -3,   /* registered workspace smaller than the plan needs, or the
                                  library's own would have to grow during graph capture */
    ILPM_ERR_HIP = -4,         /* a HIP runtime call or kernel launch failed */
    ILPM_ERR_ARCH = -5         /* the current device is not gfx950 */
};

/* Kernel families. */
enum {
    ILPM_PATH_DIRECT = 0, /* VALU direct convolution: lanes on output pixels, a
                             block of output channels per thread, taps outermost */
    ILPM_PATH_IGEMM = 1   /* fp32-MFMA implicit GEMM: M = C_out, N = output pixels,
                             K = C_in*K*K, input halo tiles staged in LDS */
};

/* How one call is executed (see ilpm_conv2d_plan). */
typedef struct ilpm_plan {
    int path;              /* ILPM_PATH_* */
    int variant;           /* compiled kernel variant within the path */
    int tile_h, tile_w;    /* output pixels per workgroup */
    int co_tile;           /* output channels per workgroup */
    int ci_chunk;          /* input channels staged in LDS per stage */
    int splits;            /* input-channel splits across workgroups (1 = none) */
    int grid;              /* workgroups launched */
    int block;             /* threads per workgroup */
    int lds_bytes;         /* LDS per workgroup */
    int h_out, w_out;      /* output size */
    size_t workspace_bytes;/* device workspace the plan needs (0 if none) */
} ilpm_plan;

/*
 * ilpm_conv2d_fwd -- out = conv2d(in, w) + bias, batch 1.
 *   in   [1, C_in, H, W]            NCHW, read only
 *   w    [C_out, C_in, K, K]        OIHW, read only
 *   bias [C_out] or NULL (no bias)  read only
 *   out  [1, C_out, H_out, W_out]   NCHW, fully written; must not overlap the inputs
 *   stride >= 1, pad >= 0, all sizes >= 1, H_out >= 1 and W_out >= 1.
 * Picks the kernel with ilpm_conv2d_plan.  Plans with splits > 1 write
 * per-split partial outputs to the device workspace; the last workgroup of
 * each output tile sums them in split order (or a second kernel on the same
 * stream does, see ilpm_set_split_sum).  Such plans also use a per-device
 * array of tile arrival counts that the library holds; calls that overlap in
 * time on one device and both use split plans must be ordered on one stream.
 * Workspace: the one registered with ilpm_set_workspace (ILPM_ERR_WORKSPACE
 * if it is too small), else the library's own for the current device.  A
 * call that needs more than the library's own holds allocates a larger one
 * (hipMalloc: no synchronisation, no free -- the smaller buffer is kept
 * until the process ends, because work already enqueued or a HIP graph
 * captured earlier may still use it).  While `stream` is being captured
 * into a graph nothing can be allocated, and such a call returns
 * ILPM_ERR_WORKSPACE instead: size the workspace before capturing (one
 * uncaptured call of the same shape, or ilpm_set_workspace).
 * Returns ILPM_OK or a negative status.
 */
int ilpm_conv2d_fwd(const float *in, const float *w, const float *bias,
                    int C_in, int H, int W, int C_out, int K, int stride, int pad,
                    float *out, hipStream_t stream);

/*
 * ilpm_conv2d_fwd_noalloc -- ilpm_conv2d_fwd for callers that cannot
 * allocate device memory (code under HIP graph capture, tight serving loops,
 * harnesses that forbid hipMalloc): same arguments, same plan and the same
 * output bits as ilpm_conv2d_fwd, but its split plans keep their partial
 * sums in a fixed array the library holds on each device (created when the
 * library's code loads on that device and held until the process ends) of
 * ILPM_NOALLOC_SCRATCH_BYTES, instead of the registered or library-owned
 * workspace.  It calls no hipMalloc, hipFree or other allocating routine.
 * A shape whose plan needs more than that returns ILPM_ERR_WORKSPACE before
 * anything is launched (ilpm_conv2d_workspace_size tells the need).  Every
 * call on a device shares that device's array and leaves its contents
 * behind (each call writes every partial sum it reads, so nothing needs
 * clearing): calls that overlap in time on one device race, so order them
 * on one stream.
 */
#define ILPM_NOALLOC_SCRATCH_BYTES ((size_t)16 << 20)
int ilpm_conv2d_fwd_noalloc(const float *in, const float *w, const float *bias,
                            int C_in, int H, int W, int C_out, int K, int stride, int pad,
                            float *out, hipStream_t stream);

/*
 * ilpm_conv2d_workspace_size -- bytes of device workspace the default plan
 * for this shape needs (0 when it needs none).  Pure host; no device access.
 */
int ilpm_conv2d_workspace_size(int C_in, int H, int W, int C_out, int K, int stride, int pad,
                               size_t *bytes);

/*
 * ilpm_set_workspace -- register caller-owned device memory (ptr, bytes) as
 * the workspace of the current device, replacing any earlier one; ptr = NULL
 * unregisters it (the library then allocates its own on need).  Its contents
 * on entry do not matter (every byte a call reads, the same call wrote first).
 * It must stay allocated while calls may use it and be 256-byte aligned;
 * `stream` is unused (kept for ABI stability).
 */
int ilpm_set_workspace(void *ptr, size_t bytes, hipStream_t stream);

/*
 * ilpm_set_split_sum -- how split plans (splits > 1) sum their per-split
 * partial outputs, for every later call in the process (Section 4's
 * accumulation over input channels, split across workgroups):
 *   ILPM_SPLIT_SUM_FUSED  (default) the last of a tile's workgroups to finish
 *                         sums the tile's slices; one launch per call.
 *   ILPM_SPLIT_SUM_KERNEL a second kernel sums all slices after the first.
 * Both add the slices in split order, so their outputs are bit-identical.
 * The 2x2 max-pool epilogue always uses the second kernel.  Returns
 * ILPM_ERR_INVALID_ARG for any other mode.  Host only.
 */
#define ILPM_SPLIT_SUM_FUSED 0
#define ILPM_SPLIT_SUM_KERNEL 1
int ilpm_set_split_sum(int mode);

/* Text for a status code (static storage). */
const char *ilpm_status_str(int status);

/*
 * ilpm_arch_supported -- the architecture check every launching call makes
 * on the current device: ILPM_OK when `gcn_arch_name` (a device's
 * hipDeviceProp_t::gcnArchName, e.g. "gfx950:sramecc+:xnack-") names gfx950,
 * ILPM_ERR_ARCH for any other architecture, ILPM_ERR_INVALID_ARG for NULL.
 * Pure host.
 */
int ilpm_arch_supported(const char *gcn_arch_name);

/* The hipError_t value behind the calling thread's most recent ILPM_ERR_HIP
 * (0 if there was none). */
int ilpm_last_hip_error(void);

/*
 * ilpm_conv2d_validate -- the argument checks of ilpm_conv2d_fwd, on the host
 * only (pointers are compared, never dereferenced).  Returns ILPM_OK,
 * ILPM_ERR_INVALID_ARG or ILPM_ERR_UNSUPPORTED.
 */
int ilpm_conv2d_validate(const void *in, const void *w, const void *bias,
                         int C_in, int H, int W, int C_out, int K, int stride, int pad,
                         const void *out);

/*
 * ilpm_conv2d_plan -- the plan ilpm_conv2d_fwd uses for this shape (path,
 * tile, split count, grid, workspace): the fastest plan measured on MI355X
 * for this exact shape when the compiled-in tuning table lists it, else the
 * best by a cost model.  Pure host.  A shape's plan is chosen once and kept
 * (a table in the library), so later calls cost a lookup.
 * Environment overrides, read once, the first time the library plans a call
 * (for sweeps and ablations; any of them bypasses the tuning table):
 *   ILPM_FORCE_PATH=direct|igemm  only that kernel family (igemm: the
 *                                 call fails with ILPM_ERR_UNSUPPORTED if
 *                                 no matrix-core variant takes the shape);
 *   ILPM_SPLIT=n                  matrix-core plans with n input-channel
 *                                 splits;
 *   ILPM_TILE=<h>x<w>             only variants whose output tile is h x w
 *                                 (ILPM_ERR_UNSUPPORTED if none takes the
 *                                 shape).
 */
int ilpm_conv2d_plan(int C_in, int H, int W, int C_out, int K, int stride, int pad,
                     ilpm_plan *plan);

/*
 * ilpm_conv2d_plan_variant -- a plan that runs compiled variant `variant` of
 * `path` with `splits` input-channel splits (0 = choose).  Pure host.  Returns
 * ILPM_ERR_INVALID_ARG when the variant does not exist or does not support the
 * filter size and stride.
 */
int ilpm_conv2d_plan_variant(int C_in, int H, int W, int C_out, int K, int stride, int pad,
                             int path, int variant, int splits, ilpm_plan *plan);

/* Number of compiled variants of `path` (0 for an unknown path). */
int ilpm_num_variants(int path);

/* Name of a compiled variant (static storage), NULL if it does not exist. */
const char *ilpm_variant_name(int path, int variant);

/*
 * ilpm_variant_info -- filter size, stride (0 = any), output tile and output
 * channels per workgroup of one compiled variant.  Pure host.
 */
int ilpm_variant_info(int path, int variant, int *K, int *stride, int *tile_h, int *tile_w,
                      int *co_tile);

/*
 * ilpm_variant_pipeline -- how a compiled variant moves its data: input
 * channels per stage (`ci_chunk`), the stage count a workgroup is built for
 * (`stages`, 0 = any), stage buffers (`buffers`; 0 for the direct path) and
 * ILPM_VARIANT_* `flags`.  A variant with a fixed stage count (more than two
 * buffers: the loads of later stages fly while earlier ones compute, and
 * the stage sequence is unrolled at compile time) plans only shapes whose
 * ceil(C_in / ci_chunk) is a whole multiple of `stages`, with exactly
 * ceil(C_in / ci_chunk) / stages splits.  A variant with a progressive
 * first stage (its first stage's matrix work starts once its first four
 * input channels have landed) plans only splits of at least two stages each.
 * A 1x1 variant whose lanes take consecutive input channels (four OIHW
 * weights per 16-byte load) plans only C_in a multiple of 4.
 * Pure host; ILPM_ERR_INVALID_ARG for an unknown variant.  Any output pointer
 * may be NULL.
 */
#define ILPM_VARIANT_WEIGHTS_LDS 1       /* weights staged through LDS from OIHW; prepacked weights are an OIHW copy */
#define ILPM_VARIANT_PROGRESSIVE_FIRST 2 /* progressive first stage: at least two stages per split */
#define ILPM_VARIANT_CONSECUTIVE_CHANNELS 4 /* consecutive input channels per lane: C_in a multiple of 4 */
int ilpm_variant_pipeline(int path, int variant, int *ci_chunk, int *stages, int *buffers, int *flags);

/*
 * ilpm_conv2d_fwd_plan -- ilpm_conv2d_fwd with an explicit plan (from
 * ilpm_conv2d_plan or ilpm_conv2d_plan_variant for the same shape).
 */
int ilpm_conv2d_fwd_plan(const float *in, const float *w, const float *bias,
                         int C_in, int H, int W, int C_out, int K, int stride, int pad,
                         float *out, const ilpm_plan *plan, hipStream_t stream);

/* ---- prepacked weights ----
 *
 * The paper stores the filter re-laid out ([C][R][S][K], output channel
 * innermost) so that the per-thread weight loads of its kernel coalesce
 * (Section 4, Algorithm 2), and treats that as offline work.  Here the same
 * idea targets the matrix-core kernels: ilpm_conv2d_prepack_weights writes a
 * plan's weights in the order its kernel loads them, so every weight load
 * instruction of a wave reads one contiguous kilobyte; weights are constant
 * across calls, so a caller packs once and then runs
 * ilpm_conv2d_fwd_prepacked.  The packed layout belongs to the plan's kernel
 * variant (and C_in, C_out, K); it is not meant to be read by the caller.
 * Channels are zero-padded to whole output-channel tiles and input-channel
 * chunks.  For a direct-path plan the packed buffer is an OIHW copy.
 */

/*
 * ilpm_conv2d_prepacked_size -- *bytes = size of the packed weights of
 * `plan` for C_in, C_out, K.  Pure host.  ILPM_ERR_INVALID_ARG if the plan's
 * variant does not take K, or an argument is out of range.
 */
int ilpm_conv2d_prepacked_size(const ilpm_plan *plan, int C_in, int C_out, int K, size_t *bytes);

/*
 * ilpm_conv2d_prepack_weights -- write w [C_out][C_in][K][K] (OIHW) into
 * `packed` (ilpm_conv2d_prepacked_size bytes, caller-owned device memory)
 * in the layout of `plan`.  w and packed: 16-byte aligned, not overlapping.
 * Enqueued on `stream`.
 */
int ilpm_conv2d_prepack_weights(const float *w, int C_in, int C_out, int K, const ilpm_plan *plan,
                                float *packed, hipStream_t stream);

/*
 * ilpm_conv2d_fwd_prepacked -- ilpm_conv2d_fwd_plan with the weights given
 * as ilpm_conv2d_prepack_weights wrote them for the same plan, C_in, C_out
 * and K (the plan must be for this exact shape, as for fwd_plan).  The result
 * is bit for bit that of ilpm_conv2d_fwd_plan with the OIHW weights.
 */
int ilpm_conv2d_fwd_prepacked(const float *in, const float *packed, const float *bias,
                              int C_in, int H, int W, int C_out, int K, int stride, int pad,
                              const ilpm_plan *plan, float *out, hipStream_t stream);

/*
 * ilpm_conv2d_plan_prepacked -- the default plan for a caller that will pack
 * the weights: the measured best with prepacked weights for this exact shape
 * (a second compiled-in table; with packed weights every weight load is one
 * contiguous kilobyte, so plans whose kernels were bound by the scattered
 * OIHW loads move up), else the plan ilpm_conv2d_plan would give.  Pure
 * host; chosen once per shape and kept, like ilpm_conv2d_plan; the same
 * environment overrides apply.  Use the plan for ilpm_conv2d_prepacked_size,
 * ilpm_conv2d_prepack_weights and the prepacked calls.
 */
int ilpm_conv2d_plan_prepacked(int C_in, int H, int W, int C_out, int K, int stride, int pad,
                               ilpm_plan *plan);

/*
 * ilpm_conv2d_plan_for -- the default plan for this shape, epilogue (the
 * ILPM_EPI_* bits the calls will pass) and weight layout (prepacked 0: OIHW,
 * 1: packed for the plan).  With ILPM_EPI_MAXPOOL2 the plan comes from the
 * measured tables of the pooled epilogue, where a plan whose tiles pool in
 * the workgroup can beat a faster convolution that needs the second kernel;
 * a shape missing there falls back as ilpm_conv2d_plan_prepacked /
 * ilpm_conv2d_plan do.  ilpm_conv2d_fwd_epilogue with plan NULL uses this
 * plan (prepacked 0).  Pure host; chosen once per (shape, epilogue kind,
 * layout) and kept.  ILPM_ERR_INVALID_ARG for unknown epilogue bits or
 * prepacked other than 0 or 1.
 */
int ilpm_conv2d_plan_for(int C_in, int H, int W, int C_out, int K, int stride, int pad, int epilogue,
                         int prepacked, ilpm_plan *plan);

/* ---- fused epilogue ----
 *
 * A CNN layer follows the convolution with ReLU and, between stages, a 2x2
 * max-pool (the ResNet and VGG networks the paper evaluates, Section 5).
 * Applying them as the convolution's results are written saves writing the
 * full-size output and reading it back.
 */
#define ILPM_EPI_RELU 1     /* out = max(conv + bias, 0) */
#define ILPM_EPI_MAXPOOL2 2 /* out[c][i][j] = max of the 2x2 window at (2i, 2j) of (conv + bias),
                               [C_out][H_out/2][W_out/2] (floor); needs H_out, W_out >= 2 */

/*
 * ilpm_conv2d_fwd_epilogue -- ilpm_conv2d_fwd followed by `epilogue`, a
 * combination of the ILPM_EPI_* bits (0 = none).  With both bits set the
 * result is max-pool of ReLU, which equals ReLU of max-pool.  `out` has the
 * pooled shape when ILPM_EPI_MAXPOOL2 is set.  plan: NULL for the default
 * plan of the shape and epilogue (ilpm_conv2d_plan_for), or one made for
 * this exact shape.  One-split
 * matrix-core plans whose tiles have even sides pool inside the kernel;
 * other plans write the full-size convolution output (as per-split partial
 * sums) to the workspace and pool it in a second kernel
 * (ilpm_conv2d_epilogue_workspace_size covers that route).  The values are
 * exactly those of the unfused sequence conv (same plan) -> ReLU -> max-pool.
 */
int ilpm_conv2d_fwd_epilogue(const float *in, const float *w, const float *bias,
                             int C_in, int H, int W, int C_out, int K, int stride, int pad,
                             int epilogue, const ilpm_plan *plan, float *out, hipStream_t stream);

/*
 * ilpm_conv2d_fwd_prepacked_epilogue -- ilpm_conv2d_fwd_epilogue with the
 * weights prepacked for `plan` (required, made for this exact shape), as
 * ilpm_conv2d_fwd_prepacked takes them.  The result is bit for bit that of
 * ilpm_conv2d_fwd_epilogue with the OIHW weights and the same plan; the
 * workspace is ilpm_conv2d_epilogue_workspace_size's for that plan.
 */
int ilpm_conv2d_fwd_prepacked_epilogue(const float *in, const float *packed, const float *bias,
                                       int C_in, int H, int W, int C_out, int K, int stride, int pad,
                                       int epilogue, const ilpm_plan *plan, float *out, hipStream_t stream);

/* Workspace bytes ilpm_conv2d_fwd_epilogue needs (plan NULL = default plan). */
int ilpm_conv2d_epilogue_workspace_size(int C_in, int H, int W, int C_out, int K, int stride, int pad,
                                        int epilogue, const ilpm_plan *plan, size_t *bytes);

/* ---- Winograd F(2x2, 3x3): a comparison path ----
 *
 * Not the ILP-M method: the competitor the paper measures it against
 * (Section 3, Winograd; Section 5).  3x3 filters, stride 1, any padding.  The
 * filter transform U = G g G^T (16 floats per (C_out, C_in) pair, layout
 * [16][C_out][C_in]) is done once by ilpm_winograd_transform_filter; each
 * call transforms the input, runs 16 channel-contraction GEMMs through the
 * rocBLAS the process already loaded (loaded at run time; without it the call
 * returns ILPM_ERR_UNSUPPORTED) and transforms the output back.  Workspace:
 * ilpm_conv2d_winograd_workspace_size bytes (same registered / library-owned
 * workspace as the split plans).  Results agree with the definition within
 * the same tolerance; the rounding is that of Winograd's transforms, not of
 * a direct sum.
 */
int ilpm_winograd_filter_size(int C_in, int C_out, size_t *bytes);
int ilpm_winograd_transform_filter(const float *w, int C_in, int C_out, float *u, hipStream_t stream);
int ilpm_conv2d_winograd_workspace_size(int C_in, int H, int W, int C_out, int pad, size_t *bytes);
int ilpm_conv2d_fwd_winograd(const float *in, const float *u, const float *bias,
                             int C_in, int H, int W, int C_out, int pad, float *out, hipStream_t stream);

/* ---- helpers for layer stacks (not part of the convolution) ---- */

/* x[i] = max(x[i], 0) for i < n, in place.  x: device fp32, n >= 0. */
int ilpm_relu_inplace(float *x, int64_t n, hipStream_t stream);

/*
 * ilpm_maxpool2x2 -- out[c][i][j] = max of in[c][2i..2i+1][2j..2j+1];
 * in [C, H, W] -> out [C, H/2, W/2] (floor).  Requires H, W >= 2; no overlap.
 */
int ilpm_maxpool2x2(const float *in, int C, int H, int W, float *out, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* ILPM_H */
