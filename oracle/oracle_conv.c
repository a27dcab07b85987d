/*
 * CPU oracle for the batch-1 2-D convolution forward pass.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the GPU library links, includes or
 * calls this file, and this file uses nothing of the GPU library: only the
 * tests, the smoke check and the benchmark's CPU-baseline leg load it.
 *
 * What it computes is the plain definition of the operation that the ILP-M
 * method evaluates (Section 4, Algorithm 2: an output pixel of output channel
 * k accumulates, over every input channel and every filter tap (r, s), the
 * filter weight times the input pixel at (y + r, x + s) -- a cross-correlation,
 * no filter flip).  ILP-M only reorders this sum (it iterates the taps in the
 * outer loop and keeps one weight in a register), so the oracle is the
 * definition written out, not the algorithm's loop order:
 *
 *   H_out = floor((H + 2p - K) / s) + 1,   W_out likewise
 *   xp[ci][i][j] = x[ci][i][j] inside [0,H) x [0,W), 0 outside (zero padding)
 *   out[co][oh][ow] = b[co] + sum_{ci, kh, kw} w[co][ci][kh][kw] * xp[ci][oh*s - p + kh][ow*s - p + kw]
 *   S[co][oh][ow]   =         sum_{ci, kh, kw} | w[co][ci][kh][kw] * xp[...] |
 *
 * Seven nested loops: image n (always 0, batch 1), co, oh, ow, ci, kh, kw.
 * Each product of two float32 values is exact in float64; terms are summed in
 * float64 in ascending (ci, kh, kw) order starting from the bias, so the
 * result does not depend on the thread count.  The bias is not part of S.
 *
 * Stride, padding and bias are not in the paper (its algorithm is stride 1 and
 * leaves the halo implicit); the readings used are the standard ones listed
 * above.
 *
 * The helpers relu and maxpool2x2 are the plain definitions used between the
 * layers of the VGG-16 stack.
 */
#include <math.h>
#include <stddef.h>
#include <stdint.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Thread count for the OpenMP loops (results do not depend on it); returns the
 * count in force afterwards, 1 in a build without OpenMP. */
int oracle_set_threads(int n)
{
#ifdef _OPENMP
    if (n > 0)
        omp_set_num_threads(n);
    return omp_get_max_threads();
#else
    (void)n;
    return 1;
#endif
}

/* floor((n + 2*pad - k) / stride) + 1, or 0 when no window fits. */
int oracle_out_size(int n, int k, int stride, int pad)
{
    long span = (long)n + 2L * pad - k;
    if (span < 0 || stride <= 0)
        return 0;
    return (int)(span / stride) + 1;
}

/* One output element (co, oh, ow) from the definition above. */
static void one_output(const float *x, const float *w, const float *b,
                       int C_in, int H, int W, int K, int stride, int pad,
                       int co, int oh, int ow, double *val, double *sabs)
{
    double acc = b ? (double)b[co] : 0.0;
    double s = 0.0;
    for (int ci = 0; ci < C_in; ++ci) {
        for (int kh = 0; kh < K; ++kh) {
            for (int kw = 0; kw < K; ++kw) {
                long ih = (long)oh * stride - pad + kh;
                long iw = (long)ow * stride - pad + kw;
                double xv = 0.0;
                if (ih >= 0 && ih < H && iw >= 0 && iw < W)
                    xv = (double)x[((size_t)ci * H + ih) * W + iw];
                double wv = (double)w[(((size_t)co * C_in + ci) * K + kh) * K + kw];
                double t = wv * xv;
                acc += t;
                s += fabs(t);
            }
        }
    }
    *val = acc;
    *sabs = s;
}

/*
 * Full output.  x: [1,C_in,H,W], w: [C_out,C_in,K,K], b: [C_out] or NULL,
 * out and sumabs: [1,C_out,H_out,W_out] float64 (sumabs may be NULL).
 * Returns 0, or -1 for a shape with no output.
 */
int oracle_conv2d_f64(const float *x, const float *w, const float *b,
                      int C_in, int H, int W, int C_out, int K, int stride, int pad,
                      double *out, double *sumabs)
{
    int Ho = oracle_out_size(H, K, stride, pad);
    int Wo = oracle_out_size(W, K, stride, pad);
    if (Ho < 1 || Wo < 1 || C_in < 1 || C_out < 1 || K < 1)
        return -1;
    for (int n = 0; n < 1; ++n) {
#pragma omp parallel for schedule(dynamic, 1)
        for (int co = 0; co < C_out; ++co) {
            for (int oh = 0; oh < Ho; ++oh) {
                for (int ow = 0; ow < Wo; ++ow) {
                    double v, s;
                    one_output(x, w, b, C_in, H, W, K, stride, pad, co, oh, ow, &v, &s);
                    size_t o = ((size_t)co * Ho + oh) * Wo + ow;
                    out[o] = v;
                    if (sumabs)
                        sumabs[o] = s;
                }
            }
        }
    }
    return 0;
}

/*
 * Selected outputs only: idx[i] is a flat index into [C_out,H_out,W_out].
 * out[i], sumabs[i] receive that element.  Returns 0, or -1 on a bad index.
 */
int oracle_conv2d_f64_points(const float *x, const float *w, const float *b,
                             int C_in, int H, int W, int C_out, int K, int stride, int pad,
                             const int64_t *idx, int64_t npts, double *out, double *sumabs)
{
    int Ho = oracle_out_size(H, K, stride, pad);
    int Wo = oracle_out_size(W, K, stride, pad);
    if (Ho < 1 || Wo < 1)
        return -1;
    int64_t total = (int64_t)C_out * Ho * Wo;
    int bad = 0;
#pragma omp parallel for schedule(dynamic, 16) reduction(| : bad)
    for (int64_t i = 0; i < npts; ++i) {
        int64_t f = idx[i];
        if (f < 0 || f >= total) {
            bad = 1;
            continue;
        }
        int co = (int)(f / ((int64_t)Ho * Wo));
        int rem = (int)(f % ((int64_t)Ho * Wo));
        double v, s;
        one_output(x, w, b, C_in, H, W, K, stride, pad, co, rem / Wo, rem % Wo, &v, &s);
        out[i] = v;
        if (sumabs)
            sumabs[i] = s;
    }
    return bad ? -1 : 0;
}

/* y[i] = x[i] if x[i] > 0, else 0. */
void oracle_relu_f32(const float *x, float *y, int64_t n)
{
    for (int64_t i = 0; i < n; ++i)
        y[i] = x[i] > 0.0f ? x[i] : 0.0f;
}

/* 2x2 window, stride 2: y[c][i][j] = max over x[c][2i+a][2j+b], a,b in {0,1};
 * output H/2 x W/2 (floor). */
void oracle_maxpool2x2_f32(const float *x, int C, int H, int W, float *y)
{
    int Ho = H / 2, Wo = W / 2;
    for (int c = 0; c < C; ++c)
        for (int i = 0; i < Ho; ++i)
            for (int j = 0; j < Wo; ++j) {
                float m = x[((size_t)c * H + 2 * i) * W + 2 * j];
                for (int a = 0; a < 2; ++a)
                    for (int bb = 0; bb < 2; ++bb) {
                        float v = x[((size_t)c * H + 2 * i + a) * W + 2 * j + bb];
                        if (v > m)
                            m = v;
                    }
                y[((size_t)c * Ho + i) * Wo + j] = m;
            }
}
