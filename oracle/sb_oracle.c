/*
 * sb_oracle.c -- fp64 CPU oracle for one SplitBrain worker's compute share
 * (arXiv 2112.15317).
 *
 * TEST INFRASTRUCTURE.  This library exists only to check the HIP path.  It
 * is loaded by the test suite, by the package smoke check and by the CPU
 * baseline leg of the benchmark, and by nothing else.  It shares no source,
 * header, table or helper with the HIP library, and never calls it.
 *
 * Every function evaluates the plain mathematical definition of one layer
 * of the paper's CNN (sec. 2.2: convolution, pooling, ReLU, fully connected
 * layers; sec. 3.1: an FC layer split to 1/K of its outputs, whose backward
 * pass yields gradients over the full input that are reduced later).  All
 * arithmetic is IEEE double; there is no blocking, reordering or fusion
 * beyond what the definition states.  Each output element is produced by one
 * small "element" function; the whole-tensor entry points loop that function
 * over every element, the "_at" entry points over a caller-given list of flat
 * output indices (used to check full-size GPU runs on a sample).
 *
 * Layout conventions (the same as the GPU library's public boundary):
 *   activations  NCHW, row-major, x[((n*C + c)*H + h)*W + w]
 *   conv weights KCRS, w[((k*C + c)*3 + r)*3 + s], 3x3 taps, stride 1, pad 1
 *   FC input     X[i*Kin + k]   (M rows = gathered batch, Kin features)
 *   FC shard     Wsh[k*Ns + j]  (the shard's Ns output columns of W)
 *   pool code    bits 0-1 = row-major position of the window maximum
 *                (0:(0,0) 1:(0,1) 2:(1,0) 3:(1,1)); bit 7 set when that
 *                maximum is <= 0 (the ReLU after the max blocks the
 *                gradient); bits 2-6 zero.
 *
 * Readings of points the paper leaves open: "convolution" is cross-
 * correlation (deep-learning convention); ReLU'(0) = 0; the pooling window
 * maximum is the first maximum in row-major order (strict ">"); the ReLU is
 * taken after the max, which gives the same value as before it.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stddef.h>

#define EXPORT __attribute__((visibility("default")))

static inline int in_range(int v, int n) { return v >= 0 && v < n; }

/* ---------------------------------------------------------------- conv ---
 * Forward (sec. 2.2, convolutional stage):
 *   Z[n,k,h,w] = b[k] + sum_{c,r,s} X[n,c,h+r-1,w+s-1] * Wt[k,c,r,s]
 * with X taken as zero outside the image (padding 1).                     */
static double conv_fwd_elem(int C, int H, int W, const double *x,
                            const double *wt, int n, int k, int h, int w)
{
    double acc = 0.0;
    for (int c = 0; c < C; ++c)
        for (int r = 0; r < 3; ++r) {
            int ih = h + r - 1;
            if (!in_range(ih, H)) continue;
            for (int s = 0; s < 3; ++s) {
                int iw = w + s - 1;
                if (!in_range(iw, W)) continue;
                acc += x[(((size_t)n * C + c) * H + ih) * W + iw] *
                       wt[(((size_t)k * C + c) * 3 + r) * 3 + s];
            }
        }
    return acc;
}

static double conv_fwd_out(int C, int H, int W, int K, const double *x,
                           const double *wt, const double *bias, int relu,
                           size_t flat)
{
    int w = (int)(flat % W);
    int h = (int)((flat / W) % H);
    int k = (int)((flat / ((size_t)W * H)) % K);
    int n = (int)(flat / ((size_t)W * H * K));
    double z = (bias ? bias[k] : 0.0) + conv_fwd_elem(C, H, W, x, wt, n, k, h, w);
    if (relu && !(z > 0.0)) z = 0.0;
    return z;
}

EXPORT void or_conv3x3_fwd(int N, int C, int H, int W, int K,
                           const double *x, const double *wt,
                           const double *bias, int relu, double *y)
{
    size_t total = (size_t)N * K * H * W;
    #pragma omp parallel for schedule(static)
    for (size_t f = 0; f < total; ++f)
        y[f] = conv_fwd_out(C, H, W, K, x, wt, bias, relu, f);
}

EXPORT void or_conv3x3_fwd_at(int N, int C, int H, int W, int K,
                              const double *x, const double *wt,
                              const double *bias, int relu,
                              int64_t count, const int64_t *flat, double *out)
{
    (void)N;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i)
        out[i] = conv_fwd_out(C, H, W, K, x, wt, bias, relu, (size_t)flat[i]);
}

/* Data gradient (sec. 2.2, backward propagation through the convolution):
 *   dX[n,c,i,j] = sum_{k,r,s} dZ[n,k,i-r+1,j-s+1] * Wt[k,c,r,s]
 * over the (r,s) whose output position lies inside the image.  With a mask
 * source S (the activation of the layer below, whose ReLU this gradient
 * passes through), dX = 0 wherever S <= 0.                               */
static double conv_bwd_data_elem(int H, int W, int K, int C, const double *dz,
                                 const double *wt, int n, int c, int i, int j)
{
    double acc = 0.0;
    for (int k = 0; k < K; ++k)
        for (int r = 0; r < 3; ++r) {
            int h = i - r + 1;
            if (!in_range(h, H)) continue;
            for (int s = 0; s < 3; ++s) {
                int w = j - s + 1;
                if (!in_range(w, W)) continue;
                acc += dz[(((size_t)n * K + k) * H + h) * W + w] *
                       wt[(((size_t)k * C + c) * 3 + r) * 3 + s];
            }
        }
    return acc;
}

static double conv_bwd_data_out(int C, int H, int W, int K, const double *dz,
                                const double *wt, const double *mask_src,
                                size_t flat)
{
    if (mask_src && !(mask_src[flat] > 0.0)) return 0.0;
    int j = (int)(flat % W);
    int i = (int)((flat / W) % H);
    int c = (int)((flat / ((size_t)W * H)) % C);
    int n = (int)(flat / ((size_t)W * H * C));
    return conv_bwd_data_elem(H, W, K, C, dz, wt, n, c, i, j);
}

EXPORT void or_conv3x3_bwd_data(int N, int C, int H, int W, int K,
                                const double *dz, const double *wt,
                                const double *mask_src, double *dx)
{
    size_t total = (size_t)N * C * H * W;
    #pragma omp parallel for schedule(static)
    for (size_t f = 0; f < total; ++f)
        dx[f] = conv_bwd_data_out(C, H, W, K, dz, wt, mask_src, f);
}

EXPORT void or_conv3x3_bwd_data_at(int N, int C, int H, int W, int K,
                                   const double *dz, const double *wt,
                                   const double *mask_src, int64_t count,
                                   const int64_t *flat, double *out)
{
    (void)N;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i)
        out[i] = conv_bwd_data_out(C, H, W, K, dz, wt, mask_src, (size_t)flat[i]);
}

/* Weight gradient (sec. 2.2 backward propagation; sec. 3.1 Modulo Layer:
 * the convolutional parameters are updated from the whole local batch):
 *   dW[k,c,r,s] = sum_{n,h,w} X[n,c,h+r-1,w+s-1] * dZ[n,k,h,w]
 *   db[k]       = sum_{n,h,w} dZ[n,k,h,w]                                 */
static double conv_bwd_weight_elem(int N, int C, int H, int W, int K,
                                   const double *x, const double *dz,
                                   int k, int c, int r, int s)
{
    double acc = 0.0;
    for (int n = 0; n < N; ++n)
        for (int h = 0; h < H; ++h) {
            int ih = h + r - 1;
            if (!in_range(ih, H)) continue;
            for (int w = 0; w < W; ++w) {
                int iw = w + s - 1;
                if (!in_range(iw, W)) continue;
                acc += x[(((size_t)n * C + c) * H + ih) * W + iw] *
                       dz[(((size_t)n * K + k) * H + h) * W + w];
            }
        }
    return acc;
}

static double conv_bwd_weight_out(int N, int C, int H, int W, int K,
                                  const double *x, const double *dz, size_t flat)
{
    int s = (int)(flat % 3);
    int r = (int)((flat / 3) % 3);
    int c = (int)((flat / 9) % C);
    int k = (int)(flat / ((size_t)9 * C));
    return conv_bwd_weight_elem(N, C, H, W, K, x, dz, k, c, r, s);
}

static double conv_bias_grad_elem(int N, int H, int W, int K,
                                  const double *dz, int k)
{
    double acc = 0.0;
    for (int n = 0; n < N; ++n)
        for (int p = 0; p < H * W; ++p)
            acc += dz[((size_t)n * K + k) * H * W + p];
    return acc;
}

EXPORT void or_conv3x3_bwd_weight(int N, int C, int H, int W, int K,
                                  const double *x, const double *dz,
                                  double *dw, double *db)
{
    size_t total = (size_t)K * C * 9;
    #pragma omp parallel for schedule(static)
    for (size_t f = 0; f < total; ++f)
        dw[f] = conv_bwd_weight_out(N, C, H, W, K, x, dz, f);
    if (db) {
        #pragma omp parallel for schedule(static)
        for (int k = 0; k < K; ++k)
            db[k] = conv_bias_grad_elem(N, H, W, K, dz, k);
    }
}

EXPORT void or_conv3x3_bwd_weight_at(int N, int C, int H, int W, int K,
                                     const double *x, const double *dz,
                                     int64_t count, const int64_t *flat,
                                     double *out)
{
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i)
        out[i] = conv_bwd_weight_out(N, C, H, W, K, x, dz, (size_t)flat[i]);
}

/* ------------------------------------------------------- ReLU + maxpool ---
 * 2x2 max pooling with stride 2 (sec. 2.2 "pooling layer downsamples"),
 * followed by the ReLU activation.  The window is scanned in row-major
 * order and the first maximum is kept.                                     */
EXPORT void or_relu_maxpool_fwd(int N, int C, int H, int W, const double *x,
                                double *y, uint8_t *idx)
{
    int Ho = H / 2, Wo = W / 2;
    size_t total = (size_t)N * C * Ho * Wo;
    #pragma omp parallel for schedule(static)
    for (size_t f = 0; f < total; ++f) {
        int ow = (int)(f % Wo);
        int oh = (int)((f / Wo) % Ho);
        size_t plane = f / ((size_t)Wo * Ho);          /* n*C + c */
        const double *p = x + plane * H * W;
        double m = p[(size_t)(2 * oh) * W + 2 * ow];
        int arg = 0;
        for (int j = 1; j < 4; ++j) {
            double v = p[(size_t)(2 * oh + j / 2) * W + 2 * ow + j % 2];
            if (v > m) { m = v; arg = j; }
        }
        y[f] = (m > 0.0) ? m : 0.0;
        idx[f] = (uint8_t)(arg | ((m > 0.0) ? 0 : 0x80));
    }
}

/* Backward: the gradient of each pooled output goes to the position that
 * held the window maximum, unless the ReLU blocked it; all else is zero.   */
EXPORT void or_relu_maxpool_bwd(int N, int C, int H, int W, const double *dy,
                                const uint8_t *idx, double *dx)
{
    int Ho = H / 2, Wo = W / 2;
    size_t total = (size_t)N * C * Ho * Wo;
    #pragma omp parallel for schedule(static)
    for (size_t f = 0; f < total; ++f) {
        int ow = (int)(f % Wo);
        int oh = (int)((f / Wo) % Ho);
        size_t plane = f / ((size_t)Wo * Ho);
        double *p = dx + plane * H * W;
        for (int j = 0; j < 4; ++j)
            p[(size_t)(2 * oh + j / 2) * W + 2 * ow + j % 2] = 0.0;
        if (!(idx[f] & 0x80)) {
            int j = idx[f] & 3;
            p[(size_t)(2 * oh + j / 2) * W + 2 * ow + j % 2] = dy[f];
        }
    }
}

/* ------------------------------------------------------------ FC shard ---
 * A LINEAR layer split to 1/K of its outputs (sec. 3.1, Layer Partitioning:
 * the FC layer is partitioned to 1/K size), run on the batch gathered by
 * the modulo layer (sec. 3.1, Modulo Layer).
 *   Y[i,j] = b[j] + sum_k X[i,k] * Wsh[k,j]          (then ReLU if asked)  */
static double fc_fwd_out(int Kin, int Ns, const double *x, const double *w,
                         const double *b, int relu, size_t flat)
{
    int j = (int)(flat % Ns);
    size_t i = flat / Ns;
    double acc = b ? b[j] : 0.0;
    for (int k = 0; k < Kin; ++k)
        acc += x[i * Kin + k] * w[(size_t)k * Ns + j];
    if (relu && !(acc > 0.0)) acc = 0.0;
    return acc;
}

EXPORT void or_fc_fwd(int M, int Kin, int Ns, const double *x, const double *w,
                      const double *b, int relu, double *y)
{
    size_t total = (size_t)M * Ns;
    #pragma omp parallel for schedule(static)
    for (size_t f = 0; f < total; ++f)
        y[f] = fc_fwd_out(Kin, Ns, x, w, b, relu, f);
}

EXPORT void or_fc_fwd_at(int M, int Kin, int Ns, const double *x,
                         const double *w, const double *b, int relu,
                         int64_t count, const int64_t *flat, double *out)
{
    (void)M;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i)
        out[i] = fc_fwd_out(Kin, Ns, x, w, b, relu, (size_t)flat[i]);
}

/* Backward of the shard (sec. 3.1, Shard Layer: a partitioned layer
 * produces gradients with respect to its full input, which the shard layer
 * later reduces across workers).  With G = dY, or dY * [S > 0] when a ReLU
 * mask source S of the shard's output is given:
 *   dXp[i,k] = sum_j G[i,j] * Wsh[k,j]      (this shard's partial sum)
 *   dW[k,j]  = (accumulate ? dW[k,j] : 0) + sum_i X[i,k] * G[i,j]
 *   db[j]    = (accumulate ? db[j]   : 0) + sum_i G[i,j]                  */
static double fc_grad(const double *dy, const double *mask, int Ns, size_t i, int j)
{
    size_t f = i * Ns + j;
    if (mask && !(mask[f] > 0.0)) return 0.0;
    return dy[f];
}

static double fc_bwd_dx_out(int Kin, int Ns, const double *w, const double *dy,
                            const double *mask, size_t flat)
{
    int k = (int)(flat % Kin);
    size_t i = flat / Kin;
    double acc = 0.0;
    for (int j = 0; j < Ns; ++j)
        acc += fc_grad(dy, mask, Ns, i, j) * w[(size_t)k * Ns + j];
    return acc;
}

static double fc_bwd_dw_sum(int M, int Kin, int Ns, const double *x,
                            const double *dy, const double *mask, size_t flat)
{
    int j = (int)(flat % Ns);
    size_t k = flat / Ns;
    double acc = 0.0;
    for (int i = 0; i < M; ++i)
        acc += x[(size_t)i * Kin + k] * fc_grad(dy, mask, Ns, (size_t)i, j);
    return acc;
}

EXPORT void or_fc_bwd(int M, int Kin, int Ns, const double *x, const double *w,
                      const double *dy, const double *mask, double *dxp,
                      double *dw, double *db, int accumulate)
{
    if (dxp) {
        size_t total = (size_t)M * Kin;
        #pragma omp parallel for schedule(static)
        for (size_t f = 0; f < total; ++f)
            dxp[f] = fc_bwd_dx_out(Kin, Ns, w, dy, mask, f);
    }
    size_t totw = (size_t)Kin * Ns;
    #pragma omp parallel for schedule(static)
    for (size_t f = 0; f < totw; ++f)
        dw[f] = (accumulate ? dw[f] : 0.0) + fc_bwd_dw_sum(M, Kin, Ns, x, dy, mask, f);
    if (db) {
        #pragma omp parallel for schedule(static)
        for (int j = 0; j < Ns; ++j) {
            double acc = 0.0;
            for (int i = 0; i < M; ++i) acc += fc_grad(dy, mask, Ns, (size_t)i, j);
            db[j] = (accumulate ? db[j] : 0.0) + acc;
        }
    }
}

EXPORT void or_fc_bwd_dx_at(int M, int Kin, int Ns, const double *w,
                            const double *dy, const double *mask,
                            int64_t count, const int64_t *flat, double *out)
{
    (void)M;
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i)
        out[i] = fc_bwd_dx_out(Kin, Ns, w, dy, mask, (size_t)flat[i]);
}

EXPORT void or_fc_bwd_dw_at(int M, int Kin, int Ns, const double *x,
                            const double *dy, const double *mask,
                            int64_t count, const int64_t *flat, double *out)
{
    #pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < count; ++i)
        out[i] = fc_bwd_dw_sum(M, Kin, Ns, x, dy, mask, (size_t)flat[i]);
}

/* ------------------------------------------------------- bf16 rounding ---
 * Round to the nearest value representable in bfloat16 (1 sign bit, 8
 * exponent bits, 7 stored fraction bits: 8 significant bits), ties to even.
 * Used at the storage points of the bf16 data path.  Written from the
 * format's definition: for |v| in [2^e, 2^(e+1)) with e >= -126 the spacing
 * of bf16 values is 2^(e-7); below 2^-126 (subnormal) it is 2^-133.  rint()
 * in the default rounding mode rounds half-way cases to even.             */
EXPORT void or_round_bf16(double *a, int64_t count)
{
    for (int64_t i = 0; i < count; ++i) {
        double v = a[i];
        if (v == 0.0 || !isfinite(v)) continue;
        int e;
        frexp(v, &e);          /* |v| = m * 2^e, m in [0.5, 1) -> |v| in [2^(e-1), 2^e) */
        int ex = e - 1;
        if (ex < -126) ex = -126;
        double q = ldexp(1.0, ex - 7);
        double r = rint(v / q) * q;
        if (fabs(r) > 3.3895313892515355e38) r = copysign(INFINITY, v);
        a[i] = r;
    }
}

/* Number of OpenMP threads the loops above run on. */
EXPORT int or_num_threads(void) { return omp_get_max_threads(); }
