/*
 * oracle.c -- plain, slow CPU oracle for restructured batch normalisation
 * (BN Fission-n-Fusion) training.  TEST INFRASTRUCTURE ONLY.
 *
 * Only the test suite, the smoke check and the benchmark's CPU-baseline leg may
 * load this library.  The GPU product path never calls, links or imports it,
 * and this file shares no code, header, table or helper with the HIP kernels.
 *
 * Every routine is the textbook definition written out with naive loops in
 * fp64 (OpenMP only splits independent outputs across threads; no blocking,
 * no fusion, no reordering of a sum beyond "left to right").  Layouts:
 *   activations  NHWC, dense:            x[((n*H + h)*W + w)*C + c]
 *   conv weights [KH][KW][C_in][C_out]:   wt[((kh*K + kw)*Ci + ci)*Co + co]
 *   per-channel vectors [C].
 *
 * What each routine follows in the paper ("Restructuring Batch Normalization
 * to Accelerate CNN Training", arXiv 1807.01702):
 *   - BN training forward/backward: Sec. 2.2 states BN as per-channel
 *     mini-batch mean and variance, then normalisation with scale gamma and
 *     shift beta (the equations themselves are those of Ioffe & Szegedy, whom
 *     the paper cites); Sec. 3.1 states the backward order (dgamma/dbeta from
 *     a sweep over the output gradient before the input gradient).
 *   - Variance: biased (divide by m), the population variance over the
 *     mini-batch that the Sec. 3.2 mean/variance-fusion identity
 *     V(X) = E(X^2) - E(X)^2 refers to.  The reference value is computed
 *     two-pass (E((X - E X)^2)); orc_mvf_stats computes the one-pass form of
 *     that identity separately.
 *   - ReLU: element-wise clip (Sec. 2.1, Sec. 3.2 ReLU-CONV fusion); the
 *     gradient is taken as 0 at exactly 0.
 *   - CONV: cross-correlation with zero padding (the usual CNN definition;
 *     DenseNet/ResNet use 1x1 and 3x3 filters, Sec. 2.2-2.3, and a 7x7 first
 *     layer, Sec. 3.1).
 *   - Pooling / FC / softmax cross-entropy: the standard DenseNet-121 head and
 *     transition (Sec. 2.3); the paper gives no equations for them.
 */
#include <math.h>
#include <stdlib.h>
#include <string.h>

#define IDX4(n, h, w, c, H, W, C) ((((long)(n) * (H) + (h)) * (W) + (w)) * (long)(C) + (c))

/* ---------------------------------------------------------------- CONV ---- */

static int out_dim(int in, int k, int stride, int pad) { return (in + 2 * pad - k) / stride + 1; }

/* out[n,oy,ox,co] = sum_{kh,kw,ci} in[n, oy*s+kh-p, ox*s+kw-p, ci] * wt[kh,kw,ci,co];
 * taps that fall outside the input image read 0. */
void orc_conv_fwd(int N, int H, int W, int Ci, int Co, int K, int stride, int pad,
                  const double *in, const double *wt, double *out)
{
    int Ho = out_dim(H, K, stride, pad), Wo = out_dim(W, K, stride, pad);
    #pragma omp parallel for collapse(3) schedule(static)
    for (int n = 0; n < N; n++)
        for (int oy = 0; oy < Ho; oy++)
            for (int ox = 0; ox < Wo; ox++)
                for (int co = 0; co < Co; co++) {
                    double acc = 0.0;
                    for (int kh = 0; kh < K; kh++)
                        for (int kw = 0; kw < K; kw++) {
                            int iy = oy * stride + kh - pad, ix = ox * stride + kw - pad;
                            if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;
                            for (int ci = 0; ci < Ci; ci++)
                                acc += in[IDX4(n, iy, ix, ci, H, W, Ci)] *
                                       wt[((long)(kh * K + kw) * Ci + ci) * Co + co];
                        }
                    out[IDX4(n, oy, ox, co, Ho, Wo, Co)] = acc;
                }
}

/* Gradient of L = sum(out * g) with respect to the input:
 * din[n,iy,ix,ci] = sum over (kh,kw,co) and the output positions (oy,ox) that
 * read input pixel (iy,ix) through tap (kh,kw) of g[n,oy,ox,co] * wt[kh,kw,ci,co]. */
void orc_conv_dgrad(int N, int H, int W, int Ci, int Co, int K, int stride, int pad,
                    const double *g, const double *wt, double *din)
{
    int Ho = out_dim(H, K, stride, pad), Wo = out_dim(W, K, stride, pad);
    #pragma omp parallel for collapse(3) schedule(static)
    for (int n = 0; n < N; n++)
        for (int iy = 0; iy < H; iy++)
            for (int ix = 0; ix < W; ix++)
                for (int ci = 0; ci < Ci; ci++) {
                    double acc = 0.0;
                    for (int kh = 0; kh < K; kh++)
                        for (int kw = 0; kw < K; kw++) {
                            int ty = iy + pad - kh, tx = ix + pad - kw;  /* = oy*stride */
                            if (ty < 0 || tx < 0 || ty % stride || tx % stride) continue;
                            int oy = ty / stride, ox = tx / stride;
                            if (oy >= Ho || ox >= Wo) continue;
                            for (int co = 0; co < Co; co++)
                                acc += g[IDX4(n, oy, ox, co, Ho, Wo, Co)] *
                                       wt[((long)(kh * K + kw) * Ci + ci) * Co + co];
                        }
                    din[IDX4(n, iy, ix, ci, H, W, Ci)] = acc;
                }
}

/* Gradient of L = sum(out * g) with respect to the weights:
 * dwt[kh,kw,ci,co] = sum_{n,oy,ox} in[n, oy*s+kh-p, ox*s+kw-p, ci] * g[n,oy,ox,co]. */
void orc_conv_wgrad(int N, int H, int W, int Ci, int Co, int K, int stride, int pad,
                    const double *in, const double *g, double *dwt)
{
    int Ho = out_dim(H, K, stride, pad), Wo = out_dim(W, K, stride, pad);
    #pragma omp parallel for collapse(3) schedule(static)
    for (int kh = 0; kh < K; kh++)
        for (int kw = 0; kw < K; kw++)
            for (int ci = 0; ci < Ci; ci++) {
                double *acc = (double *)calloc((size_t)Co, sizeof(double));
                for (int n = 0; n < N; n++)
                    for (int oy = 0; oy < Ho; oy++)
                        for (int ox = 0; ox < Wo; ox++) {
                            int iy = oy * stride + kh - pad, ix = ox * stride + kw - pad;
                            if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;
                            double a = in[IDX4(n, iy, ix, ci, H, W, Ci)];
                            const double *gr = g + IDX4(n, oy, ox, 0, Ho, Wo, Co);
                            for (int co = 0; co < Co; co++) acc[co] += a * gr[co];
                        }
                for (int co = 0; co < Co; co++)
                    dwt[((long)(kh * K + kw) * Ci + ci) * Co + co] = acc[co];
                free(acc);
            }
}

/* ------------------------------------------------------------------ BN ---- */

/* BN training forward over x[m][C] (m = N*H*W values per channel):
 *   mean = (1/m) sum x,  var = (1/m) sum (x - mean)^2  (two-pass, biased),
 *   rstd = 1/sqrt(var + eps),  xhat = (x - mean) * rstd,  y = gamma*xhat + beta. */
void orc_bn_fwd(long m, int C, const double *x, const double *gamma, const double *beta,
                double eps, double *mean, double *var, double *rstd, double *y)
{
    #pragma omp parallel for schedule(static)
    for (int c = 0; c < C; c++) {
        double s = 0.0;
        for (long i = 0; i < m; i++) s += x[i * C + c];
        double mu = s / (double)m;
        double q = 0.0;
        for (long i = 0; i < m; i++) { double d = x[i * C + c] - mu; q += d * d; }
        double v = q / (double)m;
        double r = 1.0 / sqrt(v + eps);
        mean[c] = mu; var[c] = v; rstd[c] = r;
        if (y)
            for (long i = 0; i < m; i++)
                y[i * C + c] = gamma[c] * ((x[i * C + c] - mu) * r) + beta[c];
    }
}

/* Mean/variance fusion (Sec. 3.2): E(X) and E(X^2) from one sweep, then
 * V(X) = E(X^2) - E(X)^2.  Reference for the one-pass statistics. */
void orc_mvf_stats(long m, int C, const double *x, double *mean, double *var)
{
    #pragma omp parallel for schedule(static)
    for (int c = 0; c < C; c++) {
        double s = 0.0, s2 = 0.0;
        for (long i = 0; i < m; i++) { double v = x[i * C + c]; s += v; s2 += v * v; }
        double e1 = s / (double)m, e2 = s2 / (double)m;
        mean[c] = e1;
        var[c] = e2 - e1 * e1;
    }
}

/* Shifted one-sweep statistics: the mean/variance-fusion identity of Sec. 3.2
 * applied to d = x - K for a per-channel constant K (the robust reading of
 * one-sweep statistics; the paper itself names higher precision as the
 * remedy for the cancellation of E(X^2) - E(X)^2).  With S1 = sum d and
 * S2 = sum d^2:  mean = K + S1/m,  var = S2/m - (S1/m)^2. */
void orc_mvf_stats_shifted(long m, int C, const double *x, const double *K, double *mean, double *var)
{
    #pragma omp parallel for schedule(static)
    for (int c = 0; c < C; c++) {
        double s = 0.0, s2 = 0.0;
        for (long i = 0; i < m; i++) { double d = x[i * C + c] - K[c]; s += d; s2 += d * d; }
        double d1 = s / (double)m, d2 = s2 / (double)m;
        mean[c] = K[c] + d1;
        var[c] = d2 - d1 * d1;
    }
}

/* Running statistics of BN for inference (the usual exponential moving
 * average): r = (1 - mo) r + mo * batch value, the variance taken unbiased,
 * var * m / (m - 1). */
void orc_running_update(int C, long m, double mo, const double *mean, const double *var, double *rmean, double *rvar)
{
    for (int c = 0; c < C; c++) {
        rmean[c] = (1.0 - mo) * rmean[c] + mo * mean[c];
        rvar[c] = (1.0 - mo) * rvar[c] + mo * var[c] * ((double)m / (double)(m - 1));
    }
}

/* BN training backward.  With xhat = (x - mean) * rstd recomputed from x:
 *   dbeta  = sum dy,   dgamma = sum dy * xhat,
 *   dx     = gamma * rstd * (dy - dbeta/m - xhat * dgamma/m).
 * dx may be NULL (reductions only). */
void orc_bn_bwd(long m, int C, const double *x, const double *dy, const double *gamma,
                const double *mean, const double *rstd,
                double *dgamma, double *dbeta, double *dx)
{
    #pragma omp parallel for schedule(static)
    for (int c = 0; c < C; c++) {
        double sb = 0.0, sg = 0.0;
        for (long i = 0; i < m; i++) {
            double xh = (x[i * C + c] - mean[c]) * rstd[c];
            sb += dy[i * C + c];
            sg += dy[i * C + c] * xh;
        }
        dbeta[c] = sb; dgamma[c] = sg;
        if (dx)
            for (long i = 0; i < m; i++) {
                double xh = (x[i * C + c] - mean[c]) * rstd[c];
                dx[i * C + c] = gamma[c] * rstd[c] *
                                (dy[i * C + c] - sb / (double)m - xh * sg / (double)m);
            }
    }
}

/* ---------------------------------------------------------------- ReLU ---- */

void orc_relu_fwd(long len, const double *y, double *z)
{
    #pragma omp parallel for schedule(static)
    for (long i = 0; i < len; i++) z[i] = y[i] > 0.0 ? y[i] : 0.0;
}

/* dy = dz where y > 0, else 0 (gradient 0 at y == 0). */
void orc_relu_bwd(long len, const double *dz, const double *y, double *dy)
{
    #pragma omp parallel for schedule(static)
    for (long i = 0; i < len; i++) dy[i] = y[i] > 0.0 ? dz[i] : 0.0;
}

/* ------------------------------------------------------------- pooling ---- */

/* 2x2 average pooling, stride 2 (DenseNet transition); H, W even. */
void orc_avgpool2_fwd(int N, int H, int W, int C, const double *in, double *out)
{
    int Ho = H / 2, Wo = W / 2;
    #pragma omp parallel for collapse(3) schedule(static)
    for (int n = 0; n < N; n++)
        for (int oy = 0; oy < Ho; oy++)
            for (int ox = 0; ox < Wo; ox++)
                for (int c = 0; c < C; c++)
                    out[IDX4(n, oy, ox, c, Ho, Wo, C)] =
                        0.25 * (in[IDX4(n, 2 * oy, 2 * ox, c, H, W, C)] +
                                in[IDX4(n, 2 * oy, 2 * ox + 1, c, H, W, C)] +
                                in[IDX4(n, 2 * oy + 1, 2 * ox, c, H, W, C)] +
                                in[IDX4(n, 2 * oy + 1, 2 * ox + 1, c, H, W, C)]);
}

void orc_avgpool2_bwd(int N, int H, int W, int C, const double *gout, double *gin)
{
    int Ho = H / 2, Wo = W / 2;
    #pragma omp parallel for collapse(3) schedule(static)
    for (int n = 0; n < N; n++)
        for (int iy = 0; iy < H; iy++)
            for (int ix = 0; ix < W; ix++)
                for (int c = 0; c < C; c++)
                    gin[IDX4(n, iy, ix, c, H, W, C)] = 0.25 * gout[IDX4(n, iy / 2, ix / 2, c, Ho, Wo, C)];
}

/* K x K max pooling with stride and zero-extent padding (padded taps never win). */
void orc_maxpool_fwd(int N, int H, int W, int C, int K, int stride, int pad,
                     const double *in, double *out)
{
    int Ho = out_dim(H, K, stride, pad), Wo = out_dim(W, K, stride, pad);
    #pragma omp parallel for collapse(3) schedule(static)
    for (int n = 0; n < N; n++)
        for (int oy = 0; oy < Ho; oy++)
            for (int ox = 0; ox < Wo; ox++)
                for (int c = 0; c < C; c++) {
                    double best = -INFINITY;
                    for (int kh = 0; kh < K; kh++)
                        for (int kw = 0; kw < K; kw++) {
                            int iy = oy * stride + kh - pad, ix = ox * stride + kw - pad;
                            if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;
                            double v = in[IDX4(n, iy, ix, c, H, W, C)];
                            if (v > best) best = v;
                        }
                    out[IDX4(n, oy, ox, c, Ho, Wo, C)] = best;
                }
}

/* Routes each output gradient to the first maximum of its window in row-major
 * tap order (parallel over images: windows overlap within an image). */
void orc_maxpool_bwd(int N, int H, int W, int C, int K, int stride, int pad,
                     const double *in, const double *gout, double *gin)
{
    int Ho = out_dim(H, K, stride, pad), Wo = out_dim(W, K, stride, pad);
    #pragma omp parallel for schedule(static)
    for (int n = 0; n < N; n++) {
        memset(gin + IDX4(n, 0, 0, 0, H, W, C), 0, sizeof(double) * (size_t)H * W * C);
        for (int oy = 0; oy < Ho; oy++)
            for (int ox = 0; ox < Wo; ox++)
                for (int c = 0; c < C; c++) {
                    double best = -INFINITY; long arg = -1;
                    for (int kh = 0; kh < K; kh++)
                        for (int kw = 0; kw < K; kw++) {
                            int iy = oy * stride + kh - pad, ix = ox * stride + kw - pad;
                            if (iy < 0 || iy >= H || ix < 0 || ix >= W) continue;
                            long j = IDX4(n, iy, ix, c, H, W, C);
                            if (in[j] > best) { best = in[j]; arg = j; }
                        }
                    gin[arg] += gout[IDX4(n, oy, ox, c, Ho, Wo, C)];
                }
    }
}

/* ------------------------------------------------------------ utilities ---- */

/* Round each value to the nearest bfloat16 (8 significant bits, fp32 exponent
 * range), ties to even.  Models storage of a tensor in bf16. */
void orc_round_bf16(long len, double *a)
{
    const double min_normal = ldexp(1.0, -126);
    const double max_finite = ldexp(255.0, 120);          /* (2 - 2^-7) * 2^127 */
    #pragma omp parallel for schedule(static)
    for (long i = 0; i < len; i++) {
        double v = a[i];
        if (v == 0.0 || isnan(v) || isinf(v)) continue;
        double r;
        if (fabs(v) < min_normal) {
            r = ldexp(nearbyint(ldexp(v, 133)), -133);       /* subnormal spacing 2^-133 */
        } else {
            int e;
            double f = frexp(v, &e);                          /* v = f * 2^e, 0.5 <= |f| < 1 */
            r = ldexp(nearbyint(ldexp(f, 8)), e - 8);         /* keep 8 significant bits */
        }
        if (fabs(r) > max_finite) r = v > 0 ? INFINITY : -INFINITY;
        a[i] = r;
    }
}
