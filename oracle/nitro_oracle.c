/*
 * CPU oracle for the NITRO-D integer training step: the GEMM-shaped contractions.
 *
 * TEST INFRASTRUCTURE ONLY. Nothing in the product path may link, load or call this file; only
 * the tests, the smoke check and the CPU-baseline leg of the benchmark do.
 *
 * Every function is the plain definition written out with int64 accumulators: no blocking, no
 * limb splitting, no fused epilogue. OpenMP parallelises an outer loop only; each output element
 * is owned by exactly one thread, so the sums are exact and the results do not depend on the
 * thread count. Layouts: activations and gradients NHWC, conv weights KRSC
 * [C_out][3][3][C_in], linear weights [out][in].
 *
 * Conv3x3 is the IntConv2D of section 3.2.1 (the sum over input channels j and kernel taps k of
 * a^{jk} W^{ijk}) with the Tab. 1 configuration: 3x3 kernel, stride 1, zero padding 1, no bias.
 * Linear is the IntLinear of section 3.2.1 (z^i = sum_j a^j W^{ij}).
 * The input- and weight-gradient contractions are the adjoints of those two maps: the paper uses
 * them implicitly when it back-propagates delta^{fw} through the forward layers (section 3.3,
 * training procedure) and when IntegerSGD consumes the weight gradient (Alg. 1).
 */
#include <stdint.h>

/* z[n][h][w][co] = sum_{r,s in 0..2} sum_ci x[n][h+r-1][w+s-1][ci] * W[co][r][s][ci]
 * (terms whose input position falls outside the image are zero: padding 1). */
void or_conv3x3_fwd(const int8_t *x, const int32_t *wt, int64_t *z,
                    int N, int H, int W, int C, int CO)
{
    #pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; n++)
        for (int h = 0; h < H; h++)
            for (int w = 0; w < W; w++)
                for (int co = 0; co < CO; co++) {
                    int64_t acc = 0;
                    for (int r = 0; r < 3; r++) {
                        int hh = h + r - 1;
                        if (hh < 0 || hh >= H) continue;
                        for (int s = 0; s < 3; s++) {
                            int ww = w + s - 1;
                            if (ww < 0 || ww >= W) continue;
                            const int8_t *xp = x + (((int64_t)n * H + hh) * W + ww) * C;
                            const int32_t *wp = wt + (((int64_t)co * 3 + r) * 3 + s) * C;
                            for (int ci = 0; ci < C; ci++)
                                acc += (int64_t)xp[ci] * (int64_t)wp[ci];
                        }
                    }
                    z[(((int64_t)n * H + h) * W + w) * CO + co] = acc;
                }
}

/* Input gradient, the adjoint of or_conv3x3_fwd:
 * dx[n][h][w][ci] = sum_{r,s} sum_co g[n][h-r+1][w-s+1][co] * W[co][r][s][ci]
 * (output positions outside the image contribute nothing). */
void or_conv3x3_dx(const int64_t *g, const int32_t *wt, int64_t *dx,
                   int N, int H, int W, int C, int CO)
{
    #pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; n++)
        for (int h = 0; h < H; h++)
            for (int w = 0; w < W; w++) {
                int64_t *out = dx + (((int64_t)n * H + h) * W + w) * C;
                for (int ci = 0; ci < C; ci++) out[ci] = 0;
                for (int r = 0; r < 3; r++) {
                    int ho = h - r + 1;
                    if (ho < 0 || ho >= H) continue;
                    for (int s = 0; s < 3; s++) {
                        int wo = w - s + 1;
                        if (wo < 0 || wo >= W) continue;
                        const int64_t *gp = g + (((int64_t)n * H + ho) * W + wo) * CO;
                        for (int co = 0; co < CO; co++) {
                            const int64_t gv = gp[co];
                            const int32_t *wp = wt + (((int64_t)co * 3 + r) * 3 + s) * C;
                            for (int ci = 0; ci < C; ci++)
                                out[ci] += gv * (int64_t)wp[ci];
                        }
                    }
                }
            }
}

/* Weight gradient summed over the batch:
 * dW[co][r][s][ci] = sum_{n,h,w} g[n][h][w][co] * x[n][h+r-1][w+s-1][ci]. */
void or_conv3x3_dw(const int64_t *g, const int8_t *x, int64_t *dw,
                   int N, int H, int W, int C, int CO)
{
    #pragma omp parallel for schedule(dynamic, 1)
    for (int co = 0; co < CO; co++) {
        int64_t *out = dw + (int64_t)co * 9 * C;
        for (int i = 0; i < 9 * C; i++) out[i] = 0;
        for (int n = 0; n < N; n++)
            for (int h = 0; h < H; h++)
                for (int w = 0; w < W; w++) {
                    const int64_t gv = g[(((int64_t)n * H + h) * W + w) * CO + co];
                    for (int r = 0; r < 3; r++) {
                        int hh = h + r - 1;
                        if (hh < 0 || hh >= H) continue;
                        for (int s = 0; s < 3; s++) {
                            int ww = w + s - 1;
                            if (ww < 0 || ww >= W) continue;
                            const int8_t *xp = x + (((int64_t)n * H + hh) * W + ww) * C;
                            int64_t *op = out + (r * 3 + s) * C;
                            for (int ci = 0; ci < C; ci++)
                                op[ci] += gv * (int64_t)xp[ci];
                        }
                    }
                }
    }
}

/* z[n][m] = sum_k x[n][k] * W[m][k]. */
void or_linear_fwd(const int8_t *x, const int32_t *wt, int64_t *z, int N, int K, int M)
{
    #pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; n++)
        for (int m = 0; m < M; m++) {
            int64_t acc = 0;
            const int8_t *xp = x + (int64_t)n * K;
            const int32_t *wp = wt + (int64_t)m * K;
            for (int k = 0; k < K; k++) acc += (int64_t)xp[k] * (int64_t)wp[k];
            z[(int64_t)n * M + m] = acc;
        }
}

/* Input gradient of the linear map: dx[n][k] = sum_m e[n][m] * W[m][k]. */
void or_linear_dx(const int64_t *e, const int32_t *wt, int64_t *dx, int N, int K, int M)
{
    #pragma omp parallel for schedule(static)
    for (int n = 0; n < N; n++) {
        int64_t *out = dx + (int64_t)n * K;
        for (int k = 0; k < K; k++) out[k] = 0;
        for (int m = 0; m < M; m++) {
            const int64_t ev = e[(int64_t)n * M + m];
            const int32_t *wp = wt + (int64_t)m * K;
            for (int k = 0; k < K; k++) out[k] += ev * (int64_t)wp[k];
        }
    }
}

/* Weight gradient of the linear map summed over the batch: dW[m][k] = sum_n e[n][m] * x[n][k]. */
void or_linear_dw(const int64_t *e, const int8_t *x, int64_t *dw, int N, int K, int M)
{
    #pragma omp parallel for schedule(static)
    for (int m = 0; m < M; m++) {
        int64_t *out = dw + (int64_t)m * K;
        for (int k = 0; k < K; k++) out[k] = 0;
        for (int n = 0; n < N; n++) {
            const int64_t ev = e[(int64_t)n * M + m];
            const int8_t *xp = x + (int64_t)n * K;
            for (int k = 0; k < K; k++) out[k] += ev * (int64_t)xp[k];
        }
    }
}

/* Number of OpenMP threads a parallel region uses (for reporting the CPU baseline). */
int or_num_threads(void)
{
    int n = 1;
    #pragma omp parallel
    {
        #pragma omp single
        {
#ifdef _OPENMP
            extern int omp_get_num_threads(void);
            n = omp_get_num_threads();
#endif
        }
    }
    return n;
}
