// 3x3 convolutions whose input has few channels (the first layer of an image network: 1 or 3
// channels), where K = 9 * C_in is too short for the MFMA tiles. Exact int64 VALU arithmetic.
#include "nitro_internal.h"

namespace nitro {

constexpr int SC_MAX_K = 64;             // 9 * C_in <= 64 (C_in <= 7)
constexpr int SC_MAX_W = 8192;           // int32 words of W kept in LDS

bool smallc_fwd_ok(const ConvShape &sh)
{
    return sh.c >= 1 && sh.c <= 4 && 9 * sh.c * sh.co <= SC_MAX_W && sh.co % 4 == 0;
}

// One thread per (output pixel, 4 output channels); with POOL one thread per (pooled pixel,
// 4 channels) visiting the 2x2 window in row-major order (first maximum wins).
template <int CIN, bool POOL>
__global__ __launch_bounds__(256) void k_conv_fwd_smallc(ConvShape sh, const int8_t *__restrict__ x,
                                                         const int32_t *__restrict__ w, Div sf,
                                                         Relu rp, int8_t *__restrict__ out,
                                                         uint8_t *__restrict__ code)
{
    __shared__ int32_t Ws[SC_MAX_W];
    constexpr int K = 9 * CIN;
    for (int i = threadIdx.x; i < K * sh.co; i += blockDim.x) Ws[i] = w[i];
    __syncthreads();
    const int cg = sh.co / 4;
    const int OH = POOL ? sh.h / 2 : sh.h, OW = POOL ? sh.w / 2 : sh.w;
    const int64_t total = (int64_t)sh.n * OH * OW * cg;
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total) return;
    const int c4 = (int)(i % cg) * 4;
    const int64_t op = i / cg;
    const int oq = (int)(op % OW), oh = (int)((op / OW) % OH);
    const int n = (int)(op / ((int64_t)OW * OH));
    int best[4] = {-1000, -1000, -1000, -1000}, arg[4] = {0, 0, 0, 0};
    uint8_t breg[4] = {0, 0, 0, 0};
#pragma unroll
    for (int t = 0; t < (POOL ? 4 : 1); t++) {
        const int h = POOL ? 2 * oh + (t >> 1) : oh, q = POOL ? 2 * oq + (t & 1) : oq;
        int32_t patch[K];
        for (int r = 0; r < 3; r++)
            for (int s = 0; s < 3; s++) {
                const int hh = h + r - 1, ww = q + s - 1;
                const bool ok = hh >= 0 && hh < sh.h && ww >= 0 && ww < sh.w;
                const int8_t *xp = x + (((int64_t)n * sh.h + hh) * sh.w + ww) * CIN;
                for (int c = 0; c < CIN; c++) patch[(r * 3 + s) * CIN + c] = ok ? xp[c] : 0;
            }
#pragma unroll
        for (int u = 0; u < 4; u++) {
            const int32_t *wr = Ws + (c4 + u) * K;
            int64_t z = 0;
            for (int k = 0; k < K; k++) z += (int64_t)patch[k] * wr[k];
            uint8_t reg;
            const int32_t a = relu_fwd(idiv(z, sf), rp, reg);
            if (a > best[u]) { best[u] = a; arg[u] = t; breg[u] = reg; }
        }
    }
    uint32_t av = 0, cv = 0;
#pragma unroll
    for (int u = 0; u < 4; u++) {
        av |= (uint32_t)(uint8_t)(int8_t)best[u] << (8 * u);
        cv |= (uint32_t)(POOL ? (arg[u] | (breg[u] << 2)) : breg[u]) << (8 * u);
    }
    *(uint32_t *)(out + op * sh.co + c4) = av;
    *(uint32_t *)(code + op * sh.co + c4) = cv;
}

void launch_conv_fwd_smallc(hipStream_t s, const ConvShape &sh, const int8_t *x, const int32_t *w,
                            const Div &sf, const Relu &rp, bool pool, int8_t *out, uint8_t *code)
{
    const int OH = pool ? sh.h / 2 : sh.h, OW = pool ? sh.w / 2 : sh.w;
    const int64_t total = (int64_t)sh.n * OH * OW * (sh.co / 4);
    const dim3 grid((unsigned)((total + 255) / 256));
#define NITRO_SMALLC_CASE(C)                                                                     \
    case C:                                                                                      \
        if (pool)                                                                                \
            hipLaunchKernelGGL((k_conv_fwd_smallc<C, true>), grid, dim3(256), 0, s, sh, x, w, sf, \
                               rp, out, code);                                                   \
        else                                                                                     \
            hipLaunchKernelGGL((k_conv_fwd_smallc<C, false>), grid, dim3(256), 0, s, sh, x, w, sf,\
                               rp, out, code);                                                   \
        break;
    switch (sh.c) {
        NITRO_SMALLC_CASE(1)
        NITRO_SMALLC_CASE(2)
        NITRO_SMALLC_CASE(3)
        NITRO_SMALLC_CASE(4)
    }
#undef NITRO_SMALLC_CASE
}

// ---------------------------------------------------------------------------------------------
// Weight gradient for few input channels: dW[co][t][ci] = sum_p g[p][co] x[p + shift_t][ci].
// A workgroup sums a chunk of pixels: g rows [pixels][co] and the input patches [pixels][9 ci]
// are staged in LDS; thread (co, column group) keeps SC_COLS int64 partial sums; the chunk's
// partials go to dW with int64 atomics.
constexpr int SC_PIX = 32;               // pixels staged per step
constexpr int SC_COLS = 8;               // (tap, ci) columns per thread

bool smallc_dw_ok(const ConvShape &sh)
{
    const int ngrp = (9 * sh.c + SC_COLS - 1) / SC_COLS;
    return 9 * sh.c <= SC_MAX_K && sh.co <= 256 && sh.co * ngrp <= 1024 &&
           (int64_t)sh.n * sh.h * sh.w < ((int64_t)1 << 31);
}

__global__ __launch_bounds__(256) void k_conv_dw_smallc(ConvShape sh, int chunk,
                                                        const int32_t *__restrict__ g,
                                                        const int8_t *__restrict__ x,
                                                        int64_t *__restrict__ part)
{
    __shared__ int32_t Gs[SC_PIX][256];
    __shared__ int32_t Xs[SC_PIX][SC_MAX_K];
    const int K = 9 * sh.c;
    const int ngrp = (K + SC_COLS - 1) / SC_COLS;
    const int P = sh.n * sh.h * sh.w;
    const int HW = sh.h * sh.w;
    const int p0 = blockIdx.x * chunk;
    const int p1 = p0 + chunk < P ? p0 + chunk : P;
    // work items: (co, column group); 256 threads stride over co * ngrp of them
    const int items = sh.co * ngrp;
    constexpr int MAXI = 4;                 // items per thread (co * ngrp <= 1024)
    int64_t acc[MAXI][SC_COLS];
#pragma unroll
    for (int a = 0; a < MAXI; a++)
#pragma unroll
        for (int b = 0; b < SC_COLS; b++) acc[a][b] = 0;
    for (int pb = p0; pb < p1; pb += SC_PIX) {
        __syncthreads();
        for (int e = threadIdx.x; e < SC_PIX * sh.co; e += 256) {
            const int pi = e / sh.co, co = e % sh.co;
            const int pp = pb + pi;
            Gs[pi][co] = pp < p1 ? g[(int64_t)pp * sh.co + co] : 0;
        }
        for (int e = threadIdx.x; e < SC_PIX * K; e += 256) {
            const int pi = e / K, k = e % K;
            const int pp = pb + pi;
            const int t = k / sh.c, c = k % sh.c;
            const int rem = pp % HW;
            const int hh = rem / sh.w + t / 3 - 1, ww = rem % sh.w + t % 3 - 1;
            const bool ok = pp < p1 && hh >= 0 && hh < sh.h && ww >= 0 && ww < sh.w;
            Xs[pi][k] = ok ? x[((int64_t)pp + (t / 3 - 1) * sh.w + (t % 3 - 1)) * sh.c + c] : 0;
        }
        __syncthreads();
#pragma unroll
        for (int a = 0; a < MAXI; a++) {
            const int item = threadIdx.x + 256 * a;
            if (item < items) {
                const int co = item / ngrp, c0 = (item % ngrp) * SC_COLS;
                for (int pi = 0; pi < SC_PIX; pi++) {
                    const int64_t gv = Gs[pi][co];
#pragma unroll
                    for (int b = 0; b < SC_COLS; b++)
                        if (c0 + b < K) acc[a][b] += gv * Xs[pi][c0 + b];
                }
            }
        }
    }
    int64_t *dst = part + (int64_t)blockIdx.x * sh.co * K;
#pragma unroll
    for (int a = 0; a < MAXI; a++) {
        const int item = threadIdx.x + 256 * a;
        if (item < items) {
            const int co = item / ngrp, c0 = (item % ngrp) * SC_COLS;
#pragma unroll
            for (int b = 0; b < SC_COLS; b++)
                if (c0 + b < K) dst[(int64_t)co * K + c0 + b] = acc[a][b];
        }
    }
}

static void smallc_dw_split(const ConvShape &sh, int64_t *nb_out, int64_t *chunk_out)
{
    const int64_t P = (int64_t)sh.n * sh.h * sh.w;
    int64_t nb = 128;
    int64_t chunk = (P + nb - 1) / nb;
    chunk = (chunk + SC_PIX - 1) / SC_PIX * SC_PIX;
    *chunk_out = chunk;
    *nb_out = (P + chunk - 1) / chunk;
}

int64_t smallc_dw_partial_count(const ConvShape &sh)
{
    int64_t nb, chunk;
    smallc_dw_split(sh, &nb, &chunk);
    return nb * sh.co * 9 * sh.c;
}

void launch_conv_dw_smallc(hipStream_t s, const ConvShape &sh, const int32_t *g, const int8_t *x,
                           int64_t *part, int64_t *dw)
{
    int64_t nb, chunk;
    smallc_dw_split(sh, &nb, &chunk);
    hipLaunchKernelGGL(k_conv_dw_smallc, dim3((unsigned)nb), dim3(256), 0, s, sh, (int)chunk, g, x,
                       part);
    launch_sum_partials(s, part, (int)nb, (int64_t)sh.co * 9 * sh.c, dw);
}

}  // namespace nitro
