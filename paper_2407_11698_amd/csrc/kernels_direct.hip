// Direct (non-MFMA) integer kernels for gfx950: elementwise passes, the skinny linear layers,
// and direct convolutions for layers whose channel counts are too small for the MFMA tiles.
// All accumulation is exact: int64 where a sum can leave int32.
#include "mfma_common.h"

namespace nitro {

static inline unsigned blocks_for(int64_t n, int per) { return (unsigned)((n + per - 1) / per); }

// ---------------------------------------------------------------------------------------------
__global__ void k_fill_i64(int64_t *p, int64_t count)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < count; i += stride) p[i] = 0;
}

void launch_fill_i64(hipStream_t s, int64_t *p, int64_t count)
{
    if (count <= 0) return;
    unsigned g = blocks_for(count, 256);
    if (g > 8192) g = 8192;
    hipLaunchKernelGGL(k_fill_i64, dim3(g), dim3(256), 0, s, p, count);
}

// Each workgroup: 64 consecutive outputs x 4 groups of partials (group q adds z = q, q + 4, ...),
// the groups' sums added in LDS in a fixed order (integer addition: the order does not matter).
__global__ __launch_bounds__(256) void k_sum_partials(const int64_t *__restrict__ part, int nz,
                                                      int64_t count, int64_t *__restrict__ out)
{
    __shared__ int64_t red[4][64];
    const int il = threadIdx.x & 63, q = threadIdx.x >> 6;
    const int64_t i = (int64_t)blockIdx.x * 64 + il;
    int64_t v = 0;
    if (i < count) {
        int z = q;
        for (; z + 12 < nz; z += 16)
            v += part[(int64_t)z * count + i] + part[(int64_t)(z + 4) * count + i] +
                 part[(int64_t)(z + 8) * count + i] + part[(int64_t)(z + 12) * count + i];
        for (; z < nz; z += 4) v += part[(int64_t)z * count + i];
    }
    red[q][il] = v;
    __syncthreads();
    if (q == 0 && i < count) out[i] = red[0][il] + red[1][il] + red[2][il] + red[3][il];
}

void launch_sum_partials(hipStream_t s, const int64_t *part, int nz, int64_t count, int64_t *out)
{
    if (count <= 0) return;
    hipLaunchKernelGGL(k_sum_partials, dim3((unsigned)((count + 63) / 64)), dim3(256), 0, s, part,
                       nz, count, out);
}

// Split-K sums of a conv weight gradient [co][3][3][ci] whose planes may hold g - 128 (offset
// form, max|g| in its range): output (o, r, s, c) then adds 128 S with
// S = sum_{p inside the image} x[p + (r-1, s-1)][c], from the sums xq [9][ci] of x over every
// pixel, the rows h = 0 and H-1, the columns w = 0 and W-1 and the four corners by
// inclusion-exclusion: the tap excludes row 0 when r = 2 (no p above it), row H-1 when r = 0,
// column 0 when s = 2, column W-1 when s = 0.
__global__ __launch_bounds__(256) void k_sum_partials_goff(const int64_t *__restrict__ part, int nz,
                                                           int64_t count, int64_t *__restrict__ out,
                                                           const int32_t *__restrict__ xq, int ci,
                                                           const uint32_t *gmax)
{
    __shared__ int64_t red[4][64];
    const bool off = goff_range(slot_read(gmax));
    const int il = threadIdx.x & 63, q = threadIdx.x >> 6;
    const int64_t i = (int64_t)blockIdx.x * 64 + il;
    int64_t v = 0;
    if (i < count) {
        int z = q;
        for (; z + 12 < nz; z += 16)
            v += part[(int64_t)z * count + i] + part[(int64_t)(z + 4) * count + i] +
                 part[(int64_t)(z + 8) * count + i] + part[(int64_t)(z + 12) * count + i];
        for (; z < nz; z += 4) v += part[(int64_t)z * count + i];
    }
    red[q][il] = v;
    __syncthreads();
    if (q != 0 || i >= count) return;
    int64_t sum = red[0][il] + red[1][il] + red[2][il] + red[3][il];
    if (off) {
        const int c = (int)(i % ci), t = (int)((i / ci) % 9);
        const int r = t / 3, sc = t % 3;
        const int32_t *Q = xq + c;
        int64_t S = Q[0];
        if (r == 2) S -= Q[ci];                       // row 0
        if (r == 0) S -= Q[2 * ci];                   // row H-1
        if (sc == 2) S -= Q[3 * ci];                  // column 0
        if (sc == 0) S -= Q[4 * ci];                  // column W-1
        if (r == 2 && sc == 2) S += Q[5 * ci];        // (0, 0)
        if (r == 2 && sc == 0) S += Q[6 * ci];        // (0, W-1)
        if (r == 0 && sc == 2) S += Q[7 * ci];        // (H-1, 0)
        if (r == 0 && sc == 0) S += Q[8 * ci];        // (H-1, W-1)
        sum += (int64_t)GOFF_BIAS * S;
    }
    out[i] = sum;
}

void launch_sum_partials_goff(hipStream_t s, const int64_t *part, int nz, int64_t count,
                              int64_t *out, const int32_t *xq, int ci, const uint32_t *gmax)
{
    if (count <= 0) return;
    hipLaunchKernelGGL(k_sum_partials_goff, dim3((unsigned)((count + 63) / 64)), dim3(256), 0, s, part,
                       nz, count, out, xq, ci, gmax);
}

// ---------------------------------------------------------------------------------------------
// Direct 3x3 conv, stride 1, zero padding 1: z[n][h][w][co] = sum_{r,s,ci} x[..][h+r-1][w+s-1][ci]
// * W[co][r][s][ci], then NITRO-Scaling and NITRO-ReLU.
__device__ inline int64_t conv_point(const int8_t *x, const int32_t *w, int n, int h, int q,
                                     int co, const ConvShape &sh)
{
    int64_t acc = 0;
    for (int r = 0; r < 3; r++) {
        int hh = h + r - 1;
        if (hh < 0 || hh >= sh.h) continue;
        for (int s = 0; s < 3; s++) {
            int ww = q + s - 1;
            if (ww < 0 || ww >= sh.w) continue;
            const int8_t *xp = x + (((int64_t)n * sh.h + hh) * sh.w + ww) * sh.c;
            const int32_t *wp = w + (((int64_t)co * 3 + r) * 3 + s) * sh.c;
            for (int ci = 0; ci < sh.c; ci++) acc += (int64_t)xp[ci] * (int64_t)wp[ci];
        }
    }
    return acc;
}

__global__ void k_conv_fwd_direct(ConvShape sh, const int8_t *__restrict__ x,
                                  const int32_t *__restrict__ w, Div sf, Relu rp,
                                  int8_t *__restrict__ out, uint8_t *__restrict__ code)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t total = (int64_t)sh.n * sh.h * sh.w * sh.co;
    if (i >= total) return;
    int co = (int)(i % sh.co);
    int64_t p = i / sh.co;
    int q = (int)(p % sh.w);
    int h = (int)((p / sh.w) % sh.h);
    int n = (int)(p / ((int64_t)sh.w * sh.h));
    int64_t z = conv_point(x, w, n, h, q, co, sh);
    uint8_t reg;
    int32_t a = relu_fwd(idiv(z, sf), rp, reg);
    out[i] = (int8_t)a;
    code[i] = reg;
}

// Pooled variant: one thread per pooled output; the 2x2 window is visited in row-major order
// and the first maximum wins.
__global__ void k_conv_fwd_direct_pool(ConvShape sh, const int8_t *__restrict__ x,
                                       const int32_t *__restrict__ w, Div sf, Relu rp,
                                       int8_t *__restrict__ out, uint8_t *__restrict__ code)
{
    int H2 = sh.h / 2, W2 = sh.w / 2;
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t total = (int64_t)sh.n * H2 * W2 * sh.co;
    if (i >= total) return;
    int co = (int)(i % sh.co);
    int64_t p = i / sh.co;
    int q2 = (int)(p % W2);
    int h2 = (int)((p / W2) % H2);
    int n = (int)(p / ((int64_t)W2 * H2));
    int best = -1000, arg = 0;
    uint8_t breg = 0;
    for (int t = 0; t < 4; t++) {
        int h = 2 * h2 + (t >> 1), q = 2 * q2 + (t & 1);
        int64_t z = conv_point(x, w, n, h, q, co, sh);
        uint8_t reg;
        int32_t a = relu_fwd(idiv(z, sf), rp, reg);
        if (a > best) { best = a; arg = t; breg = reg; }
    }
    out[i] = (int8_t)best;
    code[i] = (uint8_t)(arg | (breg << 2));
}

void launch_conv_fwd(hipStream_t s, const ConvShape &sh, const int8_t *x, const int32_t *w,
                     const Div &sf, const Relu &rp, bool pool, int8_t *out, uint8_t *code)
{
    if (pool) {
        int64_t total = (int64_t)sh.n * (sh.h / 2) * (sh.w / 2) * sh.co;
        hipLaunchKernelGGL(k_conv_fwd_direct_pool, dim3(blocks_for(total, 256)), dim3(256), 0, s,
                           sh, x, w, sf, rp, out, code);
    } else {
        int64_t total = (int64_t)sh.n * sh.h * sh.w * sh.co;
        hipLaunchKernelGGL(k_conv_fwd_direct, dim3(blocks_for(total, 256)), dim3(256), 0, s,
                           sh, x, w, sf, rp, out, code);
    }
}

// ---------------------------------------------------------------------------------------------
// Linear forward, one wavefront per output element: lanes stride over k, then a wave reduction.
__device__ inline int64_t wave_sum_i64(int64_t v)
{
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    return v;
}

__device__ inline int64_t linear_point(const int8_t *x, const int32_t *w, int k, int lane)
{
    int64_t acc = 0;
    if ((k & 3) == 0) {
        // (rows of a multiple of 4: each lane takes 4 inputs per step, one dword of x and four
        // weights in one 16-byte load; four steps' loads requested together)
#pragma unroll 4
        for (int t = lane; t < (k >> 2); t += 64) {
            const int xv = *(const int *)(x + 4 * t);
            const v4i wv = *(const v4i *)(w + 4 * t);
            acc += (int64_t)(int8_t)xv * wv[0] + (int64_t)(int8_t)(xv >> 8) * wv[1] +
                   (int64_t)(int8_t)(xv >> 16) * wv[2] + (int64_t)(xv >> 24) * wv[3];
        }
    } else {
        for (int t = lane; t < k; t += 64) acc += (int64_t)x[t] * (int64_t)w[t];
    }
    return wave_sum_i64(acc);
}

__global__ void k_linear_fwd_relu(int n, int k, int m, const int8_t *__restrict__ x,
                                  const int32_t *__restrict__ w, Div sf, Relu rp,
                                  int8_t *__restrict__ out, uint8_t *__restrict__ code)
{
    int64_t o = (int64_t)blockIdx.x * (blockDim.x / 64) + threadIdx.x / 64;
    int lane = threadIdx.x & 63;
    if (o >= (int64_t)n * m) return;
    int row = (int)(o / m), col = (int)(o % m);
    int64_t z = linear_point(x + (int64_t)row * k, w + (int64_t)col * k, k, lane);
    if (lane == 0) {
        uint8_t reg;
        int32_t a = relu_fwd(idiv(z, sf), rp, reg);
        out[o] = (int8_t)a;
        code[o] = reg;
    }
}

void launch_linear_fwd_relu(hipStream_t s, int n, int k, int m, const int8_t *x, const int32_t *w,
                            const Div &sf, const Relu &rp, int8_t *out, uint8_t *code)
{
    int64_t outs = (int64_t)n * m;
    hipLaunchKernelGGL(k_linear_fwd_relu, dim3(blocks_for(outs, 4)), dim3(256), 0, s,
                       n, k, m, x, w, sf, rp, out, code);
}

__global__ void k_linear_fwd_loss(int n, int k, int g, const int8_t *__restrict__ x,
                                  const int32_t *__restrict__ w, Div sf,
                                  const int32_t *__restrict__ labels, int32_t *__restrict__ yhat,
                                  int32_t *__restrict__ e, uint32_t *flags)
{
    int64_t o = (int64_t)blockIdx.x * (blockDim.x / 64) + threadIdx.x / 64;
    int lane = threadIdx.x & 63;
    if (o >= (int64_t)n * g) return;
    int row = (int)(o / g), col = (int)(o % g);
    int64_t z = linear_point(x + (int64_t)row * k, w + (int64_t)col * k, k, lane);
    if (lane == 0) {
        int64_t y = idiv(z, sf);
        if (!fits_i32(y)) raise_flag(flags, FLAG_OVERFLOW);
        yhat[o] = (int32_t)y;
        if (labels) {            // training: the loss gradient too (inference passes no labels)
            int lab = labels[row];
            if (lab < 0 || lab >= g) raise_flag(flags, FLAG_LABEL);
            int64_t ev = y - (lab == col ? 32 : 0);
            if (!fits_i32(ev)) raise_flag(flags, FLAG_OVERFLOW);
            e[o] = (int32_t)ev;
        }
    }
}

// pred[r] = the first column of row r holding the row's maximum (one wave per row).
__global__ void k_argmax_rows(int n, int g, const int32_t *__restrict__ yhat, int32_t *__restrict__ pred)
{
    const int row = blockIdx.x * (blockDim.x / 64) + threadIdx.x / 64;
    const int lane = threadIdx.x & 63;
    if (row >= n) return;
    int32_t best = INT32_MIN;
    int arg = g;
    for (int c = lane; c < g; c += 64) {
        const int32_t v = yhat[(int64_t)row * g + c];
        if (v > best) {                // strictly greater: a lane keeps its first maximum
            best = v;
            arg = c;
        }
    }
    for (int off = 32; off > 0; off >>= 1) {
        const int32_t ob = __shfl_xor(best, off, 64);
        const int oa = __shfl_xor(arg, off, 64);
        if (ob > best || (ob == best && oa < arg)) {
            best = ob;
            arg = oa;
        }
    }
    if (lane == 0) pred[row] = arg;
}

void launch_argmax_rows(hipStream_t s, int n, int g, const int32_t *yhat, int32_t *pred)
{
    hipLaunchKernelGGL(k_argmax_rows, dim3(blocks_for(n, 4)), dim3(256), 0, s, n, g, yhat, pred);
}

void launch_linear_fwd_loss(hipStream_t s, int n, int k, int g, const int8_t *x, const int32_t *w,
                            const Div &sf, const int32_t *labels, int32_t *yhat, int32_t *e,
                            uint32_t *flags)
{
    int64_t outs = (int64_t)n * g;
    hipLaunchKernelGGL(k_linear_fwd_loss, dim3(blocks_for(outs, 4)), dim3(256), 0, s,
                       n, k, g, x, w, sf, labels, yhat, e, flags);
}

// dx[n][k] = sum_m e[n][m] w[m][k]: one thread per (n, k); lanes along k read w coalesced.
__global__ void k_linear_dx(int n, int k, int m, const int32_t *__restrict__ e,
                            const int32_t *__restrict__ w, const uint8_t *__restrict__ code,
                            Relu rp, int32_t *__restrict__ out, int64_t *__restrict__ out64,
                            uint32_t *flags)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)n * k) return;
    int row = (int)(i / k), col = (int)(i % k);
    const int32_t *er = e + (int64_t)row * m;
    int64_t acc = 0;
    for (int t = 0; t < m; t++) acc += (int64_t)er[t] * (int64_t)w[(int64_t)t * k + col];
    if (out64) {
        out64[i] = acc;
        return;
    }
    bool bad = !fits_i32(acc);
    if (code) {
        acc = relu_bwd(acc, code[i], rp);
        bad |= !fits_i32(acc);
    }
    if (bad) raise_flag(flags, FLAG_OVERFLOW);
    out[i] = (int32_t)acc;
}

void launch_linear_dx(hipStream_t s, int n, int k, int m, const int32_t *e, const int32_t *w,
                      const uint8_t *code, const Relu &rp, int32_t *out, int64_t *out64,
                      uint32_t *flags)
{
    int64_t total = (int64_t)n * k;
    hipLaunchKernelGGL(k_linear_dx, dim3(blocks_for(total, 256)), dim3(256), 0, s,
                       n, k, m, e, w, code, rp, out, out64, flags);
}

// dw[m][k] = sum_n e[n][m] x[n][k]: one thread per (m, k).
__global__ void k_linear_dw(int n, int k, int m, const int32_t *__restrict__ e,
                            const int8_t *__restrict__ x, int64_t *__restrict__ dw)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= (int64_t)m * k) return;
    int row = (int)(i / k), col = (int)(i % k);
    int64_t acc = 0;
    // (unrolled: the loads of 8 samples are requested before their products)
#pragma unroll 8
    for (int t = 0; t < n; t++) acc += (int64_t)e[(int64_t)t * m + row] * (int64_t)x[(int64_t)t * k + col];
    dw[i] = acc;
}

void launch_linear_dw(hipStream_t s, int n, int k, int m, const int32_t *e, const int8_t *x,
                      int64_t *dw)
{
    int64_t total = (int64_t)m * k;
    hipLaunchKernelGGL(k_linear_dw, dim3(blocks_for(total, 256)), dim3(256), 0, s,
                       n, k, m, e, x, dw);
}

// ---------------------------------------------------------------------------------------------
// Gradient at the block output -> gradient at the last layer's z (un-pool + ReLU').
__global__ void k_unpool_relu_bwd(int n, int h, int w, int c, const int32_t *__restrict__ delta,
                                  const uint8_t *__restrict__ code, Relu rp,
                                  int32_t *__restrict__ g, uint32_t *gmax, uint32_t *flags)
{
    // pooled element i = (r * W2 + q2) * c + ch with r = n * H2 + h2 (all indices < 2^31)
    const uint32_t W2 = (uint32_t)w / 2;
    const uint32_t total = (uint32_t)n * ((uint32_t)h / 2) * W2 * (uint32_t)c;
    uint32_t mx = 0;
    bool bad = false;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const uint8_t cd = code[i];
        const int64_t v = relu_bwd(delta[i], (uint8_t)(cd >> 2), rp);
        const uint32_t a = abs_i64_sat(v);
        mx = a > mx ? a : mx;
        bad |= !fits_i32(v);
        const uint32_t ch = i % (uint32_t)c, pp = i / (uint32_t)c;
        const uint32_t q2 = pp % W2, r = pp / W2;
        const int arg = cd & 3;
#pragma unroll
        for (int t = 0; t < 4; t++) {
            const uint32_t pix = (2 * r + (t >> 1)) * (uint32_t)w + 2 * q2 + (t & 1);
            g[(int64_t)pix * c + ch] = t == arg ? (int32_t)v : 0;
        }
    }
    if (bad) raise_flag(flags, FLAG_OVERFLOW);
    if (gmax) block_slot_max(gmax, mx);
}

// g = ReLU'(delta) at the layer's region codes (int32 delta: |g| <= |delta|, so g fits). Four
// elements per thread and step (16 bytes of delta, 4 of codes) when the buffers are 16-byte
// aligned; with g16, g in the escaped 16-bit form (g then receives only the escaped values).
template <bool TR>
__global__ __launch_bounds__(256) void k_relu_bwd(uint32_t count, const int32_t *__restrict__ delta,
                                                  const uint8_t *__restrict__ code, Relu rp,
                                                  int32_t *__restrict__ g, int16_t *__restrict__ g16,
                                                  uint32_t *gmax, int vec)
{
    uint32_t mx = 0;
    const uint32_t stride = gridDim.x * blockDim.x;
    const uint32_t t0 = blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t done = 0;
    if (vec) {
        const uint32_t nq = count / 4;
        for (uint32_t q = t0; q < nq; q += stride) {
            const v4i d = *(const v4i *)(delta + 4 * (size_t)q);
            const uint32_t cd = *(const uint32_t *)(code + 4 * (size_t)q);
            v4i o;
#pragma unroll
            for (int e = 0; e < 4; e++) {
                o[e] = relu_bwd32<TR>(d[e], (cd >> (8 * e)) & 0xffu, rp);
                const uint32_t a = abs_u32(o[e]);
                mx = a > mx ? a : mx;
            }
            if (g16) {
                uint32_t h[4];
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    const bool esc = o[e] < -G16_MAX || o[e] > G16_MAX;
                    if (esc) g[4 * (size_t)q + e] = o[e];
                    h[e] = (uint32_t)(uint16_t)(esc ? G16_ESC : (int16_t)o[e]);
                }
                *(v2i *)(g16 + 4 * (size_t)q) = v2i{(int)(h[0] | (h[1] << 16)), (int)(h[2] | (h[3] << 16))};
            } else {
                *(v4i *)(g + 4 * (size_t)q) = o;
            }
        }
        done = nq * 4;
    }
    for (uint32_t i = done + t0; i < count; i += stride) {
        const int32_t v = relu_bwd32<TR>(delta[i], code[i], rp);
        const uint32_t a = abs_u32(v);
        mx = a > mx ? a : mx;
        if (g16) {
            const bool esc = v < -G16_MAX || v > G16_MAX;
            if (esc) g[i] = v;
            g16[i] = esc ? G16_ESC : (int16_t)v;
        } else {
            g[i] = v;
        }
    }
    if (gmax) block_slot_max(gmax, mx);
}

void launch_unpool_relu_bwd(hipStream_t s, int n, int h, int w, int c, bool pool,
                            const int32_t *delta, const uint8_t *code, const Relu &rp,
                            int32_t *g, uint32_t *gmax, uint32_t *flags, int16_t *g16)
{
    if (pool) {
        int64_t total = (int64_t)n * (h / 2) * (w / 2) * c;
        hipLaunchKernelGGL(k_unpool_relu_bwd, dim3(grid_stride_blocks(total)), dim3(256), 0, s,
                           n, h, w, c, delta, code, rp, g, gmax, flags);
    } else {
        const int64_t total = (int64_t)n * h * w * c;
        const int vec = (((uintptr_t)delta | (uintptr_t)code | (uintptr_t)g | (uintptr_t)g16) & 15) == 0;
        const unsigned nb = grid_stride_blocks(vec ? (total + 3) / 4 : total);
        if (rp.alpha.trunc)
            hipLaunchKernelGGL(k_relu_bwd<true>, dim3(nb), dim3(256), 0, s, (uint32_t)total, delta, code, rp,
                               g, g16, gmax, vec);
        else
            hipLaunchKernelGGL(k_relu_bwd<false>, dim3(nb), dim3(256), 0, s, (uint32_t)total, delta, code,
                               rp, g, g16, gmax, vec);
    }
}

// ---------------------------------------------------------------------------------------------
// Direct conv input gradient: dx[n][h][w][ci] = sum_{r,s,co} g[n][h-r+1][w-s+1][co] W[co][r][s][ci]
// One thread per (pixel, ci): lanes along ci read W coalesced and g as a broadcast.
__global__ void k_conv_dx_direct(ConvShape sh, const int32_t *__restrict__ g,
                                 const int32_t *__restrict__ w, const uint8_t *__restrict__ code,
                                 Relu rp, int32_t *__restrict__ out, int64_t *__restrict__ out64,
                                 uint32_t *gmax, uint32_t *flags)
{
    const int64_t total = (int64_t)sh.n * sh.h * sh.w * sh.c;
    uint32_t mx = 0;
    bool bad = false;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total;
         i += (int64_t)gridDim.x * blockDim.x) {
        const int ci = (int)(i % sh.c);
        const int64_t p = i / sh.c;
        const int q = (int)(p % sh.w);
        const int h = (int)((p / sh.w) % sh.h);
        const int n = (int)(p / ((int64_t)sh.w * sh.h));
        int64_t acc = 0;
        for (int r = 0; r < 3; r++) {
            const int ho = h - r + 1;
            if (ho < 0 || ho >= sh.h) continue;
            for (int s = 0; s < 3; s++) {
                const int wo = q - s + 1;
                if (wo < 0 || wo >= sh.w) continue;
                const int32_t *gp = g + (((int64_t)n * sh.h + ho) * sh.w + wo) * sh.co;
                const int32_t *wp = w + ((int64_t)r * 3 + s) * sh.c + ci;
                for (int co = 0; co < sh.co; co++)
                    acc += (int64_t)gp[co] * (int64_t)wp[(int64_t)co * 9 * sh.c];
            }
        }
        if (out64) {
            out64[i] = acc;
            continue;
        }
        bad |= !fits_i32(acc);
        if (code) {
            acc = relu_bwd(acc, code[i], rp);
            bad |= !fits_i32(acc);
        }
        const uint32_t a = abs_i64_sat(acc);
        mx = a > mx ? a : mx;
        out[i] = (int32_t)acc;
    }
    if (bad) raise_flag(flags, FLAG_OVERFLOW);
    if (gmax) block_slot_max(gmax, mx);
}

void launch_conv_dx(hipStream_t s, const ConvShape &sh, const int32_t *g, const int32_t *w,
                    const uint8_t *code, const Relu &rp, int32_t *out, int64_t *out64,
                    uint32_t *gmax, uint32_t *flags)
{
    int64_t total = (int64_t)sh.n * sh.h * sh.w * sh.c;
    hipLaunchKernelGGL(k_conv_dx_direct, dim3(grid_stride_blocks(total, 256, 8192)), dim3(256), 0,
                       s, sh, g, w, code, rp, out, out64, gmax, flags);
}

// ---------------------------------------------------------------------------------------------
// Direct conv weight gradient: dW[co][r][s][ci] = sum_{n,h,w} g[n][h][w][co] x[n][h+r-1][w+s-1][ci]
// Grid: (k-blocks over (r,s,ci), co, pixel chunks). Each thread owns one (r,s,ci) of one co and
// sums over its chunk of pixels; chunks are combined with int64 atomics (integer addition is
// associative, so the result does not depend on their order).
static const int DW_CHUNK_PIXELS = 4096;

__global__ void k_conv_dw_direct(ConvShape sh, int rows_per_chunk, const int32_t *__restrict__ g,
                                 const int8_t *__restrict__ x, int64_t *__restrict__ dw)
{
    int kk = blockIdx.x * blockDim.x + threadIdx.x;
    if (kk >= 9 * sh.c) return;
    int co = blockIdx.y;
    int rs = kk / sh.c, ci = kk % sh.c;
    int r = rs / 3, s = rs % 3;
    int64_t rows = (int64_t)sh.n * sh.h;
    int64_t r0 = (int64_t)blockIdx.z * rows_per_chunk;
    int64_t r1 = r0 + rows_per_chunk < rows ? r0 + rows_per_chunk : rows;
    int64_t acc = 0;
    for (int64_t row = r0; row < r1; row++) {
        int n = (int)(row / sh.h), h = (int)(row % sh.h);
        int hh = h + r - 1;
        if (hh < 0 || hh >= sh.h) continue;
        const int32_t *grow = g + row * sh.w * sh.co + co;
        const int8_t *xrow = x + (((int64_t)n * sh.h + hh) * sh.w) * sh.c + ci;
        for (int q = 0; q < sh.w; q++) {
            int ww = q + s - 1;
            if (ww < 0 || ww >= sh.w) continue;
            acc += (int64_t)grow[(int64_t)q * sh.co] * (int64_t)xrow[(int64_t)ww * sh.c];
        }
    }
    if (acc != 0)
        atomicAdd((unsigned long long *)&dw[(int64_t)co * 9 * sh.c + kk], (unsigned long long)acc);
}

void launch_conv_dw(hipStream_t s, const ConvShape &sh, const int32_t *g, const int8_t *x,
                    int64_t *dw)
{
    launch_fill_i64(s, dw, (int64_t)sh.co * 9 * sh.c);
    int64_t rows = (int64_t)sh.n * sh.h;
    int rpc = DW_CHUNK_PIXELS / sh.w > 0 ? DW_CHUNK_PIXELS / sh.w : 1;
    dim3 grid(blocks_for(9 * sh.c, 256), sh.co, blocks_for(rows, rpc));
    hipLaunchKernelGGL(k_conv_dw_direct, grid, dim3(256), 0, s, sh, rpc, g, x, dw);
}

// ---------------------------------------------------------------------------------------------
// IntegerSGD (Alg. 1) in closed form: w' = w - (dw / gamma + [eta != 0] w / eta).
__global__ void k_sgd(int32_t *__restrict__ w, const int64_t *__restrict__ dw, int64_t count,
                      Div gamma, Div eta, int decay, uint32_t *flags)
{
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < count; i += stride) {
        const int64_t wv = w[i];
        const int64_t nw = wv - (idiv(dw[i], gamma) + (decay ? idiv(wv, eta) : 0));
        if (!fits_i32(nw)) {
            raise_flag(flags, FLAG_OVERFLOW);
            continue;
        }
        w[i] = (int32_t)nw;
    }
}

void launch_sgd(hipStream_t s, int32_t *w, const int64_t *dw, int64_t count, const Div &gamma,
                const Div &eta, bool decay, uint32_t *flags)
{
    if (count <= 0) return;
    unsigned g = blocks_for(count, 256);
    if (g > 65536) g = 65536;
    hipLaunchKernelGGL(k_sgd, dim3(g), dim3(256), 0, s, w, dw, count, gamma, eta, decay ? 1 : 0,
                       flags);
}

}  // namespace nitro
