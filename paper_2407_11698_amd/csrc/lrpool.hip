// The learning layers' max-pooling: a conv block's output a_l downsampled into z^mp before its
// learning layer (section 3.3, training procedure; d^lr of Tab. 6), and the backward of that
// pooling fused with the block's own 2x2 max-pool backward and the last layer's NITRO-ReLU
// backward. Both are HBM-bound elementwise passes: one thread per output element, channels
// innermost, so the lanes of a wave touch consecutive bytes.
#include "nitro_internal.h"

namespace nitro {

// f[n][i][j][c] = the first maximum (row-major) of a's kh x kw window at (i kh, j kw), and its
// index in the window.
__global__ __launch_bounds__(256) void k_lr_pool(LrPool p, const int8_t *__restrict__ a,
                                                 int8_t *__restrict__ f, uint8_t *__restrict__ fcode)
{
    const uint32_t Hf = (uint32_t)(p.h / p.kh), Wf = (uint32_t)(p.w / p.kw), C = (uint32_t)p.c;
    const uint32_t total = (uint32_t)p.n * Hf * Wf * C;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const uint32_t c = i % C, r = i / C;
        const uint32_t j = r % Wf, r2 = r / Wf;
        const uint32_t ii = r2 % Hf, n = r2 / Hf;
        const int8_t *base = a + (((int64_t)n * p.h + ii * p.kh) * p.w + j * p.kw) * C + c;
        int best = -129, arg = 0;
        for (int t = 0; t < p.kh * p.kw; t++) {
            const int v = base[((int64_t)(t / p.kw) * p.w + t % p.kw) * C];
            if (v > best) {
                best = v;
                arg = t;
            }
        }
        f[i] = (int8_t)best;
        fcode[i] = (uint8_t)arg;
    }
}

// g at the last layer's pre-activation, one thread per element (n, y, x, c) of its full
// resolution [n][H][W][c] (H = 2 h with the block's pool, else h): zero unless the element won
// the block's 2x2 pool (if any) and then its learning-pool window; a winner takes NITRO-ReLU'
// of delta_f at its region.
__global__ __launch_bounds__(256) void k_lr_unpool_relu_bwd(LrPool p, int pool,
                                                            const int32_t *__restrict__ delta_f,
                                                            const uint8_t *__restrict__ fcode,
                                                            const uint8_t *__restrict__ code, Relu rp,
                                                            int32_t *__restrict__ g, uint32_t *gmax,
                                                            uint32_t *flags)
{
    const uint32_t C = (uint32_t)p.c;
    const uint32_t H = pool ? 2 * p.h : p.h, W = pool ? 2 * p.w : p.w;
    const uint32_t Hf = (uint32_t)(p.h / p.kh), Wf = (uint32_t)(p.w / p.kw);
    const uint32_t total = (uint32_t)p.n * H * W * C;
    uint32_t mx = 0;
    bool bad = false;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const uint32_t c = i % C, r = i / C;
        const uint32_t x = r % W, r2 = r / W;
        const uint32_t y = r2 % H, n = r2 / H;
        uint32_t hb = y, wb = x, region;
        bool win = true;
        if (pool) {
            hb = y >> 1;
            wb = x >> 1;
            const uint8_t pc = code[(((uint64_t)n * p.h + hb) * p.w + wb) * C + c];
            win = (uint32_t)(pc & 3) == ((y & 1) << 1 | (x & 1));
            region = pc >> 2;
        } else {
            region = code[i];
        }
        int64_t v = 0;
        if (win) {
            const uint32_t fi = ((n * Hf + hb / p.kh) * Wf + wb / p.kw) * C + c;
            const uint32_t t = (hb % p.kh) * p.kw + wb % p.kw;
            if (fcode[fi] == t) v = relu_bwd(delta_f[fi], (uint8_t)region, rp);
        }
        const uint32_t a = abs_i64_sat(v);
        mx = a > mx ? a : mx;
        bad |= !fits_i32(v);
        g[i] = (int32_t)v;
    }
    if (bad) raise_flag(flags, FLAG_OVERFLOW);
    if (gmax) block_slot_max(gmax, mx);
}

void launch_lr_pool(hipStream_t s, const LrPool &p, const int8_t *a, int8_t *f, uint8_t *fcode)
{
    const int64_t total = (int64_t)p.n * (p.h / p.kh) * (p.w / p.kw) * p.c;
    if (total > 0)
        hipLaunchKernelGGL(k_lr_pool, dim3(grid_stride_blocks(total)), dim3(256), 0, s, p, a, f, fcode);
}

void launch_lr_unpool_relu_bwd(hipStream_t s, const LrPool &p, bool pool, const int32_t *delta_f,
                               const uint8_t *fcode, const uint8_t *code, const Relu &rp,
                               int32_t *g, uint32_t *gmax, uint32_t *flags)
{
    const int64_t total = (int64_t)p.n * p.h * p.w * p.c * (pool ? 4 : 1);
    if (total > 0)
        hipLaunchKernelGGL(k_lr_unpool_relu_bwd, dim3(grid_stride_blocks(total)), dim3(256), 0, s, p,
                           pool ? 1 : 0, delta_f, fcode, code, rp, g, gmax, flags);
}

}  // namespace nitro

namespace nitro {

void lr_pool_window(int c, int h, int w, int d_lr, int *kh, int *kw)
{
    int a = 1, b = 1;
    bool turn_h = true;
    while (d_lr > 0 && (int64_t)c * (h / a) * (w / b) > d_lr) {
        const bool can_h = (h / a) % 2 == 0, can_w = (w / b) % 2 == 0;
        if (!can_h && !can_w) break;
        if ((turn_h && can_h) || !can_w)
            a *= 2;
        else
            b *= 2;
        turn_h = !turn_h;
    }
    *kh = a;
    *kw = b;
}

}  // namespace nitro
