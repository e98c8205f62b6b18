// The learning layers' max-pooling: a conv block's output a_l downsampled into z^mp before its
// learning layer (section 3.3, training procedure; d^lr of Tab. 6), and the backward of that
// pooling fused with the block's own 2x2 max-pool backward and the last layer's NITRO-ReLU
// backward. Both are HBM-bound elementwise passes: one thread per output element, channels
// innermost, so the lanes of a wave touch consecutive bytes.
#include "mfma_common.h"

namespace nitro {

static int log2i(int v)
{
    int l = 0;
    while ((1 << l) < v) l++;
    return l;
}

// The same two passes with 4 channels per thread (C % 4 == 0): workgroup = one output row
// (sample n, row y), its threads over the row's pixels x 4-channel groups; the windows are
// powers of two (lr_pool_window doubles them), so their divisions are shifts.
__global__ __launch_bounds__(256) void k_lr_pool4(LrPool p, int lkh, int lkw, Div32 d_c4,
                                                  const int8_t *__restrict__ a, int8_t *__restrict__ f,
                                                  uint8_t *__restrict__ fcode)
{
    const int Hf = p.h >> lkh, Wf = p.w >> lkw, C4 = p.c >> 2;
    const int n = blockIdx.x / Hf, ii = blockIdx.x - n * Hf;
    for (int it = threadIdx.x; it < Wf * C4; it += 256) {
        const int j = (int)udiv32((uint32_t)it, d_c4), c = 4 * (it - j * C4);
        const int8_t *base = a + (((int64_t)n * p.h + (ii << lkh)) * p.w + (j << lkw)) * p.c + c;
        int best[4] = {-129, -129, -129, -129}, arg[4] = {0, 0, 0, 0};
        // (unrolled: eight window loads requested before their compares)
#pragma unroll 8
        for (int t = 0; t < (1 << (lkh + lkw)); t++) {
            const uint32_t v = *(const uint32_t *)(base + ((int64_t)(t >> lkw) * p.w + (t & ((1 << lkw) - 1))) * p.c);
#pragma unroll
            for (int e = 0; e < 4; e++) {
                const int x = (int8_t)(v >> (8 * e));
                if (x > best[e]) {
                    best[e] = x;
                    arg[e] = t;
                }
            }
        }
        const int64_t o = (((int64_t)n * Hf + ii) * Wf + j) * p.c + c;
        *(uint32_t *)(f + o) = (uint32_t)(uint8_t)best[0] | (uint32_t)(uint8_t)best[1] << 8 |
                               (uint32_t)(uint8_t)best[2] << 16 | (uint32_t)(uint8_t)best[3] << 24;
        *(uint32_t *)(fcode + o) = (uint32_t)arg[0] | (uint32_t)arg[1] << 8 | (uint32_t)arg[2] << 16 |
                                   (uint32_t)arg[3] << 24;
    }
}

template <bool TR>
__global__ __launch_bounds__(256) void k_lr_unpool_relu_bwd4(LrPool p, int pool, int lkh, int lkw, Div32 d_c4,
                                                             const int32_t *__restrict__ delta_f,
                                                             const uint8_t *__restrict__ fcode,
                                                             const uint8_t *__restrict__ code, Relu rp,
                                                             int32_t *__restrict__ g, uint32_t *gmax)
{
    const int H = pool ? 2 * p.h : p.h, W = pool ? 2 * p.w : p.w, C4 = p.c >> 2;
    const int Hf = p.h >> lkh, Wf = p.w >> lkw;
    const int n = blockIdx.x / H, y = blockIdx.x - n * H;
    const int hb = pool ? y >> 1 : y;
    uint32_t mx = 0;
    for (int it = threadIdx.x; it < W * C4; it += 256) {
        const int x = (int)udiv32((uint32_t)it, d_c4), c = 4 * (it - x * C4);
        const int wb = pool ? x >> 1 : x;
        uint32_t cd = *(const uint32_t *)(code + (((int64_t)n * p.h + hb) * p.w + wb) * p.c + c);
        const int64_t fi = (((int64_t)n * Hf + (hb >> lkh)) * Wf + (wb >> lkw)) * p.c + c;
        const uint32_t t = (uint32_t)(((hb & ((1 << lkh) - 1)) << lkw) + (wb & ((1 << lkw) - 1)));
        const uint32_t fc = *(const uint32_t *)(fcode + fi);
        const v4i dv = *(const v4i *)(delta_f + fi);
        v4i o;
#pragma unroll
        for (int e = 0; e < 4; e++) {
            const uint32_t pc = (cd >> (8 * e)) & 0xffu;
            const bool win = (!pool || (pc & 3u) == (uint32_t)((y & 1) << 1 | (x & 1))) &&
                             ((fc >> (8 * e)) & 0xffu) == t;
            const int32_t v = relu_bwd32<TR>(dv[e], pool ? pc >> 2 : pc, rp);
            o[e] = win ? v : 0;
            const uint32_t a = abs_u32(o[e]);
            mx = a > mx ? a : mx;
        }
        *(v4i *)(g + (((int64_t)n * H + y) * W + x) * p.c + c) = o;
    }
    if (gmax) block_slot_max(gmax, mx);
}

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

// (the 4-channel forms where the channels allow them and the windows are powers of two, as
// lr_pool_window makes them)
static bool lr_pool4_ok(const LrPool &p)
{
    return p.c % 4 == 0 && (1 << log2i(p.kh)) == p.kh && (1 << log2i(p.kw)) == p.kw;
}

void launch_lr_pool(hipStream_t s, const LrPool &p, const int8_t *a, int8_t *f, uint8_t *fcode)
{
    const int64_t total = (int64_t)p.n * (p.h / p.kh) * (p.w / p.kw) * p.c;
    if (total <= 0) return;
    if (lr_pool4_ok(p)) {
        hipLaunchKernelGGL(k_lr_pool4, dim3((unsigned)(p.n * (p.h / p.kh))), dim3(256), 0, s, p, log2i(p.kh),
                           log2i(p.kw), make_div32((uint32_t)(p.c / 4)), a, f, fcode);
        return;
    }
    hipLaunchKernelGGL(k_lr_pool, dim3(grid_stride_blocks(total)), dim3(256), 0, s, p, a, f, fcode);
}

void launch_lr_unpool_relu_bwd(hipStream_t s, const LrPool &p, bool pool, const int32_t *delta_f,
                               const uint8_t *fcode, const uint8_t *code, const Relu &rp,
                               int32_t *g, uint32_t *gmax, uint32_t *flags)
{
    const int64_t total = (int64_t)p.n * p.h * p.w * p.c * (pool ? 4 : 1);
    if (total <= 0) return;
    if (lr_pool4_ok(p)) {
        // (an int32 delta passes NITRO-ReLU backward within int32: no overflow to flag)
        const unsigned rows = (unsigned)(p.n * (pool ? 2 * p.h : p.h));
        const Div32 dc = make_div32((uint32_t)(p.c / 4));
        if (rp.alpha.trunc)
            hipLaunchKernelGGL(k_lr_unpool_relu_bwd4<true>, dim3(rows), dim3(256), 0, s, p, pool ? 1 : 0,
                               log2i(p.kh), log2i(p.kw), dc, delta_f, fcode, code, rp, g, gmax);
        else
            hipLaunchKernelGGL(k_lr_unpool_relu_bwd4<false>, dim3(rows), dim3(256), 0, s, p, pool ? 1 : 0,
                               log2i(p.kh), log2i(p.kw), dc, delta_f, fcode, code, rp, g, gmax);
        return;
    }
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
