// Operand preparation and bookkeeping kernels shared by the training iteration: limb planes of
// int32 weight matrices (plain and transposed) in one pass, batched IntegerSGD, max-slot
// clearing, and the split-K partial sums.
#include "mfma_common.h"

namespace nitro {

// ---------------------------------------------------------------------------------------------
// X int32 [R][C] (element (r, c) at x[z zx + r xs + c]) -> balanced int8 limb planes
//   P[l][r][c] at p[z zp + l pplane + r ps + c]                          (when p != null)
//   T[l][c][r] at t[z zt + l tplane + c ts + r] for r < Rpad, zero rows r >= R  (when t != null)
// and max|X| into a max slot. One workgroup: a 64 x 64 tile, z = blockIdx.z (the taps of a
// conv weight). C, ps, ts, Rpad and the z offsets keep every 16-byte row chunk aligned.

constexpr int PACK_LS = 68;                  // LDS row stride (bytes) of the transposed tile

// One 64 x 64 tile (column tile bx, row tile by, batch z) of a pack: the four limb planes of
// every value, plain and (through LDS) transposed, and the tile's max |value| into the slot.
__device__ void pack_tile(const PackArgs &a, int bx, int by, int z, uint8_t (*L)[64][PACK_LS])
{
    const int tid = threadIdx.x;
    const int c0 = bx * 64, r0 = by * 64;
    const int r = tid >> 2, cq = (tid & 3) * 16;
    const int gr = r0 + r, gc = c0 + cq;
    const bool ok = gr < a.R && gc < a.C;
    int32_t v[16];
    uint32_t m = 0;
    const int32_t *src = a.x + z * a.zx + (int64_t)(ok ? gr : 0) * a.xs + (ok ? gc : 0);
#pragma unroll
    for (int q = 0; q < 4; q++) {
        const v4i x4 = ok ? *(const v4i *)(src + 4 * q) : v4i{0, 0, 0, 0};
#pragma unroll
        for (int e = 0; e < 4; e++) {
            v[4 * q + e] = x4[e];
            const uint32_t av = abs_u32(x4[e]);
            m = av > m ? av : m;
        }
    }
#pragma unroll
    for (int l = 0; l < 4; l++) {
        v4i d;
#pragma unroll
        for (int q = 0; q < 4; q++) d[q] = (int)limb4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3], l);
        if (a.p && ok) *(v4i *)(a.p + z * a.zp + l * a.pplane + (int64_t)gr * a.ps + gc) = d;
        if (a.t)
#pragma unroll
            for (int e = 0; e < 16; e++) L[l][cq + e][r] = (uint8_t)((uint32_t)d[e >> 2] >> (8 * (e & 3)));
    }
    if (a.t) {
        __syncthreads();
        const int c = tid >> 2, rq = (tid & 3) * 16;
        if (c0 + c < a.C && r0 + rq < a.Rpad) {
#pragma unroll
            for (int l = 0; l < 4; l++) {
                const uint32_t *s = (const uint32_t *)&L[l][c][rq];
                const v4i o = v4i{(int)s[0], (int)s[1], (int)s[2], (int)s[3]};
                *(v4i *)(a.t + z * a.zt + l * a.tplane + (int64_t)(c0 + c) * a.ts + r0 + rq) = o;
            }
        }
    }
    block_slot_max(a.wmax, m);
}

__global__ __launch_bounds__(256) void k_pack_limbs(PackArgs a)
{
    __shared__ __attribute__((aligned(16))) uint8_t L[4][64][PACK_LS];
    pack_tile(a, blockIdx.x, blockIdx.y, blockIdx.z, L);
}

// Several packs in one launch: workgroups are dealt to the packs in order (first[k] ..
// first[k+1]), each pack's tiles numbered column tile fastest, then row tile, then batch; then to
// the element-wise conv packs (each: its plain planes' workgroups, then its swapped planes').
__global__ __launch_bounds__(256) void k_pack_batch(PackBatch b)
{
    __shared__ __attribute__((aligned(16))) uint8_t L[4][64][PACK_LS];
    int wid = blockIdx.x;
    if (wid >= b.first[b.n]) {
        wid -= b.first[b.n];
        for (int k = 0; k < b.nc; k++) {
            const ConvPackArgs &c = b.c[k];
            if (wid < c.nf) {
                pack_conv_weights_part(c.w, c.co * c.taps * c.cpad, (int)c.ci, (int)c.cpad, c.wf, c.wmax,
                                       (uint32_t)wid, (uint32_t)c.nf);
                return;
            }
            wid -= c.nf;
            if (wid < c.nt) {
                pack_conv_weights_t_part(c.w, c.co, c.ci, c.wt, (uint32_t)wid);
                return;
            }
            wid -= c.nt;
        }
        return;
    }
    int k = 0;
    while (k + 1 < b.n && wid >= b.first[k + 1]) k++;
    const int loc = wid - b.first[k];
    const int bx = loc % b.gx[k], rest = loc / b.gx[k];
    pack_tile(b.t[k], bx, rest % b.gy[k], rest / b.gy[k], L);
}

static void pack_grid(const PackArgs &a, int *gx, int *gy) { *gx = (a.C + 63) / 64; *gy = (a.Rpad + 63) / 64; }

void PackList::add(hipStream_t s, const PackArgs &a, int batches)
{
    if (b.n == PACK_BATCH) flush(s);
    int gx, gy;
    pack_grid(a, &gx, &gy);
    b.t[b.n] = a;
    b.gx[b.n] = gx;
    b.gy[b.n] = gy;
    b.first[b.n + 1] = b.first[b.n] + gx * gy * batches;
    b.n++;
}

void PackList::add_conv(hipStream_t s, const int32_t *w, int co, int ci, int cpad, int8_t *wf,
                        int8_t *wt, uint32_t *wmax, int taps)
{
    if (b.nc == PACK_CONV) flush(s);
    ConvPackArgs &c = b.c[b.nc++];
    c.w = w;
    c.co = (uint32_t)co;
    c.ci = (uint32_t)ci;
    c.cpad = (uint32_t)cpad;
    c.taps = (uint32_t)taps;
    c.wf = wf;
    c.wt = taps == 9 ? wt : nullptr;
    c.wmax = wmax;
    c.nf = grid_stride_blocks((int64_t)co * taps * cpad);
    c.nt = c.wt ? (int)(((int64_t)co * 9 * ci + 255) / 256) : 0;
}

void PackList::flush(hipStream_t s)
{
    int64_t nwg = b.first[b.n];
    for (int k = 0; k < b.nc; k++) nwg += b.c[k].nf + b.c[k].nt;
    if (nwg > 0) hipLaunchKernelGGL(k_pack_batch, dim3((unsigned)nwg), dim3(256), 0, s, b);
    b.n = 0;
    b.nc = 0;
    b.first[0] = 0;
}

static void launch_pack(hipStream_t s, const PackArgs &a, int batches)
{
    const dim3 grid((unsigned)((a.C + 63) / 64), (unsigned)((a.Rpad + 63) / 64), (unsigned)batches);
    hipLaunchKernelGGL(k_pack_limbs, grid, dim3(256), 0, s, a);
}

bool pack_conv_tiled_ok(int co, int ci) { return co % 16 == 0 && ci % 16 == 0; }

PackArgs pack_conv_args(const int32_t *w, int co, int ci, int8_t *wf, int8_t *wt, uint32_t *wmax)
{
    // per tap t: X_t[o][c] = W[o][t][c]; wf = [l][o][9 ci] (tap-major K), wt = [l][c][9 co]
    PackArgs a{};
    a.x = w; a.xs = 9 * (int64_t)ci; a.zx = ci;
    a.R = co; a.C = ci; a.Rpad = co;
    a.p = wf; a.ps = 9 * (int64_t)ci; a.pplane = (int64_t)co * 9 * ci; a.zp = ci;
    a.t = wt; a.ts = 9 * (int64_t)co; a.tplane = (int64_t)ci * 9 * co; a.zt = co;
    a.wmax = wmax;
    return a;
}

PackArgs pack_matrix_args(const int32_t *w, int R, int C, int Rpad, int8_t *p, int8_t *t,
                          uint32_t *wmax)
{
    PackArgs a{};
    a.x = w; a.xs = C; a.zx = 0;
    a.R = R; a.C = C; a.Rpad = Rpad;
    a.p = p; a.ps = C; a.pplane = (int64_t)R * C; a.zp = 0;
    a.t = t; a.ts = Rpad; a.tplane = (int64_t)C * Rpad; a.zt = 0;
    a.wmax = wmax;
    return a;
}

void launch_pack_conv_tiled(hipStream_t s, const int32_t *w, int co, int ci, int8_t *wf,
                            int8_t *wt, uint32_t *wmax)
{
    // per tap t: X_t[o][c] = W[o][t][c]; wf = [l][o][9 ci] (tap-major K), wt = [l][c][9 co]
    PackArgs a{};
    a.x = w; a.xs = 9 * (int64_t)ci; a.zx = ci;
    a.R = co; a.C = ci; a.Rpad = co;
    a.p = wf; a.ps = 9 * (int64_t)ci; a.pplane = (int64_t)co * 9 * ci; a.zp = ci;
    a.t = wt; a.ts = 9 * (int64_t)co; a.tplane = (int64_t)ci * 9 * co; a.zt = co;
    a.wmax = wmax;
    launch_pack(s, a, 9);
}

void launch_pack_matrix(hipStream_t s, const int32_t *w, int R, int C, int Rpad, int8_t *p,
                        int8_t *t, uint32_t *wmax)
{
    PackArgs a{};
    a.x = w; a.xs = C; a.zx = 0;
    a.R = R; a.C = C; a.Rpad = Rpad;
    a.p = p; a.ps = C; a.pplane = (int64_t)R * C; a.zp = 0;
    a.t = t; a.ts = Rpad; a.tplane = (int64_t)C * Rpad; a.zt = 0;
    a.wmax = wmax;
    launch_pack(s, a, 1);
}

// ---------------------------------------------------------------------------------------------
// IntegerSGD (Alg. 1) over several tensors in one launch, in closed form:
// w' = w - (dw / gamma + [eta != 0] w / eta). Workgroups are dealt to tensors in order
// (first[k] .. first[k+1]).
__global__ __launch_bounds__(256) void k_sgd_batch(SgdBatch b)
{
    int k = 0;
    while (k + 1 < b.n && (int64_t)blockIdx.x >= b.first[k + 1]) k++;
    const SgdTensor &t = b.t[k];
    const int64_t base = ((int64_t)blockIdx.x - b.first[k]) * 256 * SGD_ITEMS;
    for (int q = 0; q < SGD_ITEMS; q++) {
        const int64_t i = base + q * 256 + threadIdx.x;
        if (i >= t.count) break;
        const int64_t wv = t.w[i];
        const int64_t nw = wv - (idiv(t.dw[i], t.gamma) + (t.decay ? idiv(wv, t.eta) : 0));
        if (!fits_i32(nw)) {
            raise_flag(b.flags, FLAG_OVERFLOW);
            continue;
        }
        t.w[i] = (int32_t)nw;
    }
}

void launch_sgd_batch(hipStream_t s, SgdBatch b)
{
    int64_t blocks = 0;
    for (int k = 0; k < b.n; k++) {
        b.first[k] = blocks;
        blocks += (b.t[k].count + 256 * SGD_ITEMS - 1) / (256 * SGD_ITEMS);
    }
    if (blocks == 0) return;
    hipLaunchKernelGGL(k_sgd_batch, dim3((unsigned)blocks), dim3(256), 0, s, b);
}

// ---------------------------------------------------------------------------------------------
// Zero the max slots of several blocks (one workgroup per block); the workgroups after them pad
// a network input to 16 channels (pad.P > 0).
__global__ __launch_bounds__(256) void k_zero_slots(SlotList l, int nblocks, Pad16Args pad)
{
    if ((int)blockIdx.x >= nblocks) {
        pad_channels16_part(pad.x, pad.P, pad.c, pad.xpad, (int)blockIdx.x - nblocks);
        return;
    }
    uint32_t *p = l.p[blockIdx.x];
    for (int i = threadIdx.x; i < l.words; i += 256) p[i] = 0;
}

void launch_zero_slots(hipStream_t s, const SlotList &l, int nblocks, const Pad16Args *pad)
{
    Pad16Args pa{};
    if (pad) pa = *pad;
    const int npad = pa.P > 0 ? (pa.P + 255) / 256 : 0;
    if (nblocks + npad > 0)
        hipLaunchKernelGGL(k_zero_slots, dim3((unsigned)(nblocks + npad)), dim3(256), 0, s, l, nblocks, pa);
}

// ---------------------------------------------------------------------------------------------
__global__ void k_ts_reset(uint64_t *buf, int64_t nwords)
{
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < nwords;
         i += (int64_t)gridDim.x * blockDim.x)
        buf[i] = (i % TS_WORDS) < TS_SPREAD ? ~(uint64_t)0 : 0;
}

void launch_ts_reset(hipStream_t s, uint64_t *buf, int64_t nslots)
{
    const int64_t n = nslots * TS_WORDS;
    if (n > 0) hipLaunchKernelGGL(k_ts_reset, dim3(grid_stride_blocks(n, 256, 256)), dim3(256), 0, s, buf, n);
}

}  // namespace nitro
