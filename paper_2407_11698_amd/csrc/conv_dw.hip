// Weight gradient of the 3x3 IntConv2D (section 3.2.1, 3x3 / stride 1 / pad 1 per Tab. 1) on
// gfx950 int8 MFMA, exact:
//   dW[co][r][s][ci] = sum_p g[p][co] * x[p + (r-1, s-1)][ci]          (int64)
//
// Padded pixel grid. Both operands are first rewritten on a zero-padded grid: every image row
// is followed by one zero column and every image by one zero row, so pixel (n, h, w) sits at
// position k = (n (H+1) + h) (W+1) + w and each neighbour outside the image lands on a zero. A
// tap (r, s) is then the plain position offset (r-1)(W+1) + (s-1):
//   dW[co][r][s][ci] = sum_k gp[co][k] * xr[ci][HMAX + k + (r-1)(W+1) + (s-1)]
// with no bounds test. gp holds the balanced int8 limbs of g, one plane per limb (zeros at pad
// positions), stored as the MFMA A fragments themselves: for each super-step of 256 positions,
// 16-channel block of co and K-step of 64 positions, one 1 KB fragment whose lane L = 16 q + j
// (16 bytes at 16 L) holds co row j, positions 16 q .. 16 q + 15 of the K-step. A fragment load
// is then one contiguous 1 KB read (with rows [co][kp] the four lanes sharing a 64-byte row
// segment are 16 lanes apart, and every lane is a cache access of its own). xr holds x in rows
// of 16 channels: [C_in / 16][position][16 channels], with a zero halo of HMAX >= W + 2
// positions on both sides.
//
// GEMM: M = co, N = ci (times 9 taps), K = padded positions. A workgroup owns a 64 co x 16 ci
// tile, all 9 taps, over a range of K. Its four waves run independently (no barrier in the main
// loop), each on one limb of g and one part of the range: with L limbs, Q = 4 / L parts (L = 3:
// one part, one wave idle). A fragments (g limbs) are loaded from the planes straight into
// registers, one 256-position super-step ahead. The x rows of a super-step (plus the halo) are
// staged in the wave's own double-buffered LDS slice, and the B fragment of tap (r, s) -- 16
// positions of one channel per lane -- is read from them with two transposing LDS reads
// (ds_read_b64_tr_b8) at a row offset of (r-1)(W+1) + (s-1). The waves' int32 sums, weighted
// 256^limb, are added in int64 through LDS at the end. A wave's range is at most 511 * 256
// positions, so |sum| <= 128 * 128 * 130816 < 2^31.
#include <type_traits>

#include "mfma_common.h"

namespace nitro {

constexpr int DWP_KS = 256;        // padded positions per super-step (4 MFMA K-steps of 64)
constexpr int DWP_CHUNK_MAX = 511;    // super-steps per workgroup (and per wave: <= 511 * 256)
constexpr int DWP_WIN = DWP_KS + 2 * DWP_HMAX;   // staged rows (positions) of a super-step
constexpr int DWP_NCH = DWP_WIN / 64;            // 16-byte rows per lane

struct DwpGeom {
    int wp, hp;          // W + 1, H + 1
    int64_t kraw;        // positions of the padded grid: n (H+1) (W+1)
    int64_t kp;          // positions processed (kraw rounded up to a super-step)
    int64_t xs;          // positions of an x row block: HMAX + kp + HMAX
};

DwpGeom dwp_geom(const ConvShape &sh)
{
    DwpGeom g;
    g.wp = sh.w + 1;
    g.hp = sh.h + 1;
    g.kraw = (int64_t)sh.n * g.hp * g.wp;
    g.kp = (g.kraw + DWP_KS - 1) / DWP_KS * DWP_KS;
    g.xs = g.kp + DWP_WIN - DWP_KS;   // the last super-step's window ends there
    return g;
}

// Input channels are computed in multiples of 16: a layer with C_in % 16 != 0 gets zero x
// planes up to the next multiple (their weight-gradient columns are computed and dropped).
static int dwp_c16(const ConvShape &sh) { return (sh.c + 15) / 16 * 16; }

bool dwp_ok(const ConvShape &sh)
{
    if (sh.c < 1 || sh.co % 16 || sh.w + 2 > DWP_HMAX) return false;
    const DwpGeom g = dwp_geom(sh);
    // 32-bit offsets inside the planes and in the preparation kernels
    const int64_t lim = (int64_t)1 << 31;
    return (int64_t)dwp_c16(sh) * g.xs < lim && 4 * (int64_t)sh.co * g.kp < lim &&
           (int64_t)sh.n * sh.h * sh.w * sh.co < lim && (int64_t)sh.n * sh.h * sh.w * sh.c < lim;
}

struct DwpPlan {
    int tiles_co, tiles_ci, nss, chunk, nsplit;
};

// About one workgroup per compute unit; at least 8 super-steps (2 per wave) per workgroup.
static DwpPlan dwp_plan(const ConvShape &sh)
{
    const DwpGeom g = dwp_geom(sh);
    DwpPlan p;
    p.tiles_co = (sh.co + 63) / 64;
    p.tiles_ci = dwp_c16(sh) / 16;
    p.nss = (int)(g.kp / DWP_KS);
    const int tiles = p.tiles_co * p.tiles_ci;
    int s = (256 + tiles - 1) / tiles;
    const int smax = p.nss / 8 > 1 ? p.nss / 8 : 1;
    if (s > smax) s = smax;
    p.chunk = (p.nss + s - 1) / s;
    if (p.chunk > DWP_CHUNK_MAX) p.chunk = DWP_CHUNK_MAX;
    p.nsplit = (p.nss + p.chunk - 1) / p.chunk;
    return p;
}

int64_t dwp_partial_count(const ConvShape &sh)
{
    const DwpPlan p = dwp_plan(sh);
    return p.nsplit > 1 ? (int64_t)p.nsplit * sh.co * 9 * sh.c : 0;
}

int64_t dwp_rows_stride(const ConvShape &sh) { return dwp_geom(sh).xs; }

int64_t dwp_gplane_bytes(const ConvShape &sh) { return 4 * (int64_t)sh.co * dwp_geom(sh).kp; }
int64_t dwp_xplane_bytes(const ConvShape &sh) { return (int64_t)dwp_c16(sh) * dwp_geom(sh).xs; }

// Position k of the padded grid -> NHWC pixel index, or -1 at a pad position.
__device__ inline int padded_pixel(int k, int n, int h, int w, int hp, int wp)
{
    if (k < 0) return -1;
    const int per = hp * wp;
    const int img = k / per;
    const int rem = k - img * per;
    const int hh = rem / wp, ww = rem - hh * wp;
    if (img >= n || hh >= h || ww >= w) return -1;
    return (img * h + hh) * w + ww;
}

// ---------------------------------------------------------------------------------------------
// x int8 NHWC [P][C] -> xr [C16 / 16][xs][16]: row HMAX + k holds the 16 channels of tile t at
// padded position k (zeros at pad positions, in the halo and in channels C..C16-1). One thread:
// one 16-byte row (workgroup (bx, by): rows 256 bx .., tile by).
__device__ void dwp_act_rows(const int8_t *__restrict__ x, int n, int h, int w, int c, int hp,
                             int wp, int xs, int8_t *__restrict__ xr, int bx, int by)
{
    const int i = bx * 256 + threadIdx.x;             // row within the tile's block
    const int t = by;                                 // 16-channel tile
    if (i >= xs) return;
    const int pix = padded_pixel(i - DWP_HMAX, n, h, w, hp, wp);
    const int ch = 16 * t;
    v4i v = v4i{0, 0, 0, 0};
    if (pix >= 0) {
        if ((c & 15) == 0) {
            v = *(const v4i *)(x + (int64_t)pix * c + ch);
        } else {
            for (int e = 0; e < 16 && ch + e < c; e++)
                v[e >> 2] |= (int)((uint32_t)(uint8_t)x[(int64_t)pix * c + ch + e] << (8 * (e & 3)));
        }
    }
    *(v4i *)(xr + ((int64_t)t * xs + i) * 16) = v;
}

// Zeros in the pad rows of xr (the halos, the column after every image row, the row after every
// image, the tail): the rows of the real pixels were written by the previous layer's forward.
// One thread: one pad position of one 16-channel tile (workgroup (bx, by): positions 256 bx ..,
// tile by).
__device__ void dwp_pad_rows(int n, int h, int w, int hp, int wp, int64_t kraw, int64_t xs,
                             int8_t *__restrict__ xr, int bx, int by)
{
    const int64_t i = (int64_t)bx * 256 + threadIdx.x;
    const int t = by;
    const int64_t inner = (int64_t)n * (h + w + 1);
    int64_t row;
    if (i < inner) {
        const int img = (int)(i / (h + w + 1)), j = (int)(i - (int64_t)img * (h + w + 1));
        const int hh = j < h ? j : h, ww = j < h ? w : j - h;
        row = DWP_HMAX + ((int64_t)img * hp + hh) * wp + ww;
    } else if (i < inner + DWP_HMAX) {
        row = i - inner;
    } else {
        row = DWP_HMAX + kraw + (i - inner - DWP_HMAX);
        if (row >= xs) return;
    }
    *(v4i *)(xr + ((int64_t)t * xs + row) * 16) = v4i{0, 0, 0, 0};
}

// g int32 NHWC [P][C] -> gp, limb planes l < limbs(max|g|) in fragment order: limb l of g at
// padded position k (zeros at pad positions), 16-byte chunk (channel c, positions k .. k + 15)
// at l C kp + ((k / 256 * C / 16 + c / 16) * 4 + k % 256 / 64) * 1024 + 256 (k % 64 / 16)
// + 16 (c % 16); when gn is not null also the NHWC limb planes gn [l][P][C] (the A
// operand of the input-gradient GEMM), with goff and max|g| in the offset range those of
// g - 128 (three limbs) and the indices of the entries g = 32768 appended to go.list. A
// workgroup: 64 positions x 64 channels, transposed through LDS. With pcode, g holds a 2x2-pooled layer's gradient at the pooled positions only,
// [n][h/2][w/2][C]: pixel (y, x) takes it where the pool's argmax (the code's low 2 bits) is
// window position 2 (y & 1) + (x & 1), and zero elsewhere. Workgroup (bx, by): positions
// 64 bx .., channels 64 by ...
__device__ void dwp_grad_planes(const int32_t *__restrict__ g, const int16_t *__restrict__ g16,
                                int n, int h, int w, int c, int hp,
                                int wp, int kp, const uint32_t *gmax,
                                const uint8_t *__restrict__ pcode, int8_t *__restrict__ gp,
                                int8_t *__restrict__ gn, const GOff &go, bool goff_dx,
                                bool goff_dw, int bx, int by, int32_t *lds)
{
    int32_t(*T)[65] = (int32_t(*)[65])lds;   // [64 positions][64 channels + 1]
    const int tid = threadIdx.x;
    // the max slot's word is requested with g's loads and reduced after them
    const uint32_t sw = gmax[tid & 63];
    uint32_t rmask = 0;                  // offset form: this thread's entries with g = 32768
    const int k0 = bx * 64;
    const int c0 = by * 64;
    uint32_t gm = 0;
    int LA = 0;
    bool off_n = false, off_p = false, off = false;
    {
        const int pi = tid >> 2, cq = tid & 3;
        const int pix = padded_pixel(k0 + pi, n, h, w, hp, wp);
        int src = pix;                   // pixel of g holding this position's value
        uint32_t win = 0;                // pooled g: this pixel's position in its window
        if (pcode && pix >= 0) {
            const int row = pix / w, ww = pix - row * w;   // row over all images
            const int img = row / h, hh = row - img * h;
            src = (img * (h >> 1) + (hh >> 1)) * (w >> 1) + (ww >> 1);
            win = 2u * (hh & 1) + (ww & 1);
        }
        int32_t v[16];
#pragma unroll
        for (int u = 0; u < 4; u++) {
            const int ch = c0 + 16 * cq + 4 * u;
            v4i x = v4i{0, 0, 0, 0};
            if (pix >= 0 && ch < c) {
                if (g16) {
                    // the escaped 16-bit form: an escape's value is in g at the same index
                    const v2i hv = *(const v2i *)(g16 + (int64_t)src * c + ch);
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        const int16_t v = (int16_t)((uint32_t)hv[e >> 1] >> (16 * (e & 1)));
                        x[e] = v == G16_ESC ? g[(int64_t)src * c + ch + e] : (int32_t)v;
                    }
                } else {
                    x = *(const v4i *)(g + (int64_t)src * c + ch);
                }
                if (pcode) {
                    const uint32_t cd = *(const uint32_t *)(pcode + (int64_t)src * c + ch);
#pragma unroll
                    for (int e = 0; e < 4; e++) x[e] = ((cd >> (8 * e)) & 3u) == win ? x[e] : 0;
                }
            }
#pragma unroll
            for (int e = 0; e < 4; e++) v[4 * u + e] = x[e];
        }
        gm = wave_max_u32(sw);
        LA = limbs_for(gm);
        if (LA > 4) return;              // the weight-gradient kernel flags it
        off_n = goff_dx && goff_range(gm);   // gn in the offset form
        off_p = goff_dw && goff_range(gm);   // gp in the offset form
        off = off_n || off_p;
        // (gp in the offset form: g - 128 at the image's pixels, pad positions stay zero)
        const int32_t obp = off_p && pix >= 0 ? GOFF_BIAS : 0;
#pragma unroll
        for (int u = 0; u < 4; u++) {
            const int32_t ob = c0 + 16 * cq + 4 * u < c ? obp : 0;
#pragma unroll
            for (int e = 0; e < 4; e++) T[pi][16 * cq + 4 * u + e] = v[4 * u + e] - ob;
        }
        if (off && pix >= 0) {
#pragma unroll
            for (int e = 0; e < 16; e++) rmask |= v[e] >= 32768 ? 1u << e : 0u;
        }
        if (gn && pix >= 0 && c0 + 16 * cq < c) {
            const int64_t P = (int64_t)n * h * w;
            const int32_t ob = off_n ? GOFF_BIAS : 0;
#pragma unroll
            for (int l = 0; l < 4; l++) {
                if (l < LA) {
                    v4i o;
#pragma unroll
                    for (int q = 0; q < 4; q++)
                        o[q] = (int)limb4(v[4 * q] - ob, v[4 * q + 1] - ob, v[4 * q + 2] - ob,
                                          v[4 * q + 3] - ob, l);
                    *(v4i *)(gn + (int64_t)l * P * c + (int64_t)pix * c + c0 + 16 * cq) = o;
                }
            }
        }
        // the entries g = 32768 appended to the list: one atomic per wave that has any, each
        // lane's entries at its exclusive prefix of the wave's counts (every lane is here)
        if (off && __ballot(rmask != 0)) {
            const int lane = tid & 63;
            const int k = __popc(rmask);
            int incl = k;
#pragma unroll
            for (int d = 1; d < 64; d <<= 1) {
                const int o = __shfl_up(incl, d, 64);
                if (lane >= d) incl += o;
            }
            const int total = __shfl(incl, 63, 64);
            uint32_t base = 0;
            if (lane == 0) base = atomicAdd(go.count, (uint32_t)total);
            uint32_t idx = (uint32_t)__shfl((int)base, 0, 64) + (uint32_t)(incl - k);
            for (int e = 0; e < 16; e++)
                if (rmask & (1u << e)) {
                    if (idx < GOFF_CAP) go.list[idx] = (uint32_t)pix * (uint32_t)c + (uint32_t)(c0 + 16 * cq + e);
                    idx++;
                }
        }
    }
    __syncthreads();
    // the weight-gradient kernel reads every odd block of 16 positions with its two halves of 8
    // exchanged (its transposing LDS reads take them in that order); the planes store them so
    const int cc = tid >> 2, pq = tid & 3;
    if (c0 + cc >= c) return;
    int32_t v[16];
#pragma unroll
    for (int e = 0; e < 16; e++) v[e] = T[16 * pq + (e ^ ((pq & 1) << 3))][cc];
#pragma unroll
    for (int l = 0; l < 4; l++) {
        if (l < LA) {
            v4i o;
#pragma unroll
            for (int q = 0; q < 4; q++)
                o[q] = (int)limb4(v[4 * q], v[4 * q + 1], v[4 * q + 2], v[4 * q + 3], l);
            const int co = c0 + cc;
            *(v4i *)(gp + (int64_t)l * c * kp +
                     (((int64_t)(k0 >> 8) * (c >> 4) + (co >> 4)) * 4 + ((k0 & 255) >> 6)) * 1024 +
                     256 * pq + 16 * (co & 15)) = o;
        }
    }
}

// Sums of x for the weight gradient's offset form: workgroup (image img, channels 64 cb ..
// 64 cb + 63) adds x over the image's pixels, its rows h = 0 and H-1, columns w = 0 and W-1 and
// four corners into xq [9][c] (atomic adds; xq is zero before). Thread: 4 channels (tid % 16),
// pixels tid / 16 + 16 k; the 16 pixel lanes reduced by shuffles within a wave, the waves in
// LDS. Nothing unless max|g| is in the offset range.
__device__ void dwp_xsums(const int8_t *__restrict__ x, int h, int w, int c, const uint32_t *gmax,
                          int32_t *xq, int img, int cb, int32_t *lds)
{
    int32_t(*red)[16][36] = (int32_t(*)[16][36])lds;   // [4 waves][16 lanes][36]
    if (!goff_range(slot_read(gmax))) return;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int cq = tid & 15, pl = tid >> 4;
    const int hw = h * w;
    const int8_t *base = x + (int64_t)img * hw * c + 64 * cb + 4 * cq;
    int32_t a[36];
#pragma unroll
    for (int k = 0; k < 36; k++) a[k] = 0;
    for (int p = pl; p < hw; p += 16) {
        const uint32_t v = *(const uint32_t *)(base + (int64_t)p * c);
        const int y = p / w, xx = p - y * w;
        const bool top = y == 0, bot = y == h - 1, lft = xx == 0, rgt = xx == w - 1;
        const bool on[9] = {true, top, bot, lft, rgt, top && lft, top && rgt, bot && lft, bot && rgt};
#pragma unroll
        for (int e = 0; e < 4; e++) {
            const int32_t b = (int8_t)(v >> (8 * e));
#pragma unroll
            for (int qn = 0; qn < 9; qn++) a[4 * qn + e] += on[qn] ? b : 0;
        }
    }
#pragma unroll
    for (int k = 0; k < 36; k++) {
        a[k] += __shfl_xor(a[k], 16, 64);
        a[k] += __shfl_xor(a[k], 32, 64);
    }
    if (lane < 16) {
#pragma unroll
        for (int k = 0; k < 36; k++) red[wave][lane][k] = a[k];
    }
    __syncthreads();
    for (int o = tid; o < 9 * 64; o += 256) {
        const int qn = o >> 6, cc = o & 63;
        const int k = 4 * qn + (cc & 3);
        const int32_t sum = red[0][cc >> 2][k] + red[1][cc >> 2][k] + red[2][cc >> 2][k] + red[3][cc >> 2][k];
        if (sum) atomicAdd(xq + qn * c + 64 * cb + cc, sum);
    }
}

// The independent preparations of a weight-gradient launch in one launch: workgroups
// 0 .. xs_n - 1 the sums of x for the offset form (if asked for), then x's rows (or zeros at
// their pad positions), then g's planes.
struct DwpPrep {
    int rows;                    // 1: x rows from x; 2: zeros at the pad positions of rows
                                 //    written by the previous layer's forward
    int rows_gx, rows_gy, gp_gx;
    const int8_t *x;
    int n, h, w, c, co, hp, wp, kp;
    int64_t kraw, xs;
    int8_t *xr;
    const int32_t *g;
    const int16_t *g16;          // optional: g in the escaped 16-bit form (g: the escapes)
    const uint32_t *gmax;
    const uint8_t *pcode;
    int8_t *gp, *gn;
    GOff go;                     // offset form: gn (goff_dx), gp and the sums of x (goff_dw)
    int goff_dx, goff_dw;
    int xs_n;                    // sum workgroups: n (C / 64)
};

__global__ __launch_bounds__(256) void k_dwp_prep(DwpPrep a)
{
    __shared__ int32_t lds[64 * 65];     // g planes: the transpose; sums of x: the wave sums
    const int nrows = a.rows_gx * a.rows_gy;
    int b = blockIdx.x;
    if (b < a.xs_n) {
        const int nb = a.c / 64;
        dwp_xsums(a.x, a.h, a.w, a.c, a.gmax, a.go.xq, b / nb, b % nb, lds);
        return;
    }
    b -= a.xs_n;
    if (b < nrows) {
        const int bx = b % a.rows_gx, by = b / a.rows_gx;
        if (a.rows == 1) dwp_act_rows(a.x, a.n, a.h, a.w, a.c, a.hp, a.wp, (int)a.xs, a.xr, bx, by);
        else dwp_pad_rows(a.n, a.h, a.w, a.hp, a.wp, a.kraw, a.xs, a.xr, bx, by);
        return;
    }
    const int q = b - nrows;
    dwp_grad_planes(a.g, a.g16, a.n, a.h, a.w, a.co, a.hp, a.wp, a.kp, a.gmax, a.pcode, a.gp, a.gn,
                    a.go, a.goff_dx != 0, a.goff_dw != 0, q % a.gp_gx, q / a.gp_gx, lds);
}

// ---------------------------------------------------------------------------------------------
struct DwpArgs {
    const int8_t *gp;      // LA planes of co kp, fragment order
    int64_t kp;
    const int8_t *xr;      // [ci / 16][xs][16]
    int64_t xs;
    int wp, co, ci;              // ci: computed input channels (a multiple of 16)
    int ci_out;                  // input channels of dW (<= ci)
    int tiles_ci, tiles_co, nss, chunk;
    const uint32_t *gmax;
    int64_t *out;          // [nsplit][co][9][ci_out]; dW itself when there is one split
    uint32_t *flags;
    uint64_t *ts;          // timing slot (null: untimed)
    // g's planes may be in the offset form (two limbs, or three with more than GOFF_CAP entries)
    int goff;
    const uint32_t *goff_count;
};

// Transposing LDS read (gfx950 ds_read_b64_tr_b8). Within each group of 16 lanes, output lane
// 8 h + j receives, as its byte b (b = 0..7), byte j of the 8 bytes addressed by lane 2 b + h.
__device__ inline v2i lds_read_tr8(const uint8_t *p)
{
    return __builtin_amdgcn_ds_read_tr8_b64_v2i32((__attribute__((address_space(3))) v2i *)p);
}

// Wave-local LDS hand-off: this wave's LDS writes are complete before its later reads, and the
// compiler keeps memory accesses on their side of it.
__device__ inline void wave_lds_sync() { asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory"); }

// L3: launched for long ranges (at least DWP_L3_MIN super-steps per workgroup), where g in 3 limbs
// takes all four waves (see below); a separate instance, as it needs more registers.
constexpr int DWP_L3_MIN = 32;

template <bool L3>
__global__ __launch_bounds__(256) void k_conv_dw_planes(DwpArgs p)
{
    extern __shared__ __attribute__((aligned(16))) uint8_t lds[];
    ts_start(p.ts);
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // wave-uniform (scalar)
    // (the offset form's residual count read whether or not it is used, from the max slot then,
    // so that both loads are in flight together)
    const uint32_t rn = *(p.goff ? p.goff_count : p.gmax);
    const uint32_t gm = slot_read(p.gmax);
    const bool goff = p.goff && goff_range(gm);
    const int LA = goff ? (rn <= GOFF_CAP ? 2 : 3) : limbs_for(gm);
    if (LA > 4) {
        if (tid == 0) raise_flag(p.flags, FLAG_OVERFLOW);
        return;
    }
    // Work item. Workgroups of one K range (they read the same g rows) get consecutive numbers
    // and, as the dispatcher deals workgroups round-robin to the 8 XCDs, one XCD (one L2).
    const int nwg = gridDim.x;
    int wid = blockIdx.x;
    if ((nwg & 7) == 0) wid = (wid & 7) * (nwg >> 3) + (wid >> 3);
    const int tci = wid % p.tiles_ci;
    const int rest = wid / p.tiles_ci;
    const int tco = rest % p.tiles_co;
    const int split = rest / p.tiles_co;
    const int co0 = tco * 64, ci0 = tci * 16;

    // this wave's limb and super-steps: wave w takes limb w / Q, part w % Q of the range (Q =
    // 4 / L parts for L limbs; L = 3: one part, one wave idle). With L = 3 and a long range (the
    // L3 instance) instead wave w takes part w of every limb in turn (l3), the limbs' sums folded
    // into int64 between them: a pass's set-up and fold then cost less than the idle wave.
    const bool l3 = L3 && LA == 3;
    const int Q = LA == 1 || l3 ? 4 : LA == 2 ? 2 : 1;
    const int npass = l3 ? 3 : 1;
    const int limb = l3 ? 0 : wave / Q, part = wave - limb * Q;
    const int sb = split * p.chunk;
    const int se = sb + p.chunk < p.nss ? sb + p.chunk : p.nss;
    const int per = (se - sb + Q - 1) / Q;
    const int wb = sb + part * per < se ? sb + part * per : se;
    const int nst = limb < LA ? (wb + per < se ? wb + per : se) - wb : 0;
    int64_t tot[L3 ? 3 : 1][12];   // (L3) the tile's sums, 12 per thread and 3-tap group

    constexpr int STAGE = DWP_WIN * 16;        // bytes of one staged window (rows of 16 B)
    uint8_t *wl = lds + wave * (2 * STAGE);    // this wave's two stages

    const int j = lane & 15, g4 = lane >> 4;
    // 32-bit offsets from the plane bases (the host checks that both fit)
    const uint32_t plane = (uint32_t)p.co * (uint32_t)p.kp;
    // fragment (super-step ss, co block b, K-step u) of a plane at ((ss CT + b) 4 + u) 1 KB;
    // co blocks past the end (a partial last tile) read block CT - 1, their sums not stored
    const uint32_t CT = (uint32_t)p.co / 16;
    uint32_t aoff[4];
#pragma unroll
    for (int i = 0; i < 4; i++) {
        const uint32_t blk = (uint32_t)co0 / 16 + i < CT ? (uint32_t)co0 / 16 + i : CT - 1;
        aoff[i] = blk * 4096u + 16u * (uint32_t)lane;
    }
    // this wave's x rows: the window of super-step ss is rows ss KS .. ss KS + WIN of the tile's
    // row block, contiguous; lane stages rows lane + 64 m
    const int8_t *xbase = p.xr + (int64_t)tci * p.xs * 16;
    // B fragment of tap t at K-step u: the transposing reads of lane s = 16 q + 2 b + h take row
    // HMAX + off_t + 64 u + 16 q + b (+ 8), bytes 8 h .. 8 h + 7 (the channels 8 h + j of lane
    // 8 h + j). Lane groups q odd read the rows + 8 first: in each read the two groups of 16
    // lanes that share an LDS cycle then use different halves of the banks. Their A fragments
    // hold the same order (odd 16-position blocks of the g planes have their halves exchanged).
    const int lane_row = 16 * g4 + ((lane & 15) >> 1) + 8 * (g4 & 1);
    const int lane_b = (DWP_HMAX + lane_row) * 16 + 8 * (lane & 1);
    const int second = (g4 & 1) ? -8 * 16 : 8 * 16;
    int toff[9];
#pragma unroll
    for (int t = 0; t < 9; t++) toff[t] = ((t / 3 - 1) * p.wp + (t % 3 - 1)) * 16;
    // Pipeline (per wave, super-step s): at its start the x window of s + 1 is requested; s
    // computes from LDS stage s & 1, and each K-step's A fragments are requested for s + 1 as
    // soon as that K-step has used them; at its end the window of s + 1 goes to LDS stage
    // (s + 1) & 1. The first super-step of a pass starts its accumulators from zero inside the
    // MFMAs (peeled): a loop whose accumulators enter as literal zeros is compiled with copies
    // of every accumulator on every iteration.
    v4i acc[9][4];
    v4i a[4][4];                 // A fragments [K-step][co tile]
    v4i bst[DWP_NCH];            // staged x rows

    auto load_a = [&](int u, int ss, int l) {
        const uint32_t k = (uint32_t)l * plane + (uint32_t)ss * CT * 4096u + 1024u * u;
#pragma unroll
        for (int i = 0; i < 4; i++) a[u][i] = *(const v4i *)(p.gp + (aoff[i] + k));
    };
    auto load_b = [&](int ss) {
        const int8_t *src = xbase + ((int64_t)ss * DWP_KS + lane) * 16;
#pragma unroll
        for (int m = 0; m < DWP_NCH; m++) bst[m] = *(const v4i *)(src + 64 * 16 * m);
    };
    auto store_b = [&](int stage) {
        uint8_t *dst = wl + stage * STAGE + lane * 16;
#pragma unroll
        for (int m = 0; m < DWP_NCH; m++) *(v4i *)(dst + 64 * 16 * m) = bst[m];
    };
    auto compute = [&](auto first, auto reload, int stage, int next, int l) {
        const uint8_t *base = wl + stage * STAGE + lane_b;
#pragma unroll
        for (int u = 0; u < 4; u++) {
#pragma unroll
            for (int t = 0; t < 9; t++) {
                const uint8_t *r = base + toff[t] + 64 * 16 * u;
                const v2i lo = lds_read_tr8(r), hi = lds_read_tr8(r + second);
                const v4i b = v4i{lo[0], lo[1], hi[0], hi[1]};
#pragma unroll
                for (int i = 0; i < 4; i++)
                    acc[t][i] = __builtin_amdgcn_mfma_i32_16x16x64_i8(
                        a[u][i], b, (decltype(first)::value && u == 0) ? v4i{0, 0, 0, 0} : acc[t][i],
                        0, 0, 0);
            }
            if (decltype(reload)::value) {
                load_a(u, next, l);
                // (kept here: left to itself the scheduler sinks every load of the next
                // super-step to the end of this one, and each is then waited for)
                __builtin_amdgcn_sched_barrier(0);
            }
        }
    };

    for (int pass = 0; pass < npass; pass++) {
        const int l = l3 ? pass : limb;
        if (nst > 0) {
#pragma unroll
            for (int u = 0; u < 4; u++) load_a(u, wb, l);
            load_b(wb);
            store_b(0);
            wave_lds_sync();
            // super-step 0 (peeled), then 1 .. nst - 1; the last one requests nothing
            if (nst > 1) {
                load_b(wb + 1);
                __builtin_amdgcn_sched_barrier(0);
                compute(std::true_type(), std::true_type(), 0, wb + 1, l);
                store_b(1);
                wave_lds_sync();
                for (int s = 1; s + 1 < nst; s++) {
                    load_b(wb + s + 1);
                    __builtin_amdgcn_sched_barrier(0);
                    compute(std::false_type(), std::true_type(), s & 1, wb + s + 1, l);
                    store_b((s + 1) & 1);
                    wave_lds_sync();
                }
                compute(std::false_type(), std::false_type(), (nst - 1) & 1, 0, l);
            } else {
                compute(std::true_type(), std::false_type(), 0, 0, l);
            }
        } else {
#pragma unroll
            for (int t = 0; t < 9; t++)
#pragma unroll
                for (int i = 0; i < 4; i++) acc[t][i] = v4i{0, 0, 0, 0};
        }
        // Sum of the four waves (int64), each weighted 256^limb: straight into this split's
        // tile, or (L3) into this thread's 36 values, stored after the last pass. Per 3-tap
        // group, every lane stores its accumulators whole (16 bytes: output channels
        // 16 i + 4 g4 .. + 3 of input channel j) at [wave][tap][i][g4][j][r]; then each thread
        // takes such a run of 4 output channels for the 4 waves (16-byte reads) and adds them:
        // run m of the thread is group q = tid + 256 m = (tap, i, g4, j).
        __syncthreads();
        int32_t *red = (int32_t *)lds;        // [wave][3 taps][4 i][4 g4][16 j][4 r]
#pragma unroll
        for (int t0 = 0; t0 < 9; t0 += 3) {
#pragma unroll
            for (int tt = 0; tt < 3; tt++)
#pragma unroll
                for (int i = 0; i < 4; i++)
                    *(v4i *)(red + (wave * 3 + tt) * 1024 + (i * 4 + g4) * 64 + j * 4) = acc[t0 + tt][i];
            __syncthreads();
#pragma unroll
            for (int m = 0; m < 3; m++) {
                const int q = tid + 256 * m;
                const int tt = q >> 8, cl = 4 * ((q >> 4) & 15), ci = ci0 + (q & 15);
                int64_t v[4] = {0, 0, 0, 0};
#pragma unroll
                for (int w = 0; w < 4; w++) {
                    const v4i rv = *(const v4i *)(red + (w * 3 + tt) * 1024 + (q & 255) * 4);
                    const int sh = 8 * (L3 ? (l3 ? l : w / Q) : w / Q);
#pragma unroll
                    for (int r = 0; r < 4; r++) v[r] += (int64_t)rv[r] * ((int64_t)1 << sh);
                }
                if (L3) {
#pragma unroll
                    for (int r = 0; r < 4; r++)
                        tot[L3 ? t0 / 3 : 0][4 * m + r] = pass == 0 ? v[r] : tot[L3 ? t0 / 3 : 0][4 * m + r] + v[r];
                } else {
#pragma unroll
                    for (int r = 0; r < 4; r++) {
                        const int co = co0 + cl + r;
                        if (co < p.co && ci < p.ci_out)
                            p.out[(((int64_t)split * p.co + co) * 9 + t0 + tt) * p.ci_out + ci] = v[r];
                    }
                }
            }
            __syncthreads();
        }
    }
    if (L3) {
#pragma unroll
        for (int t0 = 0; t0 < 9; t0 += 3)
#pragma unroll
            for (int m = 0; m < 3; m++) {
                const int q = tid + 256 * m;
                const int tt = q >> 8, cl = 4 * ((q >> 4) & 15), ci = ci0 + (q & 15);
#pragma unroll
                for (int r = 0; r < 4; r++) {
                    const int co = co0 + cl + r;
                    if (co < p.co && ci < p.ci_out)
                        p.out[(((int64_t)split * p.co + co) * 9 + t0 + tt) * p.ci_out + ci] =
                            tot[L3 ? t0 / 3 : 0][4 * m + r];
                }
            }
    }
    ts_end(p.ts);
}

void launch_conv_dw_planes(hipStream_t s, const ConvShape &sh, const int32_t *g,
                           const uint32_t *gmax, const int8_t *x, int8_t *gp, int8_t *xp,
                           int8_t *gn, int64_t *part, int64_t *dw, uint32_t *flags,
                           bool x_rows_ready, const uint8_t *pool_code, const int16_t *g16,
                           const GOff *goff)
{
    const DwpGeom ge = dwp_geom(sh);
    const DwpPlan pl = dwp_plan(sh);
    const int c16 = dwp_c16(sh);
    {
        DwpPrep pa{};
        pa.rows = x_rows_ready ? 2 : 1;
        const int64_t pads = (int64_t)sh.n * (sh.h + sh.w + 1) + DWP_HMAX + (ge.xs - DWP_HMAX - ge.kraw);
        pa.rows_gx = (int)(((x_rows_ready ? pads : ge.xs) + 255) / 256);
        pa.rows_gy = c16 / 16;
        pa.gp_gx = (int)(ge.kp / 64);
        pa.x = x; pa.n = sh.n; pa.h = sh.h; pa.w = sh.w; pa.c = sh.c; pa.co = sh.co;
        pa.hp = ge.hp; pa.wp = ge.wp; pa.kp = (int)ge.kp; pa.kraw = ge.kraw; pa.xs = ge.xs; pa.xr = xp;
        pa.g = g; pa.g16 = g16; pa.gmax = gmax; pa.pcode = pool_code; pa.gp = gp; pa.gn = gn;
        const bool goff_dw = goff && goff->xq && dwp_goff_ok(sh);
        if (goff) pa.go = *goff;
        pa.goff_dx = goff && gn;
        pa.goff_dw = goff_dw;
        pa.xs_n = goff_dw ? sh.n * (sh.c / 64) : 0;
        const int64_t nwg = pa.xs_n + (int64_t)pa.rows_gx * pa.rows_gy + (int64_t)pa.gp_gx * ((sh.co + 63) / 64);
        hipLaunchKernelGGL(k_dwp_prep, dim3((unsigned)nwg), dim3(256), 0, s, pa);
    }
    DwpArgs a{};
    a.gp = gp; a.kp = ge.kp;
    a.xr = xp; a.xs = ge.xs;
    a.wp = ge.wp; a.co = sh.co; a.ci = c16; a.ci_out = sh.c;
    a.tiles_ci = pl.tiles_ci; a.tiles_co = pl.tiles_co; a.nss = pl.nss; a.chunk = pl.chunk;
    a.gmax = gmax;
    a.out = pl.nsplit > 1 ? part : dw;
    a.flags = flags;
    const bool goff_dw = goff && goff->xq && dwp_goff_ok(sh);
    if (goff_dw) {
        a.goff = 1;
        a.goff_count = goff->count;
    }
    const size_t lds_stage = (size_t)4 * 2 * DWP_WIN * 16, lds_red = (size_t)4 * 3 * 1024 * 4;
    const unsigned nwg = (unsigned)(pl.tiles_co * pl.tiles_ci * pl.nsplit);
    a.ts = timer_slot(TIMED_DW);
    const size_t lds = lds_stage > lds_red ? lds_stage : lds_red;
    {
        TimedLaunch tl(TIMED_DW, s);
        if (pl.chunk >= DWP_L3_MIN)
            hipLaunchKernelGGL(k_conv_dw_planes<true>, dim3(nwg), dim3(256), lds, s, a);
        else
            hipLaunchKernelGGL(k_conv_dw_planes<false>, dim3(nwg), dim3(256), lds, s, a);
    }
    if (goff_dw)
        launch_sum_partials_goff(s, part, pl.nsplit, (int64_t)sh.co * 9 * sh.c, dw, goff->xq, sh.c, gmax);
    else if (pl.nsplit > 1)
        launch_sum_partials(s, part, pl.nsplit, (int64_t)sh.co * 9 * sh.c, dw);
}

bool dwp_goff_ok(const ConvShape &sh)
{
    return dwp_ok(sh) && sh.c % 64 == 0 && dwp_plan(sh).nsplit > 1;
}

}  // namespace nitro
