// Implicit-GEMM 3x3 IntConv2D (section 3.2.1; 3x3, stride 1, pad 1 per Tab. 1) on gfx950 int8
// MFMA with the input tile staged once per channel chunk, exact:
//   forward         z[p][co]  = sum_{r,s,ci} x[p + (r-1, s-1)][ci] * W[co][r][s][ci]
//   input gradient  dx[p][ci] = sum_{r,s,co} g[p - (r-1, s-1)][co] * W[co][r][s][ci]
//
// A workgroup computes 128 output pixels that are whole image rows (rows of one image, or several
// whole small images) times 64 GEMM columns. For each chunk of input channels it stages in LDS
// the pixels those rows need: the rows themselves, one row above and one below, and one column
// on each side, zeros outside the image. The A fragment of tap (r, s) is then the LDS pixel at
// offset (r-1)(W+2) + (s-1) from the output pixel (the opposite offset for the input gradient):
// the nine taps share one staging and need no bounds tests. The B operand (4 packed limb planes
// of W, [N][9 ck], tap-major) is read from global memory one K-step ahead. Operands wider than
// int8 are split into balanced int8 limbs; each limb pair is one pass over K accumulated in int32
// (|sum| <= 128 * 128 * 9 * 8192 < 2^31) and folded into int64 with its shift.
#include "mfma_common.h"

namespace nitro {

enum { IG_FWD = 0, IG_DX = 1 };

constexpr int CT_BM = 128;         // output pixels per workgroup
constexpr int CT_BN = 64;          // GEMM columns per workgroup
constexpr int CT_NPMAX = 320;      // largest staged pixel count (W >= 4)

template <int CC>
struct CtCfg {
    static constexpr int PS = CC == 16 ? 16 : CC == 32 ? 48 : 80;   // LDS bytes per pixel
    static constexpr int GPT = CC / 16;                 // 16-channel groups per tap and chunk
    static constexpr int KSC = (9 * GPT + 3) / 4;        // K-steps (of 4 groups) per chunk
    static constexpr int NIT = (CT_NPMAX * GPT + 255) / 256;   // staged 16-byte items per thread
};

struct TileArgs {
    int n, h, w;
    int ck;                        // channels of A; K = 9 ck (a multiple of the chunk size CC)
    int no;                        // GEMM N (a multiple of 16)
    const int8_t *a;               // forward: x NHWC; input gradient: limb planes [LA][P][ck]
    int64_t aplane;                // P * ck
    const uint32_t *a_max;         // input gradient: max|g| slot
    const int8_t *b;               // 4 limb planes [no][9 ck]
    int64_t bplane;                // no * 9 ck
    const uint32_t *b_max;
    int rt, ns, rs;                // image rows per tile; images per tile; rows per image segment
    Div32 d_w2, d_seg, d_w, d_rw;  // reciprocals of W + 2, (rs + 2)(W + 2), W and rs W
    // forward epilogue
    ScaleRelu32 sr;
    int pool;
    int8_t *out;
    uint8_t *code;
    // input-gradient epilogue
    const uint8_t *prev_code;
    Relu rp;
    int32_t *gout;
    int64_t *out64;
    uint32_t *gmax;
    uint32_t *flags;
    uint64_t *ts;                  // timing slot (null: untimed)
};

__device__ inline int32_t sat_i32(int64_t v)
{
    return v > INT32_MAX ? INT32_MAX : (v < INT32_MIN ? INT32_MIN : (int32_t)v);
}

// One tile per workgroup. B fragments are prefetched BD K-steps ahead (a ring of BD + 1 register
// sets, the K-step loop unrolled per chunk); the next chunk's A staging is loaded while the
// current chunk computes.
template <int MODE, int CC>
__global__ __launch_bounds__(256) void k_conv_tile(TileArgs p)
{
    using C = CtCfg<CC>;
    constexpr int TM = 4, TN = 2;                 // 16x16 tiles per wave: 64 pixels x 32 columns
    constexpr int BD = 3;                         // B prefetch distance (K-steps)
    constexpr int STAGE = CT_NPMAX * C::PS;
    constexpr int SMEM_A = 2 * STAGE;
    constexpr int OS = CT_BN + 16;                // epilogue byte-tile row stride (forward)
    constexpr int GS = CT_BN + 1;                 // epilogue int32-tile row stride (input gradient)
    constexpr int SMEM_EPI = MODE == IG_FWD ? 2 * CT_BM * OS : CT_BM * GS * 4;
    constexpr int SMEM = SMEM_A > SMEM_EPI ? SMEM_A : SMEM_EPI;
    __shared__ __attribute__((aligned(16))) uint8_t smem[SMEM];

    ts_start(p.ts);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int g4 = lane >> 4;
    const int W2 = p.w + 2;
    const int segpx = (p.rs + 2) * W2;
    const int np = p.ns * segpx;
    const int R0 = blockIdx.x * p.rt;              // first image row of the tile (over all images)
    const int img0 = R0 / p.h, row0 = R0 - img0 * p.h;
    const int64_t M = (int64_t)p.n * p.h * p.w;
    const int64_t m0 = (int64_t)R0 * p.w;
    const int n0 = blockIdx.y * CT_BN;
    const int K = 9 * p.ck;
    const int nchunk = p.ck / CC;

    const int LA = MODE == IG_FWD ? 1 : limbs_for(slot_read(p.a_max));
    const int LB = limbs_for(slot_read(p.b_max));
    if (LA > 4 || LB > 4) {
        if (tid == 0) raise_flag(p.flags, FLAG_OVERFLOW);
        return;
    }
    const int npass = LA * LB;

    // staged items of this thread: item tid + 256 v = (LDS pixel q, 16-channel group e); the
    // global byte offset within a chunk, or -1 for a zero (outside the image)
    int it_g[C::NIT];
#pragma unroll
    for (int v = 0; v < C::NIT; v++) {
        const int item = tid + 256 * v;
        const int q = item / C::GPT, e = item - q * C::GPT;
        it_g[v] = -1;
        if (q < np) {
            const int seg = (int)udiv32(q, p.d_seg), r = q - seg * segpx;
            const int lr = (int)udiv32(r, p.d_w2), lc = r - lr * W2;
            const int img = img0 + seg, hh = row0 + lr - 1, ww = lc - 1;
            if (img < p.n && hh >= 0 && hh < p.h && ww >= 0 && ww < p.w)
                it_g[v] = ((img * p.h + hh) * p.w + ww) * p.ck + 16 * e;
        }
    }
    int cpix[TM];
#pragma unroll
    for (int i = 0; i < TM; i++) {
        const int mloc = wm * 64 + 16 * i + (lane & 15);
        const int seg = (int)udiv32(mloc, p.d_rw), rem = mloc - seg * p.rs * p.w;
        const int row = (int)udiv32(rem, p.d_w), col = rem - row * p.w;
        cpix[i] = seg * segpx + (row + 1) * W2 + col + 1;
    }
    int brow[TN];
#pragma unroll
    for (int j = 0; j < TN; j++) {
        const int col = n0 + wn * 32 + 16 * j + (lane & 15);
        brow[j] = (col < p.no ? col : p.no - 1) * K;
    }
    const int sgn = MODE == IG_FWD ? 1 : -1;

    v4i stg[C::NIT];
    auto stage_load = [&](int la, int chunk) {
        const int8_t *src = p.a + (int64_t)la * p.aplane + chunk * CC;
#pragma unroll
        for (int v = 0; v < C::NIT; v++) stg[v] = *(const v4i *)(src + (it_g[v] >= 0 ? it_g[v] : 0));
    };
    auto stage_store = [&](int buf) {
        uint8_t *dst = smem + buf * STAGE;
#pragma unroll
        for (int v = 0; v < C::NIT; v++) {
            const int item = tid + 256 * v;
            const int q = item / C::GPT, e = item - q * C::GPT;
            if (q < np) *(v4i *)(dst + q * C::PS + 16 * e) = it_g[v] >= 0 ? stg[v] : v4i{0, 0, 0, 0};
        }
    };
    auto kslice = [&](int ks, int &t, int &c16) {
        const int G = 4 * ks + g4;
        t = G / C::GPT;
        c16 = G - t * C::GPT;
    };
    // B fragments of K-step ks of a chunk
    auto load_b = [&](v4i(&dst)[TN], int lb, int chunk, int ks) {
        int t, c16;
        kslice(ks, t, c16);
        const int tc = t < 9 ? t : 8;
        const int8_t *src = p.b + (int64_t)lb * p.bplane + tc * p.ck + chunk * CC + 16 * c16;
#pragma unroll
        for (int j = 0; j < TN; j++) dst[j] = *(const v4i *)(src + brow[j]);
    };

    int64_t acc64[TM][TN][4];
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++)
#pragma unroll
            for (int t = 0; t < 4; t++) acc64[i][j][t] = 0;
    v4i acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++) acc[i][j] = v4i{0, 0, 0, 0};

    for (int la = 0; la < LA; la++) {
        for (int lb = 0; lb < LB; lb++) {
            stage_load(la, 0);
            stage_store(0);
            __syncthreads();
            for (int chunk = 0; chunk < nchunk; chunk++) {
                const bool more = chunk + 1 < nchunk;
                if (more) stage_load(la, chunk + 1);
                v4i bq[BD + 1][TN];               // ring of prefetched B fragments
#pragma unroll
                for (int d = 0; d < BD && d < C::KSC; d++) load_b(bq[d], lb, chunk, d);
                const uint8_t *As = smem + (chunk & 1) * STAGE;
#pragma unroll
                for (int ks = 0; ks < C::KSC; ks++) {
                    if (ks + BD < C::KSC) load_b(bq[(ks + BD) % (BD + 1)], lb, chunk, ks + BD);
                    int t, c16;
                    kslice(ks, t, c16);
                    const bool valid = t < 9;
                    const int tc = valid ? t : 8;
                    const int toff = sgn * ((tc / 3 - 1) * W2 + (tc % 3 - 1));
                    v4i af[TM];
#pragma unroll
                    for (int i = 0; i < TM; i++) {
                        const v4i v = *(const v4i *)(As + (cpix[i] + toff) * C::PS + 16 * c16);
                        af[i] = valid ? v : v4i{0, 0, 0, 0};
                    }
#pragma unroll
                    for (int i = 0; i < TM; i++)
#pragma unroll
                        for (int j = 0; j < TN; j++)
                            acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bq[ks % (BD + 1)][j],
                                                                              acc[i][j], 0, 0, 0);
                }
                if (more) stage_store((chunk + 1) & 1);
                __syncthreads();
            }
            if (npass > 1) {
                // fold this limb pass into int64 with its weight 256^(la + lb)
                const int64_t sh = (int64_t)1 << (8 * (la + lb));
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int j = 0; j < TN; j++) {
#pragma unroll
                        for (int t = 0; t < 4; t++) acc64[i][j][t] += (int64_t)acc[i][j][t] * sh;
                        acc[i][j] = v4i{0, 0, 0, 0};
                    }
            }
        }
    }
    auto value = [&](int i, int j, int t) -> int64_t {
        return npass > 1 ? acc64[i][j][t] : (int64_t)acc[i][j][t];
    };

    // ---------------------------------------------------------------- epilogues
    if (MODE == IG_FWD) {
        // NITRO-Scaling + NITRO-ReLU per element into LDS, then coalesced (and pooled) stores.
        // Several passes: the int64 sum saturated to int32 still saturates z* (128 SF < 2^31).
        uint8_t *Os = smem;                   // [BM][OS] int8 activations
        uint8_t *Rs = smem + CT_BM * OS;      // [BM][OS] region codes
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++)
#pragma unroll
                for (int t = 0; t < 4; t++) {
                    const int row = wm * 64 + i * 16 + g4 * 4 + t;
                    const int col = wn * 32 + j * 16 + (lane & 15);
                    uint8_t reg;
                    const int32_t a = scale_relu32(sat_i32(value(i, j, t)), p.sr, reg);
                    Os[row * OS + col] = (uint8_t)(int8_t)a;
                    Rs[row * OS + col] = reg;
                }
        __syncthreads();
        if (!p.pool) {
            for (int c = tid; c < CT_BM * CT_BN / 16; c += 256) {
                const int row = c / (CT_BN / 16), cc = (c % (CT_BN / 16)) * 16;
                const int64_t m = m0 + row;
                if (m >= M || n0 + cc >= p.no) continue;
                const int64_t o = m * p.no + n0 + cc;
                *(v4i *)(p.out + o) = *(const v4i *)(Os + row * OS + cc);
                *(v4i *)(p.code + o) = *(const v4i *)(Rs + row * OS + cc);
            }
        } else {
            // 2x2 windows, 4 channels per thread: the tile holds rt (even) whole image rows
            const int W = p.w, Wh = p.w / 2;
            for (int c = tid; c < (CT_BM / 4) * (CT_BN / 4); c += 256) {
                const int win = c / (CT_BN / 4), col = (c % (CT_BN / 4)) * 4;
                const int wr = win / Wh, wc = win - wr * Wh;
                const int q = 2 * wr * W + 2 * wc;
                const int64_t m = m0 + q;
                if (m >= M || n0 + col >= p.no) continue;
                uint32_t ov = 0, cv = 0;
#pragma unroll
                for (int e = 0; e < 4; e++) {
                    int best = -1000, arg = 0;
                    uint8_t breg = 0;
#pragma unroll
                    for (int t = 0; t < 4; t++) {
                        const int at = q + (t >> 1) * W + (t & 1);
                        const int v = (int)(int8_t)Os[at * OS + col + e];
                        if (v > best) { best = v; arg = t; breg = Rs[at * OS + col + e]; }
                    }
                    ov |= (uint32_t)(uint8_t)(int8_t)best << (8 * e);
                    cv |= (uint32_t)(arg | (breg << 2)) << (8 * e);
                }
                const int64_t grow = m / W;
                const int64_t pp = (grow / 2) * Wh + (m % W) / 2;
                const int64_t o = pp * p.no + n0 + col;
                *(uint32_t *)(p.out + o) = ov;
                *(uint32_t *)(p.code + o) = cv;
            }
        }
    } else if (p.out64) {
        // raw int64 input gradient (the first layer of a network)
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++)
#pragma unroll
                for (int t = 0; t < 4; t++) {
                    const int64_t m = m0 + wm * 64 + i * 16 + g4 * 4 + t;
                    const int col = n0 + wn * 32 + j * 16 + (lane & 15);
                    if (m < M && col < p.no) p.out64[m * p.no + col] = value(i, j, t);
                }
    } else {
        // int32 sums into LDS, then 16 channels per thread: ReLU' with 16 codes, 64-byte rows
        int32_t *Gs = (int32_t *)smem;        // [BM][GS]
        bool bad = false;
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++)
#pragma unroll
                for (int t = 0; t < 4; t++) {
                    const int row = wm * 64 + i * 16 + g4 * 4 + t;
                    const int col = wn * 32 + j * 16 + (lane & 15);
                    const int64_t v = value(i, j, t);
                    bad |= !fits_i32(v);
                    Gs[row * GS + col] = (int32_t)v;
                }
        __syncthreads();
        uint32_t mx = 0;
        for (int c = tid; c < CT_BM * CT_BN / 16; c += 256) {
            const int row = c / (CT_BN / 16), cc = (c % (CT_BN / 16)) * 16;
            const int64_t m = m0 + row;
            if (m >= M || n0 + cc >= p.no) continue;
            const int64_t o = m * p.no + n0 + cc;
            v4i cd = v4i{0, 0, 0, 0};
            if (p.prev_code) cd = *(const v4i *)(p.prev_code + o);
            v4i outv[4];
#pragma unroll
            for (int e = 0; e < 16; e++) {
                const int32_t v = Gs[row * GS + cc + e];
                int64_t gv = v;
                if (p.prev_code) gv = relu_bwd(v, (uint8_t)((uint32_t)cd[e >> 2] >> (8 * (e & 3))), p.rp);
                outv[e >> 2][e & 3] = (int32_t)gv;
                const uint32_t ag = abs_u32((int32_t)gv);
                mx = ag > mx ? ag : mx;
            }
#pragma unroll
            for (int q = 0; q < 4; q++) *(v4i *)(p.gout + o + 4 * q) = outv[q];
        }
        if (bad) raise_flag(p.flags, FLAG_OVERFLOW);
        if (p.gmax) block_slot_max(p.gmax, mx);
    }
    ts_end(p.ts);
}

// Tile geometry: rt = 128 / W image rows; either rt divides H (one image segment) or H divides
// rt (rt / H whole images); at most CT_NPMAX staged pixels.
static bool tile_geom(int h, int w, int *rt, int *ns, int *rs)
{
    if (w < 1 || w > CT_BM || CT_BM % w) return false;
    *rt = CT_BM / w;
    if (*rt <= h) {
        if (h % *rt) return false;
        *ns = 1;
        *rs = *rt;
    } else {
        if (*rt % h) return false;
        *ns = *rt / h;
        *rs = h;
    }
    return *ns * (*rs + 2) * (w + 2) <= CT_NPMAX;
}

static bool tile_chunk_ok(int ck) { return ck == 16 || ck == 32 || (ck % 64 == 0 && ck <= 8192); }

bool tile_conv_fwd_ok(const ConvShape &sh, bool pool, int64_t sf, int alpha_inv)
{
    int rt, ns, rs;
    if (!tile_geom(sh.h, sh.w, &rt, &ns, &rs) || !tile_chunk_ok(sh.c) || sh.co % 16) return false;
    if (pool && (rt % 2 || sh.h % 2 || sh.w % 2)) return false;
    return (int64_t)sh.n * sh.h * sh.w * sh.c < ((int64_t)1 << 31) &&
           (int64_t)sh.co * 9 * sh.c < ((int64_t)1 << 31) && scale_relu32_ok(sf, alpha_inv) &&
           128 * sf < ((int64_t)1 << 31);   // a saturated int32 sum still saturates z*
}

bool tile_conv_dx_ok(const ConvShape &sh)
{
    int rt, ns, rs;
    if (!tile_geom(sh.h, sh.w, &rt, &ns, &rs) || !tile_chunk_ok(sh.co) || sh.c % 16) return false;
    return (int64_t)sh.n * sh.h * sh.w * sh.co < ((int64_t)1 << 31) &&
           (int64_t)sh.co * 9 * sh.c < ((int64_t)1 << 31);
}

template <int MODE>
static void launch_tile(hipStream_t s, TileArgs a)
{
    a.d_w2 = make_div32((uint32_t)(a.w + 2));
    a.d_seg = make_div32((uint32_t)((a.rs + 2) * (a.w + 2)));
    a.d_w = make_div32((uint32_t)a.w);
    a.d_rw = make_div32((uint32_t)(a.rs * a.w));
    const dim3 grid((unsigned)((a.n * a.h + a.rt - 1) / a.rt), (unsigned)((a.no + CT_BN - 1) / CT_BN));
    a.ts = timer_slot(MODE == IG_FWD ? TIMED_CONV_FWD : TIMED_CONV_DX);
    switch (a.ck == 16 ? 16 : a.ck == 32 ? 32 : 64) {
    case 16: hipLaunchKernelGGL((k_conv_tile<MODE, 16>), grid, dim3(256), 0, s, a); break;
    case 32: hipLaunchKernelGGL((k_conv_tile<MODE, 32>), grid, dim3(256), 0, s, a); break;
    default: hipLaunchKernelGGL((k_conv_tile<MODE, 64>), grid, dim3(256), 0, s, a); break;
    }
}

void launch_conv_fwd_tile(hipStream_t s, const ConvShape &sh, const int8_t *x, const int8_t *wf,
                          const uint32_t *wmax, int64_t sf, int alpha_inv, int round,
                          const Relu &rp, bool pool, int8_t *out, uint8_t *code, uint32_t *flags)
{
    TileArgs a{};
    a.n = sh.n; a.h = sh.h; a.w = sh.w;
    a.ck = sh.c; a.no = sh.co;
    a.a = x; a.aplane = 0; a.a_max = nullptr;
    a.b = wf; a.bplane = (int64_t)sh.co * 9 * sh.c; a.b_max = wmax;
    tile_geom(sh.h, sh.w, &a.rt, &a.ns, &a.rs);
    a.sr = make_scale_relu32(sf, alpha_inv, rp.mu, round);
    a.pool = pool ? 1 : 0;
    a.out = out; a.code = code;
    a.flags = flags;
    launch_tile<IG_FWD>(s, a);
}

void launch_conv_dx_tile(hipStream_t s, const ConvShape &sh, const int8_t *gl,
                         const uint32_t *gmax_in, const int8_t *wt, const uint32_t *wmax,
                         const uint8_t *prev_code, const Relu &rp, int32_t *gout, int64_t *out64,
                         uint32_t *gmax_out, uint32_t *flags)
{
    TileArgs a{};
    a.n = sh.n; a.h = sh.h; a.w = sh.w;
    a.ck = sh.co; a.no = sh.c;
    a.a = gl; a.aplane = (int64_t)sh.n * sh.h * sh.w * sh.co; a.a_max = gmax_in;
    a.b = wt; a.bplane = (int64_t)sh.c * 9 * sh.co; a.b_max = wmax;
    tile_geom(sh.h, sh.w, &a.rt, &a.ns, &a.rs);
    a.rp = rp;
    a.prev_code = prev_code; a.gout = gout; a.out64 = out64; a.gmax = gmax_out;
    a.flags = flags;
    launch_tile<IG_DX>(s, a);
}

}  // namespace nitro
