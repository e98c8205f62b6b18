// Implicit-GEMM 3x3 convolutions on gfx950 int8 MFMA (v_mfma_i32_16x16x64_i8), exact.
//
// Operands wider than int8 are split into balanced signed base-256 limbs: v = sum_l d_l 256^l
// with d_l in [-128, 127]. Every limb pair is one pass over K with int32 accumulators (each
// product term is at most 128*128 and K <= 9*4096, so a pass cannot overflow int32); passes are
// folded into int64 accumulators with the limb shift. The number of limbs of each operand is
// read at run time from a device-side max|.| slot written by the operand's producer, so no host
// synchronisation is needed and a pass is skipped when its limb is zero everywhere.
//
// GEMM view (rows = output pixels, K = 9 taps x channels, tap-major):
//   forward     z[p][co]  = sum_{r,s,ci} x[p + (r-1, s-1)][ci] * W[co][r][s][ci]
//   input grad  dx[p][ci] = sum_{r,s,co} g[p - (r-1, s-1)][co] * W[co][r][s][ci]
// The B operand is a packed limb plane [N][9*CK] (int8), K-contiguous, produced per call by
// k_pack_conv_weights (forward: W itself; input gradient: W with its two channel axes swapped).
#include <type_traits>

#include "mfma_common.h"

namespace nitro {

// ---------------------------------------------------------------------------------------------
// Weight packing: W int32 KRSC [co][3][3][ci] -> 4 limb planes of [co][9 cpad] (forward; input
// channels ci..cpad-1 are zeros) and, when wt != null, of [ci][9 co] with the same tap order
// (input gradient); max|W| -> the max slot wmax. Two passes, each with coalesced stores: the
// forward planes in W's own order, the swapped planes in their order (gathering W through the
// cache).
__global__ void k_pack_conv_weights(const int32_t *__restrict__ w, uint32_t total, int ci,
                                    int cpad, int8_t *__restrict__ wf, uint32_t *wmax)
{
    pack_conv_weights_part(w, total, ci, cpad, wf, wmax, blockIdx.x, gridDim.x);
}

__global__ void k_pack_conv_weights_t(const int32_t *__restrict__ w, uint32_t co, uint32_t ci,
                                      int8_t *__restrict__ wt)
{
    pack_conv_weights_t_part(w, co, ci, wt, blockIdx.x);
}

void launch_pack_conv_weights(hipStream_t s, const int32_t *w, int co, int ci, int cpad,
                              int8_t *wf, int8_t *wt, uint32_t *wmax)
{
    const uint32_t total = (uint32_t)co * 9 * (uint32_t)ci;
    const uint32_t total_pad = (uint32_t)co * 9 * (uint32_t)cpad;
    const dim3 grid((total + 255) / 256);
    hipLaunchKernelGGL(k_pack_conv_weights, dim3(grid_stride_blocks(total_pad)), dim3(256), 0, s,
                       w, total_pad, ci, cpad, wf, wmax);
    if (wt)
        hipLaunchKernelGGL(k_pack_conv_weights_t, grid, dim3(256), 0, s, w, (uint32_t)co,
                           (uint32_t)ci, wt);
}

void launch_pack_linear_weights(hipStream_t s, const int32_t *w, int co, int ci, int cpad,
                                int8_t *wf, uint32_t *wmax)
{
    // (the element-wise pack of the conv weights with one tap: row r = output, column c < ci)
    const uint32_t total_pad = (uint32_t)co * (uint32_t)cpad;
    hipLaunchKernelGGL(k_pack_conv_weights, dim3(grid_stride_blocks(total_pad)), dim3(256), 0, s,
                       w, total_pad, ci, cpad, wf, wmax);
}

// x int8 [P][c] -> [P][16] with zero channels c..15 (c < 16): the forward GEMM's K then takes
// whole 16-channel chunks per tap.
__global__ __launch_bounds__(256) void k_pad_channels16(const int8_t *__restrict__ x, int P, int c,
                                                        int8_t *__restrict__ xpad)
{
    pad_channels16_part(x, P, c, xpad, blockIdx.x);
}

void launch_pad_channels16(hipStream_t s, const int8_t *x, int P, int c, int8_t *xpad)
{
    hipLaunchKernelGGL(k_pad_channels16, dim3((unsigned)((P + 255) / 256)), dim3(256), 0, s, x, P,
                       c, xpad);
}

// ---------------------------------------------------------------------------------------------
struct IgemmArgs {
    int n, h, w;                 // image geometry (output pixels = input pixels)
    int ck;                      // channels of the A source; K = 9 * ck
    int no;                      // GEMM N: output channels of this GEMM
    const void *a;               // A source, NHWC: int8 (forward) or int32 (input gradient)
    const uint32_t *a_max;       // max|A| (input gradient only)
    const int8_t *b;             // 4 limb planes [no][9 ck]
    const uint32_t *b_max;       // max|B|
    // forward epilogue
    Div sf;
    Relu rp;
    int pool;
    int8_t *out;                 // int8 activations (pooled when pool)
    uint8_t *code;               // region codes (pooled: argmax | region << 2)
    // input-gradient epilogue
    const uint8_t *prev_code;    // region codes of the previous layer (null: raw output)
    int32_t *gout;               // int32 gradient of the previous layer
    int64_t *out64;              // raw int64 input gradient (first layer)
    uint32_t *gmax;              // max|gout|
    uint32_t *flags;
};

enum { IG_FWD = 0, IG_DX = 1 };

constexpr int IG_BK = 64;            // K per step = one MFMA K
constexpr int IG_LDS_STRIDE = 80;    // bytes per LDS row (64 + 16 pad)

// BM x BN tile per 256-thread workgroup; 4 waves in a 2 x 2 grid, each (BM/2) x (BN/2).
// K steps are software-pipelined: the global loads of step k+1 are issued before the MFMAs of
// step k, and LDS is double-buffered so each step needs one barrier.
template <int MODE, int BM, int BN>
__global__ __launch_bounds__(256) void k_igemm_conv(IgemmArgs p)
{
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int A_CHUNKS = BM * 4 / 256;       // 16-byte chunks of A per thread per step
    constexpr int B_CHUNKS = BN * 4 / 256;
    static_assert(A_CHUNKS >= 1 && B_CHUNKS >= 1, "tile too small");
    constexpr int STAGE = (BM + BN) * IG_LDS_STRIDE;
    constexpr int SMEM_AB = 2 * STAGE;
    constexpr int SMEM_EPI = 2 * BM * BN;
    constexpr int SMEM = SMEM_AB > SMEM_EPI ? SMEM_AB : SMEM_EPI;
    __shared__ __attribute__((aligned(16))) uint8_t smem[SMEM];

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int HW = p.h * p.w;
    const int64_t M = (int64_t)p.n * HW;
    const int64_t m0 = (int64_t)blockIdx.x * BM;
    const int n0 = blockIdx.y * BN;
    const int K = 9 * p.ck;
    const int ksteps = (K + IG_BK - 1) / IG_BK;

    const int LA = MODE == IG_FWD ? 1 : limbs_for(slot_read(p.a_max));
    const int LB = limbs_for(slot_read(p.b_max));
    if (LA > 4 || LB > 4) {
        if (tid == 0) raise_flag(p.flags, FLAG_OVERFLOW);
        return;
    }

    // rows this thread stages: row = tid/4 + 64 i, chunk kc = tid % 4 (fixed over K)
    const int kc = tid & 3;
    int a_h[A_CHUNKS], a_w[A_CHUNKS];
    int64_t a_pix[A_CHUNKS];                      // flattened pixel index of the output row
    for (int i = 0; i < A_CHUNKS; i++) {
        const int64_t m = m0 + (tid >> 2) + 64 * i;
        const bool ok = m < M;
        const int64_t mm = ok ? m : 0;
        const int rem = (int)(mm % HW);
        a_h[i] = ok ? rem / p.w : -100000;        // out-of-range rows never pass the bound test
        a_w[i] = rem % p.w;
        a_pix[i] = mm;
    }
    const int sgn = MODE == IG_FWD ? 1 : -1;

    typedef typename std::conditional<MODE == IG_FWD, v4i[1], v4i[4]>::type ARaw;
    ARaw ar[A_CHUNKS];
    v4i br[B_CHUNKS];

    int64_t acc64[TM][TN][4];
    for (int i = 0; i < TM; i++)
        for (int j = 0; j < TN; j++)
            for (int t = 0; t < 4; t++) acc64[i][j][t] = 0;

    const int64_t plane = (int64_t)p.no * K;
    for (int la = 0; la < LA; la++) {
        for (int lb = 0; lb < LB; lb++) {
            const int8_t *bpl = p.b + lb * plane;
            // position of this thread's 16-value chunk in K: tap and channel, advanced by 64 a step
            int ktap = 0, kci = kc * 16;
            while (kci >= p.ck) { kci -= p.ck; ktap++; }
            auto load = [&](int ks) {
                const int k = ks * IG_BK + kc * 16;
                const bool kin = k < K;
                const int dr = sgn * (ktap / 3 - 1), ds = sgn * (ktap % 3 - 1);
                for (int i = 0; i < A_CHUNKS; i++) {
                    const int hh = a_h[i] + dr, ww = a_w[i] + ds;
                    const bool ok = kin && hh >= 0 && hh < p.h && ww >= 0 && ww < p.w;
                    const int64_t pix = a_pix[i] + (int64_t)dr * p.w + ds;
                    if (MODE == IG_FWD) {
                        ar[i][0] = ok ? *(const v4i *)((const int8_t *)p.a + pix * p.ck + kci)
                                      : v4i{0, 0, 0, 0};
                    } else {
                        const v4i *src = (const v4i *)((const int32_t *)p.a + pix * p.ck + kci);
                        for (int u = 0; u < 4; u++) ar[i][u] = ok ? src[u] : v4i{0, 0, 0, 0};
                    }
                }
                for (int i = 0; i < B_CHUNKS; i++) {
                    const int nn = n0 + (tid >> 2) + 64 * i;
                    br[i] = (kin && nn < p.no) ? *(const v4i *)(bpl + (int64_t)nn * K + k)
                                               : v4i{0, 0, 0, 0};
                }
                kci += IG_BK;
                while (kci >= p.ck) { kci -= p.ck; ktap++; }
            };
            auto store = [&](int buf) {
                uint8_t *As = smem + buf * STAGE;
                uint8_t *Bs = As + BM * IG_LDS_STRIDE;
                for (int i = 0; i < A_CHUNKS; i++) {
                    v4i v;
                    if (MODE == IG_FWD) {
                        v = ar[i][0];
                    } else {
                        for (int u = 0; u < 4; u++)
                            v[u] = (int)limb4(ar[i][u][0], ar[i][u][1], ar[i][u][2], ar[i][u][3], la);
                    }
                    *(v4i *)(As + ((tid >> 2) + 64 * i) * IG_LDS_STRIDE + kc * 16) = v;
                }
                for (int i = 0; i < B_CHUNKS; i++)
                    *(v4i *)(Bs + ((tid >> 2) + 64 * i) * IG_LDS_STRIDE + kc * 16) = br[i];
            };

            v4i acc[TM][TN];
            for (int i = 0; i < TM; i++)
                for (int j = 0; j < TN; j++) acc[i][j] = v4i{0, 0, 0, 0};
            load(0);
            store(0);
            __syncthreads();
            for (int ks = 0; ks < ksteps; ks++) {
                const int cur = ks & 1;
                const bool more = ks + 1 < ksteps;
                if (more) load(ks + 1);
                const uint8_t *As = smem + cur * STAGE;
                const uint8_t *Bs = As + BM * IG_LDS_STRIDE;
                v4i af[TM], bf[TN];
                for (int i = 0; i < TM; i++)
                    af[i] = *(const v4i *)(As + (wm * WM + i * 16 + (lane & 15)) * IG_LDS_STRIDE + (lane >> 4) * 16);
                for (int j = 0; j < TN; j++)
                    bf[j] = *(const v4i *)(Bs + (wn * WN + j * 16 + (lane & 15)) * IG_LDS_STRIDE + (lane >> 4) * 16);
                for (int i = 0; i < TM; i++)
                    for (int j = 0; j < TN; j++)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
                if (more) store(cur ^ 1);
                __syncthreads();
            }
            const int sh = 8 * (la + lb);
            for (int i = 0; i < TM; i++)
                for (int j = 0; j < TN; j++)
                    for (int t = 0; t < 4; t++) acc64[i][j][t] += (int64_t)acc[i][j][t] << sh;
        }
    }

    // ---------------------------------------------------------------- epilogues
    if (MODE == IG_FWD) {
        // NITRO-Scaling + NITRO-ReLU per element into LDS, then coalesced (and pooled) stores.
        uint8_t *Os = smem;             // [BM][BN] int8 activations
        uint8_t *Rs = smem + BM * BN;   // [BM][BN] region codes
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++)
#pragma unroll
                for (int t = 0; t < 4; t++) {
                    const int row = wm * WM + i * 16 + (lane >> 4) * 4 + t;
                    const int col = wn * WN + j * 16 + (lane & 15);
                    uint8_t reg;
                    const int32_t a = relu_fwd(idiv(acc64[i][j][t], p.sf), p.rp, reg);
                    Os[row * BN + col] = (uint8_t)(int8_t)a;
                    Rs[row * BN + col] = reg;
                }
        __syncthreads();
        if (!p.pool) {
            // 16-channel chunks: BM * BN / 16 of them (vector stores need 16-byte alignment)
            const bool vec = (p.no & 15) == 0;
            for (int c = tid; c < BM * BN / 16; c += 256) {
                const int row = c / (BN / 16), cc = (c % (BN / 16)) * 16;
                const int64_t m = m0 + row;
                if (m >= M || n0 + cc >= p.no) continue;
                const int64_t o = m * p.no + n0 + cc;
                if (vec && n0 + cc + 16 <= p.no) {
                    *(v4i *)(p.out + o) = *(const v4i *)(Os + row * BN + cc);
                    *(v4i *)(p.code + o) = *(const v4i *)(Rs + row * BN + cc);
                } else {
                    for (int t = 0; t < p.no - n0 - cc; t++) {
                        p.out[o + t] = (int8_t)Os[row * BN + cc + t];
                        p.code[o + t] = Rs[row * BN + cc + t];
                    }
                }
            }
        } else {
            // windows: the tile holds BM / W whole image rows, starting at an even row
            const int W = p.w, W2 = p.w / 2;
            const int nwin = BM / 4;
            for (int c = tid; c < nwin * BN; c += 256) {
                const int win = c / BN, col = c % BN;
                const int wr = win / W2, wc = win % W2;        // window row / col inside the tile
                const int q = 2 * wr * W + 2 * wc;            // top-left local pixel
                const int64_t m = m0 + q;
                if (m >= M || n0 + col >= p.no) continue;
                int best = -1000, arg = 0;
                uint8_t breg = 0;
#pragma unroll
                for (int t = 0; t < 4; t++) {
                    const int at = q + (t >> 1) * W + (t & 1);
                    const int v = (int)(int8_t)Os[at * BN + col];
                    if (v > best) { best = v; arg = t; breg = Rs[at * BN + col]; }
                }
                const int64_t grow = m / W;                   // global image row (all images)
                const int64_t pp = (grow / 2) * W2 + (m % W) / 2;
                const int64_t o = pp * p.no + n0 + col;
                p.out[o] = (int8_t)best;
                p.code[o] = (uint8_t)(arg | (breg << 2));
            }
        }
    } else {
        uint32_t mx = 0;
        bool bad = false;
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++)
#pragma unroll
                for (int t = 0; t < 4; t++) {
                    const int64_t m = m0 + wm * WM + i * 16 + (lane >> 4) * 4 + t;
                    const int col = n0 + wn * WN + j * 16 + (lane & 15);
                    if (m >= M || col >= p.no) continue;
                    const int64_t v = acc64[i][j][t];
                    const int64_t o = m * p.no + col;
                    if (p.out64) {
                        p.out64[o] = v;
                        continue;
                    }
                    bad |= !fits_i32(v);
                    int64_t g = v;
                    if (p.prev_code) g = relu_bwd(v, p.prev_code[o], p.rp);
                    bad |= !fits_i32(g);
                    p.gout[o] = (int32_t)g;
                    const uint32_t ag = abs_u32((int32_t)g);
                    mx = ag > mx ? ag : mx;
                }
        if (bad) raise_flag(p.flags, FLAG_OVERFLOW);
        if (p.gmax) block_slot_max(p.gmax, mx);
    }
}

// One tile shape: 128 output pixels x 64 GEMM columns per workgroup.
template <int MODE>
static void launch_igemm(hipStream_t s, const IgemmArgs &a)
{
    const int64_t M = (int64_t)a.n * a.h * a.w;
    constexpr int BM = 128, BN = 64;
    dim3 grid((unsigned)((M + BM - 1) / BM), (unsigned)((a.no + BN - 1) / BN));
    hipLaunchKernelGGL((k_igemm_conv<MODE, BM, BN>), grid, dim3(256), 0, s, a);
}

// K = 9 * ck <= 9 * 8192 keeps 128 * 128 * K below 2^31 (one limb pass in int32).
bool mfma_conv_fwd_ok(const ConvShape &sh, bool pool)
{
    return sh.c % 16 == 0 && sh.c <= 8192 &&
           (!pool || (sh.w % 2 == 0 && sh.h % 2 == 0 && 128 % (2 * sh.w) == 0));
}

bool mfma_conv_dx_ok(const ConvShape &sh) { return sh.co % 16 == 0 && sh.co <= 8192; }

void launch_conv_fwd_mfma(hipStream_t s, const ConvShape &sh, const int8_t *x, const int8_t *wf,
                          const uint32_t *wmax, const Div &sf, const Relu &rp, bool pool,
                          int8_t *out, uint8_t *code, uint32_t *flags)
{
    IgemmArgs a{};
    a.n = sh.n; a.h = sh.h; a.w = sh.w;
    a.ck = sh.c; a.no = sh.co;
    a.a = x; a.a_max = nullptr;
    a.b = wf; a.b_max = wmax;
    a.sf = sf; a.rp = rp; a.pool = pool ? 1 : 0;
    a.out = out; a.code = code;
    a.flags = flags;
    launch_igemm<IG_FWD>(s, a);
}

void launch_conv_dx_mfma(hipStream_t s, const ConvShape &sh, const int32_t *g, const uint32_t *gmax_in,
                         const int8_t *wt, const uint32_t *wmax, const uint8_t *prev_code,
                         const Relu &rp, int32_t *gout, int64_t *out64, uint32_t *gmax_out,
                         uint32_t *flags)
{
    IgemmArgs a{};
    a.n = sh.n; a.h = sh.h; a.w = sh.w;
    a.ck = sh.co; a.no = sh.c;
    a.a = g; a.a_max = gmax_in;
    a.b = wt; a.b_max = wmax;
    a.rp = rp;
    a.prev_code = prev_code; a.gout = gout; a.out64 = out64; a.gmax = gmax_out;
    a.flags = flags;
    launch_igemm<IG_DX>(s, a);
}


// =============================================================================================
// Weight gradient: dW[co][r][s][ci] = sum_p g[p][co] * x[p + (r-1, s-1)][ci]  (int64 result)
//
// GEMM with M = co, N = (tap, ci), K = pixels. Both operands are stored channel-contiguous
// (NHWC), so each 4 pixel x 4 channel byte block is transposed in registers (v_perm_b32) on its
// way into LDS, where rows are K(pixel)-contiguous as the MFMA lanes read them. One workgroup owns
// 64 output channels x 16 input channels x all 9 taps over a chunk of pixels; the x tile of each
// tap is staged with its shift applied and zeros outside the image. All limbs of g are staged in
// the same pass (one accumulator set per limb). Chunks are combined with int64 atomics (integer
// addition commutes, so the result does not depend on their order). A chunk has at most 2^17
// pixels, so a limb's int32 accumulator cannot overflow (|x d| <= 128 * 128).
// =============================================================================================
struct DwArgs {
    int n, h, w, ci, co;
    const int8_t *gt;            // limb planes of g, [4][co][pstride] (pixel-contiguous rows)
    int64_t pstride;             // row length of a plane (>= P, multiple of 64)
    const uint32_t *gmax;        // max|g|
    const int8_t *x;             // NHWC [P][ci]
    int64_t *part;               // [chunks][co][9][ci]: this chunk's partial sums
    int kc;                      // pixels per chunk (multiple of 64)
    uint32_t *flags;
};

// ---------------------------------------------------------------------------------------------
// g int32 NHWC [P][C] -> limb planes [l][C][pstride] for l < limbs(max|g|), rows pixel-contiguous
// (pixels P..pstride-1 are written as zeros). One thread: 4 pixels x 4 channels.
__global__ __launch_bounds__(256) void k_grad_limb_planes(const int32_t *__restrict__ g, int P,
                                                          int C, int64_t pstride,
                                                          const uint32_t *gmax,
                                                          int8_t *__restrict__ gt)
{
    const int LA = limbs_for(slot_read(gmax));
    const int cq4 = (C + 3) / 4;
    const int64_t pq4 = pstride / 4;
    const int64_t task = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t ntask = pq4 * cq4;
    if (task >= ntask || LA > 4) return;
    // pixel quads vary fastest: the plane stores of a wave are contiguous
    const int cq = (int)(task / pq4);
    const int64_t p0 = (task % pq4) * 4;
    const int c0 = cq * 4;
    int32_t v[4][4];
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < 4; j++)
            v[i][j] = (p0 + i < P && c0 + j < C) ? g[(p0 + i) * C + c0 + j] : 0;
#pragma unroll
    for (int l = 0; l < 4; l++) {
        if (l < LA) {
            uint32_t d[4], o[4];
#pragma unroll
            for (int i = 0; i < 4; i++) d[i] = limb4(v[i][0], v[i][1], v[i][2], v[i][3], l);
            transpose4x4(d[0], d[1], d[2], d[3], o[0], o[1], o[2], o[3]);
#pragma unroll
            for (int j = 0; j < 4; j++)
                if (c0 + j < C) *(uint32_t *)(gt + ((int64_t)l * C + c0 + j) * pstride + p0) = o[j];
        }
    }
}

// ---------------------------------------------------------------------------------------------
constexpr int DW_BM = 64;          // output channels per workgroup (4 waves x 16)
constexpr int DW_BC = 16;          // input channels per workgroup
constexpr int DW_BK = 64;          // pixels per step
constexpr int DW_LDS = 80;         // LDS row stride (64 + 16 pad)
// largest chunk: 128 * 128 * DW_KC_MAX < 2^31, so a limb's int32 accumulator cannot overflow
constexpr int DW_KC_MAX = 131008;

// One workgroup: 64 output channels x 16 input channels x 9 taps over a chunk of pixels.
// A fragments (g limbs) come straight from the pixel-contiguous planes: each wave owns 16
// output channels. The x tile of each tap is staged in LDS (double-buffered, next step's global
// loads issued before this step's MFMAs). Limbs are taken two at a time: a second pass over the
// chunk handles limbs 2 and 3 when g needs them.
__global__ __launch_bounds__(256) void k_conv_dw_mfma(DwArgs p)
{
    __shared__ __attribute__((aligned(16))) uint8_t Bs[2][9][DW_BC][DW_LDS];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int LA = limbs_for(slot_read(p.gmax));
    if (LA > 4) {
        if (tid == 0) raise_flag(p.flags, FLAG_OVERFLOW);
        return;
    }
    const int HW = p.h * p.w;
    const int P = p.n * HW;
    const int co0 = blockIdx.x * DW_BM, ci0 = blockIdx.y * DW_BC;
    const int pb = blockIdx.z * p.kc;
    const int pe = pb + p.kc < P ? pb + p.kc : P;
    const int nsteps = (pe - pb + DW_BK - 1) / DW_BK;
    // one step advances every tracked pixel by DW_BK = adv_h rows + adv_w columns
    const int adv_h = DW_BK / p.w, adv_w = DW_BK % p.w;

    const int arow = co0 + wave * 16 + (lane & 15);
    const bool arow_ok = arow < p.co;
    const int8_t *abase = p.gt + (int64_t)(arow_ok ? arow : 0) * p.pstride + pb + (lane >> 4) * 16;
    const int64_t aplane = (int64_t)p.co * p.pstride;

    const int pq = (tid & 63) >> 2, cq = tid & 3;
    const int ci = ci0 + 4 * cq;
    const bool ci_ok = ci < p.ci;
    const int8_t *xci = p.x + ci;

    int64_t *part = p.part + (int64_t)blockIdx.z * p.co * 9 * p.ci;
    for (int lp = 0; lp < LA; lp += 2) {
        const bool two = lp + 1 < LA;
        int ph[4], pw[4], pidx[4];
#pragma unroll
        for (int i = 0; i < 4; i++) {
            const int pp = pb + 4 * pq + i;
            const int rem = pp % HW;
            pidx[i] = pp;
            ph[i] = rem / p.w;
            pw[i] = rem % p.w;
        }
        v4i acc[2][9];
#pragma unroll
        for (int l = 0; l < 2; l++)
#pragma unroll
            for (int t = 0; t < 9; t++) acc[l][t] = v4i{0, 0, 0, 0};

        v4i af[2][2];
        uint32_t braw[3][4];
        auto load = [&](int ks, int slot) {
            const int k0 = ks * DW_BK;
#pragma unroll
            for (int l = 0; l < 2; l++)
                af[slot][l] = (arow_ok && (l == 0 || two))
                                  ? *(const v4i *)(abase + (lp + l) * aplane + k0)
                                  : v4i{0, 0, 0, 0};
#pragma unroll
            for (int i = 0; i < 3; i++) {
                const int t = wave + 4 * i;
                const int dr = t / 3 - 1, ds = t % 3 - 1;
#pragma unroll
                for (int u = 0; u < 4; u++) {
                    const int hh = ph[u] + dr, ww = pw[u] + ds;
                    const bool ok = t < 9 && ci_ok && pidx[u] < pe && hh >= 0 && hh < p.h &&
                                    ww >= 0 && ww < p.w;
                    braw[i][u] = ok ? *(const uint32_t *)(xci + (pidx[u] + dr * p.w + ds) * p.ci) : 0u;
                }
            }
#pragma unroll
            for (int u = 0; u < 4; u++) {
                pidx[u] += DW_BK;
                pw[u] += adv_w;
                ph[u] += adv_h;
                if (pw[u] >= p.w) { pw[u] -= p.w; ph[u]++; }
                if (ph[u] >= p.h) ph[u] %= p.h;
            }
        };
        auto store = [&](int buf) {
#pragma unroll
            for (int i = 0; i < 3; i++) {
                const int t = wave + 4 * i;
                if (t < 9) {
                    uint32_t o[4];
                    transpose4x4(braw[i][0], braw[i][1], braw[i][2], braw[i][3], o[0], o[1], o[2], o[3]);
#pragma unroll
                    for (int c = 0; c < 4; c++) *(uint32_t *)&Bs[buf][t][4 * cq + c][4 * pq] = o[c];
                }
            }
        };

        load(0, 0);
        store(0);
        __syncthreads();
        for (int ks = 0; ks < nsteps; ks++) {
            const int cur = ks & 1;
            const bool more = ks + 1 < nsteps;
            if (more) load(ks + 1, cur ^ 1);
            v4i bf[9];
#pragma unroll
            for (int t = 0; t < 9; t++) bf[t] = *(const v4i *)&Bs[cur][t][lane & 15][(lane >> 4) * 16];
#pragma unroll
            for (int t = 0; t < 9; t++)
                acc[0][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[cur][0], bf[t], acc[0][t], 0, 0, 0);
            if (two) {
#pragma unroll
                for (int t = 0; t < 9; t++)
                    acc[1][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[cur][1], bf[t], acc[1][t], 0, 0, 0);
            }
            if (more) store(cur ^ 1);
            __syncthreads();
        }
        // this chunk's partial tile: the first pass stores, a second pass (limbs 2, 3) adds
#pragma unroll
        for (int t = 0; t < 9; t++)
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int co = co0 + wave * 16 + (lane >> 4) * 4 + i;
                const int cin = ci0 + (lane & 15);
                if (co < p.co && cin < p.ci) {
                    const int64_t v = ((int64_t)acc[0][t][i] << (8 * lp)) +
                                      ((int64_t)acc[1][t][i] << (8 * lp + 8));
                    int64_t *dst = part + ((int64_t)co * 9 + t) * p.ci + cin;
                    *dst = lp == 0 ? v : *dst + v;
                }
            }
    }
}

// Weight gradient for few input channels (9 * C_in <= 64): the N dimension is the flattened
// (tap, channel) column index of the KRSC weight row. Same A operand as k_conv_dw_mfma; the B tile
// [column][pixel] is gathered byte by byte (each thread: one column, four pixels).
__global__ __launch_bounds__(256) void k_conv_dw_mfma_smallc(DwArgs p)
{
    __shared__ __attribute__((aligned(16))) uint8_t Bs[2][64][DW_LDS];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int LA = limbs_for(slot_read(p.gmax));
    if (LA > 4) {
        if (tid == 0) raise_flag(p.flags, FLAG_OVERFLOW);
        return;
    }
    const int HW = p.h * p.w;
    const int P = p.n * HW;
    const int ncols = 9 * p.ci;
    const int co0 = blockIdx.x * DW_BM;
    const int pb = blockIdx.z * p.kc;
    const int pe = pb + p.kc < P ? pb + p.kc : P;
    const int nsteps = (pe - pb + DW_BK - 1) / DW_BK;
    const int adv_h = DW_BK / p.w, adv_w = DW_BK % p.w;

    const int arow = co0 + wave * 16 + (lane & 15);
    const bool arow_ok = arow < p.co;
    const int8_t *abase = p.gt + (int64_t)(arow_ok ? arow : 0) * p.pstride + pb + (lane >> 4) * 16;
    const int64_t aplane = (int64_t)p.co * p.pstride;

    // B tasks: column tid/16 + 16 i (i = 0..3), pixel quad tid % 16
    const int pq = tid & 15;
    int c_t[4], c_ci[4];
    bool c_ok[4];
#pragma unroll
    for (int i = 0; i < 4; i++) {
        const int col = (tid >> 4) + 16 * i;
        c_ok[i] = col < ncols;
        c_t[i] = c_ok[i] ? col / p.ci : 0;
        c_ci[i] = c_ok[i] ? col % p.ci : 0;
    }

    int64_t *part = p.part + (int64_t)blockIdx.z * p.co * ncols;
    for (int lp = 0; lp < LA; lp += 2) {
        const bool two = lp + 1 < LA;
        int ph[4], pw[4], pidx[4];
#pragma unroll
        for (int u = 0; u < 4; u++) {
            const int pp = pb + 4 * pq + u;
            const int rem = pp % HW;
            pidx[u] = pp;
            ph[u] = rem / p.w;
            pw[u] = rem % p.w;
        }
        v4i acc[2][4];
#pragma unroll
        for (int l = 0; l < 2; l++)
#pragma unroll
            for (int j = 0; j < 4; j++) acc[l][j] = v4i{0, 0, 0, 0};
        v4i af[2][2];
        uint32_t braw[4];
        auto load = [&](int ks, int slot) {
            const int k0 = ks * DW_BK;
#pragma unroll
            for (int l = 0; l < 2; l++)
                af[slot][l] = (arow_ok && (l == 0 || two))
                                  ? *(const v4i *)(abase + (lp + l) * aplane + k0)
                                  : v4i{0, 0, 0, 0};
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int dr = c_t[i] / 3 - 1, ds = c_t[i] % 3 - 1;
                uint32_t v = 0;
#pragma unroll
                for (int u = 0; u < 4; u++) {
                    const int hh = ph[u] + dr, ww = pw[u] + ds;
                    const bool ok = c_ok[i] && pidx[u] < pe && hh >= 0 && hh < p.h && ww >= 0 &&
                                    ww < p.w;
                    const uint32_t b = ok ? (uint32_t)(uint8_t)p.x[(pidx[u] + dr * p.w + ds) * p.ci + c_ci[i]] : 0u;
                    v |= b << (8 * u);
                }
                braw[i] = v;
            }
#pragma unroll
            for (int u = 0; u < 4; u++) {
                pidx[u] += DW_BK;
                pw[u] += adv_w;
                ph[u] += adv_h;
                if (pw[u] >= p.w) { pw[u] -= p.w; ph[u]++; }
                if (ph[u] >= p.h) ph[u] %= p.h;
            }
        };
        auto store = [&](int buf) {
#pragma unroll
            for (int i = 0; i < 4; i++)
                *(uint32_t *)&Bs[buf][(tid >> 4) + 16 * i][4 * pq] = braw[i];
        };
        load(0, 0);
        store(0);
        __syncthreads();
        const int ntile = (ncols + 15) / 16;
        for (int ks = 0; ks < nsteps; ks++) {
            const int cur = ks & 1;
            const bool more = ks + 1 < nsteps;
            if (more) load(ks + 1, cur ^ 1);
#pragma unroll
            for (int j = 0; j < 4; j++) {
                if (j < ntile) {
                    const v4i bf = *(const v4i *)&Bs[cur][16 * j + (lane & 15)][(lane >> 4) * 16];
                    acc[0][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[cur][0], bf, acc[0][j], 0, 0, 0);
                    if (two)
                        acc[1][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[cur][1], bf, acc[1][j], 0, 0, 0);
                }
            }
            if (more) store(cur ^ 1);
            __syncthreads();
        }
#pragma unroll
        for (int j = 0; j < 4; j++)
#pragma unroll
            for (int i = 0; i < 4; i++) {
                const int co = co0 + wave * 16 + (lane >> 4) * 4 + i;
                const int col = 16 * j + (lane & 15);
                if (co < p.co && col < ncols) {
                    const int64_t v = ((int64_t)acc[0][j][i] << (8 * lp)) +
                                      ((int64_t)acc[1][j][i] << (8 * lp + 8));
                    int64_t *dst = part + (int64_t)co * ncols + col;
                    *dst = lp == 0 ? v : *dst + v;
                }
            }
    }
}

bool mfma_conv_dw_smallc_ok(const ConvShape &sh)
{
    return 9 * sh.c <= 64 && sh.co % 4 == 0 &&
           ((int64_t)sh.n * sh.h * sh.w + 2 * sh.w + 2) * sh.c < ((int64_t)1 << 31);
}

bool mfma_conv_dw_ok(const ConvShape &sh)
{
    // 32-bit pixel arithmetic: every x offset (pixel * channels) stays below 2^31
    return sh.c % 4 == 0 && sh.co % 4 == 0 &&
           ((int64_t)sh.n * sh.h * sh.w + 2 * sh.w + 2) * sh.c < ((int64_t)1 << 31);
}

int64_t dw_plane_stride(const ConvShape &sh)
{
    const int64_t P = (int64_t)sh.n * sh.h * sh.w;
    return (P + DW_BK - 1) / DW_BK * DW_BK;
}

// Split of the pixel dimension: about 512 workgroups in total (128 for few input channels,
// whose partial tiles are few and short), chunks of whole 64-pixel steps.
static void dw_split(const ConvShape &sh, int64_t *nz_out, int64_t *kc_out)
{
    const int64_t P = (int64_t)sh.n * sh.h * sh.w;
    const bool smallc = !mfma_conv_dw_ok(sh);
    const int tiles = ((sh.co + DW_BM - 1) / DW_BM) * (smallc ? 1 : (sh.c + DW_BC - 1) / DW_BC);
    int64_t nz = ((smallc ? 128 : 512) + tiles - 1) / tiles;
    const int64_t steps = (P + DW_BK - 1) / DW_BK;
    if (nz > steps) nz = steps;
    int64_t kc = ((steps + nz - 1) / nz) * DW_BK;
    if (kc > DW_KC_MAX) kc = DW_KC_MAX;
    *kc_out = kc;
    *nz_out = (P + kc - 1) / kc;
}

int64_t dw_partial_count(const ConvShape &sh)
{
    int64_t nz, kc;
    dw_split(sh, &nz, &kc);
    return nz * sh.co * 9 * sh.c;
}

void launch_conv_dw_mfma(hipStream_t s, const ConvShape &sh, const int32_t *g,
                         const uint32_t *gmax, const int8_t *x, int8_t *gt, int64_t *part,
                         int64_t *dw, uint32_t *flags)
{
    const int64_t P = (int64_t)sh.n * sh.h * sh.w;
    const int64_t ps = dw_plane_stride(sh);
    {
        const int64_t ntask = (ps / 4) * ((sh.co + 3) / 4);
        hipLaunchKernelGGL(k_grad_limb_planes, dim3((unsigned)((ntask + 255) / 256)), dim3(256), 0,
                           s, g, (int)P, sh.co, ps, gmax, gt);
    }
    int64_t nz, kc;
    dw_split(sh, &nz, &kc);
    DwArgs a{};
    a.n = sh.n; a.h = sh.h; a.w = sh.w; a.ci = sh.c; a.co = sh.co;
    a.gt = gt; a.pstride = ps; a.gmax = gmax; a.x = x; a.part = part; a.kc = (int)kc;
    a.flags = flags;
    if (mfma_conv_dw_ok(sh)) {
        dim3 grid((unsigned)((sh.co + DW_BM - 1) / DW_BM), (unsigned)((sh.c + DW_BC - 1) / DW_BC),
                  (unsigned)nz);
        hipLaunchKernelGGL(k_conv_dw_mfma, grid, dim3(256), 0, s, a);
    } else {
        dim3 grid((unsigned)((sh.co + DW_BM - 1) / DW_BM), 1, (unsigned)nz);
        hipLaunchKernelGGL(k_conv_dw_mfma_smallc, grid, dim3(256), 0, s, a);
    }
    launch_sum_partials(s, part, (int)nz, (int64_t)sh.co * 9 * sh.c, dw);
}

}  // namespace nitro
