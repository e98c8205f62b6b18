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
#include "nitro_internal.h"

namespace nitro {

typedef int v4i __attribute__((ext_vector_type(4)));

__host__ __device__ inline int limbs_for(uint32_t m)
{
    return m <= 127u ? 1 : m <= 32639u ? 2 : m <= 8355711u ? 3 : m <= 2139062143u ? 4 : 5;
}

__device__ inline uint32_t abs_u32(int32_t v) { return v < 0 ? (uint32_t)(-(int64_t)v) : (uint32_t)v; }

// Limb l of four int32 values, packed into one dword (value i in byte i). Digit l of
// v + sum_{i<=l} 128*256^i is d_l + 128; xor 0x80 turns it back into the signed digit.
__device__ inline uint32_t limb4(int32_t v0, int32_t v1, int32_t v2, int32_t v3, int l)
{
    const uint32_t bias = 0x80808080u >> (24 - 8 * l);
    const int sh = 8 * l;
    uint32_t t0 = (((uint32_t)v0 + bias) >> sh) & 0xFFu;
    uint32_t t1 = (((uint32_t)v1 + bias) >> sh) & 0xFFu;
    uint32_t t2 = (((uint32_t)v2 + bias) >> sh) & 0xFFu;
    uint32_t t3 = (((uint32_t)v3 + bias) >> sh) & 0xFFu;
    return (t0 | (t1 << 8) | (t2 << 16) | (t3 << 24)) ^ 0x80808080u;
}

__device__ inline int8_t limb1(int32_t v, int l)
{
    const uint32_t bias = 0x80808080u >> (24 - 8 * l);
    return (int8_t)(((((uint32_t)v + bias) >> (8 * l)) & 0xFFu) ^ 0x80u);
}

__device__ inline uint32_t wave_max_u32(uint32_t v)
{
    for (int off = 32; off > 0; off >>= 1) {
        uint32_t o = __shfl_xor(v, off, 64);
        v = o > v ? o : v;
    }
    return v;
}

// ---------------------------------------------------------------------------------------------
// Weight packing: W int32 KRSC [co][3][3][ci] -> 4 limb planes of [co][9 ci] (forward) and,
// when wt != null, of [ci][9 co] with the same tap order (input gradient); max|W| -> *wmax.
__global__ void k_pack_conv_weights(const int32_t *__restrict__ w, int co, int ci,
                                    int8_t *__restrict__ wf, int8_t *__restrict__ wt,
                                    uint32_t *wmax)
{
    const int64_t total = (int64_t)co * 9 * ci;
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    uint32_t m = 0;
    if (i < total) {
        const int32_t v = w[i];
        m = abs_u32(v);
        const int o = (int)(i / (9 * ci));
        const int rem = (int)(i % (9 * ci));
        const int rs = rem / ci, c = rem % ci;
        const int64_t ti = (int64_t)c * 9 * co + (int64_t)rs * co + o;
        for (int l = 0; l < 4; l++) {
            const int8_t d = limb1(v, l);
            wf[l * total + i] = d;
            if (wt) wt[l * total + ti] = d;
        }
    }
    m = wave_max_u32(m);
    if ((threadIdx.x & 63) == 0) slot_max(wmax, m);
}

void launch_pack_conv_weights(hipStream_t s, const int32_t *w, int co, int ci, int8_t *wf,
                              int8_t *wt, uint32_t *wmax)
{
    const int64_t total = (int64_t)co * 9 * ci;
    hipLaunchKernelGGL(k_pack_conv_weights, dim3((unsigned)((total + 255) / 256)), dim3(256), 0,
                       s, w, co, ci, wf, wt, wmax);
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
template <int MODE, int BM, int BN>
__global__ __launch_bounds__(256) void k_igemm_conv(IgemmArgs p)
{
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int A_CHUNKS = BM * 4 / 256;       // 16-byte chunks of A per thread per step
    constexpr int B_CHUNKS = BN * 4 / 256;
    static_assert(A_CHUNKS >= 1 && B_CHUNKS >= 1, "tile too small");
    constexpr int SMEM_AB = (BM + BN) * IG_LDS_STRIDE;
    constexpr int SMEM_EPI = 2 * BM * BN;
    constexpr int SMEM = SMEM_AB > SMEM_EPI ? SMEM_AB : SMEM_EPI;
    __shared__ __attribute__((aligned(16))) uint8_t smem[SMEM];
    uint8_t *As = smem;
    uint8_t *Bs = smem + BM * IG_LDS_STRIDE;

    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int HW = p.h * p.w;
    const int64_t M = (int64_t)p.n * HW;
    const int64_t m0 = (int64_t)blockIdx.x * BM;
    const int n0 = blockIdx.y * BN;
    const int K = 9 * p.ck;
    const int ksteps = (K + IG_BK - 1) / IG_BK;

    const int LA = MODE == IG_FWD ? 1 : limbs_for(*p.a_max);
    const int LB = limbs_for(*p.b_max);
    if (LA > 4 || LB > 4) {
        if (tid == 0) raise_flag(p.flags, FLAG_OVERFLOW);
        return;
    }

    // rows this thread stages: row = tid/4 + 64 i, chunk kc = tid % 4 (fixed over K)
    const int kc = tid & 3;
    int a_n[A_CHUNKS], a_h[A_CHUNKS], a_w[A_CHUNKS];
    bool a_ok[A_CHUNKS];
    for (int i = 0; i < A_CHUNKS; i++) {
        const int64_t m = m0 + (tid >> 2) + 64 * i;
        a_ok[i] = m < M;
        const int64_t mm = a_ok[i] ? m : 0;
        a_n[i] = (int)(mm / HW);
        const int rem = (int)(mm % HW);
        a_h[i] = rem / p.w;
        a_w[i] = rem % p.w;
    }

    int64_t acc64[TM][TN][4];
    for (int i = 0; i < TM; i++)
        for (int j = 0; j < TN; j++)
            for (int t = 0; t < 4; t++) acc64[i][j][t] = 0;

    const int64_t plane = (int64_t)p.no * K;
    for (int la = 0; la < LA; la++) {
        for (int lb = 0; lb < LB; lb++) {
            v4i acc[TM][TN];
            for (int i = 0; i < TM; i++)
                for (int j = 0; j < TN; j++) acc[i][j] = v4i{0, 0, 0, 0};
            const int8_t *bpl = p.b + lb * plane;
            for (int ks = 0; ks < ksteps; ks++) {
                const int k = ks * IG_BK + kc * 16;
                const bool kin = k < K;
                const int tap = kin ? k / p.ck : 0;
                const int ci = kin ? k - tap * p.ck : 0;
                const int dr = tap / 3 - 1, ds = tap % 3 - 1;
                // ---- stage A
                for (int i = 0; i < A_CHUNKS; i++) {
                    int hh, ww;
                    if (MODE == IG_FWD) { hh = a_h[i] + dr; ww = a_w[i] + ds; }
                    else { hh = a_h[i] - dr; ww = a_w[i] - ds; }
                    const bool ok = kin && a_ok[i] && hh >= 0 && hh < p.h && ww >= 0 && ww < p.w;
                    v4i v = {0, 0, 0, 0};
                    if (ok) {
                        const int64_t pix = ((int64_t)a_n[i] * p.h + hh) * p.w + ww;
                        if (MODE == IG_FWD) {
                            v = *(const v4i *)((const int8_t *)p.a + pix * p.ck + ci);
                        } else {
                            const v4i *src = (const v4i *)((const int32_t *)p.a + pix * p.ck + ci);
                            v4i q0 = src[0], q1 = src[1], q2 = src[2], q3 = src[3];
                            v[0] = (int)limb4(q0[0], q0[1], q0[2], q0[3], la);
                            v[1] = (int)limb4(q1[0], q1[1], q1[2], q1[3], la);
                            v[2] = (int)limb4(q2[0], q2[1], q2[2], q2[3], la);
                            v[3] = (int)limb4(q3[0], q3[1], q3[2], q3[3], la);
                        }
                    }
                    *(v4i *)(As + ((tid >> 2) + 64 * i) * IG_LDS_STRIDE + kc * 16) = v;
                }
                // ---- stage B (packed limb plane lb)
                for (int i = 0; i < B_CHUNKS; i++) {
                    const int nn = n0 + (tid >> 2) + 64 * i;
                    v4i v = {0, 0, 0, 0};
                    if (kin && nn < p.no) v = *(const v4i *)(bpl + (int64_t)nn * K + k);
                    *(v4i *)(Bs + ((tid >> 2) + 64 * i) * IG_LDS_STRIDE + kc * 16) = v;
                }
                __syncthreads();
                v4i af[TM], bf[TN];
                for (int i = 0; i < TM; i++)
                    af[i] = *(const v4i *)(As + (wm * WM + i * 16 + (lane & 15)) * IG_LDS_STRIDE + (lane >> 4) * 16);
                for (int j = 0; j < TN; j++)
                    bf[j] = *(const v4i *)(Bs + (wn * WN + j * 16 + (lane & 15)) * IG_LDS_STRIDE + (lane >> 4) * 16);
                for (int i = 0; i < TM; i++)
                    for (int j = 0; j < TN; j++)
                        acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
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
        for (int i = 0; i < TM; i++)
            for (int j = 0; j < TN; j++)
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
                const int idx[4] = {q, q + 1, q + W, q + W + 1};
                int best = -1000, arg = 0;
                uint8_t breg = 0;
                for (int t = 0; t < 4; t++) {
                    const int v = (int)(int8_t)Os[idx[t] * BN + col];
                    if (v > best) { best = v; arg = t; breg = Rs[idx[t] * BN + col]; }
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
        for (int i = 0; i < TM; i++)
            for (int j = 0; j < TN; j++)
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
        if (p.gmax) {
            mx = wave_max_u32(mx);
            if (lane == 0) slot_max(p.gmax, mx);
        }
    }
}

// Tile choice: BN covers the GEMM's N when it is small (64), else 128.
template <int MODE>
static void launch_igemm(hipStream_t s, const IgemmArgs &a)
{
    const int64_t M = (int64_t)a.n * a.h * a.w;
    constexpr int BM = 128;
    if (a.no <= 64) {
        dim3 grid((unsigned)((M + BM - 1) / BM), (unsigned)((a.no + 63) / 64));
        hipLaunchKernelGGL((k_igemm_conv<MODE, BM, 64>), grid, dim3(256), 0, s, a);
    } else {
        dim3 grid((unsigned)((M + BM - 1) / BM), (unsigned)((a.no + 127) / 128));
        hipLaunchKernelGGL((k_igemm_conv<MODE, BM, 128>), grid, dim3(256), 0, s, a);
    }
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
    const int32_t *g;            // NHWC [P][co]
    const uint32_t *gmax;        // max|g|
    const int8_t *x;             // NHWC [P][ci]
    int64_t *dw;                 // [co][9][ci], zeroed before the launch
    int kc;                      // pixels per chunk (multiple of 64, <= 2^17)
    uint32_t *flags;
};

// 4x4 byte transpose: in a[i] byte j -> out[j] byte i.
__device__ inline void transpose4x4(uint32_t a0, uint32_t a1, uint32_t a2, uint32_t a3,
                                    uint32_t &o0, uint32_t &o1, uint32_t &o2, uint32_t &o3)
{
    const uint32_t t0 = __builtin_amdgcn_perm(a1, a0, 0x05010400u);   // a0.b0 a1.b0 a0.b1 a1.b1
    const uint32_t t1 = __builtin_amdgcn_perm(a1, a0, 0x07030602u);   // a0.b2 a1.b2 a0.b3 a1.b3
    const uint32_t t2 = __builtin_amdgcn_perm(a3, a2, 0x05010400u);   // a2.b0 a3.b0 a2.b1 a3.b1
    const uint32_t t3 = __builtin_amdgcn_perm(a3, a2, 0x07030602u);   // a2.b2 a3.b2 a2.b3 a3.b3
    o0 = __builtin_amdgcn_perm(t2, t0, 0x05040100u);                   // a0.b0 a1.b0 a2.b0 a3.b0
    o1 = __builtin_amdgcn_perm(t2, t0, 0x07060302u);
    o2 = __builtin_amdgcn_perm(t3, t1, 0x05040100u);
    o3 = __builtin_amdgcn_perm(t3, t1, 0x07060302u);
}

constexpr int DW_BM = 64;          // output channels per workgroup (4 waves x 16)
constexpr int DW_BC = 16;          // input channels per workgroup
constexpr int DW_BK = 64;          // pixels per step
constexpr int DW_LDS = 80;         // LDS row stride (64 + 16 pad)
// largest chunk: 128 * 128 * DW_KC_MAX < 2^31, so a limb's int32 accumulator cannot overflow
constexpr int DW_KC_MAX = 131008;

__global__ __launch_bounds__(256) void k_conv_dw_mfma(DwArgs p)
{
    __shared__ __attribute__((aligned(16))) uint8_t As[4][DW_BM][DW_LDS];
    __shared__ __attribute__((aligned(16))) uint8_t Bs[9][DW_BC][DW_LDS];
    __shared__ int pix_p[DW_BK];
    __shared__ int pix_hw[DW_BK];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int LA = limbs_for(*p.gmax);
    if (LA > 4) {
        if (tid == 0) raise_flag(p.flags, FLAG_OVERFLOW);
        return;
    }
    const int HW = p.h * p.w;
    const int P = p.n * HW;
    const int co0 = blockIdx.x * DW_BM, ci0 = blockIdx.y * DW_BC;
    const int pb = blockIdx.z * p.kc;
    const int pe = pb + p.kc < P ? pb + p.kc : P;

    v4i acc[4][9];
    for (int l = 0; l < 4; l++)
        for (int t = 0; t < 9; t++) acc[l][t] = v4i{0, 0, 0, 0};

    for (int k0 = pb; k0 < pe; k0 += DW_BK) {
        __syncthreads();                                   // previous step done with LDS
        if (tid < DW_BK) {
            const int pp = k0 + tid;
            const int rem = pp % HW;
            pix_p[tid] = pp < pe ? pp : -1;
            pix_hw[tid] = ((rem / p.w) << 16) | (rem % p.w);
        }
        __syncthreads();
        // ---- A: g[p][co0 + 4cq .. +4] for 4 pixels -> all limbs, transposed to [co][pixel]
        {
            const int cq = tid & 15, pq = tid >> 4;        // 16 x 16 tasks = 256 threads
            const int co = co0 + 4 * cq;
            v4i q[4];
            for (int i = 0; i < 4; i++) {
                const int pp = pix_p[4 * pq + i];
                q[i] = (pp >= 0 && co < p.co) ? *(const v4i *)(p.g + (int64_t)pp * p.co + co)
                                              : v4i{0, 0, 0, 0};
            }
            for (int l = 0; l < 4; l++) {
                if (l >= LA) break;
                uint32_t d[4], o[4];
                for (int i = 0; i < 4; i++) d[i] = limb4(q[i][0], q[i][1], q[i][2], q[i][3], l);
                transpose4x4(d[0], d[1], d[2], d[3], o[0], o[1], o[2], o[3]);
                for (int c = 0; c < 4; c++) *(uint32_t *)&As[l][4 * cq + c][4 * pq] = o[c];
            }
        }
        // ---- B: for each tap, x[p + shift][ci0 + 4cq .. +4] for 4 pixels, transposed
        for (int task = tid; task < 9 * 64; task += 256) {
            const int t = task >> 6, rem = task & 63;
            const int pq = rem >> 2, cq = rem & 3;
            const int dr = t / 3 - 1, ds = t % 3 - 1;
            const int ci = ci0 + 4 * cq;
            uint32_t d[4];
            for (int i = 0; i < 4; i++) {
                const int pp = pix_p[4 * pq + i];
                const int hw = pix_hw[4 * pq + i];
                const int hh = (hw >> 16) + dr, ww = (hw & 0xFFFF) + ds;
                const bool ok = pp >= 0 && ci < p.ci && hh >= 0 && hh < p.h && ww >= 0 && ww < p.w;
                d[i] = ok ? *(const uint32_t *)(p.x + (int64_t)(pp + dr * p.w + ds) * p.ci + ci) : 0u;
            }
            uint32_t o[4];
            transpose4x4(d[0], d[1], d[2], d[3], o[0], o[1], o[2], o[3]);
            for (int c = 0; c < 4; c++) *(uint32_t *)&Bs[t][4 * cq + c][4 * pq] = o[c];
        }
        __syncthreads();
        v4i bf[9];
        for (int t = 0; t < 9; t++) bf[t] = *(const v4i *)&Bs[t][lane & 15][(lane >> 4) * 16];
        for (int l = 0; l < 4; l++) {
            if (l >= LA) break;
            const v4i af = *(const v4i *)&As[l][wave * 16 + (lane & 15)][(lane >> 4) * 16];
            for (int t = 0; t < 9; t++)
                acc[l][t] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af, bf[t], acc[l][t], 0, 0, 0);
        }
    }
    // ---- combine limbs, add this chunk's partial tile into dW
    for (int t = 0; t < 9; t++)
        for (int i = 0; i < 4; i++) {
            const int co = co0 + wave * 16 + (lane >> 4) * 4 + i;
            const int ci = ci0 + (lane & 15);
            if (co >= p.co || ci >= p.ci) continue;
            int64_t v = 0;
            for (int l = 0; l < 4; l++) v += (int64_t)acc[l][t][i] << (8 * l);
            if (v != 0)
                atomicAdd((unsigned long long *)&p.dw[((int64_t)co * 9 + t) * p.ci + ci],
                          (unsigned long long)v);
        }
}

bool mfma_conv_dw_ok(const ConvShape &sh)
{
    return sh.c % 4 == 0 && sh.co % 4 == 0 && (int64_t)sh.n * sh.h * sh.w < ((int64_t)1 << 31) &&
           sh.w < 65536 && sh.h < 65536;
}

void launch_conv_dw_mfma(hipStream_t s, const ConvShape &sh, const int32_t *g,
                         const uint32_t *gmax, const int8_t *x, int64_t *dw, uint32_t *flags)
{
    launch_fill_i64(s, dw, (int64_t)sh.co * 9 * sh.c);
    DwArgs a{};
    a.n = sh.n; a.h = sh.h; a.w = sh.w; a.ci = sh.c; a.co = sh.co;
    a.g = g; a.gmax = gmax; a.x = x; a.dw = dw; a.flags = flags;
    const int64_t P = (int64_t)sh.n * sh.h * sh.w;
    const int tiles = ((sh.co + DW_BM - 1) / DW_BM) * ((sh.c + DW_BC - 1) / DW_BC);
    // about 512 workgroups in total; chunks of whole 64-pixel steps, at most 2^17 pixels
    int64_t nz = (512 + tiles - 1) / tiles;
    const int64_t steps = (P + DW_BK - 1) / DW_BK;
    if (nz > steps) nz = steps;
    int64_t kc = ((steps + nz - 1) / nz) * DW_BK;
    if (kc > DW_KC_MAX) kc = DW_KC_MAX;
    nz = (P + kc - 1) / kc;
    a.kc = (int)kc;
    dim3 grid((unsigned)((sh.co + DW_BM - 1) / DW_BM), (unsigned)((sh.c + DW_BC - 1) / DW_BC),
              (unsigned)nz);
    hipLaunchKernelGGL(k_conv_dw_mfma, grid, dim3(256), 0, s, a);
}

}  // namespace nitro
