// The learning layer of a block (an IntLinear d -> G with NITRO-Scaling, trained on the RSS
// loss) on int8 MFMA, exact:
//   forward    yhat[n][g] = floor(sum_k f[n][k] W[g][k] / 2^8 d),  e = yhat - 32 onehot(label)
//   delta      delta[n][k] = sum_g e[n][g] W[g][k]   (pre-update W), fused with the max-pool
//              routing and NITRO-ReLU backward of the block's last layer
//   gradient   dW[g][k] = sum_n e[n][g] f[n][k]
// All three are C[m][j] = sum_k A[m][k] B[j][k] with K-contiguous rows: one kernel, three
// epilogues. Wide operands use balanced int8 limbs as in the convolution kernels: the weights'
// limb planes are packed before the step, e's written by the kernel that computes e.
#include <type_traits>

#include "mfma_common.h"

namespace nitro {

enum { LIN_PART = 0, LIN_UNPOOL = 1, LIN_DW = 2 };

struct LgemmArgs {
    int M, N, K;                  // K: a multiple of 16 (zero padded rows)
    const int8_t *a;              // A rows [M][lda]; limb planes aplane apart when a_max is set
    int64_t lda, aplane;
    const uint32_t *a_max;        // limb planes of A: max|A| (null: one int8 plane)
    const int8_t *b;              // B limb planes [4][N][ldb] (one plane when b_max is null)
    int64_t ldb, bplane;
    const uint32_t *b_max;
    int kchunk;                   // K per split (a multiple of 16); grid.z = number of splits
    // LIN_PART: part[z][M][N]; LIN_DW: out64[m * ldc + j] for m < m_valid
    int64_t *out64;
    int64_t ldc;
    int m_valid;
    // LIN_UNPOOL: block output geometry (full resolution h x w, c channels, pooled or not)
    const uint8_t *code;
    Relu rp;
    int h, w, c, pool;
    int gpooled;                  // pooled: g at the pooled positions only (the argmax's value)
    int32_t *g;                   // gradient at the last layer's pre-activation, NHWC
    int32_t *delta;               // optional copy of delta (int32, pooled NHWC)
    uint32_t *gmax;
    uint32_t *flags;
};

constexpr int LG_BM = 128, LG_BN = 64, LG_BK = 64;
constexpr int LG_KC = 128;                // K per staged chunk (two MFMA K-steps)
constexpr int LG_LS = LG_KC + 16;         // LDS row stride: 16 rows of a fragment read hit
                                          // 16 different bank quads
constexpr int LG_SA = LG_BM * LG_LS;      // one A limb plane of a chunk
constexpr int LG_SB = LG_BN * LG_LS;      // one B limb plane

// A workgroup: a 128 x 64 tile of C over its K range, in chunks of 128. The limb planes of both
// operands for a chunk are staged in LDS two per operand at a time (one load round for the
// usual one or two limbs; 55 KiB of LDS, two workgroups per CU), the next round's loads issued
// before this one's MFMAs; each limb pair (la, lb) runs its two K-steps from LDS and is folded
// into int64 with its weight 256^(la + lb).
constexpr int LG_DS = LG_BN + 1;               // LIN_UNPOOL epilogue: int32-tile row stride
constexpr int LG_SMEM = 2 * LG_SA + 2 * LG_SB > LG_BM * LG_DS * 4 ? 2 * LG_SA + 2 * LG_SB : LG_BM * LG_DS * 4;

// One workgroup's tile (bx, by) of split bz; smem: LG_SMEM bytes.
template <int MODE>
__device__ void lgemm_tile(const LgemmArgs &p, uint8_t *smem, int bx, int by, int bz)
{
    constexpr int WM = LG_BM / 2, WN = LG_BN / 2;
    constexpr int TM = WM / 16, TN = WN / 16;
    constexpr int AU = LG_BM * (LG_KC / 16) / 256, BU = LG_BN * (LG_KC / 16) / 256;  // units/thread
    constexpr int DS = LG_DS;

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int m0 = bx * LG_BM, n0 = by * LG_BN;
    const int kb = bz * p.kchunk;
    const int ke = kb + p.kchunk < p.K ? kb + p.kchunk : p.K;
    const int nck = (ke - kb + LG_KC - 1) / LG_KC;
    uint8_t *As = smem, *Bs = smem + 2 * LG_SA;

    // unit u of a thread: row (tid >> 3) + 32 u, 16-byte column tid & 7. Round r = (chunk, A
    // plane pair, B plane pair); limb plane 0 of the first round is requested before the limb
    // counts are known.
    const int ur = tid >> 3, uc = (tid & 7) * 16;
    v4i ar[2][AU], br[2][BU];
    int LA = 1, LB = 1, NA = 1, NB = 1;
    auto load = [&](int r, int lmin) {
        const int ck = r / (NA * NB), pa = (r / NB) % NA, pb = r % NB;
        const int k = kb + ck * LG_KC + uc;
        const bool kin = k < ke;
#pragma unroll
        for (int h = 0; h < 2; h++) {
            const int la = 2 * pa + h, lb = 2 * pb + h;
            if (la >= lmin && la < LA) {
                const int8_t *apl = p.a + la * p.aplane;
#pragma unroll
                for (int u = 0; u < AU; u++) {
                    const int m = m0 + ur + 32 * u;
                    ar[h][u] = kin && m < p.M ? *(const v4i *)(apl + (int64_t)m * p.lda + k) : v4i{0, 0, 0, 0};
                }
            }
            if (lb >= lmin && lb < LB) {
                const int8_t *bpl = p.b + lb * p.bplane;
#pragma unroll
                for (int u = 0; u < BU; u++) {
                    const int nn = n0 + ur + 32 * u;
                    br[h][u] = kin && nn < p.N ? *(const v4i *)(bpl + (int64_t)nn * p.ldb + k) : v4i{0, 0, 0, 0};
                }
            }
        }
    };
    auto store = [&](int r) {
        const int pa = (r / NB) % NA, pb = r % NB;
#pragma unroll
        for (int h = 0; h < 2; h++) {
            if (2 * pa + h < LA)
#pragma unroll
                for (int u = 0; u < AU; u++) *(v4i *)(As + h * LG_SA + (ur + 32 * u) * LG_LS + uc) = ar[h][u];
            if (2 * pb + h < LB)
#pragma unroll
                for (int u = 0; u < BU; u++) *(v4i *)(Bs + h * LG_SB + (ur + 32 * u) * LG_LS + uc) = br[h][u];
        }
    };

    int64_t acc64[TM][TN][4];
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++)
#pragma unroll
            for (int t = 0; t < 4; t++) acc64[i][j][t] = 0;

    if (nck > 0) load(0, 0);                     // (LA = LB = 1: plane 0 only)
    LA = p.a_max ? limbs_for(slot_read(p.a_max)) : 1;
    LB = p.b_max ? limbs_for(slot_read(p.b_max)) : 1;
    if (LA > 4 || LB > 4) {
        if (tid == 0) raise_flag(p.flags, FLAG_OVERFLOW);
        return;
    }
    NA = (LA + 1) / 2;
    NB = (LB + 1) / 2;
    const int nr = nck * NA * NB;
    if (nck > 0) load(0, 1);
    // (LIN_UNPOOL: the epilogue's region codes, requested now)
    constexpr int EIT = MODE == LIN_UNPOOL ? LG_BM * (LG_BN / 16) / 256 : 1;
    v4i cdp[EIT];
    if (MODE == LIN_UNPOOL) {
#pragma unroll
        for (int q = 0; q < EIT; q++) {
            const int it = tid + 256 * q;
            const int m = m0 + it / (LG_BN / 16), col = n0 + (it % (LG_BN / 16)) * 16;
            cdp[q] = m < p.M && col < p.N ? *(const v4i *)(p.code + (int64_t)m * p.N + col) : v4i{0, 0, 0, 0};
        }
    }
    // (the codes are consumed here, by nothing: left alone, the compiler issues their loads
    // only in the epilogue, where each then waits for the memory; this wait coincides with the
    // first round's own)
    if (MODE == LIN_UNPOOL) {
#pragma unroll
        for (int q = 0; q < EIT; q++) asm volatile("" : "+v"(cdp[q]));
    }
    for (int r = 0; r < nr; r++) {
        __syncthreads();                          // every wave is done with the previous round
        store(r);
        __syncthreads();
        if (r + 1 < nr) load(r + 1, 0);
        const int pa = (r / NB) % NA, pb = r % NB;
        for (int ha = 0; ha < 2 && 2 * pa + ha < LA; ha++) {
            for (int hb = 0; hb < 2 && 2 * pb + hb < LB; hb++) {
                const uint8_t *Ap = As + ha * LG_SA, *Bp = Bs + hb * LG_SB;
                v4i acc[TM][TN];
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int j = 0; j < TN; j++) acc[i][j] = v4i{0, 0, 0, 0};
#pragma unroll
                for (int ks = 0; ks < LG_KC / LG_BK; ks++) {
                    v4i af[TM], bf[TN];
#pragma unroll
                    for (int i = 0; i < TM; i++)
                        af[i] = *(const v4i *)(Ap + (wm * WM + i * 16 + (lane & 15)) * LG_LS + ks * LG_BK + (lane >> 4) * 16);
#pragma unroll
                    for (int j = 0; j < TN; j++)
                        bf[j] = *(const v4i *)(Bp + (wn * WN + j * 16 + (lane & 15)) * LG_LS + ks * LG_BK + (lane >> 4) * 16);
#pragma unroll
                    for (int i = 0; i < TM; i++)
#pragma unroll
                        for (int j = 0; j < TN; j++)
                            acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(af[i], bf[j], acc[i][j], 0, 0, 0);
                }
                const int sh = 8 * (2 * pa + ha + 2 * pb + hb);
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int j = 0; j < TN; j++)
#pragma unroll
                        for (int t = 0; t < 4; t++) acc64[i][j][t] += (int64_t)acc[i][j][t] << sh;
            }
        }
    }
    __syncthreads();                              // (the epilogue reuses the LDS)

    if (MODE != LIN_UNPOOL) {
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++)
#pragma unroll
                for (int t = 0; t < 4; t++) {
                    const int m = m0 + wm * WM + i * 16 + (lane >> 4) * 4 + t;
                    const int col = n0 + wn * WN + j * 16 + (lane & 15);
                    if (m >= p.M || col >= p.N) continue;
                    const int64_t v = acc64[i][j][t];
                    if (MODE == LIN_PART) p.out64[((int64_t)bz * p.M + m) * p.N + col] = v;
                    else if (m < p.m_valid) p.out64[(int64_t)m * p.ldc + col] = v;
                }
        return;
    }
    // LIN_UNPOOL. m = sample, col = index in the block output. delta (int32: it must fit) goes
    // through LDS; then each thread takes 16 consecutive outputs of one sample (one pooled pixel,
    // 16 channels: N and c are multiples of 16), applies NITRO-ReLU backward with their 16 region
    // codes and writes the 2x2 window of each (the gradient at the argmax, 0 elsewhere) as
    // 64-byte rows.
    bool bad = false;
    int32_t *Ds = (int32_t *)smem;            // [LG_BM][DS]
#pragma unroll
    for (int i = 0; i < TM; i++)
#pragma unroll
        for (int j = 0; j < TN; j++)
#pragma unroll
            for (int t = 0; t < 4; t++) {
                const int row = wm * WM + i * 16 + (lane >> 4) * 4 + t;
                const int col = wn * WN + j * 16 + (lane & 15);
                const int64_t v = acc64[i][j][t];
                bad |= !fits_i32(v);
                Ds[row * DS + col] = (int32_t)v;
            }
    __syncthreads();
    uint32_t mx = 0;
    const uint32_t W2 = (uint32_t)p.w / 2;
    auto emit = [&](auto trunc_tag) {
        constexpr bool TR = decltype(trunc_tag)::value;
#pragma unroll
        for (int q = 0; q < EIT; q++) {
            const int it = tid + 256 * q;
            const int row = it / (LG_BN / 16), cc = (it % (LG_BN / 16)) * 16;
            const int m = m0 + row, col = n0 + cc;
            if (m >= p.M || col >= p.N) continue;
            const int64_t o = (int64_t)m * p.N + col;
            const v4i cd = cdp[q];
            v4i dv[4], gv[4];
#pragma unroll
            for (int e = 0; e < 16; e++) {
                // |g| <= |delta|, and delta was checked to fit int32
                const int32_t v = Ds[row * DS + cc + e];
                const uint32_t c8 = ((uint32_t)cd[e >> 2] >> (8 * (e & 3))) & 0xFFu;
                const int32_t g = relu_bwd32<TR>(v, p.pool ? c8 >> 2 : c8, p.rp);
                const uint32_t a = abs_u32(g);
                mx = a > mx ? a : mx;
                dv[e >> 2][e & 3] = v;
                gv[e >> 2][e & 3] = g;
            }
            if (p.delta)
#pragma unroll
                for (int q = 0; q < 4; q++) *(v4i *)(p.delta + o + 4 * q) = dv[q];
            if (!p.pool || p.gpooled) {
#pragma unroll
                for (int q = 0; q < 4; q++) *(v4i *)(p.g + o + 4 * q) = gv[q];
                continue;
            }
            const uint32_t ch = (uint32_t)col % (uint32_t)p.c, pp = (uint32_t)col / (uint32_t)p.c;
            const uint32_t q2 = pp % W2, h2 = pp / W2;
            int32_t *gb = p.g + (int64_t)m * p.h * p.w * p.c + ch;
#pragma unroll
            for (int u = 0; u < 4; u++) {
                const uint32_t pix = (2 * h2 + (u >> 1)) * (uint32_t)p.w + 2 * q2 + (u & 1);
#pragma unroll
                for (int q = 0; q < 4; q++) {
                    v4i o4;
#pragma unroll
                    for (int r = 0; r < 4; r++) {
                        const int e = 4 * q + r;
                        const uint32_t arg = ((uint32_t)cd[e >> 2] >> (8 * (e & 3))) & 3u;
                        o4[r] = arg == (uint32_t)u ? gv[q][r] : 0;
                    }
                    *(v4i *)(gb + (int64_t)pix * p.c + 4 * q) = o4;
                }
            }
        }
    };
    if (p.rp.alpha.trunc) emit(std::true_type{});
    else emit(std::false_type{});
    if (bad) raise_flag(p.flags, FLAG_OVERFLOW);
    block_slot_max(p.gmax, mx);
}


// ---------------------------------------------------------------------------------------------
// Learning weights W [G][d] int32 -> limb planes [4][G][d] and [4][d][gp] (zero rows g >= G);
// max|W| -> *wmax.
__global__ void k_pack_learning_weights(const int32_t *__restrict__ w, uint32_t G, uint32_t d,
                                        uint32_t gp, int8_t *__restrict__ wf,
                                        int8_t *__restrict__ wt, uint32_t *wmax)
{
    const uint32_t total = G * d;
    uint32_t m = 0;
    for (uint32_t i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const int32_t v = w[i];
        const uint32_t a = abs_u32(v);
        m = a > m ? a : m;
#pragma unroll
        for (int l = 0; l < 4; l++) wf[(int64_t)l * total + i] = limb1(v, l);
    }
    // transposed planes in their own order (coalesced stores)
    const uint32_t ttotal = d * gp;
    for (uint32_t ti = blockIdx.x * blockDim.x + threadIdx.x; ti < ttotal; ti += gridDim.x * blockDim.x) {
        const uint32_t g = ti % gp, k = ti / gp;
        const int32_t v = g < G ? w[g * d + k] : 0;
#pragma unroll
        for (int l = 0; l < 4; l++) wt[(int64_t)l * ttotal + ti] = limb1(v, l);
    }
    block_slot_max(wmax, m);
}

// f [n][d] int8 -> fT [d][np] (zero columns n >= N), tile (bx, by) = features 64 bx ..,
// samples 64 by ..: each thread transposes one 4 x 4 byte block in registers (four dword loads
// of 4 samples' 4 features, byte permutes, four dword stores of 4 features' 4 samples; d and np
// are multiples of 16).
__device__ void transpose_i8_tile(const int8_t *__restrict__ f, int N, int d, int np,
                                  int8_t *__restrict__ ft, int bx, int by)
{
    const int t = threadIdx.x;
    const int r0 = by * 64 + 4 * (t >> 4);             // first of the block's 4 samples
    const int c0 = bx * 64 + 4 * (t & 15);             // first of its 4 features
    if (c0 >= d || r0 >= np) return;
    uint32_t a[4];
#pragma unroll
    for (int i = 0; i < 4; i++)
        a[i] = r0 + i < N ? *(const uint32_t *)(f + (int64_t)(r0 + i) * d + c0) : 0u;
    uint32_t o[4];
    transpose4x4(a[0], a[1], a[2], a[3], o[0], o[1], o[2], o[3]);
#pragma unroll
    for (int j = 0; j < 4; j++) *(uint32_t *)(ft + (int64_t)(c0 + j) * np + r0) = o[j];
}

// Forward of the learning layer in one launch: workgroups 0 .. ngemm - 1 compute the split-K
// partial tiles (x fastest, then y, then split), the rest transpose f (for the weight gradient);
// the tiles come first, so that their longer chains start before the short transposes.
__global__ __launch_bounds__(256) void k_lgemm_fwd(LgemmArgs p, const int8_t *f, int N, int d, int np,
                                                   int8_t *ft, int tgx, int tgy)
{
    __shared__ __attribute__((aligned(16))) uint8_t smem[LG_SMEM];
    const int b = blockIdx.x;
    const int gx = (p.M + LG_BM - 1) / LG_BM, gy = (p.N + LG_BN - 1) / LG_BN;
    const int ngemm = (int)gridDim.x - tgx * tgy;
    if (b < ngemm) {
        lgemm_tile<LIN_PART>(p, smem, b % gx, (b / gx) % gy, b / (gx * gy));
        return;
    }
    const int q = b - ngemm;
    transpose_i8_tile(f, N, d, np, ft, q % tgx, q / tgx);
}

// Backward of the learning layer in one launch (both read e only): workgroups 0 .. ndw - 1 the
// weight-gradient tiles, the rest delta's (with the un-pool and ReLU' epilogue).
__global__ __launch_bounds__(256) void k_lgemm_bwd(LgemmArgs dw, LgemmArgs up)
{
    __shared__ __attribute__((aligned(16))) uint8_t smem[LG_SMEM];
    const int dgx = (dw.M + LG_BM - 1) / LG_BM, dgy = (dw.N + LG_BN - 1) / LG_BN;
    const int b = blockIdx.x;
    if (b < dgx * dgy) {
        lgemm_tile<LIN_DW>(dw, smem, b % dgx, b / dgx, 0);
        return;
    }
    const int q = b - dgx * dgy;
    const int ugx = (up.M + LG_BM - 1) / LG_BM;
    lgemm_tile<LIN_UNPOOL>(up, smem, q % ugx, q / ugx, 0);
}

// yhat and e from the split-K partial sums; also e padded to [n][gp] and transposed to [gp][np]
// (zeros in the padding), max|e| -> *emax.
__global__ void k_loss_from_partials(const int64_t *__restrict__ part, int nz, int N, int G, int gp,
                                     int np, Div sf, const int32_t *__restrict__ labels,
                                     int32_t *__restrict__ yhat, int32_t *__restrict__ e,
                                     int8_t *__restrict__ epad, int8_t *__restrict__ et,
                                     uint32_t *emax, uint32_t *flags)
{
    uint32_t m = 0;
    bool bad = false, badlab = false;
    const int total = np * gp;
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const int n = i / gp, g = i % gp;
        int64_t ev = 0;
        if (n < N && g < G) {
            // (four independent sums: the split partials are read four loads at a time)
            const int64_t st = (int64_t)N * G;
            const int64_t *pp = part + (int64_t)n * G + g;
            int64_t z0 = 0, z1 = 0, z2 = 0, z3 = 0;
            int s = 0;
            for (; s + 3 < nz; s += 4) {
                z0 += pp[s * st];
                z1 += pp[(s + 1) * st];
                z2 += pp[(s + 2) * st];
                z3 += pp[(s + 3) * st];
            }
            for (; s < nz; s++) z0 += pp[s * st];
            const int64_t z = (z0 + z1) + (z2 + z3);
            const int64_t y = idiv(z, sf);
            const int lab = labels[n];
            badlab |= lab < 0 || lab >= G;
            ev = y - (lab == g ? 32 : 0);
            bad |= !fits_i32(y) || !fits_i32(ev);
            yhat[n * G + g] = (int32_t)y;
            e[n * G + g] = (int32_t)ev;
            const uint32_t a = abs_i64_sat(ev);
            m = a > m ? a : m;
        }
        // e's four balanced limb planes in both layouts (a value outside int32 is flagged above)
        const int32_t e32 = (int32_t)ev;
        const int64_t plane = (int64_t)np * gp;
#pragma unroll
        for (int l = 0; l < 4; l++) {
            const int8_t d = limb1(e32, l);
            if (n < N) epad[l * plane + n * gp + g] = d;
            et[l * plane + (int64_t)g * np + n] = d;
        }
    }
    if (bad) raise_flag(flags, FLAG_OVERFLOW);
    if (badlab) raise_flag(flags, FLAG_LABEL);
    block_slot_max(emax, m);
}

// ---------------------------------------------------------------------------------------------
// IntLinear forward layers and their weight gradients on the same tile.

// Split-K partial tiles of C = A B^T (grid: x fastest, then y, then split).
__global__ __launch_bounds__(256) void k_lgemm_part(LgemmArgs p)
{
    __shared__ __attribute__((aligned(16))) uint8_t smem[LG_SMEM];
    const int gx = (p.M + LG_BM - 1) / LG_BM, gy = (p.N + LG_BN - 1) / LG_BN;
    const int b = blockIdx.x;
    lgemm_tile<LIN_PART>(p, smem, b % gx, (b / gx) % gy, b / (gx * gy));
}

// C = A B^T written as int64 rows (no split).
__global__ __launch_bounds__(256) void k_lgemm_dw(LgemmArgs p)
{
    __shared__ __attribute__((aligned(16))) uint8_t smem[LG_SMEM];
    const int gx = (p.M + LG_BM - 1) / LG_BM;
    lgemm_tile<LIN_DW>(p, smem, blockIdx.x % gx, blockIdx.x / gx, 0);
}

// x int8 [n][ci] -> xpad [n][cip] with zero columns ci..cip-1: thread = 16 bytes of one row.
__global__ __launch_bounds__(256) void k_pad_rows(const int8_t *__restrict__ x, int n, int ci, int cip,
                                                  int8_t *__restrict__ xpad)
{
    const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
    const int per = cip / 16;
    if (u >= (int64_t)n * per) return;
    const int r = (int)(u / per), c0 = (int)(u - (int64_t)r * per) * 16;
    v4i v = v4i{0, 0, 0, 0};
    const int8_t *src = x + (int64_t)r * ci + c0;
    if ((ci & 3) == 0) {
        // (dword loads: rows of a multiple of 4 bytes keep them aligned)
#pragma unroll
        for (int q = 0; q < 4; q++)
            if (c0 + 4 * q < ci) v[q] = *(const int *)(src + 4 * q);
    } else {
        for (int e = 0; e < 16 && c0 + e < ci; e++)
            v[e >> 2] |= (int)((uint32_t)(uint8_t)src[e] << (8 * (e & 3)));
    }
    *(v4i *)(xpad + (int64_t)r * cip + c0) = v;
}

// NITRO-Scaling and NITRO-ReLU of z = the sum of the split partials [nz][n][co] (as the direct
// kernel: floor or truncated z / SF, then the NITRO-ReLU map and its region code).
__global__ __launch_bounds__(256) void k_linear_relu_from_partials(const int64_t *__restrict__ part, int nz,
                                                                   int64_t count, Div sf, Relu rp,
                                                                   int8_t *__restrict__ out,
                                                                   uint8_t *__restrict__ code)
{
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < count; i += (int64_t)gridDim.x * 256) {
        int64_t z0 = 0, z1 = 0;
        int s = 0;
        for (; s + 1 < nz; s += 2) {
            z0 += part[(int64_t)s * count + i];
            z1 += part[(int64_t)(s + 1) * count + i];
        }
        if (s < nz) z0 += part[(int64_t)s * count + i];
        uint8_t reg;
        const int32_t a = relu_fwd(idiv(z0 + z1, sf), rp, reg);
        out[i] = (int8_t)a;
        code[i] = reg;
    }
}

// The weight gradient's operands: workgroups 0 .. ng - 1 write g^T's balanced limb planes
// gt [4][co][np] (thread: one output channel, 16 samples; zero for samples >= n) and fold max|g|
// into gmax; the rest write x^T [ci][np] (thread: one input channel, 16 samples).
__global__ __launch_bounds__(256) void k_linear_dw_prep(const int32_t *__restrict__ g, int n, int co,
                                                        int np, int8_t *__restrict__ gt, uint32_t *gmax,
                                                        const int8_t *__restrict__ x, int ci,
                                                        int8_t *__restrict__ xt, int ng)
{
    const int q = np / 16;
    if ((int)blockIdx.x < ng) {
        const int64_t u = (int64_t)blockIdx.x * 256 + threadIdx.x;
        uint32_t mx = 0;
        if (u < (int64_t)co * q) {
            const int o = (int)(u % co), s0 = (int)(u / co) * 16;
            int32_t v[16];
#pragma unroll
            for (int e = 0; e < 16; e++) {
                v[e] = s0 + e < n ? g[(int64_t)(s0 + e) * co + o] : 0;
                const uint32_t a = abs_u32(v[e]);
                mx = a > mx ? a : mx;
            }
            const int64_t plane = (int64_t)co * np;
#pragma unroll
            for (int l = 0; l < 4; l++) {
                v4i d;
#pragma unroll
                for (int k = 0; k < 4; k++) d[k] = (int)limb4(v[4 * k], v[4 * k + 1], v[4 * k + 2], v[4 * k + 3], l);
                *(v4i *)(gt + l * plane + (int64_t)o * np + s0) = d;
            }
        }
        block_slot_max(gmax, mx);
        return;
    }
    const int64_t u = (int64_t)(blockIdx.x - ng) * 256 + threadIdx.x;
    if (u >= (int64_t)ci * q) return;
    const int c = (int)(u % ci), s0 = (int)(u / ci) * 16;
    v4i d = v4i{0, 0, 0, 0};
#pragma unroll
    for (int e = 0; e < 16; e++)
        if (s0 + e < n) d[e >> 2] |= (int)((uint32_t)(uint8_t)x[(int64_t)(s0 + e) * ci + c] << (8 * (e & 3)));
    *(v4i *)(xt + (int64_t)c * np + s0) = d;
}

bool linear_mfma_ok(int n, int ci, int co)
{
    const int64_t cip = (ci + 15) / 16 * 16, np = (n + 15) / 16 * 16;
    const int64_t lim = (int64_t)1 << 31;
    return n >= 1 && ci >= 1 && co >= 1 && 4 * (int64_t)co * cip < lim && (int64_t)n * cip < lim &&
           4 * (int64_t)co * np < lim && (int64_t)ci * np < lim && (int64_t)n * co < lim;
}

LinearScratch linear_scratch(int n, int ci, int co)
{
    LinearScratch s{};
    s.cip = (ci + 15) / 16 * 16;
    s.np = (n + 15) / 16 * 16;
    // forward split-K as the learning layer's: about 256 of K per workgroup, at most 1024
    // workgroups
    int splits = (s.cip + 255) / 256;
    const int tiles = ((n + LG_BM - 1) / LG_BM) * ((co + LG_BN - 1) / LG_BN);
    if (splits * tiles > 1024) splits = (1024 + tiles - 1) / tiles;
    if (splits < 1) splits = 1;
    int kchunk = (s.cip + splits - 1) / splits;
    kchunk = (kchunk + LG_KC - 1) / LG_KC * LG_KC;
    s.kchunk = kchunk;
    s.splits = (s.cip + kchunk - 1) / kchunk;
    s.wf_bytes = 4 * (int64_t)co * s.cip;
    s.xpad_bytes = ci % 16 ? (int64_t)n * s.cip : 0;
    s.part_bytes = 8 * (int64_t)s.splits * n * co;
    s.gt_bytes = 4 * (int64_t)co * s.np;
    s.xt_bytes = (int64_t)ci * s.np;
    return s;
}

void launch_linear_fwd_mfma(hipStream_t s, int n, int ci, int co, const int8_t *x, int8_t *xpad,
                            const int8_t *wf, const uint32_t *wmax, const Div &sf, const Relu &rp,
                            int8_t *out, uint8_t *code, int64_t *part, uint32_t *flags)
{
    const LinearScratch sc = linear_scratch(n, ci, co);
    const int8_t *a = x;
    if (ci % 16) {
        const int64_t units = (int64_t)n * (sc.cip / 16);
        hipLaunchKernelGGL(k_pad_rows, dim3((unsigned)((units + 255) / 256)), dim3(256), 0, s, x, n, ci,
                           sc.cip, xpad);
        a = xpad;
    }
    LgemmArgs p{};
    p.M = n; p.N = co; p.K = sc.cip;
    p.a = a; p.lda = sc.cip;
    p.b = wf; p.ldb = sc.cip; p.bplane = (int64_t)co * sc.cip; p.b_max = wmax;
    p.kchunk = sc.kchunk;
    p.out64 = part;
    p.flags = flags;
    const int64_t nwg = (int64_t)((n + LG_BM - 1) / LG_BM) * ((co + LG_BN - 1) / LG_BN) * sc.splits;
    hipLaunchKernelGGL(k_lgemm_part, dim3((unsigned)nwg), dim3(256), 0, s, p);
    const int64_t count = (int64_t)n * co;
    hipLaunchKernelGGL(k_linear_relu_from_partials, dim3(grid_stride_blocks(count)), dim3(256), 0, s,
                       part, sc.splits, count, sf, rp, out, code);
}

void launch_linear_dw_mfma(hipStream_t s, int n, int ci, int co, const int32_t *g, uint32_t *gmax,
                           const int8_t *x, int8_t *gt, int8_t *xt, int64_t *dw, uint32_t *flags)
{
    const LinearScratch sc = linear_scratch(n, ci, co);
    const int q = sc.np / 16;
    const int ng = (int)(((int64_t)co * q + 255) / 256), nx = (int)(((int64_t)ci * q + 255) / 256);
    hipLaunchKernelGGL(k_linear_dw_prep, dim3((unsigned)(ng + nx)), dim3(256), 0, s, g, n, co, sc.np,
                       gt, gmax, x, ci, xt, ng);
    // dW[o][c] = sum_k gt[o][k] xt[c][k]: M = co, N = ci, K = np (one split)
    LgemmArgs p{};
    p.M = co; p.N = ci; p.K = sc.np;
    p.a = gt; p.lda = sc.np; p.aplane = (int64_t)co * sc.np; p.a_max = gmax;
    p.b = xt; p.ldb = sc.np; p.bplane = 0; p.b_max = nullptr;
    p.kchunk = sc.np;
    p.out64 = dw; p.ldc = ci; p.m_valid = co;
    p.flags = flags;
    const int64_t nwg = (int64_t)((co + LG_BM - 1) / LG_BM) * ((ci + LG_BN - 1) / LG_BN);
    hipLaunchKernelGGL(k_lgemm_dw, dim3((unsigned)nwg), dim3(256), 0, s, p);
}

// ---------------------------------------------------------------------------------------------
bool mfma_learning_ok(int n, int64_t d, int G, int c)
{
    // c: channels of the block output (its 16-column epilogue groups stay inside one pixel)
    return d % 16 == 0 && c % 16 == 0 && n >= 1 && G >= 1 && (int64_t)n * d < ((int64_t)1 << 31) &&
           (int64_t)G * d < ((int64_t)1 << 31) && G <= 4096;
}

LearningScratch learning_scratch(int n, int64_t d, int G)
{
    LearningScratch s{};
    s.gp = (G + 15) / 16 * 16;
    s.np = (n + 15) / 16 * 16;
    // forward split-K: about two staged chunks (256 of K) per workgroup, at most 1024 workgroups
    int splits = (int)((d + 255) / 256);
    if (splits < 1) splits = 1;
    const int tiles = ((n + LG_BM - 1) / LG_BM) * ((G + LG_BN - 1) / LG_BN);
    if (splits * tiles > 1024) splits = (1024 + tiles - 1) / tiles;
    int64_t kchunk = (d + splits - 1) / splits;
    kchunk = (kchunk + LG_KC - 1) / LG_KC * LG_KC;
    s.kchunk = kchunk;
    s.splits = (int)((d + kchunk - 1) / kchunk);
    s.wf_bytes = 4 * (int64_t)G * d;
    s.wt_bytes = 4 * d * s.gp;
    s.part_bytes = 8 * (int64_t)s.splits * n * G;
    s.epad_bytes = 4 * (int64_t)s.np * s.gp;
    s.et_bytes = 4 * (int64_t)s.gp * s.np;
    s.ft_bytes = d * s.np;
    return s;
}

void launch_learning_mfma(hipStream_t s, int n, int64_t d, int G, const int8_t *f,
                          const int32_t *w, const Div &sf, const int32_t *labels,
                          const LearningBuffers &b, const uint8_t *code, const Relu &rp, int h,
                          int wdt, int c, bool pool, int32_t *g, int32_t *delta_copy,
                          int32_t *yhat, int32_t *e, int64_t *dw, uint32_t *flags,
                          bool prepacked, bool g_pooled)
{
    const LearningScratch sc = learning_scratch(n, d, G);
    // operands: learning-weight limb planes (unless the caller packed them), the transposed
    // block output
    if (!prepacked) launch_pack_matrix(s, w, G, (int)d, sc.gp, b.wf, b.wt, b.wmax);
    // forward: the transposed block output and the split-K partials (one launch), then yhat / e
    {
        LgemmArgs a{};
        a.M = n; a.N = G; a.K = (int)d;
        a.a = f; a.lda = d;
        a.b = b.wf; a.ldb = d; a.bplane = (int64_t)G * d; a.b_max = b.wmax;
        a.kchunk = (int)sc.kchunk;
        a.out64 = b.part;
        a.flags = flags;
        const int tgx = (int)((d + 63) / 64), tgy = (sc.np + 63) / 64;
        const int64_t nwg = (int64_t)tgx * tgy + (int64_t)((n + LG_BM - 1) / LG_BM) * ((G + LG_BN - 1) / LG_BN) * sc.splits;
        hipLaunchKernelGGL(k_lgemm_fwd, dim3((unsigned)nwg), dim3(256), 0, s, a, f, n, (int)d, sc.np, b.ft, tgx, tgy);
        hipLaunchKernelGGL(k_loss_from_partials, dim3(grid_stride_blocks((int64_t)sc.np * sc.gp, 256, 256)),
                           dim3(256), 0, s, b.part, sc.splits, n, G, sc.gp, sc.np, sf, labels, yhat,
                           e, b.epad, b.et, b.emax, flags);
    }
    // weight gradient dW[g][k] = sum_n e[n][g] f[n][k] (M = gp, N = d, K = np) and delta = e W
    // (pre-update), routed through the pool and NITRO-ReLU backward into g: one launch
    LgemmArgs da{}, ua{};
    {
        LgemmArgs &a = da;
        a.M = sc.gp; a.N = (int)d; a.K = sc.np;
        a.a = b.et; a.lda = sc.np; a.aplane = (int64_t)sc.gp * sc.np; a.a_max = b.emax;
        a.b = b.ft; a.ldb = sc.np; a.bplane = 0; a.b_max = nullptr;
        a.kchunk = sc.np;
        a.out64 = dw; a.ldc = d; a.m_valid = G;
        a.flags = flags;
    }
    {
        LgemmArgs &a = ua;
        a.M = n; a.N = (int)d; a.K = sc.gp;
        a.a = b.epad; a.lda = sc.gp; a.aplane = (int64_t)sc.np * sc.gp; a.a_max = b.emax;
        a.b = b.wt; a.ldb = sc.gp; a.bplane = d * sc.gp; a.b_max = b.wmax;
        a.kchunk = sc.gp;
        a.code = code; a.rp = rp; a.h = h; a.w = wdt; a.c = c; a.pool = pool ? 1 : 0;
        a.gpooled = pool && g_pooled ? 1 : 0;
        a.g = g; a.delta = delta_copy; a.gmax = b.gmax;
        a.flags = flags;
    }
    const int64_t nwg = (int64_t)((da.M + LG_BM - 1) / LG_BM) * ((da.N + LG_BN - 1) / LG_BN) +
                        (int64_t)((ua.M + LG_BM - 1) / LG_BM) * ((ua.N + LG_BN - 1) / LG_BN);
    hipLaunchKernelGGL(k_lgemm_bwd, dim3((unsigned)nwg), dim3(256), 0, s, da, ua);
}

}  // namespace nitro
