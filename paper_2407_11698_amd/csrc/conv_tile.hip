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
// of W, [N][9 ck], tap-major) is staged beside it, the nine taps of the chunk for the tile's 64
// columns. Operands wider than int8 are split into balanced int8 limbs; each limb pair is one
// pass over K accumulated in int32 (|sum| <= 128 * 128 * 9 * 8192 < 2^31) and folded into int64
// with its shift.
#include <type_traits>

#include "mfma_common.h"

namespace nitro {

enum { IG_FWD = 0, IG_DX = 1 };

constexpr int CT_BN = 64;          // GEMM columns per workgroup

// Tile shapes. WM = 2: 128 output pixels, 4 waves, one LDS stage (two workgroups per CU).
// WM = 4: 256 output pixels, 8 waves, two LDS stages (one workgroup per CU), the next phase's
// operands written to the idle stage while the current one computes.
template <int WM>
struct CtShape {
    static constexpr int BM = 64 * WM;                  // output pixels per workgroup
    static constexpr int NT = 128 * WM;                 // threads
    static constexpr int NPMAX = WM == 2 ? 320 : 448;   // largest staged pixel count
    static constexpr int NBUF = WM == 2 ? 1 : 2;        // LDS stages
};

// LDS stages. A: [pixel][PS bytes], PS = 96 for chunks of 32 or 64 channels (a fragment read,
// 16 consecutive pixels by 4 lane groups, then touches every bank once per cycle). B:
// [tap][column][CC bytes]; with 64 channels the 16-byte unit u of column c sits in slot
// u ^ ((c >> 1) & 3), which keeps both its fragment reads and the staging writes (4 lanes per
// column) free of bank conflicts.
template <int CC, int WM>
struct CtCfg {
    static constexpr int PS = CC == 16 ? 16 : 96;      // LDS bytes per staged pixel
    static constexpr int GPT = CC / 16;                 // 16-channel groups per tap and chunk
    static constexpr int KSC = (9 * GPT + 3) / 4;        // K-steps (of 4 groups) per chunk
    static constexpr int NIT = (CtShape<WM>::NPMAX * GPT + CtShape<WM>::NT - 1) / CtShape<WM>::NT;
};

__host__ __device__ constexpr int ct_bswz(int cc, int c) { return cc == 64 ? (c >> 1) & 3 : 0; }

// A straight into LDS (64-channel chunks, W a multiple of 16, two stages): staged rows of apitch
// pixels (W + 2 used); LDS unit 4 q + (e ^ ((q >> 1) & 3)) holds 16-channel group e of staged
// pixel q. The load is lane-linear, four consecutive lanes taking one pixel's 64 contiguous bytes
// (one cache access), and a fragment read (16 consecutive pixels, one group, from any first
// pixel) runs without bank conflicts (measured; the swizzle (q >> 2) & 3 costs about 4 conflict
// cycles per read).
constexpr int CT_NPMAX_DIRECT = 576;           // staged pixels
__device__ __attribute__((aligned(16))) const int8_t ct_zero16[16] = {};   // source of zero units

struct TileArgs {
    int n, h, w;
    int ck;                        // channels of A; K = 9 ck (a multiple of the chunk size CC)
    int no;                        // GEMM N (a multiple of 16)
    int ntiles;                    // output tiles (the grid may be smaller: persistent workgroups)
    const int8_t *a;               // forward: x NHWC; input gradient: limb planes [LA][P][ck]
    int64_t aplane;                // P * ck
    const uint32_t *a_max;         // input gradient: max|g| slot
    const int8_t *b;               // 4 limb planes [no][9 ck]
    int64_t bplane;                // no * 9 ck
    const uint32_t *b_max;
    int rt, ns, rs;                // image rows per tile; images per tile; rows per image segment
    int apitch;                    // A loaded straight into LDS: staged row pitch (a multiple of 16)
    Div32 d_apitch, d_aseg;        // its reciprocals of apitch and (rs + 2) apitch
    Div32 d_w2, d_seg, d_w, d_rw;  // reciprocals of W + 2, (rs + 2)(W + 2), W and rs W
    // forward epilogue
    ScaleFast sf;
    int pool;
    int8_t *out;
    uint8_t *code;
    int8_t *xr;                    // optional (not pooled): the next layer's weight-gradient x rows
    int64_t xs;                    // their stride (positions per 16-channel tile)
    Div32 d_h;                     // reciprocal of H
    // input-gradient epilogue
    const uint8_t *prev_code;
    Relu rp;
    int32_t *gout;
    int16_t *gout16;               // optional: g in the escaped 16-bit form (gout: escapes only)
    int64_t *out64;
    uint32_t *gmax;
    uint32_t *flags;
    uint64_t *ts;                  // timing slot (null: untimed)
    // out64: g may be in the offset form (two limbs of g - 128, or three with more than
    // GOFF_CAP entries g = 32768), its term from the border-class table goff_bias [16][no]
    int goff;
    const uint32_t *goff_count;
    const int64_t *goff_bias;
};

__device__ inline int32_t sat_i32(int64_t v)
{
    return v > INT32_MAX ? INT32_MAX : (v < INT32_MIN ? INT32_MIN : (int32_t)v);
}

// One tile per workgroup. Both operands go through LDS: each phase (a limb pair and a chunk of CC
// channels) stages the A pixels and the B block of 9 taps x 64 columns x CC. The next phase's
// global loads are issued before the current phase computes; the fragments of the next K-step
// are read from LDS while the MFMAs of the current one run.
template <int MODE, int CC, int WM, bool PERSIST, bool ADMA>
__global__ __launch_bounds__(128 * WM) __attribute__((amdgpu_waves_per_eu(2, 2)))
void k_conv_tile(TileArgs p)
{
    using S = CtShape<WM>;
    using C = CtCfg<CC, WM>;
    static_assert(!ADMA || (CC == 64 && S::NBUF == 2), "A straight into LDS: 64 channels, two stages");
    constexpr int BM = S::BM, NT = S::NT;
    constexpr int TM = 4, TN = 2;                 // 16x16 tiles per wave: 64 pixels x 32 columns
    constexpr int NU = CC / 16;                   // 16-byte units per (tap, column) row of B
    constexpr int SA = ADMA ? CT_NPMAX_DIRECT * 64 : S::NPMAX * C::PS;   // A stage bytes
    constexpr int NIA = ADMA ? (CT_NPMAX_DIRECT * 4 + NT - 1) / NT : C::NIT;   // A items per thread
    constexpr int BITEMS = 9 * CT_BN * NU;        // 16-byte units of a B stage
    constexpr int BIT = (BITEMS + NT - 1) / NT;   // B units per thread
    constexpr int SAB = SA + BITEMS * 16;         // one stage
    constexpr int OS = CT_BN + 16;                // forward epilogue: LDS row stride in bytes
    constexpr int SMEM_EPI = MODE == IG_FWD ? 2 * BM * OS : 0;
    // the forward epilogue's LDS: one stage; two stages: the one the last phase computed from
    // (the other holds the next tile's first phase), or after both where it does not fit one
    constexpr bool EPI_IN_STAGE = S::NBUF == 1 || SMEM_EPI <= SAB;
    constexpr int SMEM_MAIN = S::NBUF == 1 ? (SAB > SMEM_EPI ? SAB : SMEM_EPI)
                                           : 2 * SAB + (EPI_IN_STAGE ? 0 : SMEM_EPI);
    constexpr int SMEM_SINK = SMEM_MAIN + (MODE == IG_FWD ? 528 : 0);   // after the NITRO-ReLU table
    constexpr int SMEM = SMEM_SINK + 1024;        // + a sink for staging lanes with nothing to store
    __shared__ __attribute__((aligned(16))) uint8_t smem[SMEM];

    ts_start(p.ts);
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int g4 = lane >> 4;
    uint16_t *const tab = (uint16_t *)(smem + SMEM_MAIN);   // forward: entry for zs = -128 .. 128
    if (MODE == IG_FWD)
        for (int k = tid; k < 257; k += NT) tab[k] = relu_table_entry(k - 128, p.sf);
    const int ntile_n = (p.no + CT_BN - 1) / CT_BN;
    const int ntiles = p.ntiles;
    const int W2 = p.w + 2;
    const int segpx = (p.rs + 2) * W2;
    const int aseg = (p.rs + 2) * p.apitch;       // A straight into LDS: staged pixels per segment
    const int np = ADMA ? p.ns * aseg : p.ns * segpx;
    const int64_t M = (int64_t)p.n * p.h * p.w;
    const int K = 9 * p.ck;
    const int nchunk = p.ck / CC;

    // (input gradient: the residual count of the offset form is read whether or not it is
    // used, from the max slot then, so that both loads are in flight together)
    bool goff = false;
    int LA = 1;
    if (MODE == IG_DX) {
        const uint32_t rn = *(p.goff ? p.goff_count : p.a_max);
        const uint32_t am = slot_read(p.a_max);
        goff = p.goff && goff_range(am);
        LA = goff ? (rn <= GOFF_CAP ? 2 : 3) : limbs_for(am);
    }
    const int LB = limbs_for(slot_read(p.b_max));
    if (LA > 4 || LB > 4) {
        if (tid == 0) raise_flag(p.flags, FLAG_OVERFLOW);
        return;
    }
    const int npass = LA * LB;
    const int nph = npass * nchunk;

    // staged A items of this thread: item tid + NT v = (LDS pixel q, 16-channel group e), the
    // groups of one pixel on consecutive lanes
    auto a_item = [&](int item, int &q, int &e) {
        q = item / C::GPT;
        e = item - q * C::GPT;
    };
    // staged B units of this thread: unit tid + NT v is (tap t, column c, unit u), the units of a
    // column on consecutive lanes; c and u are fixed by tid and t = v TPV + t0
    constexpr int TPV = NT / (CT_BN * NU);        // taps per NT units
    const int b_c = (tid % (CT_BN * NU)) / NU, b_u = tid % NU, b_t0 = tid / (CT_BN * NU);
    const int b_l0 = (b_t0 * CT_BN + b_c) * CC + 16 * (b_u ^ ct_bswz(CC, b_c));

    // The current tile: its first output pixel m0 and column n0; the global byte offset within a
    // chunk of each staged A item (-1: a zero, outside the image) and of this thread's B units.
    // Tile order: each of the eight XCDs takes a contiguous range of tiles, so the column tiles of
    // one pixel tile run together and share their A rows in that XCD's L2.
    int64_t m0;
    int n0, b_g0;
    int it_g[NIA];
    auto set_tile = [&](int v) {
        const int tile = (ntiles & 7) == 0 ? (v & 7) * (ntiles >> 3) + (v >> 3) : v;
        const int mt = tile / ntile_n, nt = tile - mt * ntile_n;
        const int R0 = mt * p.rt;                  // first image row of the tile (over all images)
        const int img0 = (int)udiv32((uint32_t)R0, p.d_h), row0 = R0 - img0 * p.h;
        m0 = (int64_t)R0 * p.w;
        n0 = nt * CT_BN;
#pragma unroll
        for (int u = 0; u < NIA; u++) {
            int q, e;
            if (ADMA) {
                const int unit = tid + NT * u;
                q = unit >> 2;
                e = (unit & 3) ^ ((q >> 1) & 3);
            } else {
                a_item(tid + NT * u, q, e);
            }
            it_g[u] = -1;
            if (q < np) {
                int seg, lr, lc;
                if (ADMA) {
                    seg = (int)udiv32(q, p.d_aseg);
                    const int r = q - seg * aseg;
                    lr = (int)udiv32(r, p.d_apitch);
                    lc = r - lr * p.apitch;
                } else {
                    seg = (int)udiv32(q, p.d_seg);
                    const int r = q - seg * segpx;
                    lr = (int)udiv32(r, p.d_w2);
                    lc = r - lr * W2;
                }
                const int img = img0 + seg, hh = row0 + lr - 1, ww = lc - 1;
                if (img < p.n && hh >= 0 && hh < p.h && ww >= 0 && ww < p.w)
                    it_g[u] = ((img * p.h + hh) * p.w + ww) * p.ck + 16 * e;
                else if (ADMA && ww > p.w)
                    it_g[u] = -2;                  // row padding: never read, not loaded
            }
        }
        // A and B straight into LDS: lane-linear, so B's unit swizzle is applied to the source;
        // otherwise through registers, swizzled on the store
        const int bu = ADMA ? b_u ^ ct_bswz(CC, b_c) : b_u;
        b_g0 = (n0 + b_c < p.no ? n0 + b_c : p.no - 1) * K + b_t0 * p.ck + 16 * bu;
    };
    // LDS byte offset of this lane's A pixel in fragment i (tap (1, 1)). A straight into LDS:
    // the fragment's 16 pixels lie in one image row, from a column that is a multiple of 16, so
    // the offset is that 16-pixel block's; the lane's pixel l = lane % 16 + s in the block for
    // column offset s - 1 (s = 0, 1, 2) and its channel group give alast[s] (row offsets are
    // whole blocks, so the swizzle depends on l only).
    int cpix[TM], alast[3];
#pragma unroll
    for (int i = 0; i < TM; i++) {
        const int mloc = wm * 64 + 16 * i + (ADMA ? 0 : (lane & 15));
        const int seg = (int)udiv32(mloc, p.d_rw), rem = mloc - seg * p.rs * p.w;
        const int row = (int)udiv32(rem, p.d_w), col = rem - row * p.w;
        if (ADMA)
            cpix[i] = (seg * aseg + (row + 1) * p.apitch + col) * 64;
        else
            cpix[i] = (seg * segpx + (row + 1) * W2 + col + 1) * C::PS;
    }
#pragma unroll
    for (int t = 0; t < 3; t++) {
        const int l = (lane & 15) + t;
        alast[t] = 64 * l + 16 * (g4 ^ ((l >> 1) & 3));
    }
    // LDS byte offset of this lane's B unit in each column tile (tap 0): column c, unit c16 of
    // the lane's group (fixed per lane: 4 ks + g4 = g4 modulo GPT)
    const int c16l = g4 % C::GPT;
    int bcol[TN];
#pragma unroll
    for (int j = 0; j < TN; j++) {
        const int c = wn * 32 + 16 * j + (lane & 15);
        bcol[j] = c * CC + 16 * (c16l ^ ct_bswz(CC, c));
    }
    const int sgn = MODE == IG_FWD ? 1 : -1;

    // operands of phase ph: limb pair (la, lb) and the chunk of CC channels
    auto src_a = [&](int ph) {
        const int chunk = ph % nchunk, pass = ph / nchunk;
        return p.a + (int64_t)(pass / LB) * p.aplane + chunk * CC;
    };
    auto src_b = [&](int ph) {
        const int chunk = ph % nchunk, pass = ph / nchunk;
        return p.b + (int64_t)(pass % LB) * p.bplane + chunk * CC + b_g0;
    };
    v4i stga[NIA], stgb[BIT];
    auto a_load = [&](const int8_t *srca, int v) {
        stga[v] = *(const v4i *)(srca + (it_g[v] >= 0 ? it_g[v] : 0));
    };
    // (branch-free: a lane whose item lies past the staged pixels stores into the sink)
    auto a_store = [&](int buf, int v) {
        int q, e;
        a_item(tid + NT * v, q, e);
        const int off = q < np ? buf * SAB + q * C::PS + 16 * e : SMEM_SINK + 16 * lane;
        *(v4i *)(smem + off) = it_g[v] >= 0 ? stga[v] : v4i{0, 0, 0, 0};
    };
    // B unit tid + NT v straight into LDS byte 16 (tid + NT v) (A straight into LDS): a wave's
    // 64 units are contiguous (its tap, b_t0 + v TPV, is the same on every lane); a wave past the
    // ninth tap has nothing to load
    typedef __attribute__((address_space(3))) void *LdsPtr;
    const int wave_u = __builtin_amdgcn_readfirstlane(wave);
    const int b_t0u = __builtin_amdgcn_readfirstlane(b_t0);
    auto b_direct = [&](int buf, const int8_t *srcb, int v) {
        if (b_t0u + v * TPV < 9)
            __builtin_amdgcn_global_load_lds((const void *)(srcb + v * TPV * p.ck),
                                             (LdsPtr)(smem + buf * SAB + SA + 16 * (NT * v + 64 * wave_u)),
                                             16, 0, 0);
    };
    // A unit tid + NT v straight into LDS (A straight into LDS): a wave's 64 units are
    // contiguous and all staged, or (past the staged pixels) none; a zero unit is read from
    // ct_zero16; a lane on row padding loads nothing
    const int npa4u = __builtin_amdgcn_readfirstlane(4 * np);
    auto a_direct = [&](int buf, const int8_t *srca, int v) {
        if (NT * v + 64 * wave_u < npa4u && it_g[v] != -2) {
            const int8_t *src = it_g[v] >= 0 ? srca + it_g[v] : ct_zero16;
            __builtin_amdgcn_global_load_lds((const void *)src,
                                             (LdsPtr)(smem + buf * SAB + 16 * (NT * v + 64 * wave_u)), 16, 0, 0);
        }
    };
    // one stage: the whole phase through registers, loaded before the compute, stored after it
    auto stage_load = [&](int ph) {
        const int8_t *srca = src_a(ph), *srcb = src_b(ph);
#pragma unroll
        for (int v = 0; v < NIA; v++) a_load(srca, v);
#pragma unroll
        for (int v = 0; v < BIT; v++)
            if (b_t0 + v * TPV < 9) stgb[v] = *(const v4i *)(srcb + v * TPV * p.ck);
    };
    auto stage_store = [&](int buf) {
#pragma unroll
        for (int v = 0; v < NIA; v++) a_store(buf, v);
#pragma unroll
        for (int v = 0; v < BIT; v++)
            if (b_t0 + v * TPV < 9) *(v4i *)(smem + buf * SAB + SA + b_l0 + v * NT * 16) = stgb[v];
    };
    // fragments of K-step ks: group G = 4 ks + g4 is (tap t, 16-channel group c16); a K-step past
    // the ninth tap (chunks of 16 or 32 channels) has zero A fragments
    auto load_frags = [&](const uint8_t *As, v4i(&af)[TM], v4i(&bf)[TN], int ks) {
        const uint8_t *Bs = As + SA;
        const int G = 4 * ks + g4;
        const int t = G / C::GPT, c16 = G - t * C::GPT;
        const bool valid = t < 9;
        const int tc = valid ? t : 8;
        if (ADMA) {
            // (64 channels: tap ks, group g4 on every lane)
            const int dr = sgn * (ks / 3 - 1), dc = sgn * (ks % 3 - 1);
            const int roff = dr * p.apitch * 64;
#pragma unroll
            for (int i = 0; i < TM; i++) af[i] = *(const v4i *)(As + cpix[i] + alast[1 + dc] + roff);
        } else {
            const int toff = sgn * ((tc / 3 - 1) * W2 + (tc % 3 - 1)) * C::PS + 16 * c16;
#pragma unroll
            for (int i = 0; i < TM; i++) {
                const v4i v = *(const v4i *)(As + cpix[i] + toff);
                af[i] = valid ? v : v4i{0, 0, 0, 0};
            }
        }
#pragma unroll
        for (int j = 0; j < TN; j++) bf[j] = *(const v4i *)(Bs + tc * CT_BN * CC + bcol[j]);
    };

    int64_t acc64[TM][TN][4];
    v4i acc[TM][TN];

    // A straight into LDS: while a phase computes, the other stage receives the next phase's
    // operands, their LDS-direct loads spread over all but the last K-step so that the address
    // unit takes them alongside the MFMAs.
    constexpr int NLD = NIA + BIT;                // loads per thread and phase
    constexpr int LDK = C::KSC - 1;               // K-steps issuing them
    auto compute = [&](auto stage_tag, const uint8_t *As, int sbuf, const int8_t *sa, const int8_t *sb) {
        constexpr bool STG = decltype(stage_tag)::value;
        v4i af[2][TM], bf[2][TN];
        load_frags(As, af[0], bf[0], 0);
        // the next K-step's fragment reads are issued before this K-step's MFMAs, and the
        // scheduling barriers keep them there: left to itself the scheduler issues each read just
        // before its first use and then waits for it. (The 128-pixel input-gradient kernel has
        // no registers left for the second set of fragments.)
        constexpr bool PIPE = !(WM == 2 && MODE == IG_DX);
#pragma unroll
        for (int ks = 0; ks < C::KSC; ks++) {
            if (ADMA && STG) {
#pragma unroll
                for (int i = 0; i < NLD; i++)
                    if (i * LDK / NLD == ks) {
                        if (i < NIA) a_direct(sbuf, sa, i);
                        else b_direct(sbuf, sb, i - NIA);
                    }
            }
            if (ks + 1 < C::KSC) load_frags(As, af[(ks + 1) & 1], bf[(ks + 1) & 1], ks + 1);
            if (PIPE) __builtin_amdgcn_sched_barrier(0);
#pragma unroll
            for (int i = 0; i < TM; i++)
#pragma unroll
                for (int j = 0; j < TN; j++)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(bf[ks & 1][j], af[ks & 1][i],
                                                                      acc[i][j], 0, 0, 0);
            if (PIPE) __builtin_amdgcn_sched_barrier(0);
        }
    };
    auto fold = [&](int ph) {
        if (npass > 1 && (ph + 1) % nchunk == 0) {
            // fold this limb pass into int64 with its weight 256^(la + lb)
            const int pass = ph / nchunk, la = pass / LB, lb = pass - la * LB;
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
    };

    // Persistent (two stages, one workgroup per CU): workgroup b takes tiles b, b + G, b + 2G, ...
    // (G = the grid size), its set-up done once, and the global loads of the next tile's first
    // phase are issued before the epilogue and overlap it. Otherwise one tile per workgroup.
    // (input gradient: the previous layer's region codes of this thread's outputs, requested
    // all at once as the tile's last phase starts, so that they arrive under its MFMAs; read
    // one by one between the epilogue's stores, each read would wait for the memory in turn)
    uint32_t cdv[MODE == IG_DX ? TM : 1][MODE == IG_DX ? TN : 1];
    // The loads are issued whether or not there are codes (then from a zero block): this loop
    // also loads straight into LDS, and the compiler counts outstanding loads statically, so a
    // load skipped on one path would let its wait before the next barrier count too few.
    auto codes_load = [&](int64_t tm0, int tn0) {
        if (MODE != IG_DX) return;
        const int pxp = (tid >> 7) * 64 + (tid & 15);
        const int cbp = ((tid >> 6) & 1) * 32 + 4 * ((tid >> 4) & 3);
        const bool have = p.prev_code != nullptr;
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++) {
                const int64_t m = tm0 + pxp + 16 * i;
                const int col = tn0 + cbp + 16 * j;
                const bool in = have && m < M && col < p.no;
                const uint8_t *src = in ? p.prev_code + m * p.no + col : (const uint8_t *)ct_zero16;
                cdv[MODE == IG_DX ? i : 0][MODE == IG_DX ? j : 0] = *(const uint32_t *)src;
            }
    };
    uint32_t mx = 0;                              // input gradient: max |g| over this workgroup
    bool bad = false;                             // input gradient: a sum outside int32
    int v = blockIdx.x;
    int gph = 0;                                  // phases computed: stage gph & 1 is current
    set_tile(v);
    if (ADMA) {
        const int8_t *sa = src_a(0), *sb = src_b(0);
#pragma unroll
        for (int u = 0; u < NIA; u++) a_direct(0, sa, u);
#pragma unroll
        for (int u = 0; u < BIT; u++) b_direct(0, sb, u);
    } else {
        stage_load(0);
        if (S::NBUF == 2) stage_store(0);
    }
    for (;;) {
        const int vn = v + (int)gridDim.x;
        const bool more = PERSIST && vn < ntiles;
        const int64_t em0 = m0;                   // this tile's, for the epilogue
        const int en0 = n0;
#pragma unroll
        for (int i = 0; i < TM; i++)
#pragma unroll
            for (int j = 0; j < TN; j++) {
                acc[i][j] = v4i{0, 0, 0, 0};
#pragma unroll
                for (int t = 0; t < 4; t++) acc64[i][j][t] = 0;
            }
        if (S::NBUF == 1) {
            for (int ph = 0; ph < nph; ph++) {
                __syncthreads();                  // every wave is done with the previous stage
                stage_store(0);
                __syncthreads();
                if (ph + 1 < nph) stage_load(ph + 1);
                if (ph + 1 == nph) codes_load(em0, en0);
                compute(std::false_type{}, smem, 0, nullptr, nullptr);
                fold(ph);
                gph++;
            }
        } else {
            // the barrier publishes stage gph & 1 (staged during the previous phase, of this tile
            // or the one before) and ends every read of the other stage, which then receives
            // this tile's next phase or, in its last phase, the next tile's first. A straight
            // into LDS: during the compute. Otherwise loaded into registers before the compute
            // and stored after it; the next tile's first phase loaded after the last compute and
            // stored after the epilogue.
            for (int ph = 0; ph < nph; ph++) {
                __syncthreads();
                const int cb = gph & 1;
                if (ph + 1 == nph) codes_load(em0, en0);
                if (ADMA) {
                    const int8_t *sa = nullptr, *sb = nullptr;
                    if (ph + 1 < nph) {
                        sa = src_a(ph + 1);
                        sb = src_b(ph + 1);
                    } else if (more) {
                        set_tile(vn);
                        sa = src_a(0);
                        sb = src_b(0);
                    }
                    if (sa) compute(std::true_type{}, smem + cb * SAB, cb ^ 1, sa, sb);
                    else compute(std::false_type{}, smem + cb * SAB, 0, nullptr, nullptr);
                } else {
                    if (ph + 1 < nph) stage_load(ph + 1);
                    compute(std::false_type{}, smem + cb * SAB, 0, nullptr, nullptr);
                }
                fold(ph);
                if (!ADMA && ph + 1 < nph) stage_store(cb ^ 1);
                gph++;
            }
            if (!ADMA && more) {
                set_tile(vn);
                stage_load(0);
            }
        }
        __syncthreads();                          // the epilogue reuses the stages' LDS
        // ------------------------------------------------------------ epilogues
        // The MFMAs took B as the first operand: lane l of tile (i, j) holds output channels
        // cb = wn 32 + 16 j + 4 g4 .. cb + 3 of pixel wm 64 + 16 i + l % 16. The thread index is
        // taken through an opaque copy so that the epilogue's address terms are recomputed per
        // tile rather than held in registers across the tile loop.
        int etid = tid;
        asm volatile("" : "+v"(etid));
        const int pxl = (etid >> 7) * 64 + (etid & 15);
        const int cbl = ((etid >> 6) & 1) * 32 + 4 * ((etid >> 4) & 3);
        // (input gradient, register staging: the next tile's first phase to its stage before
        // the epilogue's global stores, as in the forward epilogue)
        if (MODE == IG_DX && !ADMA && S::NBUF == 2 && more) stage_store(gph & 1);
        if (MODE == IG_FWD) {
            // NITRO-Scaling (shift, clamp, one multiply-high) and the table's NITRO-ReLU per
            // element; four channels packed per dword into LDS, then 16-byte (or pooled) stores.
            // Several limb passes: the int64 sum saturated to int32 still saturates z*
            // (128 SF < 2^31).
            if (npass > 1) {
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int j = 0; j < TN; j++)
#pragma unroll
                        for (int t = 0; t < 4; t++) acc[i][j][t] = sat_i32(acc64[i][j][t]);
            }
            constexpr int OW = OS / 4;                // row stride in dwords
            const int epi = !EPI_IN_STAGE ? 2 * SAB : S::NBUF == 2 ? ((gph - 1) & 1) * SAB : 0;
            uint32_t *Ov = (uint32_t *)(smem + epi);  // [BM][OW] packed activations
            uint32_t *Rv = Ov + BM * OW;              // [BM][OW] packed region codes
            // (every table read is issued before the first is used; each entry is the output
            // byte | region << 8, and two byte permutes gather four entries' outputs and regions)
            auto pack = [&](auto trunc_tag) {
                constexpr bool TR = decltype(trunc_tag)::value;
                uint32_t ent[TM][TN][4];
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int j = 0; j < TN; j++)
#pragma unroll
                        for (int t = 0; t < 4; t++) ent[i][j][t] = tab[scale_fast<TR>(acc[i][j][t], p.sf) + 128];
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int j = 0; j < TN; j++) {
                        const uint32_t x01 = ent[i][j][0] | (ent[i][j][1] << 16);
                        const uint32_t x23 = ent[i][j][2] | (ent[i][j][3] << 16);
                        const int o = (pxl + 16 * i) * OW + (cbl + 16 * j) / 4;
                        Ov[o] = __builtin_amdgcn_perm(x23, x01, 0x06040200u);
                        Rv[o] = __builtin_amdgcn_perm(x23, x01, 0x07050301u);
                    }
            };
            if (p.sf.trunc) pack(std::true_type{});
            else pack(std::false_type{});
            // register staging: the next tile's first phase goes to its stage now (its loads
            // were issued before this epilogue), ahead of the epilogue's global stores
            if (!ADMA && S::NBUF == 2 && more) stage_store(gph & 1);
            __syncthreads();
            if (!p.pool) {
                for (int c = etid; c < BM * CT_BN / 16; c += NT) {
                    const int row = c / (CT_BN / 16), q = c % (CT_BN / 16);
                    const int64_t m = em0 + row;
                    if (m >= M || en0 + 16 * q >= p.no) continue;
                    const int64_t o = m * p.no + en0 + 16 * q;
                    const v4i av = *(const v4i *)(Ov + row * OW + 4 * q);
                    *(v4i *)(p.out + o) = av;
                    *(v4i *)(p.code + o) = *(const v4i *)(Rv + row * OW + 4 * q);
                    if (p.xr) {
                        // padded position of pixel m: (n (H+1) + h)(W+1) + w
                        // = (R + R / H)(W+1) + w, R = m / W its row over all images
                        const uint32_t R = udiv32((uint32_t)m, p.d_w);
                        const uint32_t ww = (uint32_t)m - R * (uint32_t)p.w;
                        const int64_t k = (int64_t)(R + udiv32(R, p.d_h)) * (p.w + 1) + ww;
                        const int64_t row16 = (int64_t)((en0 >> 4) + q) * p.xs + DWP_HMAX + k;
                        *(v4i *)(p.xr + row16 * 16) = av;
                    }
                }
            } else {
                // 2x2 windows, 4 channels per thread: the tile holds rt (even) whole image rows;
                // the first maximum in (0,0), (0,1), (1,0), (1,1) order wins
                const int W = p.w, Wh = p.w / 2;
                for (int c = etid; c < (BM / 4) * (CT_BN / 4); c += NT) {
                    const int win = c / (CT_BN / 4), cw = c % (CT_BN / 4);
                    const int wr = win / Wh, wc = win - wr * Wh;
                    const int q = 2 * wr * W + 2 * wc;
                    const int64_t m = em0 + q;
                    if (m >= M || en0 + 4 * cw >= p.no) continue;
                    uint32_t va[4], ra[4];
#pragma unroll
                    for (int t = 0; t < 4; t++) {
                        const int at = q + (t >> 1) * W + (t & 1);
                        va[t] = Ov[at * OW + cw];
                        ra[t] = Rv[at * OW + cw];
                    }
                    uint32_t ov = 0, cv = 0;
#pragma unroll
                    for (int e = 0; e < 4; e++) {
                        int best = (int)(int8_t)(va[0] >> (8 * e));
                        uint32_t code = (ra[0] >> (8 * e)) & 0xffu;
                        code <<= 2;
#pragma unroll
                        for (int t = 1; t < 4; t++) {
                            const int v = (int)(int8_t)(va[t] >> (8 * e));
                            if (v > best) {
                                best = v;
                                code = (((ra[t] >> (8 * e)) & 0xffu) << 2) | (uint32_t)t;
                            }
                        }
                        ov |= (uint32_t)(uint8_t)(int8_t)best << (8 * e);
                        cv |= code << (8 * e);
                    }
                    const int64_t grow = m / W;
                    const int64_t pp = (grow / 2) * Wh + (m % W) / 2;
                    const int64_t o = pp * p.no + en0 + 4 * cw;
                    *(uint32_t *)(p.out + o) = ov;
                    *(uint32_t *)(p.code + o) = cv;
                }
            }
        } else if (p.out64) {
            // raw int64 input gradient (the first layer of a network): 4 channels per lane and
            // tile; the offset form adds its term for the pixel's border class
#pragma unroll
            for (int i = 0; i < TM; i++)
#pragma unroll
                for (int j = 0; j < TN; j++) {
                    const int64_t m = em0 + pxl + 16 * i;
                    const int col = en0 + cbl + 16 * j;
                    if (m >= M || col >= p.no) continue;
                    int64_t *dst = p.out64 + m * p.no + col;
                    int64_t bv[4] = {0, 0, 0, 0};
                    if (goff) {
                        const uint32_t R = udiv32((uint32_t)m, p.d_w);
                        const int ww = (int)((uint32_t)m - R * (uint32_t)p.w);
                        const int hh = (int)(R - udiv32(R, p.d_h) * (uint32_t)p.h);
                        const int cls = (hh == 0) | (hh == p.h - 1) << 1 | (ww == 0) << 2 | (ww == p.w - 1) << 3;
                        const int64_t *bp = p.goff_bias + cls * p.no + col;
#pragma unroll
                        for (int t = 0; t < 4; t++) bv[t] = bp[t];
                    }
#pragma unroll
                    for (int t = 0; t < 4; t++)
                        dst[t] = (npass > 1 ? acc64[i][j][t] : (int64_t)acc[i][j][t]) + bv[t];
                }
        } else {
            // int32 sums, ReLU' of the previous layer with its 4 region codes, one 16-byte store
            // per lane and tile
            if (npass > 1) {
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int j = 0; j < TN; j++)
#pragma unroll
                        for (int t = 0; t < 4; t++) {
                            bad |= !fits_i32(acc64[i][j][t]);
                            acc[i][j][t] = (int32_t)acc64[i][j][t];
                        }
            }
            auto emit = [&](auto trunc_tag) {
                constexpr bool TR = decltype(trunc_tag)::value;
#pragma unroll
                for (int i = 0; i < TM; i++)
#pragma unroll
                    for (int j = 0; j < TN; j++) {
                        const int64_t m = em0 + pxl + 16 * i;
                        const int col = en0 + cbl + 16 * j;
                        if (m >= M || col >= p.no) continue;
                        const int64_t o = m * p.no + col;
                        v4i g = acc[i][j];
                        if (p.prev_code) {
                            const uint32_t cd = cdv[MODE == IG_DX ? i : 0][MODE == IG_DX ? j : 0];
#pragma unroll
                            for (int t = 0; t < 4; t++)
                                g[t] = relu_bwd32<TR>(g[t], (cd >> (8 * t)) & 0xffu, p.rp);
                        }
#pragma unroll
                        for (int t = 0; t < 4; t++) {
                            const uint32_t ag = abs_u32(g[t]);
                            mx = ag > mx ? ag : mx;
                        }
                        if (p.gout16) {
                            uint32_t h[4];
#pragma unroll
                            for (int t = 0; t < 4; t++) {
                                const bool esc = g[t] < -G16_MAX || g[t] > G16_MAX;
                                if (esc) p.gout[o + t] = g[t];
                                h[t] = (uint32_t)(uint16_t)(esc ? G16_ESC : (int16_t)g[t]);
                            }
                            *(v2i *)(p.gout16 + o) = v2i{(int)(h[0] | (h[1] << 16)), (int)(h[2] | (h[3] << 16))};
                        } else {
                            *(v4i *)(p.gout + o) = g;
                        }
                    }
            };
            if (p.rp.alpha.trunc) emit(std::true_type{});
            else emit(std::false_type{});
        }
        if (!more) break;
        v = vn;
    }
    if (MODE == IG_DX && !p.out64) {
        if (bad) raise_flag(p.flags, FLAG_OVERFLOW);
        if (p.gmax) block_slot_max(p.gmax, mx);
    }
    ts_end(p.ts);
}

// Tile geometry: rt = BM / W image rows; either rt divides H (one image segment) or H divides
// rt (rt / H whole images); at most NPMAX staged pixels.
template <int WM>
static bool tile_geom(int h, int w, int *rt, int *ns, int *rs)
{
    constexpr int BM = CtShape<WM>::BM;
    if (w < 1 || w > BM || BM % w) return false;
    *rt = BM / w;
    if (*rt <= h) {
        if (h % *rt) return false;
        *ns = 1;
        *rs = *rt;
    } else {
        if (*rt % h) return false;
        *ns = *rt / h;
        *rs = h;
    }
    return *ns * (*rs + 2) * (w + 2) <= CtShape<WM>::NPMAX;
}

static bool tile_chunk_ok(int ck) { return ck == 16 || ck == 32 || (ck % 64 == 0 && ck <= 8192); }

bool tile_conv_fwd_ok(const ConvShape &sh, bool pool, int64_t sf, int alpha_inv)
{
    int rt, ns, rs;
    if (!tile_geom<2>(sh.h, sh.w, &rt, &ns, &rs) || !tile_chunk_ok(sh.c) || sh.co % 16) return false;
    if (pool && (rt % 2 || sh.h % 2 || sh.w % 2)) return false;
    return (int64_t)sh.n * sh.h * sh.w * sh.c < ((int64_t)1 << 31) &&
           (int64_t)sh.co * 9 * sh.c < ((int64_t)1 << 31) && scale_fast_ok(sf) && alpha_inv >= 2 &&
           128 * sf < ((int64_t)1 << 31);   // a saturated int32 sum still saturates z*
}

bool tile_conv_dx_ok(const ConvShape &sh)
{
    int rt, ns, rs;
    if (!tile_geom<2>(sh.h, sh.w, &rt, &ns, &rs) || !tile_chunk_ok(sh.co) || sh.c % 16) return false;
    return (int64_t)sh.n * sh.h * sh.w * sh.co < ((int64_t)1 << 31) &&
           (int64_t)sh.co * 9 * sh.c < ((int64_t)1 << 31);
}

// The 256-pixel tile where it fits (pooling needs an even number of rows per tile) and, chosen by
// shape, where it still gives at least one tile per two CUs (measured on the VGG-style layers:
// even at 8x8 images with 128 to 256 tiles it beats two 128-pixel workgroups per CU).
static bool use_wide_tile(int pref, int n, int h, int w, int no, bool pool)
{
    int rt, ns, rs;
    if (pref == 128 || !tile_geom<4>(h, w, &rt, &ns, &rs) || (pool && rt % 2)) return false;
    if (pref == 256) return true;
    const int64_t tiles = ((int64_t)n * h / rt) * ((no + CT_BN - 1) / CT_BN);
    return tiles >= 128;
}

// Compute units of the current device (cached per device).
static int device_cu_count()
{
    static int cached[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
    if (!cached[dev]) {
        int n = 0;
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 1)
            n = 256;
        cached[dev] = n;
    }
    return cached[dev];
}

// Launches of at least this many tiles per CU take the persistent 256-pixel kernel (forced
// persistent launches: about this many tiles per workgroup).
constexpr int CT_PERSIST_TILES_PER_CU = 4;

template <int MODE, int WM, bool PERSIST>
static void launch_tile_cc(hipStream_t s, const TileArgs &a, dim3 grid, bool adma)
{
    const dim3 block(CtShape<WM>::NT);
    switch (a.ck == 16 ? 16 : a.ck == 32 ? 32 : 64) {
    case 16: hipLaunchKernelGGL((k_conv_tile<MODE, 16, WM, PERSIST, false>), grid, block, 0, s, a); break;
    case 32: hipLaunchKernelGGL((k_conv_tile<MODE, 32, WM, PERSIST, false>), grid, block, 0, s, a); break;
    default:
        if (WM == 4 && adma)
            hipLaunchKernelGGL((k_conv_tile<MODE, 64, WM, PERSIST, WM == 4>), grid, block, 0, s, a);
        else
            hipLaunchKernelGGL((k_conv_tile<MODE, 64, WM, PERSIST, false>), grid, block, 0, s, a);
        break;
    }
}

// One workgroup per tile, or (256-pixel tiles, many of them) one persistent workgroup per CU:
// its two LDS stages take the whole LDS.
template <int MODE, int WM>
static void launch_tile(hipStream_t s, int persist, TileArgs a)
{
    tile_geom<WM>(a.h, a.w, &a.rt, &a.ns, &a.rs);
    a.d_w2 = make_div32((uint32_t)(a.w + 2));
    a.d_seg = make_div32((uint32_t)((a.rs + 2) * (a.w + 2)));
    a.d_w = make_div32((uint32_t)a.w);
    a.d_rw = make_div32((uint32_t)(a.rs * a.w));
    a.d_h = make_div32((uint32_t)a.h);
    a.ntiles = ((a.n * a.h + a.rt - 1) / a.rt) * ((a.no + CT_BN - 1) / CT_BN);
    a.ts = timer_slot(MODE == IG_FWD ? TIMED_CONV_FWD : TIMED_CONV_DX);
    // A straight into LDS: 256-pixel tiles, 64-channel chunks, rows of whole 16-pixel blocks
    a.apitch = (a.w + 2 + 15) / 16 * 16;
    const bool adma = WM == 4 && a.ck % 64 == 0 && a.w % 16 == 0 &&
                      a.ns * (a.rs + 2) * a.apitch <= CT_NPMAX_DIRECT;
    a.d_apitch = make_div32((uint32_t)a.apitch);
    a.d_aseg = make_div32((uint32_t)((a.rs + 2) * a.apitch));
    const int cus = device_cu_count();
    const bool big = a.ntiles >= CT_PERSIST_TILES_PER_CU * cus;
    TimedLaunch tl(MODE == IG_FWD ? TIMED_CONV_FWD : TIMED_CONV_DX, s);
    if (WM == 4 && (persist > 0 || (persist == 0 && big))) {
        int g = (a.ntiles + CT_PERSIST_TILES_PER_CU - 1) / CT_PERSIST_TILES_PER_CU;
        if (g > cus) g = cus;
        launch_tile_cc<MODE, WM, WM == 4>(s, a, dim3((unsigned)g), adma);
    } else {
        launch_tile_cc<MODE, WM, false>(s, a, dim3((unsigned)a.ntiles), adma);
    }
}

void launch_conv_fwd_tile(hipStream_t s, int tile, int persist, const ConvShape &sh, const int8_t *x, const int8_t *wf,
                          const uint32_t *wmax, int64_t sf, int alpha_inv, int round,
                          const Relu &rp, bool pool, int8_t *out, uint8_t *code, uint32_t *flags,
                          int8_t *xr, int64_t xs)
{
    TileArgs a{};
    a.n = sh.n; a.h = sh.h; a.w = sh.w;
    a.ck = sh.c; a.no = sh.co;
    a.a = x; a.aplane = 0; a.a_max = nullptr;
    a.b = wf; a.bplane = (int64_t)sh.co * 9 * sh.c; a.b_max = wmax;
    a.sf = make_scale_fast(sf, alpha_inv, rp.mu, round);
    a.pool = pool ? 1 : 0;
    a.out = out; a.code = code;
    a.xr = pool ? nullptr : xr; a.xs = xs;
    a.flags = flags;
    if (use_wide_tile(tile, sh.n, sh.h, sh.w, sh.co, pool)) launch_tile<IG_FWD, 4>(s, persist, a);
    else launch_tile<IG_FWD, 2>(s, persist, a);
}

void launch_conv_dx_tile(hipStream_t s, int tile, int persist, const ConvShape &sh, const int8_t *gl,
                         const uint32_t *gmax_in, const int8_t *wt, const uint32_t *wmax,
                         const uint8_t *prev_code, const Relu &rp, int32_t *gout, int64_t *out64,
                         uint32_t *gmax_out, uint32_t *flags, int16_t *gout16, const GOff *goff)
{
    TileArgs a{};
    a.n = sh.n; a.h = sh.h; a.w = sh.w;
    a.ck = sh.co; a.no = sh.c;
    a.a = gl; a.aplane = (int64_t)sh.n * sh.h * sh.w * sh.co; a.a_max = gmax_in;
    a.b = wt; a.bplane = (int64_t)sh.c * 9 * sh.co; a.b_max = wmax;
    a.rp = rp;
    a.prev_code = prev_code; a.gout = gout; a.out64 = out64; a.gmax = gmax_out;
    a.gout16 = gout ? gout16 : nullptr;
    if (goff && out64) {
        a.goff = 1;
        a.goff_count = goff->count;
        a.goff_bias = goff->bias;
    }
    a.flags = flags;
    if (use_wide_tile(tile, sh.n, sh.h, sh.w, sh.c, false)) launch_tile<IG_DX, 4>(s, persist, a);
    else launch_tile<IG_DX, 2>(s, persist, a);
}

// ---------------------------------------------------------------------------------------------
// Offset form of g: the bias table and the corrections of the listed entries.

// bias[cls][ci] = 128 sum_co sum_{(r,s) allowed by cls} W[co][r][s][ci]: a pixel on the top row
// (cls bit 0) has no g position above it to take tap r = 2 from (g at p - (r-1, s-1)), the
// bottom row (bit 1) none for r = 0, the first column (bit 2) none for s = 2, the last column
// (bit 3) none for s = 0. W is read from the input gradient's limb planes wt [4][ci][9 co] (all
// four limbs: W exactly). One wave per input channel c: its lanes take the dwords of row c of
// each plane, every (limb, tap) load issued before the sums, then the 36 tap sums are reduced
// across the wave by shuffles and lanes 0..15 form the 16 classes.
__global__ __launch_bounds__(256) void k_goff_bias(const int8_t *__restrict__ wt, int co, int ci,
                                                   const uint32_t *gmax, int64_t *__restrict__ bias)
{
    if (!goff_range(slot_read(gmax))) return;
    const int lane = threadIdx.x & 63;
    const int c = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (c >= ci) return;
    const int64_t row = 9 * (int64_t)co, plane = (int64_t)ci * row;
    const int nd = co / 4;                        // dwords per tap row
    int32_t acc[36];
#pragma unroll
    for (int k = 0; k < 36; k++) acc[k] = 0;
    for (int d0 = 0; d0 < nd; d0 += 64) {
        const int d = d0 + lane;
        const bool in = d < nd;
        uint32_t v[36];
#pragma unroll
        for (int k = 0; k < 36; k++)
            v[k] = in ? *(const uint32_t *)(wt + (k / 9) * plane + c * row + (k % 9) * co + 4 * d) : 0u;
#pragma unroll
        for (int k = 0; k < 36; k++)
            acc[k] += (int8_t)v[k] + (int8_t)(v[k] >> 8) + (int8_t)(v[k] >> 16) + (int8_t)(v[k] >> 24);
    }
#pragma unroll
    for (int k = 0; k < 36; k++)
        for (int off = 32; off > 0; off >>= 1) acc[k] += __shfl_xor(acc[k], off, 64);
    if (lane >= 16) return;
    const int cls = lane;
    int64_t b = 0;
#pragma unroll
    for (int t = 0; t < 9; t++) {
        const int r = t / 3, sc = t % 3;
        const bool ok = !(((cls & 1) && r == 2) || ((cls & 2) && r == 0) || ((cls & 4) && sc == 2) ||
                          ((cls & 8) && sc == 0));
#pragma unroll
        for (int l = 0; l < 4; l++)
            if (ok) b += (int64_t)acc[9 * l + t] * ((int64_t)1 << (8 * l));
    }
    bias[(int64_t)cls * ci + c] = (int64_t)GOFF_BIAS * b;
}

void launch_goff_bias(hipStream_t s, const int8_t *wt, int co, int ci, const uint32_t *gmax,
                      int64_t *bias)
{
    hipLaunchKernelGGL(k_goff_bias, dim3((unsigned)((ci + 3) / 4)), dim3(256), 0, s, wt, co, ci, gmax,
                       bias);
}

// Entry (g = 32768 at pixel p, channel o, its third limb 1): dx[p + (r-1, s-1)][ci] +=
// 65536 W[o][r][s][ci] for the taps whose pixel is inside the image, and (dw) dW[o][r][s][ci] +=
// 65536 x[p + (r-1, s-1)][ci] for the same taps (atomic adds: entries near each other reach the
// same outputs). Workgroups take entries e = blockIdx.x + gridDim.x k, threads the input
// channels; a thread's nine W (or x) values are loaded before its adds.
__global__ __launch_bounds__(256) void k_goff_fix(GOff go, const int32_t *__restrict__ w, int h,
                                                  int wd, int co, int ci, int64_t *__restrict__ dx,
                                                  const int8_t *__restrict__ x, int64_t *__restrict__ dw)
{
    const uint32_t cnt = *go.count;
    if (cnt == 0 || cnt > GOFF_CAP) return;
    const uint32_t hw = (uint32_t)h * (uint32_t)wd;
    for (uint32_t e = blockIdx.x; e < cnt; e += gridDim.x) {
        const uint32_t idx = go.list[e];
        const uint32_t pix = idx / (uint32_t)co, o = idx - pix * (uint32_t)co;
        const uint32_t img = pix / hw, rem = pix - img * hw;
        const int y = (int)(rem / (uint32_t)wd), xc = (int)(rem - (uint32_t)y * (uint32_t)wd);
        bool in[9];
        int64_t q[9];
#pragma unroll
        for (int t = 0; t < 9; t++) {
            const int qy = y + t / 3 - 1, qx = xc + t % 3 - 1;
            in[t] = qy >= 0 && qy < h && qx >= 0 && qx < wd;
            q[t] = ((int64_t)img * h + qy) * wd + qx;
        }
        for (int c = threadIdx.x; c < ci; c += 256) {
            if (dx) {
                int64_t v[9];
#pragma unroll
                for (int t = 0; t < 9; t++) v[t] = (int64_t)w[((int64_t)o * 9 + t) * ci + c] * 65536;
#pragma unroll
                for (int t = 0; t < 9; t++)
                    if (in[t]) atomicAdd((unsigned long long *)(dx + q[t] * ci + c), (unsigned long long)v[t]);
            }
            if (dw) {
                int64_t v[9];
#pragma unroll
                for (int t = 0; t < 9; t++) v[t] = in[t] ? (int64_t)x[q[t] * ci + c] * 65536 : 0;
#pragma unroll
                for (int t = 0; t < 9; t++)
                    if (v[t]) atomicAdd((unsigned long long *)(dw + ((int64_t)o * 9 + t) * ci + c), (unsigned long long)v[t]);
            }
        }
    }
}

void launch_goff_fix(hipStream_t s, const ConvShape &sh, const GOff &go, const int32_t *w,
                     int64_t *dx, const int8_t *x, int64_t *dw)
{
    hipLaunchKernelGGL(k_goff_fix, dim3(1024), dim3(256), 0, s, go, w, sh.h, sh.w, sh.co, sh.c, dx,
                       x, dw);
}

}  // namespace nitro
