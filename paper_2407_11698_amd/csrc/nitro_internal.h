// Internal declarations of the NITRO-D HIP library (gfx950). Not part of the C ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "nitro.h"

namespace nitro {

// ------------------------------------------------------------------------------------------
// Division by an invariant positive divisor.
//
// Every division in the method has a divisor fixed for the whole launch (SF, alpha_inv,
// gamma_inv, eta). The kernels multiply by a precomputed reciprocal instead of dividing:
// the round-up method of Granlund and Montgomery, "Division by invariant integers using
// multiplication" (PLDI 1994, section 4), for unsigned 64-bit numerators below 2^63:
//   l = ceil(log2 d), m = floor(2^64 (2^l - d) / d) + 1,  q = (mulhi(m, n) + n) >> l.
// (t = mulhi(m, n) <= n < 2^63, so t + n cannot wrap.) Signed numerators are reduced to that
// case: floor(n/d) = n >= 0 ? q(n) : ~q(~n)  and  trunc(n/d) = n >= 0 ? q(n) : -q(-n).
// ------------------------------------------------------------------------------------------
struct Div {
    int64_t d;        // the divisor, >= 1
    uint64_t m;       // magic multiplier
    int32_t l;        // shift
    int32_t trunc;    // 0: round toward minus infinity, 1: toward zero
};

inline Div make_div(int64_t d, int round)
{
    Div r;
    r.d = d;
    int l = 0;
    while (l < 63 && ((int64_t)1 << l) < d) l++;
    unsigned __int128 num = ((unsigned __int128)(((uint64_t)1 << l) - (uint64_t)d)) << 64;
    r.m = (uint64_t)(num / (uint64_t)d) + 1;
    r.l = l;
    r.trunc = round == NITRO_ROUND_TRUNC;
    return r;
}

__host__ __device__ inline uint64_t mulhi_u64(uint64_t a, uint64_t b)
{
#if defined(__HIP_DEVICE_COMPILE__)
    return __umul64hi(a, b);
#else
    return (uint64_t)(((unsigned __int128)a * b) >> 64);
#endif
}

__host__ __device__ inline uint64_t udiv_magic(uint64_t n, const Div &v)
{
    uint64_t t = mulhi_u64(v.m, n);
    return (t + n) >> v.l;
}

__host__ __device__ inline int64_t idiv(int64_t n, const Div &v)
{
    if (n >= 0) return (int64_t)udiv_magic((uint64_t)n, v);
    if (v.trunc) return -(int64_t)udiv_magic((uint64_t)(-n), v);
    return ~(int64_t)udiv_magic((uint64_t)(~n), v);
}

// ------------------------------------------------------------------------------------------
// NITRO-ReLU parameters and region codes.
// Region of a rescaled pre-activation z*: 0 = identity segment (0 <= z* <= 127),
// 1 = leaky segment (-127 <= z* < 0), 2 = saturated (z* > 127 or z* < -127).
// ------------------------------------------------------------------------------------------
struct Relu {
    Div alpha;        // alpha_inv
    int32_t mu;
    uint32_t a32_m;   // 32-bit reciprocal of alpha_inv (Div32 fields), for |values| < 2^32
    int32_t a32_l;
};

enum : uint8_t { REG_PASS = 0, REG_SLOPE = 1, REG_ZERO = 2 };

__device__ inline int32_t relu_fwd(int64_t zs, const Relu &rp, uint8_t &region)
{
    if (zs < 0) {
        region = zs >= -127 ? REG_SLOPE : REG_ZERO;
        int64_t c = zs < -127 ? -127 : zs;
        return (int32_t)(idiv(c, rp.alpha) - rp.mu);
    }
    region = zs <= 127 ? REG_PASS : REG_ZERO;
    int64_t c = zs > 127 ? 127 : zs;
    return (int32_t)(c - rp.mu);
}


// The same method for 32-bit numerators (n < 2^32, 1 <= d < 2^32): m fits 32 bits and the sum
// t + n is formed in 64 bits. Used where a value is known to be small.
struct Div32 {
    uint32_t m;
    int32_t l;
};

inline Div32 make_div32(uint32_t d)
{
    Div32 r;
    int l = 0;
    while (l < 32 && ((uint64_t)1 << l) < d) l++;
    r.m = (uint32_t)((((uint64_t)1 << 32) * (((uint64_t)1 << l) - d)) / d + 1);
    r.l = l;
    return r;
}

__host__ __device__ inline uint32_t udiv32(uint32_t n, const Div32 &v)
{
#if defined(__HIP_DEVICE_COMPILE__)
    const uint32_t t = __umulhi(v.m, n);
#else
    const uint32_t t = (uint32_t)(((uint64_t)v.m * n) >> 32);
#endif
    return (uint32_t)(((uint64_t)t + n) >> v.l);
}

// NITRO-Scaling followed by NITRO-ReLU, with 32-bit division. The quotient z / SF only matters
// exactly while it lies in [-128, 128]; beyond, both rounding modes give a saturated region and
// the clamped value. So z >= 128 SF and z <= -128 SF are decided by comparison, and every other
// z has |z| < 128 SF <= 2^32 (required of SF by make_scale_relu's caller).
struct ScaleRelu {
    Div32 sf, alpha;
    int64_t lim;          // 128 * SF
    int32_t mu;
    int32_t trunc;
};

inline ScaleRelu make_scale_relu(int64_t sf, int64_t alpha_inv, int32_t mu, int round)
{
    ScaleRelu q;
    q.sf = make_div32((uint32_t)sf);
    q.alpha = make_div32((uint32_t)alpha_inv);
    q.lim = 128 * sf;
    q.mu = mu;
    q.trunc = round == NITRO_ROUND_TRUNC;
    return q;
}

inline bool scale_relu_ok(int64_t sf, int64_t alpha_inv)
{
    return sf >= 1 && 128 * sf <= ((int64_t)1 << 32) && alpha_inv >= 1 && alpha_inv < ((int64_t)1 << 31);
}

// floor or trunc of -n / d for 0 < n < 2^32
__host__ __device__ inline int32_t neg_div32(uint32_t n, const Div32 &d, int trunc)
{
    return trunc ? -(int32_t)udiv32(n, d) : -1 - (int32_t)udiv32(n - 1, d);
}

__host__ __device__ inline int32_t scale_relu(int64_t z, const ScaleRelu &q, uint8_t &region)
{
    int32_t zs;
    if (z >= q.lim) zs = 128;
    else if (z <= -q.lim) zs = -128;
    else if (z >= 0) zs = (int32_t)udiv32((uint32_t)z, q.sf);
    else zs = neg_div32((uint32_t)(-z), q.sf, q.trunc);
    if (zs < 0) {
        region = zs >= -127 ? REG_SLOPE : REG_ZERO;
        const int32_t c = zs < -127 ? -127 : zs;
        return neg_div32((uint32_t)(-c), q.alpha, q.trunc) - q.mu;
    }
    region = zs <= 127 ? REG_PASS : REG_ZERO;
    return (zs > 127 ? 127 : zs) - q.mu;
}

inline Relu make_relu_params(int64_t alpha_inv, int32_t mu, int round)
{
    Relu r;
    r.alpha = make_div(alpha_inv, round);
    r.mu = mu;
    const Div32 a = make_div32((uint32_t)alpha_inv);
    r.a32_m = a.m;
    r.a32_l = a.l;
    return r;
}

__device__ inline int64_t relu_bwd(int64_t delta, uint8_t region, const Relu &rp)
{
    if (region == REG_PASS) return delta;
    if (region == REG_SLOPE) {
        const Div32 a{rp.a32_m, rp.a32_l};
        const int64_t lim = (int64_t)1 << 32;
        if (delta >= 0 && delta < lim) return udiv32((uint32_t)delta, a);
        if (delta < 0 && delta > -lim) return neg_div32((uint32_t)(-delta), a, rp.alpha.trunc);
        return idiv(delta, rp.alpha);
    }
    return 0;
}

// Branch-free NITRO-Scaling + NITRO-ReLU of an int32 pre-activation (the workgroup's sums fit
// int32). Both divisions use the round-up method without the 33-bit sum:
// q = (t + ((n - t) >> 1)) >> (l - 1), t = mulhi(m, n), valid for divisors >= 2.
struct ScaleRelu32 {
    uint32_t sf_m, a_m;
    int32_t sf_l, a_l;
    int32_t mu;
    int32_t trunc;
};

inline ScaleRelu32 make_scale_relu32(int64_t sf, int64_t alpha_inv, int32_t mu, int round)
{
    const Div32 a = make_div32((uint32_t)sf), b = make_div32((uint32_t)alpha_inv);
    return ScaleRelu32{a.m, b.m, a.l, b.l, mu, round == NITRO_ROUND_TRUNC};
}

inline bool scale_relu32_ok(int64_t sf, int64_t alpha_inv)
{
    return sf >= 2 && sf < ((int64_t)1 << 31) && alpha_inv >= 2 && alpha_inv < ((int64_t)1 << 31);
}

__host__ __device__ inline uint32_t udiv32_nf(uint32_t n, uint32_t m, int l)
{
#if defined(__HIP_DEVICE_COMPILE__)
    const uint32_t t = __umulhi(m, n);
#else
    const uint32_t t = (uint32_t)(((uint64_t)m * n) >> 32);
#endif
    return (t + ((n - t) >> 1)) >> (l - 1);
}

__host__ __device__ inline int32_t scale_relu32(int32_t z, const ScaleRelu32 &q, uint8_t &region)
{
    const int32_t sg = z >> 31;                                   // 0 or -1
    // floor: n = ~z for z < 0 and zs = ~q; trunc: n = -z and zs = -q
    const uint32_t n = q.trunc ? (uint32_t)((z ^ sg) - sg) : (uint32_t)(z ^ sg);
    const uint32_t d = udiv32_nf(n, q.sf_m, q.sf_l);
    const int32_t zs = q.trunc ? (((int32_t)d ^ sg) - sg) : ((int32_t)d ^ sg);
    const int32_t c = zs < -127 ? -127 : (zs > 127 ? 127 : zs);
    region = c != zs ? REG_ZERO : (c < 0 ? REG_SLOPE : REG_PASS);
    const uint32_t n2 = q.trunc ? (uint32_t)(-c) : (uint32_t)(~c);  // used only when c < 0
    const int32_t d2 = (int32_t)udiv32_nf(n2, q.a_m, q.a_l);
    const int32_t neg = q.trunc ? -d2 : ~d2;
    return (c < 0 ? neg : c) - q.mu;
}

// NITRO-Scaling of an int32 sum for the tile epilogue, clamped to [-128, 128]. SF = 2^e D with D
// odd: floor(z / 2^e) is an arithmetic shift (truncation: the shift after adding 2^e - 1 to a
// negative z), and clamping that to [-128 D, 128 D] keeps its quotient by D inside [-128, 128]
// and saturates it to -128 or 128 outside. The clamped quotient is exact with one multiply-high
// by m = ceil(2^32 / D): for n <= 128 D, n (m D - 2^32) < 128 D^2 < 2^32. The NITRO-ReLU of the
// result (and its region) is a lookup in a 257-entry table.
struct ScaleFast {
    int32_t e;
    uint32_t m;        // ceil(2^32 / D)
    int32_t lo, hi;    // -128 D, 128 D
    int32_t alpha, mu, trunc;
};

// SF a power of two is taken as 2^(e-1) * 2, so that D >= 2 and m is a 32-bit number.
inline bool scale_fast_ok(int64_t sf)
{
    if (sf < 2 || sf >= ((int64_t)1 << 31)) return false;
    int64_t d = sf;
    while (!(d & 1)) d >>= 1;
    return 128 * d * d < ((int64_t)1 << 32);
}

inline ScaleFast make_scale_fast(int64_t sf, int32_t alpha_inv, int32_t mu, int round)
{
    ScaleFast q{};
    int64_t d = sf;
    while (!(d & 1)) {
        d >>= 1;
        q.e++;
    }
    if (d == 1) {
        d = 2;
        q.e--;
    }
    q.m = (uint32_t)((((uint64_t)1 << 32) + (uint64_t)d - 1) / (uint64_t)d);
    q.lo = (int32_t)(-128 * d);
    q.hi = (int32_t)(128 * d);
    q.alpha = alpha_inv;
    q.mu = mu;
    q.trunc = round == NITRO_ROUND_TRUNC;
    return q;
}

template <bool TRUNC>
__host__ __device__ inline int32_t scale_fast(int32_t z, const ScaleFast &q)
{
    int32_t s = TRUNC ? (z + ((z >> 31) & ((1 << q.e) - 1))) >> q.e : z >> q.e;
    s = max(min(s, q.hi), q.lo);
    const int32_t sg = s >> 31;
    const uint32_t n = TRUNC ? (uint32_t)((s ^ sg) - sg) : (uint32_t)(s ^ sg);
#if defined(__HIP_DEVICE_COMPILE__)
    const uint32_t dq = __umulhi(n, q.m);
#else
    const uint32_t dq = (uint32_t)(((uint64_t)n * q.m) >> 32);
#endif
    return TRUNC ? (((int32_t)dq ^ sg) - sg) : ((int32_t)dq ^ sg);
}

// Table entry for a scaled value zs in [-128, 128]: the NITRO-ReLU output byte | region << 8.
__host__ __device__ inline uint16_t relu_table_entry(int32_t zs, const ScaleFast &q)
{
    const int32_t c = zs < -127 ? -127 : (zs > 127 ? 127 : zs);
    const uint32_t reg = c != zs ? REG_ZERO : (c < 0 ? REG_SLOPE : REG_PASS);
    int32_t a = c;
    if (c < 0) {
        a = c / q.alpha;
        if (!q.trunc && a * q.alpha != c) a -= 1;
    }
    a -= q.mu;
    return (uint16_t)((uint32_t)(uint8_t)(int8_t)a | (reg << 8));
}

// NITRO-ReLU backward of an int32 gradient, branch-free (same result as relu_bwd).
template <bool TRUNC>
__device__ inline int32_t relu_bwd32(int32_t d, uint32_t region, const Relu &rp)
{
    const int32_t sg = d >> 31;
    const uint32_t n = TRUNC ? (uint32_t)((d ^ sg) - sg) : (uint32_t)(d ^ sg);
    const uint32_t qd = udiv32_nf(n, rp.a32_m, rp.a32_l);
    const int32_t s = TRUNC ? (((int32_t)qd ^ sg) - sg) : ((int32_t)qd ^ sg);
    return region == REG_PASS ? d : (region == REG_SLOPE ? s : 0);
}

// Sticky status flags written by kernels (bit or).
enum : uint32_t { FLAG_OVERFLOW = 1u, FLAG_LABEL = 2u };

__device__ inline bool fits_i32(int64_t v) { return v >= INT32_MIN && v <= INT32_MAX; }

__device__ inline void raise_flag(uint32_t *flags, uint32_t f) { atomicOr(flags, f); }

// Running maximum in a device slot: one atomic max, its result unused (a workgroup's last act:
// reading the slot first to skip the atomic costs the workgroup a memory round trip).
__device__ inline void slot_max(uint32_t *slot, uint32_t m)
{
    if (m) atomicMax(slot, m);
}

__device__ inline uint32_t wave_max_u32(uint32_t v)
{
    for (int off = 32; off > 0; off >>= 1) {
        const uint32_t o = __shfl_xor(v, off, 64);
        v = o > v ? o : v;
    }
    return v;
}

// A max slot is SLOT_WORDS words: a workgroup folds its maximum into word (workgroup index mod
// SLOT_WORDS), so that concurrent workgroups seldom meet on one address (same-address device
// atomics serialise across the XCDs), and a reader takes the maximum over the words.
constexpr int SLOT_WORDS = 64;

// Workgroup-wide maximum folded into a max slot with one atomic per workgroup. Every thread of
// the workgroup must call it (it contains a barrier); at most 1024 threads.
__device__ inline void block_slot_max(uint32_t *slot, uint32_t m)
{
    __shared__ uint32_t red[16];
    m = wave_max_u32(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = 0;
        for (unsigned w = 0; w < (blockDim.x + 63) / 64; w++) r = red[w] > r ? red[w] : r;
        const unsigned b = blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
        slot_max(slot + b % SLOT_WORDS, r);
    }
}

// The value of a max slot. Every lane of the calling wave must be active.
__device__ inline uint32_t slot_read(const uint32_t *slot)
{
    static_assert(SLOT_WORDS == 64, "one word per lane");
    return wave_max_u32(slot[threadIdx.x & 63]);
}

__device__ inline uint32_t abs_u32(int32_t v) { return v < 0 ? (uint32_t)(-(int64_t)v) : (uint32_t)v; }

// |v| for a value meant for int32 (anything outside int32 maps to the largest code, which no
// limb count accepts)
__device__ inline uint32_t abs_i64_sat(int64_t v)
{
    return (v >= INT32_MIN && v <= INT32_MAX) ? abs_u32((int32_t)v) : 0xFFFFFFFFu;
}

// Grid size for a grid-stride elementwise kernel: enough workgroups to fill the GPU, few
// enough that per-workgroup reductions stay cheap.
inline unsigned grid_stride_blocks(int64_t n, int per = 256, unsigned cap = 2048)
{
    const int64_t b = (n + per - 1) / per;
    return (unsigned)(b < 1 ? 1 : (b > cap ? cap : b));
}

// ------------------------------------------------------------------------------------------
// Optional per-kernel timing, measured on the device so that it also works inside a replayed
// graph. A timed launch gets a slot of TS_WORDS uint64 words in a context-owned buffer: words
// [0, TS_SPREAD) take the minimum start time of its workgroups and [TS_SPREAD, 2 TS_SPREAD) the
// maximum end time (the constant-rate wall clock), each workgroup folding into word
// (workgroup id mod TS_SPREAD). Slots are assigned when launches are enqueued (also while a graph
// is being captured); the API entry points install the calling context's timer for the duration
// of a call (thread-local, so concurrent contexts on other threads are not affected).
// classes: 0 k_conv_tile forward, 1 k_conv_tile input gradient, 2 k_conv_dw_planes
enum { TIMED_CONV_FWD = 0, TIMED_CONV_DX = 1, TIMED_DW = 2, TIMED_CLASSES = 3 };
constexpr int TS_SPREAD = 16, TS_WORDS = 2 * TS_SPREAD;
struct LaunchTimer {
    virtual uint64_t *slot(int cls) = 0;
    // event timing (eager launches only): events recorded on the launch's stream around it
    virtual void ev_begin(int cls, hipStream_t s) {}
    virtual void ev_end(int cls, hipStream_t s) {}
    virtual ~LaunchTimer() {}
};
extern thread_local LaunchTimer *g_timer;
inline uint64_t *timer_slot(int cls) { return g_timer ? g_timer->slot(cls) : nullptr; }
// Brackets one timed kernel launch with the installed timer's events (when it times by events).
struct TimedLaunch {
    int cls;
    hipStream_t s;
    TimedLaunch(int c, hipStream_t st) : cls(c), s(st)
    {
        if (g_timer) g_timer->ev_begin(cls, s);
    }
    ~TimedLaunch()
    {
        if (g_timer) g_timer->ev_end(cls, s);
    }
};

__device__ inline unsigned ts_block_id()
{
    return blockIdx.x + gridDim.x * (blockIdx.y + gridDim.y * blockIdx.z);
}
// first statement of a timed kernel
__device__ inline void ts_start(uint64_t *ts)
{
    if (ts && threadIdx.x == 0)
        atomicMin((unsigned long long *)&ts[ts_block_id() % TS_SPREAD], (unsigned long long)wall_clock64());
}
// last statement of a timed kernel; every thread of the workgroup must reach it
__device__ inline void ts_end(uint64_t *ts)
{
    if (ts) {
        __syncthreads();
        if (threadIdx.x == 0)
            atomicMax((unsigned long long *)&ts[TS_SPREAD + ts_block_id() % TS_SPREAD],
                      (unsigned long long)wall_clock64());
    }
}
// reset n slots: starts to the largest value, ends to 0
void launch_ts_reset(hipStream_t s, uint64_t *buf, int64_t nslots);

// ------------------------------------------------------------------------------------------
// Kernel launchers (each enqueues on `s`; shapes are validated by the caller).
// ------------------------------------------------------------------------------------------
struct ConvShape {
    int n, h, w, c, co;    // input NHWC [n][h][w][c], output channels co
};

void launch_fill_i64(hipStream_t s, int64_t *p, int64_t count);
// out[i] = sum_{z < nz} part[z * count + i]  (split-K partial sums, fixed order)
void launch_sum_partials(hipStream_t s, const int64_t *part, int nz, int64_t count, int64_t *out);
// The same for a conv weight gradient [co][9][ci] whose g may be in the offset form: when
// max|g| (gmax) is in the offset range, each output adds the offset's term from xq.
void launch_sum_partials_goff(hipStream_t s, const int64_t *part, int nz, int64_t count,
                              int64_t *out, const int32_t *xq, int ci, const uint32_t *gmax);

// forward conv + Scaling + ReLU; POOL variant writes the pooled output and per pooled element
// code = argmax | region << 2; the plain variant writes the full-resolution output and region.
void launch_conv_fwd(hipStream_t s, const ConvShape &sh, const int8_t *x, const int32_t *w,
                     const Div &sf, const Relu &rp, bool pool, int8_t *out, uint8_t *code);
// forward linear + Scaling + ReLU: x [n][k], w [m][k] -> a [n][m], region codes [n][m].
void launch_linear_fwd_relu(hipStream_t s, int n, int k, int m, const int8_t *x, const int32_t *w,
                            const Div &sf, const Relu &rp, int8_t *out, uint8_t *code);
// learning / output layer: yhat = x w^T / sf, e = yhat - 32 onehot(labels) (labels NULL: yhat
// only).
void launch_linear_fwd_loss(hipStream_t s, int n, int k, int g, const int8_t *x, const int32_t *w,
                            const Div &sf, const int32_t *labels, int32_t *yhat, int32_t *e,
                            uint32_t *flags);
// pred[r] = first argmax of yhat's row r ([n][g])
void launch_argmax_rows(hipStream_t s, int n, int g, const int32_t *yhat, int32_t *pred);
// dx[n][k] = sum_m e[n][m] w[m][k]; optional ReLU' with `code` -> int32 out (overflow flagged),
// or the raw sum into out64 (int64) when out64 is not null.
void launch_linear_dx(hipStream_t s, int n, int k, int m, const int32_t *e, const int32_t *w,
                      const uint8_t *code, const Relu &rp, int32_t *out, int64_t *out64,
                      uint32_t *flags);
// dw[m][k] = sum_n e[n][m] x[n][k], int64, overwritten.
void launch_linear_dw(hipStream_t s, int n, int k, int m, const int32_t *e, const int8_t *x,
                      int64_t *dw);
// gradient at the block output -> gradient at the last layer's pre-activation; max|g| -> *gmax
// (when not null).
// g16 (not pooled): g in the escaped 16-bit form below (g then receives only the escapes).
void launch_unpool_relu_bwd(hipStream_t s, int n, int h, int w, int c, bool pool,
                            const int32_t *delta, const uint8_t *code, const Relu &rp,
                            int32_t *g, uint32_t *gmax, uint32_t *flags, int16_t *g16 = nullptr);
// conv input gradient; with `code` applies ReLU' of the previous layer and writes int32 `out`
// (overflow flagged, max|out| -> *gmax when not null); with out64 writes the raw int64 sum.
void launch_conv_dx(hipStream_t s, const ConvShape &sh, const int32_t *g, const int32_t *w,
                    const uint8_t *code, const Relu &rp, int32_t *out, int64_t *out64,
                    uint32_t *gmax, uint32_t *flags);

// ---- learning layer on int8 MFMA (linear_mfma.hip)
struct LearningScratch {
    int gp, np, splits;            // G and n rounded up to 16; split-K count of the forward GEMM
    int64_t kchunk;
    int64_t wf_bytes, wt_bytes, part_bytes, epad_bytes, et_bytes, ft_bytes;
};
struct LearningBuffers {
    int8_t *wf, *wt, *ft;          // weight limb planes [4][G][d], [4][d][gp]; f^T [d][np]
    int64_t *part;                 // forward split-K partial sums
    int8_t *epad, *et;             // e's 4 limb planes as [np][gp] and [gp][np] (zero padded)
    uint32_t *wmax, *emax, *gmax;  // max|W|, max|e|, max|g| slots (zeroed before the call)
};
bool mfma_learning_ok(int n, int64_t d, int G, int c);   // c: block output channels
// IntLinear forward layers (section 3.2.1) on the same GEMM: z = x W^T in split-K partials, then
// NITRO-Scaling and NITRO-ReLU; their weight gradient dW = g^T x (int64). K (c_in, and the batch
// for dW) is zero-padded to a multiple of 16.
struct LinearScratch {
    int cip, np, splits, kchunk;   // c_in and n rounded up to 16; forward split-K
    int64_t wf_bytes;              // the weight's limb planes [4][co][cip]
    int64_t xpad_bytes;            // x with its rows padded to cip (0 when c_in % 16 == 0)
    int64_t part_bytes;            // forward partials [splits][n][co] int64
    int64_t gt_bytes, xt_bytes;    // weight gradient: g^T limb planes [4][co][np], x^T [ci][np]
};
bool linear_mfma_ok(int n, int ci, int co);
LinearScratch linear_scratch(int n, int ci, int co);
// out (int8 [n][co]) and code from x (int8 [n][ci]); wf / wmax from launch_pack_linear_weights.
void launch_linear_fwd_mfma(hipStream_t s, int n, int ci, int co, const int8_t *x, int8_t *xpad,
                            const int8_t *wf, const uint32_t *wmax, const Div &sf, const Relu &rp,
                            int8_t *out, uint8_t *code, int64_t *part, uint32_t *flags);
// dw (int64 [co][ci], overwritten) = g^T x for g int32 [n][co]; max|g| folded into gmax (a slot
// that is zero, or already holds max|g|, before the call).
void launch_linear_dw_mfma(hipStream_t s, int n, int ci, int co, const int32_t *g, uint32_t *gmax,
                           const int8_t *x, int8_t *gt, int8_t *xt, int64_t *dw, uint32_t *flags);
LearningScratch learning_scratch(int n, int64_t d, int G);
// yhat, e, dW of the learning layer on f = the block output [n][d], and the gradient g at the
// last forward layer's pre-activation (un-pool and NITRO-ReLU backward of delta = e W).
// g_pooled (pooled block): g is left at the pooled positions, [n][h/2][w/2][c], the value of each
// window's argmax (the others are zero); launch_conv_dw_planes un-pools it with the codes.
void launch_learning_mfma(hipStream_t s, int n, int64_t d, int G, const int8_t *f,
                          const int32_t *w, const Div &sf, const int32_t *labels,
                          const LearningBuffers &b, const uint8_t *code, const Relu &rp, int h,
                          int wdt, int c, bool pool, int32_t *g, int32_t *delta_copy,
                          int32_t *yhat, int32_t *e, int64_t *dw, uint32_t *flags, bool prepacked = false,
                          bool g_pooled = false);

// ---- learning layers' max-pooling (lrpool.hip)
struct LrPool {
    int n, h, w, c;       // the block output [n][h][w][c] (after the block's own pool)
    int kh, kw;           // window; the pooled input of the learning layer is [n][h/kh][w/kw][c]
};
// Window of the learning layers' pooling for a block output c x h x w and d_lr (0: none):
// kh, kw doubled in turn (kh first) while c (h/kh)(w/kw) > d_lr and a side can be halved.
void lr_pool_window(int c, int h, int w, int d_lr, int *kh, int *kw);
void launch_lr_pool(hipStream_t s, const LrPool &p, const int8_t *a, int8_t *f, uint8_t *fcode);
// g (the last layer's pre-activation gradient, full resolution) from delta_f (the gradient at the
// pooled learning-layer input), fcode, and the last layer's codes (pooled: argmax | region << 2)
void launch_lr_unpool_relu_bwd(hipStream_t s, const LrPool &p, bool pool, const int32_t *delta_f,
                               const uint8_t *fcode, const uint8_t *code, const Relu &rp,
                               int32_t *g, uint32_t *gmax, uint32_t *flags);

// ---- integer pre-processing of a uint8 dataset (preprocess.hip)
constexpr int PRE_MAX_GROUPS = 1024;
int preprocess_groups(int64_t count);
size_t preprocess_workspace(int64_t count);          // bytes: partial histograms and the table
// out = clamp((x - mu) 51 / omega) with mu, omega of the whole dataset; stats = {mu, omega,
// saturated count} (device, int64); out may be x itself
void launch_preprocess(hipStream_t s, const uint8_t *x, int64_t count, int round, int8_t *out,
                       int64_t *stats, void *workspace);

// ---- dropout of a block output (dropout.hip)
struct Dropout {
    uint64_t threshold;   // floor(p 2^32); 0: no dropout
    uint64_t seed, step;
    int32_t block;
    int32_t pooled;       // codes are argmax | region << 2
};
void launch_dropout(hipStream_t s, int8_t *a, uint8_t *code, int64_t count, const Dropout &d);

// ---- few input channels (conv_smallc.hip)
bool smallc_fwd_ok(const ConvShape &sh);
bool smallc_dw_ok(const ConvShape &sh);
void launch_conv_fwd_smallc(hipStream_t s, const ConvShape &sh, const int8_t *x, const int32_t *w,
                            const Div &sf, const Relu &rp, bool pool, int8_t *out, uint8_t *code);
int64_t smallc_dw_partial_count(const ConvShape &sh);
void launch_conv_dw_smallc(hipStream_t s, const ConvShape &sh, const int32_t *g, const int8_t *x,
                           int64_t *part, int64_t *dw);

// ---- int8 MFMA implicit-GEMM path (conv_mfma.hip)
bool mfma_conv_fwd_ok(const ConvShape &sh, bool pool);
bool mfma_conv_dx_ok(const ConvShape &sh);
// W int32 KRSC -> 4 balanced int8 limb planes [co][9 cpad] (wf; channels ci..cpad-1 zero) and
// [ci][9 co] (wt, optional); max|W| -> the max slot wmax (zeroed first).
void launch_pack_conv_weights(hipStream_t s, const int32_t *w, int co, int ci, int cpad,
                              int8_t *wf, int8_t *wt, uint32_t *wmax);
// Linear weight W int32 [co][ci] -> 4 limb planes [co][cpad] (columns ci..cpad-1 zero), max|W|.
void launch_pack_linear_weights(hipStream_t s, const int32_t *w, int co, int ci, int cpad,
                                int8_t *wf, uint32_t *wmax);
// x int8 [P][c] (c < 16) -> [P][16], channels c..15 zero.
void launch_pad_channels16(hipStream_t s, const int8_t *x, int P, int c, int8_t *xpad);
void launch_conv_fwd_mfma(hipStream_t s, const ConvShape &sh, const int8_t *x, const int8_t *wf,
                          const uint32_t *wmax, const Div &sf, const Relu &rp, bool pool,
                          int8_t *out, uint8_t *code, uint32_t *flags);
bool mfma_conv_dw_ok(const ConvShape &sh);
bool mfma_conv_dw_smallc_ok(const ConvShape &sh);   // few input channels (9 C_in <= 64)
// Row length of the pixel-contiguous gradient limb planes used by the weight gradient; the
// scratch `gt` holds 4 * sh.co * dw_plane_stride(sh) bytes.
int64_t dw_plane_stride(const ConvShape &sh);
// int64 words of split-K partial sums the weight gradient needs as scratch
int64_t dw_partial_count(const ConvShape &sh);
// dW (int64) from g int32 NHWC (max|g| in *gmax) and x int8 NHWC; `gt`, `part` are scratch.
void launch_conv_dw_mfma(hipStream_t s, const ConvShape &sh, const int32_t *g,
                         const uint32_t *gmax, const int8_t *x, int8_t *gt, int64_t *part,
                         int64_t *dw, uint32_t *flags);
// ---- weight gradient over zero-padded pixel planes (conv_dw.hip): C_in and C_out multiples of
// 16, W <= 62. Scratch: gp (dwp_gplane_bytes), xp (dwp_xplane_bytes), part (dwp_partial_count
// int64 words; none when the pixel range is not split).
bool dwp_ok(const ConvShape &sh);
int64_t dwp_gplane_bytes(const ConvShape &sh);
int64_t dwp_xplane_bytes(const ConvShape &sh);
int64_t dwp_partial_count(const ConvShape &sh);
// gn (optional): also write g's NHWC limb planes [4][P][co] (the input-gradient tile kernel's A).
// x rows [C16 / 16][xs][16] of the weight-gradient kernel: a zero halo of DWP_HMAX positions,
// then padded position k = (n (H+1) + h)(W+1) + w at row DWP_HMAX + k. With x_rows_ready the
// caller has written every real pixel's row (the forward epilogue of the previous layer) and
// only the pad rows are zeroed here.
constexpr int DWP_HMAX = 64;
int64_t dwp_rows_stride(const ConvShape &sh);   // xs
// pool_code (a pooled layer's codes, [n][h/2][w/2][co]): g is given at the pooled positions only
// (launch_learning_mfma with g_pooled) and each window's argmax takes the value
// g16: g in the escaped 16-bit form (g then holds the escaped values only).
// goff: gn (if any) may take the offset form below, and with goff->xq (dwp_goff_ok) the weight
// gradient too.
struct GOff;
void launch_conv_dw_planes(hipStream_t s, const ConvShape &sh, const int32_t *g,
                           const uint32_t *gmax, const int8_t *x, int8_t *gp, int8_t *xp,
                           int8_t *gn, int64_t *part, int64_t *dw, uint32_t *flags,
                           bool x_rows_ready = false, const uint8_t *pool_code = nullptr,
                           const int16_t *g16 = nullptr, const GOff *goff = nullptr);

// g one value past two limbs. Two balanced int8 limbs hold the 65536 integers [-32896, 32639];
// a gradient with max|g| = 32768 (the 16-bit error signal of the single-layer case passed
// through NITRO-ReLU) spans 65537 and would take a third limb pass in the input-gradient GEMM.
// Offset form, for the int64 input gradient of a block's first layer: when
// 32639 < max|g| <= 32768, g's NHWC limb planes hold the three balanced limbs of g - 128 at
// every pixel, whose third limb is 1 where g = 32768 and 0 elsewhere. The GEMM runs limbs 0
// and 1 only, and the input gradient gets back
//   + 128 sum_{co, (r,s) with p - (r-1, s-1) inside the image} W[co][r][s][ci]
// (a function of ci and of the pixel's border class, from a table) and, for each g = 32768
// (listed by the preparation, at most GOFF_CAP of them), 65536 W[co][r][s][ci] at the pixels
// p + (r-1, s-1) inside the image (atomic adds). With more than GOFF_CAP such entries the GEMM
// runs all three limbs instead. Exact either way.
constexpr int32_t GOFF_BIAS = 128;
constexpr uint32_t GOFF_CAP = 16384;
__host__ __device__ inline bool goff_range(uint32_t m) { return m > 32639u && m <= 32768u; }
struct GOff {
    uint32_t *count;       // entries with g = 32768 (a word that is zero before the preparation)
    uint32_t *list;        // [GOFF_CAP] their indices p co + c in g
    int64_t *bias;         // [16][ci]: the offset's term for border class
                           // (h == 0) | (h == H-1) << 1 | (w == 0) << 2 | (w == W-1) << 3
    int32_t *xq;           // (weight gradient in the form too) [9][ci], zero before the
                           // preparation: x summed over every pixel, over the rows h = 0 and
                           // h = H-1, the columns w = 0 and w = W-1, and the four corners
};
// The weight gradient takes the offset form too where the layer's shape allows it (C_in a
// multiple of 64, split-K): its planes hold g - 128, the split-K sums add
// 128 sum_{p inside} x[p + (r-1, s-1)][ci] (from xq) and the fix adds 65536 x rows per entry.
bool dwp_goff_ok(const ConvShape &sh);
// The bias table from W's input-gradient limb planes wt [4][ci][9 co] (the workgroups return
// at once unless max|g| is in the offset range).
void launch_goff_bias(hipStream_t s, const int8_t *wt, int co, int ci, const uint32_t *gmax,
                      int64_t *bias);
// The listed entries' 65536 W terms added into dx int64 NHWC [n][h][w][ci] and (dw not null)
// their 65536 x terms into dW int64 KRSC (nothing unless 0 < count <= GOFF_CAP).
void launch_goff_fix(hipStream_t s, const ConvShape &sh, const GOff &go, const int32_t *w,
                     int64_t *dx, const int8_t *x = nullptr, int64_t *dw = nullptr);

// ---- implicit-GEMM conv with the input tile staged once (conv_tile.hip)
bool tile_conv_fwd_ok(const ConvShape &sh, bool pool, int64_t sf, int alpha_inv);
bool tile_conv_dx_ok(const ConvShape &sh);
// tile: 0 by shape, 128 or 256 pixels forced where that tile fits (nitro_set_conv_tile);
// persist: persistent 256-pixel workgroups by size (0), always (1), never (-1)
// (nitro_set_conv_persistent); xr (not pooled): also write the output into the next layer's
// weight-gradient x rows
void launch_conv_fwd_tile(hipStream_t s, int tile, int persist, const ConvShape &sh, const int8_t *x, const int8_t *wf,
                          const uint32_t *wmax, int64_t sf, int alpha_inv, int round,
                          const Relu &rp, bool pool, int8_t *out, uint8_t *code, uint32_t *flags,
                          int8_t *xr = nullptr, int64_t xs = 0);
// gl: g's NHWC limb planes [LA][P][co] (max|g| in gmax_in); otherwise as launch_conv_dx_mfma.
// gout16 (with gout): the result in the escaped 16-bit form below instead of int32 (gout then
// receives only the escaped values).
// goff (out64 only): gl may hold g in the offset form (as launch_conv_dw_planes wrote it).
void launch_conv_dx_tile(hipStream_t s, int tile, int persist, const ConvShape &sh, const int8_t *gl,
                         const uint32_t *gmax_in, const int8_t *wt, const uint32_t *wmax,
                         const uint8_t *prev_code, const Relu &rp, int32_t *gout, int64_t *out64,
                         uint32_t *gmax_out, uint32_t *flags, int16_t *gout16 = nullptr,
                         const GOff *goff = nullptr);

// A gradient stored in 16 bits with an escape: g16[i] = g[i] where |g[i]| <= G16_MAX, else
// G16_ESC, and then the int32 array beside it holds g[i] at the same index (written, and read,
// only there).
constexpr int32_t G16_MAX = 32767;
constexpr int16_t G16_ESC = -32768;
void launch_conv_dx_mfma(hipStream_t s, const ConvShape &sh, const int32_t *g, const uint32_t *gmax_in,
                         const int8_t *wt, const uint32_t *wmax, const uint8_t *prev_code,
                         const Relu &rp, int32_t *gout, int64_t *out64, uint32_t *gmax_out,
                         uint32_t *flags);
// conv weight gradient, int64 KRSC, overwritten.
void launch_conv_dw(hipStream_t s, const ConvShape &sh, const int32_t *g, const int8_t *x,
                    int64_t *dw);
// ---- preparation and bookkeeping (prep.hip)
// Conv weight W [co][9][ci] -> wf [4][co][9 ci] and wt [4][ci][9 co] in one pass (co, ci % 16 == 0).
bool pack_conv_tiled_ok(int co, int ci);
// int32 values -> 4 balanced int8 limb planes, plain p and transposed t (rows padded to Rpad),
// in 64 x 64 tiles, batched over z; max |value| into wmax
struct PackArgs {
    const int32_t *x;
    int64_t xs, zx;
    int R, C, Rpad;
    int8_t *p;
    int64_t ps, pplane, zp;
    int8_t *t;
    int64_t ts, tplane, zt;
    uint32_t *wmax;
};
PackArgs pack_conv_args(const int32_t *w, int co, int ci, int8_t *wf, int8_t *wt, uint32_t *wmax);
PackArgs pack_matrix_args(const int32_t *w, int R, int C, int Rpad, int8_t *p, int8_t *t,
                          uint32_t *wmax);
constexpr int PACK_BATCH = 16;
// Conv weights packed element-wise (C_in not a multiple of 16, or zero-padded to 16): the planes
// of k_pack_conv_weights and k_pack_conv_weights_t as entries of a batched launch.
constexpr int PACK_CONV = 4;
struct ConvPackArgs {
    const int32_t *w;
    uint32_t co, ci, cpad;
    uint32_t taps;                 // 9 (conv KRSC) or 1 (linear [co][ci])
    int8_t *wf, *wt;
    uint32_t *wmax;
    int nf, nt;                    // workgroups of the plain and of the swapped planes
};
struct PackBatch {
    PackArgs t[PACK_BATCH];
    int gx[PACK_BATCH], gy[PACK_BATCH];
    int first[PACK_BATCH + 1];
    int n;
    ConvPackArgs c[PACK_CONV];     // dealt the workgroups after first[n], in order
    int nc;
};
// packs gathered on the host and enqueued as one launch (flushed when full)
struct PackList {
    PackBatch b{};
    void add(hipStream_t s, const PackArgs &a, int batches);   // batches: 9 for a conv weight
    // a conv weight packed element-wise (launch_pack_conv_weights' planes and max)
    void add_conv(hipStream_t s, const int32_t *w, int co, int ci, int cpad, int8_t *wf, int8_t *wt,
                  uint32_t *wmax, int taps = 9);
    void flush(hipStream_t s);
};
void launch_pack_conv_tiled(hipStream_t s, const int32_t *w, int co, int ci, int8_t *wf,
                            int8_t *wt, uint32_t *wmax);
// Matrix X [R][C] (C % 16 == 0, Rpad % 16 == 0) -> limb planes P [4][R][C] and T [4][C][Rpad].
void launch_pack_matrix(hipStream_t s, const int32_t *w, int R, int C, int Rpad, int8_t *p,
                        int8_t *t, uint32_t *wmax);
constexpr int SGD_MAX = 24;
constexpr int SGD_ITEMS = 2;
struct SgdTensor {
    int32_t *w;
    const int64_t *dw;
    int64_t count;
    Div gamma, eta;
    int32_t decay;
};
struct SgdBatch {
    SgdTensor t[SGD_MAX];
    int64_t first[SGD_MAX];       // first workgroup of each tensor (set by the launcher)
    int n;
    uint32_t *flags;
};
void launch_sgd_batch(hipStream_t s, SgdBatch b);
struct SlotList {
    uint32_t *p[NITRO_MAX_BLOCKS];
    int words;
};
// pad (optional): in the same launch, a network input zero-padded to 16 channels
// (launch_pad_channels16).
struct Pad16Args {
    const int8_t *x;
    int P, c;
    int8_t *xpad;
};
void launch_zero_slots(hipStream_t s, const SlotList &l, int nblocks, const Pad16Args *pad = nullptr);

// IntegerSGD (Alg. 1) in place.
void launch_sgd(hipStream_t s, int32_t *w, const int64_t *dw, int64_t count, const Div &gamma,
                const Div &eta, bool decay, uint32_t *flags);

}  // namespace nitro
