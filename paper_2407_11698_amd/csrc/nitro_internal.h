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

__device__ inline int64_t relu_bwd(int64_t delta, uint8_t region, const Relu &rp)
{
    if (region == REG_PASS) return delta;
    if (region == REG_SLOPE) return idiv(delta, rp.alpha);
    return 0;
}

// Sticky status flags written by kernels (bit or).
enum : uint32_t { FLAG_OVERFLOW = 1u, FLAG_LABEL = 2u };

__device__ inline bool fits_i32(int64_t v) { return v >= INT32_MIN && v <= INT32_MAX; }

__device__ inline void raise_flag(uint32_t *flags, uint32_t f) { atomicOr(flags, f); }

// Running maximum in a device slot. The plain read first skips the atomic whenever the slot
// already holds a value at least as large (a stale read only costs an extra atomic).
__device__ inline void slot_max(uint32_t *slot, uint32_t m)
{
    if (m && m > __hip_atomic_load(slot, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT))
        atomicMax(slot, m);
}

__device__ inline uint32_t wave_max_u32(uint32_t v)
{
    for (int off = 32; off > 0; off >>= 1) {
        const uint32_t o = __shfl_xor(v, off, 64);
        v = o > v ? o : v;
    }
    return v;
}

// Workgroup-wide maximum folded into a device slot with one atomic per workgroup. Every thread
// of the workgroup must call it (it contains a barrier); at most 1024 threads.
__device__ inline void block_slot_max(uint32_t *slot, uint32_t m)
{
    __shared__ uint32_t red[16];
    m = wave_max_u32(m);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = m;
    __syncthreads();
    if (threadIdx.x == 0) {
        uint32_t r = 0;
        for (unsigned w = 0; w < (blockDim.x + 63) / 64; w++) r = red[w] > r ? red[w] : r;
        slot_max(slot, r);
    }
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
// Optional per-kernel timing: launchers bracket the launches of the timed kernel classes with
// begin/end; the API entry points install the calling context's timer for the duration of a
// call (thread-local, so concurrent contexts on other threads are not affected).
// classes: 0 k_igemm_conv forward, 1 k_igemm_conv input gradient, 2 k_conv_dw_planes
enum { TIMED_IGEMM_FWD = 0, TIMED_IGEMM_DX = 1, TIMED_DW_MFMA = 2, TIMED_CLASSES = 3 };
struct LaunchTimer {
    virtual void begin(int cls) = 0;
    virtual void end(int cls) = 0;
    virtual ~LaunchTimer() {}
};
extern thread_local LaunchTimer *g_timer;
inline void timer_begin(int cls) { if (g_timer) g_timer->begin(cls); }
inline void timer_end(int cls) { if (g_timer) g_timer->end(cls); }

// ------------------------------------------------------------------------------------------
// Kernel launchers (each enqueues on `s`; shapes are validated by the caller).
// ------------------------------------------------------------------------------------------
struct ConvShape {
    int n, h, w, c, co;    // input NHWC [n][h][w][c], output channels co
};

void launch_fill_i64(hipStream_t s, int64_t *p, int64_t count);
// out[i] = sum_{z < nz} part[z * count + i]  (split-K partial sums, fixed order)
void launch_sum_partials(hipStream_t s, const int64_t *part, int nz, int64_t count, int64_t *out);

// forward conv + Scaling + ReLU; POOL variant writes the pooled output and per pooled element
// code = argmax | region << 2; the plain variant writes the full-resolution output and region.
void launch_conv_fwd(hipStream_t s, const ConvShape &sh, const int8_t *x, const int32_t *w,
                     const Div &sf, const Relu &rp, bool pool, int8_t *out, uint8_t *code);
// forward linear + Scaling + ReLU: x [n][k], w [m][k] -> a [n][m], region codes [n][m].
void launch_linear_fwd_relu(hipStream_t s, int n, int k, int m, const int8_t *x, const int32_t *w,
                            const Div &sf, const Relu &rp, int8_t *out, uint8_t *code);
// learning / output layer: yhat = x w^T / sf, e = yhat - 32 onehot(labels).
void launch_linear_fwd_loss(hipStream_t s, int n, int k, int g, const int8_t *x, const int32_t *w,
                            const Div &sf, const int32_t *labels, int32_t *yhat, int32_t *e,
                            uint32_t *flags);
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
void launch_unpool_relu_bwd(hipStream_t s, int n, int h, int w, int c, bool pool,
                            const int32_t *delta, const uint8_t *code, const Relu &rp,
                            int32_t *g, uint32_t *gmax, uint32_t *flags);
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
    int32_t *epad, *et;            // e as [np][gp] and [gp][np] (zero padded)
    uint32_t *wmax, *emax, *gmax;  // max|W|, max|e|, max|g| slots (zeroed before the call)
};
bool mfma_learning_ok(int n, int64_t d, int G);
LearningScratch learning_scratch(int n, int64_t d, int G);
// yhat, e, dW of the learning layer on f = the block output [n][d], and the gradient g at the
// last forward layer's pre-activation (un-pool and NITRO-ReLU backward of delta = e W).
void launch_learning_mfma(hipStream_t s, int n, int64_t d, int G, const int8_t *f,
                          const int32_t *w, const Div &sf, const int32_t *labels,
                          const LearningBuffers &b, const uint8_t *code, const Relu &rp, int h,
                          int wdt, int c, bool pool, int32_t *g, int32_t *delta_copy,
                          int32_t *yhat, int32_t *e, int64_t *dw, uint32_t *flags);

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
// W int32 KRSC -> 4 balanced int8 limb planes [co][9 ci] (wf) and [ci][9 co] (wt, optional);
// max|W| -> *wmax (atomic max: the slot must be zeroed first).
void launch_pack_conv_weights(hipStream_t s, const int32_t *w, int co, int ci, int8_t *wf,
                              int8_t *wt, uint32_t *wmax);
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
void launch_conv_dw_planes(hipStream_t s, const ConvShape &sh, const int32_t *g,
                           const uint32_t *gmax, const int8_t *x, int8_t *gp, int8_t *xp,
                           int64_t *part, int64_t *dw, uint32_t *flags);
void launch_conv_dx_mfma(hipStream_t s, const ConvShape &sh, const int32_t *g, const uint32_t *gmax_in,
                         const int8_t *wt, const uint32_t *wmax, const uint8_t *prev_code,
                         const Relu &rp, int32_t *gout, int64_t *out64, uint32_t *gmax_out,
                         uint32_t *flags);
// conv weight gradient, int64 KRSC, overwritten.
void launch_conv_dw(hipStream_t s, const ConvShape &sh, const int32_t *g, const int8_t *x,
                    int64_t *dw);
// IntegerSGD (Alg. 1) in place.
void launch_sgd(hipStream_t s, int32_t *w, const int64_t *dw, int64_t count, const Div &gamma,
                const Div &eta, bool decay, uint32_t *flags);

}  // namespace nitro
