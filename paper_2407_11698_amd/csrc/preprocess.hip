// Integer-only pre-processing of an unsigned 8-bit dataset (Appendix A):
//   mu = sum x / N,  omega = sum |x - mu| / N,  xhat = (x - mu) 51 / omega.
// A byte has only 256 values, so both sums follow from the dataset's histogram and xhat is a
// 256-entry table: three passes, of which two stream the data.
//   1. k_pre_hist: per-workgroup histograms (16 LDS copies each, so that the lanes of an atomic
//      rarely collide), 16 bytes per thread and load, written as partial histograms (no global
//      atomics), at most one workgroup per compute unit;
//   2. k_pre_stats (one workgroup of 1024 threads): the histogram, mu, omega and the table; the
//      divisions by N and omega are done once, here;
//   3. k_pre_map: out = table[x], 16 bytes per thread and load/store, the table in LDS.
// HBM traffic: N bytes read twice, N written.
#include "nitro_internal.h"

namespace nitro {

namespace {

// [0, head) and [head + 16 nvec, count) are handled byte by byte; the middle as 16-byte vectors
struct Span {
    int64_t head, nvec;
};

__host__ __device__ inline Span span_of(const void *p, int64_t count)
{
    const int64_t mis = (int64_t)((uintptr_t)p & 15);
    int64_t head = mis ? 16 - mis : 0;
    if (head > count) head = count;
    return Span{head, (count - head) / 16};
}

}  // namespace

// 16 copies of the histogram per workgroup, lane l counting into copy l mod 16, each copy padded
// to 257 words: the lanes of one LDS atomic instruction then meet on one address only when four
// of them hold the same byte, and copies of one bin fall on different banks.
constexpr int PRE_COPIES = 16, PRE_STRIDE = 257;

__global__ __launch_bounds__(256) void k_pre_hist(const uint8_t *__restrict__ x, int64_t count,
                                                  uint32_t *__restrict__ part)
{
    __shared__ uint32_t h[PRE_COPIES * PRE_STRIDE];
    for (int i = threadIdx.x; i < PRE_COPIES * PRE_STRIDE; i += 256) h[i] = 0;
    __syncthreads();
    uint32_t *mine = h + (threadIdx.x % PRE_COPIES) * PRE_STRIDE;
    const Span sp = span_of(x, count);
    const uint4 *xv = (const uint4 *)(x + sp.head);
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x; v < sp.nvec; v += stride) {
        const uint4 q = xv[v];
        const uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int k = 0; k < 4; k++) {
#pragma unroll
            for (int b = 0; b < 4; b++) atomicAdd(&mine[(w[k] >> (8 * b)) & 0xffu], 1u);
        }
    }
    const int64_t tail0 = sp.head + 16 * sp.nvec;
    const int64_t rest = sp.head + (count - tail0);
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < rest; i += stride) {
        const int64_t e = i < sp.head ? i : tail0 + (i - sp.head);
        atomicAdd(&mine[x[e]], 1u);
    }
    __syncthreads();
    const int v = threadIdx.x;
    uint32_t t = 0;
#pragma unroll
    for (int c = 0; c < PRE_COPIES; c++) t += h[c * PRE_STRIDE + v];
    part[(int64_t)blockIdx.x * 256 + v] = t;
}

// Sum of a uint64 over the workgroup's 1024 threads (every thread gets it).
__device__ inline uint64_t block_sum_u64(uint64_t v, uint64_t *red)
{
    for (int off = 32; off > 0; off >>= 1) v += __shfl_xor(v, off, 64);
    __syncthreads();
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    uint64_t t = 0;
#pragma unroll
    for (int w = 0; w < 16; w++) t += red[w];
    return t;
}

__device__ inline int64_t div_round(int64_t n, int64_t d, int trunc)
{
    const int64_t q = n / d;                      // rounds toward zero
    return (!trunc && (n % d) != 0 && (n < 0)) ? q - 1 : q;
}

// 1024 threads: thread t adds bin t mod 256 of the partial histograms of groups t / 256, + 4, ...
// (independent accumulators, so the loads overlap); then threads 0..255 own one bin each.
__global__ __launch_bounds__(1024) void k_pre_stats(const uint32_t *__restrict__ part, int groups,
                                                    int64_t count, int trunc,
                                                    int64_t *__restrict__ stats,
                                                    int8_t *__restrict__ table)
{
    __shared__ uint64_t red[16];
    __shared__ uint64_t slice[4][256];
    const int v = threadIdx.x & 255, sl = threadIdx.x >> 8;
    uint64_t acc[4] = {0, 0, 0, 0};
    int g = sl;
    for (; g + 12 < groups; g += 16) {
#pragma unroll
        for (int k = 0; k < 4; k++) acc[k] += part[(int64_t)(g + 4 * k) * 256 + v];
    }
    for (; g < groups; g += 4) acc[0] += part[(int64_t)g * 256 + v];
    slice[sl][v] = acc[0] + acc[1] + acc[2] + acc[3];
    __syncthreads();
    const bool own = threadIdx.x < 256;
    const uint64_t hv = own ? slice[0][v] + slice[1][v] + slice[2][v] + slice[3][v] : 0;
    const uint64_t s1 = block_sum_u64(hv * (uint64_t)v, red);
    const int64_t mu = div_round((int64_t)s1, count, trunc);
    const int64_t dev = v > mu ? v - mu : mu - v;
    const uint64_t s2 = block_sum_u64(hv * (uint64_t)dev, red);
    int64_t omega = div_round((int64_t)s2, count, trunc);
    if (omega < 1) omega = 1;
    const int64_t q = div_round(((int64_t)v - mu) * 51, omega, trunc);
    const bool sat = q < -127 || q > 127;
    if (own) table[v] = (int8_t)(q < -127 ? -127 : (q > 127 ? 127 : q));
    const uint64_t ns = block_sum_u64(sat ? hv : 0, red);
    if (threadIdx.x == 0) {
        stats[0] = mu;
        stats[1] = omega;
        stats[2] = (int64_t)ns;
    }
}

__global__ __launch_bounds__(256) void k_pre_map(const uint8_t *x, int64_t count,
                                                 const int8_t *__restrict__ table, int8_t *out)
{
    __shared__ uint8_t t[256];
    t[threadIdx.x] = (uint8_t)table[threadIdx.x];
    __syncthreads();
    // x and out may be the same buffer: every element is read before it is written, by the same
    // thread; the 16-byte vectors are aligned for both only when the two alignments agree
    const bool vec = (((uintptr_t)x ^ (uintptr_t)out) & 15) == 0;
    const Span sp = vec ? span_of(x, count) : Span{count, 0};
    const uint4 *xv = (const uint4 *)(x + sp.head);
    uint4 *ov = (uint4 *)(out + sp.head);
    const int64_t stride = (int64_t)gridDim.x * 256;
    for (int64_t v = (int64_t)blockIdx.x * 256 + threadIdx.x; v < sp.nvec; v += stride) {
        const uint4 q = xv[v];
        uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
        for (int k = 0; k < 4; k++) {
            uint32_t r = 0;
#pragma unroll
            for (int b = 0; b < 4; b++) r |= (uint32_t)t[(w[k] >> (8 * b)) & 0xffu] << (8 * b);
            w[k] = r;
        }
        ov[v] = make_uint4(w[0], w[1], w[2], w[3]);
    }
    const int64_t tail0 = sp.head + 16 * sp.nvec;
    const int64_t rest = sp.head + (count - tail0);
    for (int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x; i < rest; i += stride) {
        const int64_t e = i < sp.head ? i : tail0 + (i - sp.head);
        out[e] = (int8_t)t[x[e]];
    }
}

// About 4 vectors per thread for small datasets, at most 256 workgroups (one per compute unit)
// for large ones; beyond 2^38 bytes, enough groups that no group counts 2^30 bytes or more (its
// 32-bit bins cannot overflow).
int preprocess_groups(int64_t count)
{
    int64_t g = (count + 16 * 256 * 4 - 1) / (16 * 256 * 4);
    if (g > 256) g = 256;
    const int64_t need = (count + ((int64_t)1 << 30) - 1) >> 30;
    if (g < need) g = need;
    return (int)(g < 1 ? 1 : (g > PRE_MAX_GROUPS ? PRE_MAX_GROUPS : g));
}

size_t preprocess_workspace(int64_t count)
{
    return (size_t)preprocess_groups(count) * 256 * 4 + 256;
}

void launch_preprocess(hipStream_t s, const uint8_t *x, int64_t count, int round, int8_t *out,
                       int64_t *stats, void *workspace)
{
    const int groups = preprocess_groups(count);
    uint32_t *part = (uint32_t *)workspace;
    int8_t *table = (int8_t *)((uint8_t *)workspace + (size_t)groups * 256 * 4);
    hipLaunchKernelGGL(k_pre_hist, dim3(groups), dim3(256), 0, s, x, count, part);
    hipLaunchKernelGGL(k_pre_stats, dim3(1), dim3(1024), 0, s, part, groups, count,
                       round == NITRO_ROUND_TRUNC ? 1 : 0, stats, table);
    int64_t mg = (count + 16 * 256 * 4 - 1) / (16 * 256 * 4);      // about 4 vectors per thread
    mg = mg < 1 ? 1 : (mg > 2048 ? 2048 : mg);
    hipLaunchKernelGGL(k_pre_map, dim3((unsigned)mg), dim3(256), 0, s, x, count, table, out);
}

}  // namespace nitro
