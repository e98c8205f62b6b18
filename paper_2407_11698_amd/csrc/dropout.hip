// Dropout of a block's output in a training iteration (rates p_c, p_l of Tab. 6), with masks
// drawn from the counter-based generator Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11):
// element i takes 64-bit word i mod 4 of Philox4x64-10 at counter (i div 4 + 1, block, step, 0)
// and key (seed, 0), and is dropped when the word's upper 32 bits are below the threshold
// floor(p 2^32). A dropped element becomes 0 and its NITRO-ReLU region code becomes "saturated",
// so every backward path (which applies NITRO-ReLU' from the codes) passes it no gradient.
#include "nitro_internal.h"

namespace nitro {

// Philox4x64 with 10 rounds: each round forms the 128-bit products of counter words 0 and 2 with
// two fixed constants and recombines their halves with words 1 and 3 and the key; the key is
// bumped by two Weyl constants between rounds.
__device__ inline void philox4x64_10(uint64_t c[4], uint64_t k0, uint64_t k1)
{
    const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
    const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
    for (int r = 0; r < 10; r++) {
        const uint64_t hi0 = __umul64hi(M0, c[0]), lo0 = M0 * c[0];
        const uint64_t hi1 = __umul64hi(M1, c[2]), lo1 = M1 * c[2];
        const uint64_t n0 = hi1 ^ c[1] ^ k0, n2 = hi0 ^ c[3] ^ k1;
        c[0] = n0;
        c[1] = lo1;
        c[2] = n2;
        c[3] = lo0;
        k0 += W0;
        k1 += W1;
    }
}

// one thread per group of four elements (one generator call)
__global__ __launch_bounds__(256) void k_dropout(int8_t *__restrict__ a, uint8_t *__restrict__ code,
                                                 int64_t count, Dropout d)
{
    const int64_t j = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (4 * j >= count) return;
    uint64_t c[4] = {(uint64_t)j + 1, (uint64_t)d.block, d.step, 0};
    philox4x64_10(c, d.seed, 0);
#pragma unroll
    for (int e = 0; e < 4; e++) {
        const int64_t i = 4 * j + e;
        if (i < count && (c[e] >> 32) < d.threshold) {
            a[i] = 0;
            code[i] = d.pooled ? (uint8_t)((code[i] & 3u) | (REG_ZERO << 2)) : (uint8_t)REG_ZERO;
        }
    }
}

void launch_dropout(hipStream_t s, int8_t *a, uint8_t *code, int64_t count, const Dropout &d)
{
    const int64_t groups = (count + 3) / 4;
    if (groups > 0 && d.threshold > 0)
        hipLaunchKernelGGL(k_dropout, dim3((unsigned)((groups + 255) / 256)), dim3(256), 0, s, a, code,
                           count, d);
}

}  // namespace nitro
