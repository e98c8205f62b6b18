// Rate probe of the int8 matrix cores: the dense rate that the conv kernels' figures are priced
// against, measured rather than taken from a data sheet. Every wave runs MR_CHAINS independent
// accumulator chains of v_mfma_i32_16x16x64_i8 on operands held in registers; the only memory
// access is one 4-byte store per thread at the end, which keeps the chains live.
#include "mfma_common.h"
#include "probe.h"

namespace nitro {

constexpr int MR_CHAINS = 8;

__global__ __launch_bounds__(256) void k_mfma_rate(int iters, int32_t *out)
{
    const int tid = threadIdx.x;
    const v4i a = v4i{tid, 3 * tid + 1, tid ^ 0x55, tid + 7};
    const v4i b = v4i{5 * tid, tid + 11, tid ^ 0x33, 7 * tid + 2};
    v4i acc[MR_CHAINS];
#pragma unroll
    for (int c = 0; c < MR_CHAINS; c++) acc[c] = v4i{c, tid, 0, 0};
    for (int it = 0; it < iters; it++)
#pragma unroll
        for (int c = 0; c < MR_CHAINS; c++)
            acc[c] = __builtin_amdgcn_mfma_i32_16x16x64_i8(a, b, acc[c], 0, 0, 0);
    int32_t s = 0;
#pragma unroll
    for (int c = 0; c < MR_CHAINS; c++) s += acc[c][0] + acc[c][1] + acc[c][2] + acc[c][3];
    out[(int64_t)blockIdx.x * 256 + tid] = s;
}

int64_t mfma_rate_ops(int grid, int iters) { return (int64_t)grid * 4 * MR_CHAINS * iters * (2 * 16 * 16 * 64); }

void launch_mfma_rate(hipStream_t s, int grid, int iters, int32_t *out)
{
    hipLaunchKernelGGL(k_mfma_rate, dim3((unsigned)grid), dim3(256), 0, s, iters, out);
}

}  // namespace nitro
