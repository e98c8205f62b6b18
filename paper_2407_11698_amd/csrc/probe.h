// int8 matrix-core rate probe (probe.hip): `grid` workgroups of 4 waves, `iters` MFMAs per
// chain; out holds grid * 256 int32. mfma_rate_ops: the int8 ops one such launch executes.
#pragma once

#include <hip/hip_runtime.h>
#include <cstdint>

namespace nitro {

void launch_mfma_rate(hipStream_t s, int grid, int iters, int32_t *out);
int64_t mfma_rate_ops(int grid, int iters);

}  // namespace nitro
