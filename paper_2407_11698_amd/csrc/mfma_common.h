// Helpers shared by the int8 MFMA kernels (gfx950): balanced int8 limbs, limb counts, byte
// transposes.
#pragma once

#include "nitro_internal.h"

namespace nitro {

typedef int v4i __attribute__((ext_vector_type(4)));

__host__ __device__ inline int limbs_for(uint32_t m)
{
    return m <= 127u ? 1 : m <= 32639u ? 2 : m <= 8355711u ? 3 : m <= 2139062143u ? 4 : 5;
}

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

}  // namespace nitro
