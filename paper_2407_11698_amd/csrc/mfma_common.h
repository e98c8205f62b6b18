// Helpers shared by the int8 MFMA kernels (gfx950): balanced int8 limbs, limb counts, byte
// transposes.
#pragma once

#include "nitro_internal.h"

namespace nitro {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v2i __attribute__((ext_vector_type(2)));

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

// ---------------------------------------------------------------------------------------------
// Bodies shared by the per-call kernels and the training iteration's batched launches.

// Conv weight W int32 KRSC [co][3][3][ci] -> 4 limb planes of [co][9 cpad] (channels ci..cpad-1
// zero), elements i = bid 256 + tid, stepping nb 256; max|W| into the slot wmax.
__device__ inline void pack_conv_weights_part(const int32_t *__restrict__ w, uint32_t total, int ci,
                                              int cpad, int8_t *__restrict__ wf, uint32_t *wmax,
                                              uint32_t bid, uint32_t nb)
{
    uint32_t m = 0;
    if ((ci & 3) == 0 && (cpad & 3) == 0) {
        // four elements of one row per step: 16-byte loads, one dword per limb plane
        for (uint32_t i = (bid * 256 + threadIdx.x) * 4; i < total; i += nb * 256 * 4) {
            const uint32_t c = i % (uint32_t)cpad, row = i / (uint32_t)cpad;
            v4i v = v4i{0, 0, 0, 0};
            if ((int)c < ci) v = *(const v4i *)(w + (int64_t)row * ci + c);
#pragma unroll
            for (int e = 0; e < 4; e++) {
                const uint32_t a = abs_u32(v[e]);
                m = a > m ? a : m;
            }
#pragma unroll
            for (int l = 0; l < 4; l++)
                *(uint32_t *)(wf + (int64_t)l * total + i) = limb4(v[0], v[1], v[2], v[3], l);
        }
    } else {
        for (uint32_t i = bid * 256 + threadIdx.x; i < total; i += nb * 256) {
            int32_t v;
            if (cpad == ci) {
                v = w[i];
            } else {
                const uint32_t c = i % (uint32_t)cpad, row = i / (uint32_t)cpad;
                v = (int)c < ci ? w[row * ci + c] : 0;
            }
            const uint32_t a = abs_u32(v);
            m = a > m ? a : m;
#pragma unroll
            for (int l = 0; l < 4; l++) wf[(int64_t)l * total + i] = limb1(v, l);
        }
    }
    block_slot_max(wmax, m);
}

// The same weight's channel-swapped planes [ci][9 co] (input gradient), element
// (c 9 + rs) co + o = bid 256 + tid.
__device__ inline void pack_conv_weights_t_part(const int32_t *__restrict__ w, uint32_t co,
                                                uint32_t ci, int8_t *__restrict__ wt, uint32_t bid)
{
    const uint32_t total = co * 9 * ci;
    const uint32_t ti = bid * 256 + threadIdx.x;
    if (ti >= total) return;
    const uint32_t o = ti % co, crs = ti / co;
    const uint32_t rs = crs % 9, c = crs / 9;
    const int32_t v = w[(o * 9 + rs) * ci + c];
#pragma unroll
    for (int l = 0; l < 4; l++) wt[(int64_t)l * total + ti] = limb1(v, l);
}

// x int8 [P][c] -> [P][16] with zero channels c..15 (c < 16): pixel p = bid 256 + tid.
__device__ inline void pad_channels16_part(const int8_t *__restrict__ x, int P, int c,
                                           int8_t *__restrict__ xpad, int bid)
{
    const int p = bid * 256 + threadIdx.x;
    if (p >= P) return;
    v4i v = v4i{0, 0, 0, 0};
    for (int e = 0; e < c; e++)
        v[e >> 2] |= (int)((uint32_t)(uint8_t)x[(int64_t)p * c + e] << (8 * (e & 3)));
    *(v4i *)(xpad + (int64_t)p * 16) = v;
}

}  // namespace nitro
