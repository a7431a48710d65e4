// quant.hpp -- the group quantizer of Sec. 2.2 as the append and the
// generation-phase kernels run it: one 32-dim group spread over a 16-lane row,
// two values per lane, bit-exact with the IEEE fp32 definition.
#pragma once

#include "common.hpp"

namespace dkv {

// Min / max over a 16-lane row with DPP (quad swaps, then half-row and row mirrors).
template <int CTRL>
__device__ __forceinline__ float dpp_f32(float x)
{
    return __int_as_float(__builtin_amdgcn_mov_dpp(__float_as_int(x), CTRL, 0xF, 0xF, false));
}
__device__ __forceinline__ float row16_min(float x)
{
    x = fminf(x, dpp_f32<0xB1>(x));   // quad_perm [1,0,3,2]
    x = fminf(x, dpp_f32<0x4E>(x));   // quad_perm [2,3,0,1]
    x = fminf(x, dpp_f32<0x141>(x));  // row_half_mirror
    return fminf(x, dpp_f32<0x140>(x));  // row_mirror
}
__device__ __forceinline__ float row16_max(float x)
{
    x = fmaxf(x, dpp_f32<0xB1>(x));
    x = fmaxf(x, dpp_f32<0x4E>(x));
    x = fmaxf(x, dpp_f32<0x141>(x));
    return fmaxf(x, dpp_f32<0x140>(x));
}

// clamp(rint(d / s), 0, lb) for two values, with d / s the IEEE fp32
// quotient.  The quotient through the hardware reciprocal (v_rcp_f32, within
// 1 ulp) and one rounded product is within 1.5 * 2^-23 relative, i.e. 2^-13
// absolute for |d/s| <= 2^9; larger quotients clamp the same way either way.
// It rounds to another integer than the IEEE quotient only if it lies within
// that distance of a half-integer, so lanes within 2^-12 of one (about 1 in
// 2^11) divide exactly, in a branch the compiler may not flatten.
__device__ __forceinline__ void codes_of(float d0, float d1, float s, float lb, uint32_t& c0, uint32_t& c1)
{
#pragma clang fp contract(off)
    const float rs = __builtin_amdgcn_rcpf(s);
    float q0 = d0 * rs, q1 = d1 * rs;
    const bool n0 = fabsf(q0 - rintf(q0)) > 0.5f - 0x1p-12f;
    const bool n1 = fabsf(q1 - rintf(q1)) > 0.5f - 0x1p-12f;
    if (n0 || n1) {
        asm volatile("" ::: "memory");
        if (n0) q0 = d0 / s;
        if (n1) q1 = d1 / s;
    }
    c0 = (uint32_t)fminf(fmaxf(rintf(q0), 0.0f), lb);
    c1 = (uint32_t)fminf(fmaxf(rintf(q1), 0.0f), lb);
}

// Quantize one 32-dim group spread over a 16-lane row (2 values per lane).
// Arithmetic is IEEE fp32 with no contraction, identical to the text of the
// quantizer: s = fp16((max-min)/L), z = fp16(min), code = clamp(rint((x-z)/s)).
__device__ __forceinline__ void quant_pair(uint32_t xbits, int lb, uint32_t& sz, uint32_t& c0,
                                           uint32_t& c1)
{
#pragma clang fp contract(off)
    float x0 = h2f(xbits & 0xffffu) + 0.0f;
    float x1 = h2f(xbits >> 16) + 0.0f;
    float mn = row16_min(fminf(x0, x1));
    float mx = row16_max(fmaxf(x0, x1));
    float s32 = (mx - mn) / (float)lb;
    uint32_t s16 = f2h_rne(s32);
    uint32_t z16 = f2h_rne(mn);
    float s = h2f(s16), z = h2f(z16);
    if (s16 == 0) {
        c0 = c1 = 0;
    } else {
        codes_of(x0 - z, x1 - z, s, (float)lb, c0, c1);
    }
    sz = s16 | (z16 << 16);
}

}  // namespace dkv
