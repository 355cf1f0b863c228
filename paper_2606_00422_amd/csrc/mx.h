// MXFP8 encoding helpers (device code, header-only).
//
// The fp8 projection variant (paper Sec. 3, "FP8 quantization": E4M3 in the
// forward pass) stores each operand row as OCP microscaling blocks: 32
// consecutive values along the contraction axis share one scale 2^e (an E8M0
// byte e + 127) and each value is an E4M3 code.  e = floor(log2 max|v|) - 8,
// at least -127; a value is v / 2^e rounded to the nearest E4M3 value, ties
// to even, saturated to +-448.  gfx950's v_cvt_pk_fp8_f32 rounds to nearest
// even in the OCP E4M3 format but turns magnitudes above 464 into NaN, so
// values are clamped to +-448 first (values in (448, 464] round to 448
// either way).
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

namespace upr {

constexpr int kMxBlock = 32;

// Shared exponent of a block whose largest magnitude is amax (finite, >= 0):
// the biased fp32 exponent field gives floor(log2 amax) for normal amax;
// zero and subnormal maxima land at the -127 floor.
__device__ __forceinline__ int mx_block_exp(float amax) {
    const int eb = (int)((__float_as_uint(amax) >> 23) & 0xFFu);
    return eb - 135 > -127 ? eb - 135 : -127;
}

// 2^-e as a float; e <= 119 for any finite fp32 block maximum, so the
// result is a normal number and multiplying by it is exact.
__device__ __forceinline__ float mx_inv_scale(int e) {
    return __uint_as_float((uint32_t)(127 - e) << 23);
}

// Four values already divided by their block scale -> E4M3 codes, value k in
// byte k.
__device__ __forceinline__ uint32_t mx_pack4(float a, float b, float c, float d) {
    a = fminf(fmaxf(a, -448.0f), 448.0f);
    b = fminf(fmaxf(b, -448.0f), 448.0f);
    c = fminf(fmaxf(c, -448.0f), 448.0f);
    d = fminf(fmaxf(d, -448.0f), 448.0f);
    const int lo = __builtin_amdgcn_cvt_pk_fp8_f32(a, b, 0, false);
    return (uint32_t)__builtin_amdgcn_cvt_pk_fp8_f32(c, d, lo, true);
}

}  // namespace upr
