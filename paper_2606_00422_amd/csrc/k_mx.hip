// MXFP8 encoding of row-major activations (the library's upr_mx_quantize
// call, and the fp8 projection variant's attention output when the
// reference attention kernel computed it).
//
// One wave per row.  A lane takes eight consecutive values per 512-value
// stretch of the row, so one 32-value block is four consecutive lanes: the
// block maximum takes two lane exchanges, each lane writes its eight codes
// (8 bytes) and the block's first lane the scale byte.
#include "mx.h"
#include "upr_internal.h"

namespace upr {

namespace {

constexpr int kRowsPerBlock = 4;

template <typename T> struct Load8;
template <> struct Load8<float> {
    __device__ __forceinline__ static void get(const float* p, float (&v)[8]) {
        const float4 a = *reinterpret_cast<const float4*>(p);
        const float4 b = *reinterpret_cast<const float4*>(p + 4);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    }
};
template <> struct Load8<f16> {
    __device__ __forceinline__ static void get(const f16* p, float (&v)[8]) {
        typedef __attribute__((ext_vector_type(8))) _Float16 h8;
        const h8 a = *reinterpret_cast<const h8*>(p);
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = (float)a[i];
    }
};
template <> struct Load8<bf16> {
    __device__ __forceinline__ static void get(const bf16* p, float (&v)[8]) {
        typedef __attribute__((ext_vector_type(8))) __bf16 b8;
        const b8 a = *reinterpret_cast<const b8*>(p);
#pragma unroll
        for (int i = 0; i < 8; ++i) v[i] = (float)a[i];
    }
};

template <typename T>
__global__ __launch_bounds__(256) void k_mx_quantize(const T* __restrict__ x, int64_t rows, int k,
                                                     uint8_t* __restrict__ codes,
                                                     uint8_t* __restrict__ scales) {
    const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    const T* xr = x + row * k;
    uint8_t* cr = codes + row * k;
    uint8_t* sr = scales + row * (k / kMxBlock);
    for (int c0 = 0; c0 < k; c0 += 512) {           // uniform trip count: every lane shuffles
        const int c = c0 + 8 * lane;
        const bool active = c < k;                  // k is a multiple of 32: whole blocks
        float v[8];
        if (active) {
            Load8<T>::get(xr + c, v);
        } else {
#pragma unroll
            for (int i = 0; i < 8; ++i) v[i] = 0.f;
        }
        float amax = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i) amax = fmaxf(amax, fabsf(v[i]));
        amax = fmaxf(amax, __shfl_xor(amax, 1, 64));
        amax = fmaxf(amax, __shfl_xor(amax, 2, 64));
        const int e = mx_block_exp(amax);
        const float inv = mx_inv_scale(e);
        if (active) {
            const uint32_t lo = mx_pack4(v[0] * inv, v[1] * inv, v[2] * inv, v[3] * inv);
            const uint32_t hi = mx_pack4(v[4] * inv, v[5] * inv, v[6] * inv, v[7] * inv);
            *reinterpret_cast<uint2*>(cr + c) = make_uint2(lo, hi);
            if ((lane & 3) == 0) sr[c / kMxBlock] = (uint8_t)(e + 127);
        }
    }
}

}  // namespace

template <typename T>
hipError_t launch_mx_quantize(const T* x, int64_t rows, int k, uint8_t* codes, uint8_t* scales,
                              hipStream_t s) {
    if (rows == 0) return hipSuccess;
    if (k <= 0 || k % kMxBlock != 0) return hipErrorInvalidValue;
    k_mx_quantize<T><<<(unsigned)((rows + kRowsPerBlock - 1) / kRowsPerBlock), 256, 0, s>>>(
        x, rows, k, codes, scales);
    return hipGetLastError();
}

template hipError_t launch_mx_quantize<float>(const float*, int64_t, int, uint8_t*, uint8_t*,
                                              hipStream_t);
template hipError_t launch_mx_quantize<f16>(const f16*, int64_t, int, uint8_t*, uint8_t*,
                                            hipStream_t);
template hipError_t launch_mx_quantize<bf16>(const bf16*, int64_t, int, uint8_t*, uint8_t*,
                                             hipStream_t);

}  // namespace upr
