// Row-wise kernels: residual-stream initialisation, LayerNorm, score head.
//
// One 64-lane wave owns one row of d features (d a multiple of 64, at most
// 1024).  For d a multiple of 256 a lane holds float4 groups j*256 + 4*lane
// (16-byte loads, 8-byte half stores); otherwise features lane + 64 i.
// Statistics are two-pass in fp32 over the registers: mean, then the mean
// of squared deviations (population variance), as LayerNorm defines them.
#include "mx.h"
#include "upr_internal.h"

namespace upr {

namespace {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}

template <typename T> __device__ __forceinline__ float to_f(T v) { return (float)v; }

// Four consecutive token values (8 bytes for bf16, 16 for fp32) as floats.
template <typename T>
__device__ __forceinline__ void load4(const T* __restrict__ p, float* v) {
    typedef __attribute__((ext_vector_type(4))) T t4;
    const t4 x = *reinterpret_cast<const t4*>(p);
#pragma unroll
    for (int t = 0; t < 4; ++t) v[t] = (float)x[t];
}

constexpr int kRowsPerBlock = 4;     // 4 waves, one row each
constexpr int kMaxPerLane = 16;      // d <= 1024

// Per-lane feature index of register slot i.
template <bool VEC>
__device__ __forceinline__ int feat(int lane, int i) {
    return VEC ? (i >> 2) * 256 + 4 * lane + (i & 3) : lane + 64 * i;
}

template <bool VEC>
__device__ __forceinline__ void load_row(const float* __restrict__ x, int d, int lane,
                                         float (&v)[kMaxPerLane]) {
    const int per = d >> 6;
    if (VEC) {
#pragma unroll
        for (int j = 0; j < kMaxPerLane / 4; ++j)
            if (4 * j < per) {
                const float4 q = *reinterpret_cast<const float4*>(x + j * 256 + 4 * lane);
                v[4 * j] = q.x; v[4 * j + 1] = q.y; v[4 * j + 2] = q.z; v[4 * j + 3] = q.w;
            }
    } else {
#pragma unroll
        for (int i = 0; i < kMaxPerLane; ++i)
            if (i < per) v[i] = x[lane + 64 * i];
    }
}

// (mean, 1/sqrt(var + eps)) of the row held in v.
__device__ __forceinline__ void row_stats(const float (&v)[kMaxPerLane], int d, float eps,
                                          float& mu, float& rstd) {
    const int per = d >> 6;
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxPerLane; ++i)
        if (i < per) s += v[i];
    mu = wave_sum(s) / (float)d;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxPerLane; ++i)
        if (i < per) { const float t = v[i] - mu; q = fmaf(t, t, q); }
    rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + eps);
}

// Writes LN(v) (gain/shift) for the row to out (model operand type TA).
template <bool VEC, typename TA>
__device__ __forceinline__ void store_normed(TA* __restrict__ out, const float (&v)[kMaxPerLane],
                                             int d, int lane, float mu, float rstd,
                                             const float* __restrict__ gain,
                                             const float* __restrict__ shift) {
    const int per = d >> 6;
    if constexpr (VEC && sizeof(TA) == 2) {
        typedef __attribute__((ext_vector_type(4))) TA t4;
#pragma unroll
        for (int j = 0; j < kMaxPerLane / 4; ++j)
            if (4 * j < per) {
                const int c = j * 256 + 4 * lane;
                const float4 gq = *reinterpret_cast<const float4*>(gain + c);
                const float4 bq = *reinterpret_cast<const float4*>(shift + c);
                t4 o;
                o[0] = (TA)keep_f32(fmaf((v[4 * j] - mu) * rstd, gq.x, bq.x));
                o[1] = (TA)keep_f32(fmaf((v[4 * j + 1] - mu) * rstd, gq.y, bq.y));
                o[2] = (TA)keep_f32(fmaf((v[4 * j + 2] - mu) * rstd, gq.z, bq.z));
                o[3] = (TA)keep_f32(fmaf((v[4 * j + 3] - mu) * rstd, gq.w, bq.w));
                *reinterpret_cast<t4*>(out + c) = o;
            }
    } else {
#pragma unroll
        for (int i = 0; i < kMaxPerLane; ++i)
            if (i < per) {
                const int c = feat<VEC>(lane, i);
                out[c] = (TA)keep_f32(fmaf((v[i] - mu) * rstd, gain[c], shift[c]));
            }
    }
}

// Writes LN(v) for the row as MXFP8 (fp8 projection inputs): the VEC layout
// gives a lane four consecutive features per 256-feature group, so one
// 32-feature block is eight consecutive lanes; codes[c] is feature c's E4M3
// code, scales[c / 32] its block's E8M0 byte.
__device__ __forceinline__ void store_normed_mx(uint8_t* __restrict__ codes,
                                                uint8_t* __restrict__ scales,
                                                const float (&v)[kMaxPerLane], int d, int lane,
                                                float mu, float rstd,
                                                const float* __restrict__ gain,
                                                const float* __restrict__ shift) {
    const int per = d >> 6;
#pragma unroll
    for (int j = 0; j < kMaxPerLane / 4; ++j)
        if (4 * j < per) {
            const int c = j * 256 + 4 * lane;
            const float4 gq = *reinterpret_cast<const float4*>(gain + c);
            const float4 bq = *reinterpret_cast<const float4*>(shift + c);
            const float y0 = keep_f32(fmaf((v[4 * j] - mu) * rstd, gq.x, bq.x));
            const float y1 = keep_f32(fmaf((v[4 * j + 1] - mu) * rstd, gq.y, bq.y));
            const float y2 = keep_f32(fmaf((v[4 * j + 2] - mu) * rstd, gq.z, bq.z));
            const float y3 = keep_f32(fmaf((v[4 * j + 3] - mu) * rstd, gq.w, bq.w));
            float amax = fmaxf(fmaxf(fabsf(y0), fabsf(y1)), fmaxf(fabsf(y2), fabsf(y3)));
            amax = fmaxf(amax, __shfl_xor(amax, 1, 64));
            amax = fmaxf(amax, __shfl_xor(amax, 2, 64));
            amax = fmaxf(amax, __shfl_xor(amax, 4, 64));
            const int e = mx_block_exp(amax);
            const float inv = mx_inv_scale(e);
            *reinterpret_cast<uint32_t*>(codes + c) = mx_pack4(y0 * inv, y1 * inv, y2 * inv, y3 * inv);
            if ((lane & 7) == 0) scales[c >> 5] = (uint8_t)(e + 127);
        }
}

// g = float(x); a = LN(g)  (residual stream initialisation fused with the
// first layer's LayerNorm).  g may be null: the first residual update then
// reads x itself.
template <bool VEC, typename TKV, typename TA>
__global__ __launch_bounds__(256) void k_init_layernorm(const TKV* __restrict__ x,
                                                        float* __restrict__ g, TA* __restrict__ a,
                                                        int64_t rows, int d,
                                                        const float* __restrict__ gain,
                                                        const float* __restrict__ shift, float eps) {
    const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    const int per = d >> 6;
    float v[kMaxPerLane];
    const TKV* xr = x + row * d;
    float* gr = g + row * d;
    if (VEC) {
#pragma unroll
        for (int j = 0; j < kMaxPerLane / 4; ++j)
            if (4 * j < per) load4(xr + j * 256 + 4 * lane, v + 4 * j);
    } else {
#pragma unroll
        for (int i = 0; i < kMaxPerLane; ++i)
            if (i < per) v[i] = to_f(xr[lane + 64 * i]);
    }
    if (g == nullptr) {
    } else if (VEC) {
#pragma unroll
        for (int j = 0; j < kMaxPerLane / 4; ++j)
            if (4 * j < per)
                *reinterpret_cast<float4*>(gr + j * 256 + 4 * lane) =
                    make_float4(v[4 * j], v[4 * j + 1], v[4 * j + 2], v[4 * j + 3]);
    } else {
#pragma unroll
        for (int i = 0; i < kMaxPerLane; ++i)
            if (i < per) gr[lane + 64 * i] = v[i];
    }
    float mu, rstd;
    row_stats(v, d, eps, mu, rstd);
    store_normed<VEC>(a + row * d, v, d, lane, mu, rstd, gain, shift);
}

template <bool VEC, typename TA>
__global__ __launch_bounds__(256) void k_layernorm(const float* __restrict__ g, TA* __restrict__ a,
                                                   int64_t rows, int d,
                                                   const float* __restrict__ gain,
                                                   const float* __restrict__ shift, float eps) {
    const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    float v[kMaxPerLane], mu, rstd;
    load_row<VEC>(g + row * d, d, lane, v);
    row_stats(v, d, eps, mu, rstd);
    store_normed<VEC>(a + row * d, v, d, lane, mu, rstd, gain, shift);
}

// MXFP8 LayerNorm outputs (d a multiple of 256).  INIT: the residual stream
// starts here, g = float(x).
template <bool INIT, typename TKV>
__global__ __launch_bounds__(256) void k_layernorm_mx(const TKV* __restrict__ x,
                                                      float* __restrict__ g,
                                                      uint8_t* __restrict__ codes,
                                                      uint8_t* __restrict__ scales, int64_t rows,
                                                      int d, const float* __restrict__ gain,
                                                      const float* __restrict__ shift, float eps) {
    const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    const int per = d >> 6;
    float v[kMaxPerLane], mu, rstd;
    if constexpr (INIT) {
        const TKV* xr = x + row * d;
        float* gr = g + row * d;
#pragma unroll
        for (int j = 0; j < kMaxPerLane / 4; ++j)
            if (4 * j < per) {
                const int c = j * 256 + 4 * lane;
                load4(xr + c, v + 4 * j);
                if (g != nullptr)      // null: the first residual update reads x
                    *reinterpret_cast<float4*>(gr + c) =
                        make_float4(v[4 * j], v[4 * j + 1], v[4 * j + 2], v[4 * j + 3]);
            }
    } else {
        load_row<true>(g + row * d, d, lane, v);
    }
    row_stats(v, d, eps, mu, rstd);
    store_normed_mx(codes + row * d, scales + row * (d / kMxBlock), v, d, lane, mu, rstd, gain,
                    shift);
}

template <bool VEC>
__global__ __launch_bounds__(256) void k_score_head(const float* __restrict__ g,
                                                    float* __restrict__ scores, int64_t rows, int d,
                                                    const float* __restrict__ gain,
                                                    const float* __restrict__ shift,
                                                    const float* __restrict__ w,
                                                    const float* __restrict__ b, float eps) {
    const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    float v[kMaxPerLane], mu, rstd;
    load_row<VEC>(g + row * d, d, lane, v);
    row_stats(v, d, eps, mu, rstd);
    const int per = d >> 6;
    float acc = 0.f;
    if (VEC) {
#pragma unroll
        for (int j = 0; j < kMaxPerLane / 4; ++j)
            if (4 * j < per) {
                const int c = j * 256 + 4 * lane;
                const float4 gq = *reinterpret_cast<const float4*>(gain + c);
                const float4 bq = *reinterpret_cast<const float4*>(shift + c);
                const float4 wq = *reinterpret_cast<const float4*>(w + c);
                acc = fmaf(fmaf((v[4 * j] - mu) * rstd, gq.x, bq.x), wq.x, acc);
                acc = fmaf(fmaf((v[4 * j + 1] - mu) * rstd, gq.y, bq.y), wq.y, acc);
                acc = fmaf(fmaf((v[4 * j + 2] - mu) * rstd, gq.z, bq.z), wq.z, acc);
                acc = fmaf(fmaf((v[4 * j + 3] - mu) * rstd, gq.w, bq.w), wq.w, acc);
            }
    } else {
#pragma unroll
        for (int i = 0; i < kMaxPerLane; ++i)
            if (i < per) {
                const int c = lane + 64 * i;
                acc = fmaf(fmaf((v[i] - mu) * rstd, gain[c], shift[c]), w[c], acc);
            }
    }
    acc = wave_sum(acc);
    if (lane == 0) scores[row] = acc + b[0];
}

inline unsigned grid_rows(int64_t rows) {
    return (unsigned)((rows + kRowsPerBlock - 1) / kRowsPerBlock);
}

}  // namespace

template <typename TKV, typename TA>
hipError_t launch_init_layernorm(const TKV* x, float* g, TA* a, int64_t rows, int d,
                                 const float* gain, const float* shift, float eps, hipStream_t s) {
    if (rows == 0) return hipSuccess;
    if (d % 256 == 0)
        k_init_layernorm<true, TKV, TA><<<grid_rows(rows), 256, 0, s>>>(x, g, a, rows, d, gain,
                                                                       shift, eps);
    else
        k_init_layernorm<false, TKV, TA><<<grid_rows(rows), 256, 0, s>>>(x, g, a, rows, d, gain,
                                                                        shift, eps);
    return hipGetLastError();
}

template <typename TA>
hipError_t launch_layernorm(const float* g, TA* a, int64_t rows, int d, const float* gain,
                            const float* shift, float eps, hipStream_t s) {
    if (rows == 0) return hipSuccess;
    if (d % 256 == 0)
        k_layernorm<true, TA><<<grid_rows(rows), 256, 0, s>>>(g, a, rows, d, gain, shift, eps);
    else
        k_layernorm<false, TA><<<grid_rows(rows), 256, 0, s>>>(g, a, rows, d, gain, shift, eps);
    return hipGetLastError();
}

template <typename TKV>
hipError_t launch_init_layernorm_mx(const TKV* x, float* g, uint8_t* codes, uint8_t* scales,
                                    int64_t rows, int d, const float* gain, const float* shift,
                                    float eps, hipStream_t s) {
    if (rows == 0) return hipSuccess;
    if (d % 256 != 0) return hipErrorInvalidValue;
    k_layernorm_mx<true, TKV><<<grid_rows(rows), 256, 0, s>>>(x, g, codes, scales, rows, d, gain,
                                                             shift, eps);
    return hipGetLastError();
}

hipError_t launch_layernorm_mx(const float* g, uint8_t* codes, uint8_t* scales, int64_t rows,
                               int d, const float* gain, const float* shift, float eps,
                               hipStream_t s) {
    if (rows == 0) return hipSuccess;
    if (d % 256 != 0) return hipErrorInvalidValue;
    k_layernorm_mx<false, float><<<grid_rows(rows), 256, 0, s>>>(nullptr, const_cast<float*>(g),
                                                                codes, scales, rows, d, gain,
                                                                shift, eps);
    return hipGetLastError();
}

hipError_t launch_score_head(const float* g, float* scores, int64_t rows, int d,
                             const FinalWeights& fw, float eps, hipStream_t s) {
    if (rows == 0) return hipSuccess;
    if (d % 256 == 0)
        k_score_head<true><<<grid_rows(rows), 256, 0, s>>>(g, scores, rows, d, fw.lnf_g, fw.lnf_b,
                                                           fw.w_score, fw.b_score, eps);
    else
        k_score_head<false><<<grid_rows(rows), 256, 0, s>>>(g, scores, rows, d, fw.lnf_g,
                                                            fw.lnf_b, fw.w_score, fw.b_score, eps);
    return hipGetLastError();
}

template hipError_t launch_init_layernorm<float, float>(const float*, float*, float*, int64_t, int,
                                                        const float*, const float*, float,
                                                        hipStream_t);
template hipError_t launch_init_layernorm<bf16, f16>(const bf16*, float*, f16*, int64_t, int,
                                                     const float*, const float*, float,
                                                     hipStream_t);
template hipError_t launch_init_layernorm_mx<bf16>(const bf16*, float*, uint8_t*, uint8_t*,
                                                   int64_t, int, const float*, const float*,
                                                   float, hipStream_t);
template hipError_t launch_layernorm<float>(const float*, float*, int64_t, int, const float*,
                                            const float*, float, hipStream_t);
template hipError_t launch_layernorm<f16>(const float*, f16*, int64_t, int, const float*,
                                          const float*, float, hipStream_t);

}  // namespace upr
