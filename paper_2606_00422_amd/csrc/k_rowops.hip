// Row-wise kernels: residual-stream initialisation, LayerNorm, score head.
//
// One 64-lane wave owns one row of d features (d a multiple of 64, at most
// 1024); lane j holds features j, j+64, ... so every load is a coalesced
// 256-byte (fp32) run.  Statistics are two-pass in fp32: mean, then the mean of
// squared deviations (population variance), as the LayerNorm definition has it.
#include "upr_internal.h"

namespace upr {

namespace {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}

template <typename T> __device__ __forceinline__ float to_f(T v) { return (float)v; }
template <typename T> __device__ __forceinline__ T from_f(float v) { return (T)v; }

constexpr int kRowsPerBlock = 4;     // 4 waves, one row each
constexpr int kMaxPerLane = 16;      // d <= 1024

// Loads one row into registers and returns (mean, 1/sqrt(var + eps)).
__device__ __forceinline__ void row_stats(const float* __restrict__ x, int d, int lane,
                                          float (&v)[kMaxPerLane], float eps, float& mu,
                                          float& rstd) {
    const int per = d >> 6;
    float s = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxPerLane; ++i)
        if (i < per) { v[i] = x[lane + 64 * i]; s += v[i]; }
    mu = wave_sum(s) / (float)d;
    float q = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxPerLane; ++i)
        if (i < per) { float t = v[i] - mu; q += t * t; }
    rstd = 1.0f / sqrtf(wave_sum(q) / (float)d + eps);
}

template <typename T>
__global__ __launch_bounds__(256) void k_resid_init(const T* __restrict__ x, float* __restrict__ g,
                                                    int64_t n) {
    int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (; i < n; i += stride) g[i] = to_f(x[i]);
}

template <typename T>
__global__ __launch_bounds__(256) void k_layernorm(const float* __restrict__ g, T* __restrict__ a,
                                                   int64_t rows, int d,
                                                   const float* __restrict__ gain,
                                                   const float* __restrict__ shift, float eps) {
    const int64_t row = (int64_t)blockIdx.x * kRowsPerBlock + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    float v[kMaxPerLane], mu, rstd;
    row_stats(g + row * d, d, lane, v, eps, mu, rstd);
    T* out = a + row * d;
    const int per = d >> 6;
#pragma unroll
    for (int i = 0; i < kMaxPerLane; ++i)
        if (i < per) {
            const int c = lane + 64 * i;
            out[c] = from_f<T>((v[i] - mu) * rstd * gain[c] + shift[c]);
        }
}

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
    row_stats(g + row * d, d, lane, v, eps, mu, rstd);
    const int per = d >> 6;
    float acc = 0.f;
#pragma unroll
    for (int i = 0; i < kMaxPerLane; ++i)
        if (i < per) {
            const int c = lane + 64 * i;
            acc += ((v[i] - mu) * rstd * gain[c] + shift[c]) * w[c];
        }
    acc = wave_sum(acc);
    if (lane == 0) scores[row] = acc + b[0];
}

inline unsigned grid_rows(int64_t rows) {
    return (unsigned)((rows + kRowsPerBlock - 1) / kRowsPerBlock);
}

}  // namespace

template <typename T>
hipError_t launch_resid_init(const T* x, float* g, int64_t rows, int d, hipStream_t s) {
    const int64_t n = rows * d;
    if (n == 0) return hipSuccess;
    int64_t blocks = (n + 255) / 256;
    if (blocks > 65536) blocks = 65536;
    k_resid_init<T><<<(unsigned)blocks, 256, 0, s>>>(x, g, n);
    return hipGetLastError();
}

template <typename T>
hipError_t launch_layernorm(const float* g, T* a, int64_t rows, int d, const float* gain,
                            const float* shift, float eps, hipStream_t s) {
    if (rows == 0) return hipSuccess;
    k_layernorm<T><<<grid_rows(rows), 256, 0, s>>>(g, a, rows, d, gain, shift, eps);
    return hipGetLastError();
}

hipError_t launch_score_head(const float* g, float* scores, int64_t rows, int d,
                             const FinalWeights& fw, float eps, hipStream_t s) {
    if (rows == 0) return hipSuccess;
    k_score_head<<<grid_rows(rows), 256, 0, s>>>(g, scores, rows, d, fw.lnf_g, fw.lnf_b,
                                                 fw.w_score, fw.b_score, eps);
    return hipGetLastError();
}

template hipError_t launch_resid_init<float>(const float*, float*, int64_t, int, hipStream_t);
template hipError_t launch_resid_init<bf16>(const bf16*, float*, int64_t, int, hipStream_t);
template hipError_t launch_layernorm<float>(const float*, float*, int64_t, int, const float*,
                                            const float*, float, hipStream_t);
template hipError_t launch_layernorm<f16>(const float*, f16*, int64_t, int, const float*,
                                          const float*, float, hipStream_t);

}  // namespace upr
