// Plain kernels: a tiled FMA GEMM with the projection epilogues, and
// per-(row, head) attention for ranking and for history encoding.  They run
// the fp32 models (all arithmetic fp32) and the shapes the MFMA kernels do
// not take (head_dim 32).  Like every kernel here they are tested against
// the CPU oracle.
#include <cmath>

#include "epilogue.h"
#include "upr_internal.h"
#include "upr_plan.h"

namespace upr {

namespace {

template <typename T> __device__ __forceinline__ float to_f(T v) { return (float)v; }

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v = fmaxf(v, __shfl_xor(v, m, 64));
    return v;
}

// ---------------------------------------------------------------------------
// GEMM: 64x64 output tile per 256-thread block, K in steps of 16 through LDS,
// each thread a 4x4 register tile.
// ---------------------------------------------------------------------------
template <typename TA, typename TKV>
__global__ __launch_bounds__(256) void k_gemm_simple(const TA* __restrict__ A, int64_t lda,
                                                     const TA* __restrict__ W, int64_t M, int N,
                                                     int K, Epilogue epi) {
    __shared__ float As[16][68];
    __shared__ float Ws[16][68];
    const int tx = threadIdx.x & 15, ty = threadIdx.x >> 4;
    const int64_t m0 = (int64_t)blockIdx.y * 64;
    const int n0 = blockIdx.x * 64;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += 16) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int idx = threadIdx.x + 256 * i;
            const int r = idx >> 4, kk = idx & 15;
            const int64_t gm = m0 + r;
            const int gn = n0 + r, gk = k0 + kk;
            As[kk][r] = (gm < M && gk < K) ? to_f(A[gm * lda + gk]) : 0.f;
            Ws[kk][r] = (gn < N && gk < K) ? to_f(W[(int64_t)gn * K + gk]) : 0.f;
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < 16; ++kk) {
            float a[4], b[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) a[i] = As[kk][ty + 16 * i];
#pragma unroll
            for (int j = 0; j < 4; ++j) b[j] = Ws[kk][tx + 16 * j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(a[i], b[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int64_t m = m0 + ty + 16 * i;
            const int n = n0 + tx + 16 * j;
            if (m < M && n < N) epilogue_apply<TKV, TA>(epi, m, n, acc[i][j]);
        }
}

// Index of the segment holding absolute row `row`: the largest u in [0, U)
// with offsets[u] <= row (empty segments before it are skipped this way).
__device__ __forceinline__ int find_segment(const int32_t* __restrict__ offsets, int U, int64_t row) {
    int lo = 0, hi = U - 1;
    while (lo < hi) {
        const int mid = (lo + hi + 1) >> 1;
        if ((int64_t)offsets[mid] <= row) lo = mid; else hi = mid - 1;
    }
    return lo;
}

// ---------------------------------------------------------------------------
// Ranking attention, one wave per (candidate row, head).  Lane 0 starts the
// online softmax from the candidate's own key/value; lanes then take history
// keys t = lane, lane+64, ...; the 64 partial states are merged at the end.
// ---------------------------------------------------------------------------
template <typename T, typename TA, int D>
__global__ __launch_bounds__(256) void k_attn_rank_simple(
    const T* __restrict__ qkv, TA* __restrict__ o, int64_t rows, int64_t row0, int H,
    const int32_t* __restrict__ cand_offsets, const int32_t* __restrict__ hist_offsets, int U,
    const T* __restrict__ cache_k, const T* __restrict__ cache_v, int64_t cap) {
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int h = blockIdx.y;
    const int lane = threadIdx.x & 63;
    if (r >= rows) return;
    const int u = find_segment(cand_offsets, U, r + row0);
    const int64_t hb = hist_offsets[u];
    int n = hist_offsets[u + 1] - hist_offsets[u];
    // device offsets that disagree with the validated host ones (a caller
    // error) must not move the key range outside the cache
    if (hb < 0 || n < 0 || hb + n > cap) n = 0;
    const int d = H * D;
    const T* qrow = qkv + r * 3 * d + h * D;
    float q[D];
#pragma unroll
    for (int e = 0; e < D; ++e) q[e] = to_f(qrow[e]);
    float m = -INFINITY, l = 0.f, acc[D];
    if (lane == 0) {
        const T* ks = qrow + d;
        const T* vs = qrow + 2 * d;
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < D; ++e) s = fmaf(q[e], to_f(ks[e]), s);
        m = s;
        l = 1.f;
#pragma unroll
        for (int e = 0; e < D; ++e) acc[e] = to_f(vs[e]);
    } else {
#pragma unroll
        for (int e = 0; e < D; ++e) acc[e] = 0.f;
    }
    const T* Kb = cache_k + ((int64_t)h * cap + hb) * D;
    const T* Vb = cache_v + ((int64_t)h * cap + hb) * D;
    for (int t = lane; t < n; t += 64) {
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < D; ++e) s = fmaf(q[e], to_f(Kb[(int64_t)t * D + e]), s);
        const float mn = fmaxf(m, s);
        const float alpha = exp2f(m - mn);
        const float p = exp2f(s - mn);
        l = l * alpha + p;
#pragma unroll
        for (int e = 0; e < D; ++e) acc[e] = fmaf(p, to_f(Vb[(int64_t)t * D + e]), acc[e] * alpha);
        m = mn;
    }
    const float M = wave_max(m);
    const float sc = (m == -INFINITY) ? 0.f : exp2f(m - M);
    const float L = wave_sum(l * sc);
    float mine = 0.f;
#pragma unroll
    for (int e = 0; e < D; ++e) {
        const float v = wave_sum(acc[e] * sc);
        if (lane == e) mine = v;
    }
    if (lane < D) o[r * d + h * D + lane] = (TA)keep_f32(mine / L);
}

// ---------------------------------------------------------------------------
// Causal history attention, one wave per (history row, head): position i of
// its user attends to positions 0..i, whose keys/values are already in the
// cache plane of this layer.
// ---------------------------------------------------------------------------
template <typename T, typename TA, int D>
__global__ __launch_bounds__(256) void k_attn_encode_simple(
    const T* __restrict__ qbuf, TA* __restrict__ o, int64_t rows, int64_t row0, int H,
    const int32_t* __restrict__ hist_offsets, int U, const T* __restrict__ cache_k,
    const T* __restrict__ cache_v, int64_t cap) {
    const int64_t r = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int h = blockIdx.y;
    const int lane = threadIdx.x & 63;
    if (r >= rows) return;
    const int64_t arow = r + row0;
    const int u = find_segment(hist_offsets, U, arow);
    const int64_t hb = hist_offsets[u];
    // (-1, no keys, for device offsets that disagree with the host ones)
    const int i = hb < 0 || arow < hb || arow >= cap ? -1 : (int)(arow - hb);
    const int d = H * D;
    const T* qrow = qbuf + r * d + h * D;
    float q[D];
#pragma unroll
    for (int e = 0; e < D; ++e) q[e] = to_f(qrow[e]);
    float m = -INFINITY, l = 0.f, acc[D];
#pragma unroll
    for (int e = 0; e < D; ++e) acc[e] = 0.f;
    const T* Kb = cache_k + ((int64_t)h * cap + hb) * D;
    const T* Vb = cache_v + ((int64_t)h * cap + hb) * D;
    for (int t = lane; t <= i; t += 64) {
        float s = 0.f;
#pragma unroll
        for (int e = 0; e < D; ++e) s = fmaf(q[e], to_f(Kb[(int64_t)t * D + e]), s);
        const float mn = fmaxf(m, s);
        const float alpha = exp2f(m - mn);
        const float p = exp2f(s - mn);
        l = l * alpha + p;
#pragma unroll
        for (int e = 0; e < D; ++e) acc[e] = fmaf(p, to_f(Vb[(int64_t)t * D + e]), acc[e] * alpha);
        m = mn;
    }
    const float M = wave_max(m);
    const float sc = (m == -INFINITY) ? 0.f : exp2f(m - M);
    const float L = wave_sum(l * sc);
    float mine = 0.f;
#pragma unroll
    for (int e = 0; e < D; ++e) {
        const float v = wave_sum(acc[e] * sc);
        if (lane == e) mine = v;
    }
    if (lane < D) o[r * d + h * D + lane] = (TA)keep_f32(mine / L);
}

}  // namespace

template <typename TA, typename TKV>
hipError_t launch_gemm_simple(const TA* A, int64_t lda, const TA* W, int64_t M, int N, int K,
                              const Epilogue& epi, hipStream_t s) {
    if (M == 0) return hipSuccess;
    dim3 grid((unsigned)((N + 63) / 64), (unsigned)((M + 63) / 64));
    k_gemm_simple<TA, TKV><<<grid, 256, 0, s>>>(A, lda, W, M, N, K, epi);
    return hipGetLastError();
}

template <typename TKV, typename TA>
hipError_t launch_attn_rank_simple(const TKV* qkv, TA* o, int64_t rows, int64_t row0, int H,
                                   int D, const int32_t* cand_offsets,
                                   const int32_t* hist_offsets, int num_users, const TKV* cache_k,
                                   const TKV* cache_v, int64_t cache_cap, hipStream_t s) {
    if (rows == 0) return hipSuccess;
    dim3 grid((unsigned)((rows + 3) / 4), (unsigned)H);
    if (D == 32)
        k_attn_rank_simple<TKV, TA, 32><<<grid, 256, 0, s>>>(qkv, o, rows, row0, H, cand_offsets,
                                                            hist_offsets, num_users, cache_k,
                                                            cache_v, cache_cap);
    else
        k_attn_rank_simple<TKV, TA, 64><<<grid, 256, 0, s>>>(qkv, o, rows, row0, H, cand_offsets,
                                                            hist_offsets, num_users, cache_k,
                                                            cache_v, cache_cap);
    return hipGetLastError();
}

template <typename TKV, typename TA>
hipError_t launch_attn_encode_simple(const TKV* q, TA* o, int64_t rows, int64_t row0, int H,
                                     int D, const int32_t* hist_offsets, int num_users,
                                     const TKV* cache_k, const TKV* cache_v, int64_t cache_cap,
                                     hipStream_t s) {
    if (rows == 0) return hipSuccess;
    dim3 grid((unsigned)((rows + 3) / 4), (unsigned)H);
    if (D == 32)
        k_attn_encode_simple<TKV, TA, 32><<<grid, 256, 0, s>>>(q, o, rows, row0, H, hist_offsets,
                                                              num_users, cache_k, cache_v,
                                                              cache_cap);
    else
        k_attn_encode_simple<TKV, TA, 64><<<grid, 256, 0, s>>>(q, o, rows, row0, H, hist_offsets,
                                                              num_users, cache_k, cache_v,
                                                              cache_cap);
    return hipGetLastError();
}

#define UPR_INST(TKV, TA)                                                                       \
    template hipError_t launch_gemm_simple<TA, TKV>(const TA*, int64_t, const TA*, int64_t, int, \
                                                    int, const Epilogue&, hipStream_t);         \
    template hipError_t launch_attn_rank_simple<TKV, TA>(                                      \
        const TKV*, TA*, int64_t, int64_t, int, int, const int32_t*, const int32_t*, int,       \
        const TKV*, const TKV*, int64_t, hipStream_t);                                          \
    template hipError_t launch_attn_encode_simple<TKV, TA>(const TKV*, TA*, int64_t, int64_t,  \
                                                           int, int, const int32_t*, int,       \
                                                           const TKV*, const TKV*, int64_t,     \
                                                           hipStream_t);
UPR_INST(float, float)
UPR_INST(bf16, f16)
#undef UPR_INST
// fp32 models: every projection runs on the FMA GEMM (fp32 residual rows only)
template <>
hipError_t launch_gemm<float, float>(const float* A, int64_t lda, const float* W, int64_t M,
                                     int N, int K, const Epilogue& epi, hipStream_t s) {
    if (epi.resid_src != nullptr) return hipErrorInvalidValue;
    return launch_gemm_simple<float, float>(A, lda, W, M, N, K, epi, s);
}

// the fp8 projection variant's fallback attention: bf16 queries/keys/values
// and cache, fp32 output for the MXFP8 encoder
template hipError_t launch_attn_rank_simple<bf16, float>(const bf16*, float*, int64_t, int64_t,
                                                         int, int, const int32_t*, const int32_t*,
                                                         int, const bf16*, const bf16*, int64_t,
                                                         hipStream_t);

}  // namespace upr
