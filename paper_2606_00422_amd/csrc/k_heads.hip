// Per-action ranking heads (output layer) and per-user utility top-K.
//
// Paper Sec. 3: every action type c has its own MLP head producing a scalar
// logit from the hidden state (action prediction objective); the serving
// node returns the top K candidates by the heads' utility.  The heads' first
// layer (all C heads stacked, GELU) runs on the projection GEMM; this file
// holds the rest.
#include "upr_plan.h"

namespace upr {

namespace {

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int m = 32; m >= 1; m >>= 1) v += __shfl_xor(v, m, 64);
    return v;
}

__device__ __forceinline__ float sigmoid(float x) {
    const float e = expf(-fabsf(x));
    return x >= 0.f ? 1.0f / (1.0f + e) : e / (1.0f + e);
}

template <typename TA> struct Vec8;
template <> struct Vec8<f16> {
    typedef __attribute__((ext_vector_type(8))) _Float16 type;
};
template <> struct Vec8<float> {
    typedef __attribute__((ext_vector_type(8))) float type;
};

// One wave per candidate row: logit_c = w2_c . hid[c*Fh .. c*Fh+Fh) + b2_c,
// p_c = sigmoid(logit_c), utility = sum_c u_c p_c (c in order).  Each lane
// takes 8 consecutive hidden values per step (Fh is a multiple of 8, so they
// belong to one head).
template <typename TA>
__global__ __launch_bounds__(256) void k_heads_out(const TA* __restrict__ hid, int64_t ldh,
                                                   int64_t rows, int C, int Fh,
                                                   const float* __restrict__ w2,
                                                   const float* __restrict__ b2, HeadUtility uw,
                                                   float* __restrict__ probs,
                                                   float* __restrict__ util) {
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (row >= rows) return;
    float part[kMaxActions];
#pragma unroll
    for (int c = 0; c < kMaxActions; ++c) part[c] = 0.f;
    const TA* hr = hid + row * ldh;
    const int n = C * Fh;
    for (int e = lane * 8; e < n; e += 64 * 8) {
        const typename Vec8<TA>::type v = *reinterpret_cast<const typename Vec8<TA>::type*>(hr + e);
        const float4 wa = *reinterpret_cast<const float4*>(w2 + e);
        const float4 wb = *reinterpret_cast<const float4*>(w2 + e + 4);
        float s = (float)v[0] * wa.x;
        s = fmaf((float)v[1], wa.y, s);
        s = fmaf((float)v[2], wa.z, s);
        s = fmaf((float)v[3], wa.w, s);
        s = fmaf((float)v[4], wb.x, s);
        s = fmaf((float)v[5], wb.y, s);
        s = fmaf((float)v[6], wb.z, s);
        s = fmaf((float)v[7], wb.w, s);
        const int head = e / Fh;
#pragma unroll
        for (int c = 0; c < kMaxActions; ++c)
            if (c == head) part[c] += s;
    }
    float u = 0.f;
#pragma unroll
    for (int c = 0; c < kMaxActions; ++c) {
        if (c >= C) break;
        const float p = sigmoid(wave_sum(part[c]) + b2[c]);
        if (lane == 0 && probs) probs[row * C + c] = p;
        u = fmaf(uw.u[c], p, u);
    }
    if (lane == 0 && util) util[row] = u;
}

constexpr int kTopkThreads = 1024;

// Sort key of one candidate: ascending order of the key is descending
// utility (NaN after every number, -0 equal to +0), then ascending row.
__device__ __forceinline__ uint64_t topk_key(float f, uint32_t local_row) {
    uint32_t hi;
    if (__builtin_isnan(f)) {
        hi = 0xFFFFFFFFu;
    } else {
        if (f == 0.f) f = 0.f;
        const uint32_t b = __float_as_uint(f);
        const uint32_t ord = (b & 0x80000000u) ? ~b : (b | 0x80000000u);   // increasing in f
        hi = ~ord;
    }
    return ((uint64_t)hi << 32) | local_row;
}

// One workgroup per user: bitonic sort of the user's keys in LDS (padded to
// a power of two with all-ones keys), then the first K entries out.
__global__ __launch_bounds__(kTopkThreads) void k_topk(const float* __restrict__ util,
                                                       const int32_t* __restrict__ coffs, int K,
                                                       int32_t* __restrict__ out_rows,
                                                       float* __restrict__ out_util, int64_t row_first,
                                                       int64_t row_last) {
    __shared__ uint64_t keys[kTopkMaxCandidates];
    const int u = blockIdx.x, tid = threadIdx.x;
    const int32_t r0 = coffs[u];
    int k = coffs[u + 1] - r0;
    // device offsets that disagree with the validated host ones (a caller
    // error): no entries rather than reads outside the utility rows
    if (r0 < row_first || k < 0 || r0 + (int64_t)k > row_last || k > kTopkMaxCandidates) k = 0;
    int N = 1;
    while (N < k) N <<= 1;
    for (int i = tid; i < N; i += kTopkThreads)
        keys[i] = i < k ? topk_key(util[r0 + i], (uint32_t)i) : ~0ull;
    __syncthreads();
    for (int size = 2; size <= N; size <<= 1)
        for (int stride = size >> 1; stride > 0; stride >>= 1) {
            for (int i = tid; i < (N >> 1); i += kTopkThreads) {
                const int lo = 2 * stride * (i / stride) + (i % stride), hi = lo + stride;
                const bool up = (lo & size) == 0;
                const uint64_t a = keys[lo], b = keys[hi];
                if ((a > b) == up) {
                    keys[lo] = b;
                    keys[hi] = a;
                }
            }
            __syncthreads();
        }
    int32_t* rows = out_rows + (int64_t)u * K;
    float* vals = out_util ? out_util + (int64_t)u * K : nullptr;
    for (int j = tid; j < K; j += kTopkThreads) {
        if (j < k) {
            const uint32_t lr = (uint32_t)(keys[j] & 0xFFFFFFFFu);
            rows[j] = r0 + (int32_t)lr;
            if (vals) vals[j] = util[r0 + lr];
        } else {
            rows[j] = -1;
            if (vals) vals[j] = __builtin_nanf("");
        }
    }
}

}  // namespace

template <typename TA>
hipError_t launch_heads_out(const TA* hid, int64_t ldh, int64_t rows, int C, int Fh,
                            const float* w2, const float* b2, const HeadUtility& uw, float* probs,
                            float* util, hipStream_t s) {
    if (rows == 0) return hipSuccess;
    if (C < 1 || C > kMaxActions || Fh % 8 != 0 || ldh % 8 != 0) return hipErrorInvalidValue;
    k_heads_out<TA><<<(unsigned)((rows + 3) / 4), 256, 0, s>>>(hid, ldh, rows, C, Fh, w2, b2, uw,
                                                              probs, util);
    return hipGetLastError();
}

hipError_t launch_topk(const float* util, const int32_t* coffs_dev, int U, int K,
                       int32_t* out_rows, float* out_util, int64_t row_first, int64_t row_last,
                       hipStream_t s) {
    if (U == 0) return hipSuccess;
    if (K < 1) return hipErrorInvalidValue;
    k_topk<<<(unsigned)U, kTopkThreads, 0, s>>>(util, coffs_dev, K, out_rows, out_util, row_first,
                                                row_last);
    return hipGetLastError();
}

template hipError_t launch_heads_out<float>(const float*, int64_t, int64_t, int, int, const float*,
                                            const float*, const HeadUtility&, float*, float*,
                                            hipStream_t);
template hipError_t launch_heads_out<f16>(const f16*, int64_t, int64_t, int, int, const float*,
                                          const float*, const HeadUtility&, float*, float*,
                                          hipStream_t);

}  // namespace upr
