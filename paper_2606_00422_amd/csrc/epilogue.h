// Per-element epilogue of the projection GEMMs (device code, header-only).
#pragma once

#include "upr_internal.h"

namespace upr {

__device__ __forceinline__ float gelu_tanh_f(float x) {
    // 0.5 x (1 + tanh(sqrt(2/pi) (x + 0.044715 x^3)))
    const float k0 = 0.7978845608028654f;
    const float y = k0 * (x + 0.044715f * x * x * x);
    return 0.5f * x * (1.0f + tanhf(y));
}

// Applies the epilogue to the accumulated value v = sum_k A[m,k] W[n,k] of
// output element (m, n); m is relative to the call's first row.  kv-typed
// outputs (queries/keys/values, cache) are TKV, the FFN hidden is TA.
template <typename TKV, typename TA>
__device__ __forceinline__ void epilogue_apply(const Epilogue& e, int64_t m, int n, float v) {
    v = v * e.acc_scale + e.bias[n];
    switch (e.mode) {
        case EPI_STORE:
            if (n < e.scale_cols) v *= e.col_scale;
            static_cast<TKV*>(e.out)[m * e.ldo + n] = (TKV)keep_f32(v);
            break;
        case EPI_GELU:
            static_cast<TA*>(e.out)[m * e.ldo + n] = (TA)keep_f32(gelu_tanh_f(v));
            break;
        case EPI_RESID:
            e.resid[m * e.ldr + n] += v;
            break;
        case EPI_QKV_CACHE: {
            const int d = e.d_model;
            if (n < d) {
                static_cast<TKV*>(e.out)[m * e.ldo + n] = (TKV)keep_f32(v * e.col_scale);
            } else {
                const int part = n >= 2 * d ? 2 : 1;
                const int c = n - part * d;
                const int h = c / e.head_dim;
                const int ee = c - h * e.head_dim;
                TKV* plane = static_cast<TKV*>(part == 1 ? e.cache_k : e.cache_v);
                plane[((int64_t)h * e.cache_cap + (e.row0 + m)) * e.head_dim + ee] = (TKV)keep_f32(v);
            }
            break;
        }
        default:
            break;
    }
}

}  // namespace upr
