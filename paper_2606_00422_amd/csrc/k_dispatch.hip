// GEMM dispatch by model family.
#include "upr_plan.h"

namespace upr {

template <>
hipError_t launch_gemm<float, float>(const float* A, int64_t lda, const float* W, int64_t M,
                                     int N, int K, const Epilogue& epi, hipStream_t s) {
    return launch_gemm_simple<float, float>(A, lda, W, M, N, K, epi, s);
}

template <>
hipError_t launch_gemm<f16, bf16>(const f16* A, int64_t lda, const f16* W, int64_t M, int N,
                                  int K, const Epilogue& epi, hipStream_t s) {
    return launch_gemm_simple<f16, bf16>(A, lda, W, M, N, K, epi, s);
}

hipError_t launch_rank_worklist(const int32_t*, const int32_t*, int, int, int, int32_t*, int64_t,
                                hipStream_t) {
    return hipErrorNotSupported;
}

hipError_t launch_attn_rank(const bf16*, f16*, int64_t, int, int, const int32_t*,
                            const int32_t*, const int32_t*, int64_t, int, const bf16*,
                            const bf16*, int64_t, hipStream_t) {
    return hipErrorNotSupported;
}

}  // namespace upr
