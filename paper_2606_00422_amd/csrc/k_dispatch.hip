// GEMM dispatch by model family.
#include "upr_plan.h"

namespace upr {

template <>
hipError_t launch_gemm<float, float>(const float* A, int64_t lda, const float* W, int64_t M,
                                     int N, int K, const Epilogue& epi, hipStream_t s) {
    if (epi.resid_src != nullptr) return hipErrorInvalidValue;   // fp32 rows only
    return launch_gemm_simple<float, float>(A, lda, W, M, N, K, epi, s);
}

template <>
hipError_t launch_gemm<f16, bf16>(const f16* A, int64_t lda, const f16* W, int64_t M, int N,
                                  int K, const Epilogue& epi, hipStream_t s) {
    return launch_gemm_mfma(A, lda, W, M, N, K, epi, s);
}

}  // namespace upr
