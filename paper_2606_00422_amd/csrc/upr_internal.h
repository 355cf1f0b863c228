// Internal declarations shared by the library's host code and kernels.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "upr.h"

namespace upr {

typedef __bf16 bf16;
typedef _Float16 f16;

// Storage types of the two model families.
//   fp32 models: everything fp32.
//   bf16 models: tokens, queries/keys/values, the cache and softmax
//     probabilities are bf16; the operands of the projection GEMMs (LayerNorm
//     outputs, attention output, FFN hidden, weights) are fp16, whose 11-bit
//     significand holds every bf16 weight exactly and rounds activations 8x
//     finer at the same MFMA rate; the residual stream and all accumulation
//     are fp32.
struct F32Types {
    using kv = float;       // tokens, q/k/v, cache
    using act = float;      // projection operands (activations and weights)
};
struct Bf16Types {
    using kv = bf16;
    using act = f16;
};

// Device copy of one layer's weights.  Matrices are [out, in] row-major in the
// projection operand type; Wqkv stacks the rows of Wq, Wk and Wv ([3d, d]).
// For bf16 models each matrix is stored multiplied by 2^k (an exact power of
// two chosen so its largest magnitude lands in [2^14, 2^15)); the matching
// s_* factor 2^-k undoes it on the fp32 accumulator.  Vectors are fp32.
struct LayerWeights {
    const void* Wqkv;
    const void* Wo;
    const void* W1;
    const void* W2;
    // fused FFN (bf16 models, supported shapes): Wo, W1 and W2 again in the
    // fragment-major layout of the fused kernel (same values and scales);
    // null when not built
    const void* WoP;
    const void* W1p;
    const void* W2p;
    // W2's columns are stored in the EPI_GELU_PERM order (with W1p/W2p):
    // the FFN-up GEMM must then write its GELU output in that order
    bool w2_perm;
    float s_qkv, s_o, s_1, s_2;
    // fp8 projection variant: the same matrices as MXFP8 (E4M3 codes
    // [out, in], E8M0 scales [out, in / 32]); null for other models
    const uint8_t *mx_qkv, *mx_qkv_s, *mx_o, *mx_o_s, *mx_1, *mx_1_s, *mx_2, *mx_2_s;
    const float* ln1_g;
    const float* ln1_b;
    const float* bqkv;      // [3d]: bq, bk, bv
    const float* bo;
    const float* ln2_g;
    const float* ln2_b;
    const float* b1;
    const float* b2;
};

struct FinalWeights {
    const float* lnf_g;
    const float* lnf_b;
    const float* w_score;
    const float* b_score;   // one value
};

constexpr int kMaxLayers = 64;

// Materialises x as an fp32 register value.  Used right before an fp32 ->
// fp16/bf16 conversion in code whose unrolled copies serve different rows:
// without it the compiler may fold the producing multiply into a
// mixed-precision instruction (one rounding) in some copies and not in others
// (two roundings), so a row's result would depend on its position.  Not
// volatile: a volatile statement would also fence the scheduler, keeping
// loads behind it from being issued early.
__device__ __forceinline__ float keep_f32(float x) {
    asm("" : "+v"(x));
    return x;
}

// Epilogue modes of the projection GEMMs, out = A W^T + bias, then:
enum EpiMode : int {
    EPI_STORE = 0,      // out[m, n] (kv type); columns < scale_cols are multiplied by col_scale
    EPI_GELU = 1,       // out[m, n] = gelu_tanh(.)  (projection operand type)
    EPI_RESID = 2,      // resid[m, n] += .           (fp32, in place)
    EPI_QKV_CACHE = 3,  // columns [0,d): query -> out (scaled); [d,2d): keys and
                        // [2d,3d): values -> cache plane of the layer
    EPI_GELU_MX = 4,    // gelu_tanh(.) as MXFP8: E4M3 codes -> out (ldo bytes per
                        // row), one E8M0 byte per 32 columns -> out_scales
    EPI_RESID_LN = 5,   // EPI_RESID, then ln_out[m, :] = LayerNorm(resid[m, :])
                        // (ln_gain, ln_shift, ln_eps; projection operand type);
                        // the tile spans whole rows, so N <= 512
    EPI_RESID_LN_MX = 6,  // EPI_RESID_LN with the LayerNorm written as MXFP8:
                          // codes -> ln_out (ln_ldo bytes per row), one E8M0
                          // byte per 32 columns -> ln_scales (ln_ldo / 32 per row)
    EPI_RESID_SCORE = 7,  // the last residual update, then the score head:
                          // score_out[m] = LN(resid[m, :]) . score_w + *score_b
                          // (ln_gain, ln_shift, ln_eps = LN_f); the updated
                          // residual itself is not stored; N <= 512
    EPI_GELU_PERM = 8,    // EPI_GELU with the columns of each 16-column group
                          // stored in the order 0-3, 8-11, 4-7, 12-15 (position
                          // p holds column kHidPerm[p]): the order in which the
                          // fused FFN feeds the hidden values to the FFN-down
                          // MFMAs, which a W2 with the same column order then
                          // matches product for product
};

// The column order of EPI_GELU_PERM within a 16-column group (its own
// inverse).
constexpr int kHidPerm[16] = {0, 1, 2, 3, 8, 9, 10, 11, 4, 5, 6, 7, 12, 13, 14, 15};

// Widest row (N) the residual update with LayerNorm (EPI_RESID_LN) handles.
constexpr int kResidLnMaxN = 512;

struct Epilogue {
    int mode;
    float acc_scale;        // multiplies the accumulator first (weight scale)
    const float* bias;      // [N]
    void* out;              // EPI_STORE / EPI_GELU / EPI_QKV_CACHE (query part)
    int64_t ldo;            // leading dimension of out (elements)
    float* resid;           // EPI_RESID, leading dimension ldr
    int64_t ldr;
    float col_scale;        // applied to columns < scale_cols
    int scale_cols;
    // EPI_QKV_CACHE: cache plane of the layer and the absolute row of A's row 0
    void* cache_k;          // &cache[l][0][0][0][0]
    void* cache_v;          // &cache[l][1][0][0][0]
    int64_t cache_cap;
    int64_t row0;
    int d_model;
    int head_dim;
    // EPI_GELU_MX: block scales, ldo / 32 bytes per row
    void* out_scales;
    // EPI_RESID_LN: LayerNorm of the updated rows -> ln_out (leading dimension ln_ldo)
    const float* ln_gain;
    const float* ln_shift;
    float ln_eps;
    void* ln_out;
    int64_t ln_ldo;
    void* ln_scales;        // EPI_RESID_LN_MX
    // EPI_RESID*: when set, the residual is read from these bf16 rows
    // (leading dimension ldr) instead of resid, and the sum still goes to
    // resid: the first layer's update reads the tokens themselves
    const void* resid_src;
    // EPI_RESID_LN / EPI_RESID_SCORE with fp16 operands: nonzero when the
    // accumulators start at resid / acc_scale instead of zero (acc_scale a
    // power of two, so the division is exact).  The update is then
    // acc * acc_scale + bias, with no residual read in the epilogue: the FFN
    // down accumulates onto the residual that the O projection produced.
    int acc_resid;
    // EPI_RESID_SCORE
    const float* score_w;   // [N]
    const float* score_b;   // one value
    float* score_out;       // [M]
};

// ---------------------------------------------------------------------------
// Launchers (all enqueue on `stream`; they return hipGetLastError()).
// Row-wise kernels.
// ---------------------------------------------------------------------------
// g = float(x) and a = LN(g) in one pass (first layer's LayerNorm).
template <typename TKV, typename TA>
hipError_t launch_init_layernorm(const TKV* x, float* g, TA* a, int64_t rows, int d,
                                 const float* gain, const float* shift, float eps, hipStream_t s);
template <typename TA>
hipError_t launch_layernorm(const float* g, TA* a, int64_t rows, int d, const float* gain,
                            const float* shift, float eps, hipStream_t s);
hipError_t launch_score_head(const float* g, float* scores, int64_t rows, int d,
                             const FinalWeights& fw, float eps, hipStream_t s);

// MXFP8 variants of the LayerNorm launches (d a multiple of 256): codes
// [rows, d], scales [rows, d / 32].
template <typename TKV>
hipError_t launch_init_layernorm_mx(const TKV* x, float* g, uint8_t* codes, uint8_t* scales,
                                    int64_t rows, int d, const float* gain, const float* shift,
                                    float eps, hipStream_t s);
hipError_t launch_layernorm_mx(const float* g, uint8_t* codes, uint8_t* scales, int64_t rows,
                               int d, const float* gain, const float* shift, float eps,
                               hipStream_t s);
// MXFP8 encoding of x [rows, k] (k a multiple of 32) along its rows.
template <typename T>
hipError_t launch_mx_quantize(const T* x, int64_t rows, int k, uint8_t* codes, uint8_t* scales,
                              hipStream_t s);
// MXFP8 projection GEMM: out = A W^T + epilogue with A [M, K] and W [N, K]
// E4M3 codes and their E8M0 scales ([M, K/32], [N, K/32]); K a multiple of
// 128; epilogue modes EPI_STORE, EPI_RESID, EPI_GELU_MX and EPI_RESID_LN_MX.
// EPI_RESID_LN_MX may write its LayerNorm into A itself (same rows, same
// layout): a tile spans whole rows and writes them only after its last read
// of A, and no other tile reads those rows.
hipError_t launch_gemm_mx(const uint8_t* A, const uint8_t* A_scales, const uint8_t* W,
                          const uint8_t* W_scales, int64_t M, int N, int K, const Epilogue& epi,
                          hipStream_t s);

// Reference-quality GEMM: out = A[M,K] W[N,K]^T + epilogue; A and W are of the
// projection operand type TA, kv-typed epilogue outputs of type TKV.
template <typename TA, typename TKV>
hipError_t launch_gemm_simple(const TA* A, int64_t lda, const TA* W, int64_t M, int N, int K,
                              const Epilogue& epi, hipStream_t s);

// Reference-quality attention.  qkv / q rows are relative to the call's first
// row `row0`; offsets are absolute.  Logits use exp2 with queries pre-scaled by
// log2(e)/sqrt(D).  The output o is of the projection operand type TA.
template <typename TKV, typename TA>
hipError_t launch_attn_rank_simple(const TKV* qkv, TA* o, int64_t rows, int64_t row0, int H,
                                   int D, const int32_t* cand_offsets,
                                   const int32_t* hist_offsets, int num_users, const TKV* cache_k,
                                   const TKV* cache_v, int64_t cache_cap, hipStream_t s);
template <typename TKV, typename TA>
hipError_t launch_attn_encode_simple(const TKV* q, TA* o, int64_t rows, int64_t row0, int H,
                                     int D, const int32_t* hist_offsets, int num_users,
                                     const TKV* cache_k, const TKV* cache_v, int64_t cache_cap,
                                     hipStream_t s);

// Error reporting shared by the C-interface source files: records a
// formatted message for upr_last_error() and returns st (report_ok clears
// it and returns UPR_OK); validate_config checks a upr_config as every
// entry point does.
upr_status report_error(upr_status st, const char* fmt, ...);
upr_status report_ok();
upr_status validate_config(const upr_config* c);

// Device address, on the current device, of the library's scratch array
// for upr_rank_candidates_noalloc (UPR_NOALLOC_SCRATCH_BYTES, 256-byte
// aligned; looked up once per device).
hipError_t noalloc_scratch(void** ptr);

}  // namespace upr
