// Workspace plans of encode and rank, and the launchers they dispatch to.
#pragma once

#include <algorithm>
#include <cstddef>
#include <cstdint>

#include "upr_internal.h"

namespace upr {

inline size_t align256(size_t x) { return (x + 255) & ~size_t(255); }

// Query rows per work item of the MFMA attention (one workgroup handles this
// many history rows, in the causal encode pass, or candidates, in ranking,
// of one user for one head).
constexpr int kAttnTile = 128;
constexpr int kRankAttnTile = 128;
constexpr int kSmallRankAttnTile = 64;      // ranking calls with few work items
constexpr int64_t kSmallRankItems = 512;    // fewer 128-candidate items than this
// Ranking calls whose candidates see long histories (on average at least
// kLongHistory rows each) take 256-candidate items, eight waves per
// workgroup: each K/V stage then serves twice the queries.
constexpr int kLongRankAttnTile = 256;
constexpr double kLongHistory = 4096.0;
constexpr bool kHaveMfmaAttn = true;

struct EncodePlan {
    int64_t row0 = 0, rows = 0;
    size_t off_g = 0, off_a = 0, off_q = 0, off_o = 0, off_h = 0, off_work = 0;
    int64_t work_items = 0;
    int attn_tile = kAttnTile;
    bool use_mfma_attn = false;
    size_t bytes = 0;
};

struct RankPlan {
    int64_t row0 = 0, rows = 0;
    size_t off_g = 0, off_a = 0, off_qkv = 0, off_o = 0, off_h = 0, off_work = 0;
    int64_t work_items = 0;
    int attn_tile = kRankAttnTile;
    bool use_mfma_attn = false;
    size_t bytes = 0;
};

inline bool bf16_storage(const upr_config& c) {
    return c.dtype == UPR_BF16 || c.dtype == UPR_BF16_MXFP8;
}
inline size_t dtype_bytes(const upr_config& c) { return bf16_storage(c) ? 2 : 4; }

// Number of MFMA attention work items over the rows of `offs`: one per
// (user, head, tile of up to `tile` rows).
inline int64_t attn_items(const upr_config& c, int U, const int32_t* offs, int tile) {
    int64_t items = 0;
    for (int u = 0; u < U; ++u) items += ((int64_t)offs[u + 1] - offs[u] + tile - 1) / tile;
    return items * c.n_heads;
}

inline bool use_mfma_attn(const upr_config& c) {
    return kHaveMfmaAttn && bf16_storage(c) && c.head_dim == 64;
}

// Workspace of encode for the history rows of `hoffs` (host offsets): fp32
// residual stream, then LayerNorm output, queries, attention output and FFN
// hidden (model dtype), and (bf16 models) the attention work list.
inline EncodePlan plan_encode(const upr_config& c, int U, const int32_t* hoffs) {
    EncodePlan p;
    p.row0 = hoffs[0];
    p.rows = (int64_t)hoffs[U] - hoffs[0];
    if (p.rows <= 0) { p.rows = 0; return p; }
    const size_t es = dtype_bytes(c), R = (size_t)p.rows, d = c.d_model, F = c.d_ff;
    p.use_mfma_attn = use_mfma_attn(c);
    if (p.use_mfma_attn) p.work_items = attn_items(c, U, hoffs, p.attn_tile);
    size_t o = 0;
    p.off_g = o; o = align256(o + R * d * 4);
    p.off_a = o; o = align256(o + R * d * es);
    p.off_q = o; o = align256(o + R * d * es);
    p.off_o = o; o = align256(o + R * d * es);
    p.off_h = o; o = align256(o + R * F * es);
    p.off_work = o; o = align256(o + (size_t)p.work_items * 4 * sizeof(int32_t));
    p.bytes = o;
    return p;
}

// Workspace of rank for the candidate rows of `coffs` (host offsets):
// residual, LayerNorm output, fused q|k|v rows, attention output, FFN hidden
// (at least head_cols wide: the action heads' hidden layer reuses it), and
// (bf16 models) the attention work list.  The fp8-projection variant keeps
// MXFP8 encodings in the LayerNorm-output and FFN-hidden buffers (codes,
// then scales at the next 256-byte boundary: rows x cols x 2 bytes hold
// both for rows x cols >= 256).
inline RankPlan plan_rank(const upr_config& c, int U, const int32_t* coffs, const int32_t* hoffs,
                          int head_cols = 0) {
    RankPlan p;
    p.row0 = coffs[0];
    p.rows = (int64_t)coffs[U] - coffs[0];
    if (p.rows <= 0) { p.rows = 0; return p; }
    const size_t es = dtype_bytes(c), R = (size_t)p.rows, d = c.d_model, F = c.d_ff;
    p.use_mfma_attn = use_mfma_attn(c);
    if (p.use_mfma_attn) {
        double seen = 0.0;                  // history rows seen, summed over candidates
        for (int u = 0; u < U; ++u)
            seen += (double)((int64_t)coffs[u + 1] - coffs[u]) * (double)((int64_t)hoffs[u + 1] - hoffs[u]);
        const int64_t long_items = attn_items(c, U, coffs, kLongRankAttnTile);
        if (seen >= kLongHistory * (double)p.rows && long_items >= kSmallRankItems) {
            p.attn_tile = kLongRankAttnTile;
            p.work_items = long_items;
        } else {
            p.work_items = attn_items(c, U, coffs, p.attn_tile);
            if (p.work_items < kSmallRankItems) {
                p.attn_tile = kSmallRankAttnTile;
                p.work_items = attn_items(c, U, coffs, p.attn_tile);
            }
        }
    }
    size_t o = 0;
    p.off_g = o; o = align256(o + R * d * 4);
    p.off_a = o; o = align256(o + R * d * es);
    p.off_qkv = o; o = align256(o + R * 3 * d * es);
    // (the fp8 variant's fallback attention, head_dim 32, writes fp32 here
    // before the MXFP8 encoder reads it)
    const size_t o_es = c.dtype == UPR_BF16_MXFP8 ? 4 : es;
    p.off_o = o; o = align256(o + R * d * o_es);
    p.off_h = o; o = align256(o + R * std::max<size_t>(F, (size_t)head_cols) * es);
    p.off_work = o; o = align256(o + (size_t)p.work_items * 4 * sizeof(int32_t));
    p.bytes = o;
    return p;
}

// Projection GEMM, out = A[M,K] W[N,K]^T + epilogue: fp32 models use the
// reference FMA kernel, bf16 models the fp16 MFMA kernel.
template <typename TA, typename TKV>
hipError_t launch_gemm(const TA* A, int64_t lda, const TA* W, int64_t M, int N, int K,
                       const Epilogue& epi, hipStream_t s);

// fp16 MFMA GEMM (K a multiple of 64, lda a multiple of 8).  (The MXFP8
// GEMM, launch_gemm_mx, is declared with the other launchers.)
hipError_t launch_gemm_mfma(const f16* A, int64_t lda, const f16* W, int64_t M, int N, int K,
                            const Epilogue& epi, hipStream_t s);

// Fused layer tail (k_ffn_fused.hip) on the fp32 residual g:
//   g += O Wo^T + bo;  a = LN2(g);  g += gelu(a W1^T + b1) W2^T + b2
// then the LayerNorm (epi.mode EPI_RESID_LN) or the score head
// (EPI_RESID_SCORE).  O [M, d] fp16 attention output rows (leading dimension
// d); epa: the O projection's EPI_RESID_LN epilogue (Wo's scale, bo, LN2,
// the same residual; resid_src in the first layer), epi: the FFN down's
// (W2's scale, b2, the following LayerNorm or score head).  WoP [d, d],
// W1p [F, d] and W2p [d, F] in the fragment-major layout the model image
// builds; s1 = W1's scale.
bool ffn_fused_supported(int d, int F);
// Whether a call of M rows takes the fused kernel: its 128-row tiles must
// fill the device.  Smaller calls run the unfused sequence on short tiles,
// with bit-identical results (same products in the same order).
bool ffn_fused_rows(int64_t M);
hipError_t launch_ffn_fused(const f16* O, const f16* WoP, const Epilogue& epa, const f16* W1p,
                            const f16* W2p, const float* b1, float s1, int64_t M, int d, int F,
                            const Epilogue& epi, hipStream_t s);

// Work list of the MFMA attention: entries (first history row of the user,
// history length, first query row, head | query count << 16) over the rows
// of `row_offsets` (candidates, or the history itself for encode), users
// with the longest history first; `reverse` lists
// each user's tiles last-first (encode: the costliest causal tiles first).
// row_first / row_last: the host values of row_offsets[0] and [U]; cap: the
// cache rows.  Device offsets that disagree with them yield empty items.
hipError_t launch_attn_worklist(const int32_t* row_offsets, const int32_t* hist_offsets, int U,
                                int H, int tile, bool reverse, int32_t* work, int64_t items,
                                int64_t row_first, int64_t row_last, int64_t cap, hipStream_t s);

// MFMA ranking attention (bf16 q|k|v rows and cache, head_dim 64), fp16 output.
hipError_t launch_attn_rank(const bf16* qkv, f16* o, int64_t row0, int H, int D,
                            const int32_t* work, int64_t items,
                            int tile, const bf16* cache_k, const bf16* cache_v, int64_t cache_cap,
                            hipStream_t s);

// The same with the output as MXFP8 (codes [rows, H*64], one E8M0 scale byte
// per 32-value block [rows, H*2]), encoded from the normalised fp32 values:
// the fp8 projection variant's input of the O projection.
hipError_t launch_attn_rank_mx(const bf16* qkv, uint8_t* codes, uint8_t* scales, int64_t row0,
                               int H, int D, const int32_t* work,
                               int64_t items, int tile, const bf16* cache_k, const bf16* cache_v,
                               int64_t cache_cap, hipStream_t s);

// MFMA causal encode attention (bf16 query rows and cache, head_dim 64),
// fp16 output.
hipError_t launch_attn_encode(const bf16* q, f16* o, int64_t row0, int H, int D,
                              const int32_t* work, int64_t items,
                              int tile, const bf16* cache_k, const bf16* cache_v,
                              int64_t cache_cap, hipStream_t s);

// Host MXFP8 encoding of x [rows, k] (k a multiple of 32): the weights of
// the fp8-projection variant, and upr_mx_quantize_host.
void mx_quantize_host(const float* x, int64_t rows, int k, uint8_t* codes, uint8_t* scales);

// Per-action heads: at most kMaxActions heads; utility weights by value.
constexpr int kMaxActions = 8;
struct HeadUtility {
    float u[kMaxActions];
};

// logit_c = w2_c . hid[:, c*Fh .. c*Fh+Fh) + b2_c, probs[r, c] = sigmoid(logit_c)
// (if probs), util[r] = sum_c u_c probs[r, c] (if util); hid rows of ldh
// elements, Fh a multiple of 8.
template <typename TA>
hipError_t launch_heads_out(const TA* hid, int64_t ldh, int64_t rows, int C, int Fh,
                            const float* w2, const float* b2, const HeadUtility& uw, float* probs,
                            float* util, hipStream_t s);

// Per-user top K by utility (one workgroup per user, at most
// kTopkMaxCandidates candidates per user: the caller checks).  A user whose
// device offsets leave [row_first, row_last] or that limit gets no entries.
constexpr int kTopkMaxCandidates = 16384;
hipError_t launch_topk(const float* util, const int32_t* coffs_dev, int U, int K,
                       int32_t* out_rows, float* out_util, int64_t row_first, int64_t row_last,
                       hipStream_t s);

}  // namespace upr
