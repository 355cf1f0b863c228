// Host side of the C interface: argument validation, model creation,
// workspace carving and the encode / rank launch sequences.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <string>
#include <type_traits>
#include <vector>

#include "upr_internal.h"
#include "upr_plan.h"
#include "upr_profile.h"

using upr::bf16;

struct upr_model {
    upr_config cfg;
    void* dev = nullptr;
    size_t dev_bytes = 0;
    upr::LayerWeights layers[upr::kMaxLayers];
    upr::FinalWeights fin;
};

// Per-action heads: stacked first layers W1 [C*Fh, d] (model matrix type,
// scaled by 2^k for bf16 models: s_w1 = 2^-k), b1 [C*Fh], w2 [C*Fh], b2 [C].
struct upr_heads {
    upr_config cfg;             // of the model the heads were made for
    int32_t C = 0, Fh = 0;
    void* dev = nullptr;
    const void* W1 = nullptr;
    float s_w1 = 1.0f;
    const float* b1 = nullptr;
    const float* w2 = nullptr;
    const float* b2 = nullptr;
};

namespace {

thread_local std::string g_last_error;

upr_status fail(upr_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

upr_status ok() {
    g_last_error.clear();
    return UPR_OK;
}

// Discards a HIP error left pending by the caller's earlier work, so that a
// launch check of this call reports only this call's own failures.
void clear_pending_error() { (void)hipGetLastError(); }

// bf16 storage (tokens, cache): UPR_BF16 and its fp8-projection variant
bool bf16_family(int32_t dt) { return dt == UPR_BF16 || dt == UPR_BF16_MXFP8; }

upr_status check_config(const upr_config* c) {
    if (!c) return fail(UPR_ERR_NULL, "config is NULL");
    if (c->dtype != UPR_F32 && !bf16_family(c->dtype))
        return fail(UPR_ERR_DTYPE, "dtype %d is not UPR_F32, UPR_BF16 or UPR_BF16_MXFP8", c->dtype);
    if (c->dtype == UPR_BF16_MXFP8 && (c->d_model % 256 != 0 || c->d_ff % 128 != 0))
        return fail(UPR_ERR_CONFIG, "UPR_BF16_MXFP8 needs d_model %% 256 == 0 and d_ff %% 128 == 0 "
                    "(got %d, %d)", c->d_model, c->d_ff);
    if (c->head_dim != 32 && c->head_dim != 64)
        return fail(UPR_ERR_CONFIG, "head_dim %d not supported (32 or 64)", c->head_dim);
    if (c->n_heads <= 0 || (int64_t)c->n_heads * c->head_dim != c->d_model)
        return fail(UPR_ERR_CONFIG, "d_model %d != n_heads %d * head_dim %d", c->d_model,
                    c->n_heads, c->head_dim);
    if (c->d_model % 64 != 0 || c->d_model > 1024)
        return fail(UPR_ERR_CONFIG, "d_model %d must be a multiple of 64 and <= 1024", c->d_model);
    if (c->d_ff <= 0 || c->d_ff % 64 != 0 || c->d_ff > 8192)
        return fail(UPR_ERR_CONFIG, "d_ff %d must be a positive multiple of 64, <= 8192", c->d_ff);
    if (c->n_layers < 1 || c->n_layers > upr::kMaxLayers)
        return fail(UPR_ERR_CONFIG, "n_layers %d outside [1, %d]", c->n_layers, upr::kMaxLayers);
    if (!(c->ln_eps > 0.f) || !std::isfinite(c->ln_eps))
        return fail(UPR_ERR_CONFIG, "ln_eps must be positive and finite");
    return UPR_OK;
}

int64_t weights_count(const upr_config& c) {
    const int64_t d = c.d_model, F = c.d_ff;
    return c.n_layers * (4 * d * d + 2 * F * d + 9 * d + F) + 3 * d + 1;
}

uint16_t f32_to_bf16_rne(float f) {
    uint32_t u;
    std::memcpy(&u, &f, 4);
    if ((u & 0x7F800000u) == 0x7F800000u && (u & 0x007FFFFFu))
        return (uint16_t)((u >> 16) | 0x0040u);           // quiet NaN
    u += 0x7FFFu + ((u >> 16) & 1u);
    return (uint16_t)(u >> 16);
}

float bf16_value(uint16_t b) {
    const uint32_t u = (uint32_t)b << 16;
    float f;
    std::memcpy(&f, &u, 4);
    return f;
}

// Validates one segment descriptor; on success [*first, *last) is its row range.
upr_status check_segments(const upr_segments* s, const char* name, int64_t* first, int64_t* last) {
    if (!s) return fail(UPR_ERR_NULL, "%s segments pointer is NULL", name);
    if (s->num_users < 0) return fail(UPR_ERR_OFFSETS, "%s num_users %d < 0", name, s->num_users);
    if (!s->offsets_host) return fail(UPR_ERR_NULL, "%s offsets_host is NULL", name);
    const int32_t* o = s->offsets_host;
    if (o[0] < 0) return fail(UPR_ERR_OFFSETS, "%s offsets[0] = %d < 0", name, o[0]);
    for (int u = 0; u < s->num_users; ++u)
        if (o[u + 1] < o[u])
            return fail(UPR_ERR_OFFSETS, "%s offsets decrease at user %d (%d -> %d)", name, u, o[u],
                        o[u + 1]);
    if (s->num_users > 0 && !s->offsets_dev)
        return fail(UPR_ERR_NULL, "%s offsets_dev is NULL", name);
    *first = o[0];
    *last = o[s->num_users];
    return UPR_OK;
}

// Device image under construction: pieces start on 256-byte boundaries.
// Matrices: fp32 models copy them; bf16 models round each value to bf16
// (nearest, ties to even), multiply by an exact power of two 2^k that puts
// the largest magnitude in [2^14, 2^15), and store fp16 -- exact for every
// value within 2^29 of that maximum.  *scale receives 2^-k.  Vectors stay
// fp32.
struct ImageBuilder {
    std::vector<char> img;
    upr_dtype dtype;
    static size_t align(size_t x) { return (x + 255) & ~size_t(255); }
    // perm_row > 0: the matrix has rows of perm_row values whose columns are
    // stored in the EPI_GELU_PERM order within each 16-column group.
    size_t add_mat(const float* src, int64_t n, float* scale, int64_t perm_row = 0) {
        const bool bf = bf16_family(dtype);
        const size_t es = bf ? 2 : 4;
        size_t off = align(img.size());
        img.resize(off + n * es);
        *scale = 1.0f;
        if (bf) {
            float maxabs = 0.f;
            for (int64_t i = 0; i < n; ++i)
                maxabs = std::fmax(maxabs, std::fabs(bf16_value(f32_to_bf16_rne(src[i]))));
            int k = 0;
            if (maxabs > 0.f && std::isfinite(maxabs)) {
                int ex;
                std::frexp(maxabs, &ex);               // maxabs in [2^(ex-1), 2^ex)
                k = std::min(100, std::max(-100, 15 - ex));
            }
            const float up = std::ldexp(1.0f, k);
            *scale = std::ldexp(1.0f, -k);
            _Float16* dst = reinterpret_cast<_Float16*>(img.data() + off);
            for (int64_t i = 0; i < n; ++i) {
                const int64_t j = perm_row > 0 ? i - i % 16 + upr::kHidPerm[i % 16] : i;
                dst[i] = (_Float16)(bf16_value(f32_to_bf16_rne(src[j])) * up);
            }
        } else {
            std::memcpy(img.data() + off, src, n * 4);
        }
        return off;
    }
    // Fragment-major copy, for the fused FFN, of the fp16 matrix at `off`
    // ([N, K] row-major, N a multiple of 32, K of 16): fragment (t, kk) is
    // 64 lanes x 8 values, lane l taking row 32t + l % 32 at K positions
    // 16kk + 8(l / 32) + e, e = 0..7 (the MFMA operand layout).
    size_t add_frag(size_t off, int64_t N, int64_t K) {
        const size_t dst_off = align(img.size());
        img.resize(dst_off + N * K * 2);
        const _Float16* src = reinterpret_cast<const _Float16*>(img.data() + off);
        _Float16* dst = reinterpret_cast<_Float16*>(img.data() + dst_off);
        const int64_t ksteps = K / 16;
        for (int64_t t = 0; t < N / 32; ++t)
            for (int64_t kk = 0; kk < ksteps; ++kk)
                for (int l = 0; l < 64; ++l)
                    for (int e = 0; e < 8; ++e) {
                        const int64_t row = 32 * t + l % 32;
                        const int64_t k = 16 * kk + 8 * (l / 32) + e;
                        dst[((t * ksteps + kk) * 64 + l) * 8 + e] = src[row * K + k];
                    }
        return dst_off;
    }
    size_t add_vec(const float* src, int64_t n) {
        size_t off = align(img.size());
        img.resize(off + n * 4);
        std::memcpy(img.data() + off, src, n * 4);
        return off;
    }
    // MXFP8 encoding of a [rows, k] matrix, its values first rounded to bf16
    // (the model's weights): codes at *codes_off, scales at *scales_off.
    void add_mx(const float* src, int64_t rows, int k, size_t* codes_off, size_t* scales_off) {
        std::vector<float> w(src, src + rows * k);
        for (float& v : w) v = bf16_value(f32_to_bf16_rne(v));
        *codes_off = align(img.size());
        *scales_off = align(*codes_off + rows * k);
        img.resize(*scales_off + rows * (k / 32));
        upr::mx_quantize_host(w.data(), rows, k, reinterpret_cast<uint8_t*>(img.data() + *codes_off),
                              reinterpret_cast<uint8_t*>(img.data() + *scales_off));
    }
    // Copies the image to new device memory (*dev) or fails.
    upr_status upload(void** dev) {
        img.resize(align(img.size()));
        hipError_t e = hipMalloc(dev, img.size());
        if (e != hipSuccess)
            return fail(UPR_ERR_HIP, "hipMalloc(%zu) failed: %s", img.size(), hipGetErrorString(e));
        e = hipMemcpy(*dev, img.data(), img.size(), hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            (void)hipFree(*dev);
            *dev = nullptr;
            return fail(UPR_ERR_HIP, "hipMemcpy of weights failed: %s", hipGetErrorString(e));
        }
        return UPR_OK;
    }
};

upr_status check_workspace(void* ws, size_t ws_bytes, size_t need) {
    if (need == 0) return UPR_OK;
    if (!ws) return fail(UPR_ERR_NULL, "workspace is NULL (%zu bytes needed)", need);
    if (ws_bytes < need)
        return fail(UPR_ERR_WORKSPACE, "workspace has %zu bytes, %zu needed", ws_bytes, need);
    if (reinterpret_cast<uintptr_t>(ws) % 256 != 0)
        return fail(UPR_ERR_WORKSPACE, "workspace is not 256-byte aligned");
    return UPR_OK;
}

#define UPR_HIP(...)                                                                            \
    do {                                                                                        \
        hipError_t e_ = (__VA_ARGS__);                                                          \
        if (e_ != hipSuccess)                                                                   \
            return fail(UPR_ERR_HIP, "%s failed: %s", #__VA_ARGS__, hipGetErrorString(e_));     \
    } while (0)

// Testing hook.  With UPR_STOP_AFTER=n in the environment, an encode or
// rank call enqueues only the first n launches of its sequence (those made
// through UPR_LAUNCH) and returns UPR_OK, leaving the workspace as they
// wrote it, so that a test can check one stage at a time against the oracle
// on the GPU's own inputs of that stage.  Unset: no limit.
thread_local int64_t g_launches_left = -1;

void arm_stop_hook() {
    const char* e = std::getenv("UPR_STOP_AFTER");
    g_launches_left = (e != nullptr && *e != '\0') ? std::strtoll(e, nullptr, 10) : -1;
}

// Launch with a named timing scope (a no-op unless profiling is enabled).
#define UPR_LAUNCH(name, ...)                                                                   \
    do {                                                                                        \
        if (g_launches_left == 0) return UPR_OK;                                                \
        ProfScope ps_(name, s);                                                                 \
        UPR_HIP(__VA_ARGS__);                                                                   \
        if (g_launches_left > 0) --g_launches_left;                                             \
    } while (0)

size_t elem_size(const upr_config& c) { return bf16_family(c.dtype) ? 2 : 4; }

void* plane_ptr(const upr_config& c, const upr_kv_cache* cache, int layer, int kv) {
    const size_t off = (size_t)(layer * 2 + kv) * c.n_heads * cache->capacity_rows * c.head_dim;
    return static_cast<char*>(cache->data) + off * elem_size(c);
}

}  // namespace

// ---------------------------------------------------------------------------
// Encode / rank sequences
// ---------------------------------------------------------------------------
namespace upr {

upr_status report_error(upr_status st, const char* fmt, ...) {
    char buf[512];
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(buf, sizeof(buf), fmt, ap);
    va_end(ap);
    g_last_error = buf;
    return st;
}

upr_status report_ok() { return ok(); }

upr_status validate_config(const upr_config* c) { return check_config(c); }

// ---- MXFP8 on the host

// E4M3 code of s (finite): nearest value, ties to even (nearbyint in the
// default rounding mode), magnitudes above 448 saturated, the sign bit kept
// for negative values that round to zero.  Scaling by powers of two is exact.
static uint8_t e4m3_code(float s) {
    const uint8_t sign = std::signbit(s) ? 0x80 : 0x00;
    const float a = std::fabs(s);
    if (a >= 448.0f) return sign | 0x7E;
    if (a < 0.015625f)                                 // below 2^-6: steps of 2^-9,
        return sign | (uint8_t)std::nearbyint(a * 512.0f);   // 8 is the code of 2^-6
    int ex;
    std::frexp(a, &ex);                                // a in [2^(ex-1), 2^ex)
    int e = ex - 1;                                    // in [-6, 8]
    int m = (int)std::nearbyint(std::ldexp(a, 3 - e)); // in [8, 16]
    if (m == 16) {
        e += 1;
        m = 8;
    }
    return sign | (uint8_t)(((e + 7) << 3) | (m - 8));
}

void mx_quantize_host(const float* x, int64_t rows, int k, uint8_t* codes, uint8_t* scales) {
    for (int64_t r = 0; r < rows; ++r)
        for (int b = 0; b < k / 32; ++b) {
            const float* v = x + r * k + b * 32;
            float amax = 0.f;
            for (int i = 0; i < 32; ++i) amax = std::fmax(amax, std::fabs(v[i]));
            int e = -127;
            if (amax >= 0x1p-126f) {                    // normal: floor(log2 amax) = ex - 1
                int ex;
                std::frexp(amax, &ex);
                e = std::max(ex - 1 - 8, -127);
            }
            scales[r * (k / 32) + b] = (uint8_t)(e + 127);
            for (int i = 0; i < 32; ++i) codes[r * k + b * 32 + i] = e4m3_code(std::ldexp(v[i], -e));
        }
}

// Candidate layers of the fp8-projection variant: the bf16 sequence with
// MXFP8 projection operands (LayerNorms write MXFP8 directly, the attention
// kernel encodes its fp32 output, the FFN-up GEMM writes its GELU output as
// MXFP8).
static upr_status rank_layers_mx(const upr_model* m, const upr_kv_cache* cache,
                                 const upr_segments* hist, const bf16* cand_emb,
                                 const upr_segments* cand, const RankPlan& p, char* ws,
                                 hipStream_t s) {
    const upr_config& c = m->cfg;
    const int d = c.d_model, F = c.d_ff, H = c.n_heads, D = c.head_dim;
    const int64_t R = p.rows;
    float* g = reinterpret_cast<float*>(ws + p.off_g);
    uint8_t* ac = reinterpret_cast<uint8_t*>(ws + p.off_a);
    uint8_t* asc = ac + align256((size_t)R * d);
    bf16* qkv = reinterpret_cast<bf16*>(ws + p.off_qkv);
    float* o32 = reinterpret_cast<float*>(ws + p.off_o);
    uint8_t* hc = reinterpret_cast<uint8_t*>(ws + p.off_h);
    uint8_t* hsc = hc + align256((size_t)R * F);
    const float qscale = 1.4426950408889634f / std::sqrt((float)D);
    // the first O projection reads the residual from the tokens
    UPR_LAUNCH("rank.init_ln1",
               launch_init_layernorm_mx<bf16>(cand_emb + p.row0 * d, nullptr, ac, asc, R, d,
                                              m->layers[0].ln1_g, m->layers[0].ln1_b, c.ln_eps, s));
    if (p.use_mfma_attn)
        UPR_LAUNCH("rank.worklist",
                   launch_attn_worklist(cand->offsets_dev, hist->offsets_dev, cand->num_users, H,
                                        p.attn_tile, false, reinterpret_cast<int32_t*>(ws + p.off_work),
                                        p.work_items, cand->offsets_host[0],
                                        cand->offsets_host[cand->num_users], cache->capacity_rows, s));
    // LN2 is folded into the O projection (EPI_RESID_LN_MX) when a row fits
    // its tile; it then writes LN2 over its own operand (the attention
    // output): each tile owns whole rows and overwrites them after its last
    // read.  LN1 stays a row kernel: folded into FFN down (K = d_ff) the
    // 64-row tiles would re-read all of W2 per 64 rows (measured 0.22 ->
    // 0.32 ms for that GEMM).
    const bool fuse = d <= kResidLnMaxN && d % 64 == 0;
    auto resid_epilogue = [&](const float* bias, const float* ln_g, const float* ln_b) {
        Epilogue r{};
        r.mode = ln_g != nullptr ? EPI_RESID_LN_MX : EPI_RESID;
        r.acc_scale = 1.0f;
        r.bias = bias;
        r.resid = g;
        r.ldr = d;
        r.ln_gain = ln_g;
        r.ln_shift = ln_b;
        r.ln_eps = c.ln_eps;
        r.ln_out = ac;
        r.ln_ldo = d;
        r.ln_scales = asc;
        return r;
    };
    for (int l = 0; l < c.n_layers; ++l) {
        const LayerWeights& w = m->layers[l];
        if (l > 0)
            UPR_LAUNCH("rank.ln1",
                       launch_layernorm_mx(g, ac, asc, R, d, w.ln1_g, w.ln1_b, c.ln_eps, s));
        Epilogue e{};
        e.mode = EPI_STORE;
        e.acc_scale = 1.0f;
        e.bias = w.bqkv;
        e.out = qkv;
        e.ldo = 3 * d;
        e.col_scale = qscale;
        e.scale_cols = d;
        UPR_LAUNCH("rank.gemm_qkv", launch_gemm_mx(ac, asc, w.mx_qkv, w.mx_qkv_s, R, 3 * d, d, e, s));
        const bf16* ck = static_cast<const bf16*>(plane_ptr(c, cache, l, 0));
        const bf16* cv = static_cast<const bf16*>(plane_ptr(c, cache, l, 1));
        if (p.use_mfma_attn) {
            // attention writes the O projection's MXFP8 operand directly
            UPR_LAUNCH("rank.attn", launch_attn_rank_mx(qkv, ac, asc, p.row0, H, D,
                                                        reinterpret_cast<const int32_t*>(ws + p.off_work),
                                                        p.work_items, p.attn_tile, ck, cv,
                                                        cache->capacity_rows, s));
        } else {
            // fp32 attention output, then the MXFP8 encoder
            UPR_LAUNCH("rank.attn",
                       launch_attn_rank_simple<bf16, float>(qkv, o32, R, p.row0, H, D, cand->offsets_dev,
                                                            hist->offsets_dev, cand->num_users, ck, cv,
                                                            cache->capacity_rows, s));
            UPR_LAUNCH("rank.quant_o", launch_mx_quantize<float>(o32, R, d, ac, asc, s));
        }
        Epilogue r = resid_epilogue(w.bo, fuse ? w.ln2_g : nullptr, w.ln2_b);
        if (l == 0) r.resid_src = cand_emb + p.row0 * d;
        UPR_LAUNCH("rank.gemm_o", launch_gemm_mx(ac, asc, w.mx_o, w.mx_o_s, R, d, d, r, s));
        if (!fuse)
            UPR_LAUNCH("rank.ln2", launch_layernorm_mx(g, ac, asc, R, d, w.ln2_g, w.ln2_b, c.ln_eps, s));
        Epilogue up{};
        up.mode = EPI_GELU_MX;
        up.acc_scale = 1.0f;
        up.bias = w.b1;
        up.out = hc;
        up.ldo = F;
        up.out_scales = hsc;
        UPR_LAUNCH("rank.gemm_up", launch_gemm_mx(ac, asc, w.mx_1, w.mx_1_s, R, F, d, up, s));
        const Epilogue dn = resid_epilogue(w.b2, nullptr, nullptr);
        UPR_LAUNCH("rank.gemm_down", launch_gemm_mx(hc, hsc, w.mx_2, w.mx_2_s, R, d, F, dn, s));
    }
    return UPR_OK;
}

// The fp16 projection path folds each LayerNorm that follows a residual
// update into that update's GEMM (EPI_RESID_LN) when a row fits its tile.
template <typename Types>
static bool fused_layernorm(const upr_config& c) {
    return std::is_same_v<Types, Bf16Types> && c.d_model <= kResidLnMaxN;
}

// Attention-output projection and FFN of one layer, on the fp32 residual g:
// g += o Wo^T + bo;  a = LN2(g);  h = gelu(a W1^T + b1);  g += h W2^T + b2;
// then, when next_g is given and the LayerNorm is fused, a = LN(g) with
// (next_g, next_b).  resid_src (first layer, bf16 models): g is not yet
// written and the O projection reads the residual from these token rows.
// scores (last ranking layer, fused LayerNorms): FFN down ends in the score
// head, scores[m] = LN_f(g[m]) . w + b with score_fin, and g is left stale.
// Timing scopes are named "<stage>.gemm_o" etc.; the one-kernel tail is
// "<stage>.oproj_ffn".
template <typename Types>
static hipError_t launch_ffn_block(const char* const names[5], const upr_config& c,
                                   const LayerWeights& w, const typename Types::act* o,
                                   typename Types::act* a, typename Types::act* h, float* g,
                                   int64_t R, const float* next_g, const float* next_b,
                                   const void* resid_src, const FinalWeights* score_fin,
                                   float* scores, hipStream_t s) {
    using T = typename Types::kv;
    using TA = typename Types::act;
    const int d = c.d_model, F = c.d_ff;
    const float eps = c.ln_eps;
    const bool fuse = fused_layernorm<Types>(c);
    hipError_t e = hipSuccess;
    Epilogue r{};
    r.mode = fuse ? EPI_RESID_LN : EPI_RESID;
    r.acc_scale = w.s_o;
    r.bias = w.bo;
    r.resid = g;
    r.ldr = d;
    r.ln_gain = w.ln2_g;
    r.ln_shift = w.ln2_b;
    r.ln_eps = eps;
    r.ln_out = a;
    r.ln_ldo = d;
    r.resid_src = resid_src;
    // the layer's tail in one kernel (O projection, residual update, LN2,
    // FFN with its hidden rows on chip, then the next LayerNorm or the score
    // head) for calls whose 128-row tiles fill the device
    const bool tail = std::is_same_v<Types, Bf16Types> && fuse && w.WoP != nullptr && w.W1p != nullptr &&
                      (next_g != nullptr || scores != nullptr) && ffn_fused_rows(R);
    if (!tail) {
        ProfScope ps(names[0], s);
        e = launch_gemm<TA, T>(o, d, static_cast<const TA*>(w.Wo), R, d, d, r, s);
    }
    if (e != hipSuccess) return e;
    if (!fuse) {
        ProfScope ps(names[1], s);
        e = launch_layernorm<TA>(g, a, R, d, w.ln2_g, w.ln2_b, eps, s);
    }
    if (e != hipSuccess) return e;
    if constexpr (std::is_same_v<Types, Bf16Types>) {
        if (tail) {
            const Epilogue oproj = r;
            r.mode = scores != nullptr ? EPI_RESID_SCORE : EPI_RESID_LN;
            r.resid_src = nullptr;
            r.acc_resid = 1;
            r.acc_scale = w.s_2;
            r.bias = w.b2;
            if (scores != nullptr) {
                r.ln_gain = score_fin->lnf_g;
                r.ln_shift = score_fin->lnf_b;
                r.score_w = score_fin->w_score;
                r.score_b = score_fin->b_score;
                r.score_out = scores;
            } else {
                r.ln_gain = next_g;
                r.ln_shift = next_b;
            }
            ProfScope ps(names[4], s);
            return launch_ffn_fused(reinterpret_cast<const f16*>(o), static_cast<const f16*>(w.WoP), oproj,
                                    static_cast<const f16*>(w.W1p), static_cast<const f16*>(w.W2p), w.b1,
                                    w.s_1, R, d, F, r, s);
        }
    }
    Epilogue up{};
    up.mode = w.w2_perm ? EPI_GELU_PERM : EPI_GELU;
    up.acc_scale = w.s_1;
    up.bias = w.b1;
    up.out = h;
    up.ldo = F;
    {
        ProfScope ps(names[2], s);
        e = launch_gemm<TA, T>(a, d, static_cast<const TA*>(w.W1), R, F, d, up, s);
    }
    if (e != hipSuccess) return e;
    r.mode = fuse && next_g ? EPI_RESID_LN : EPI_RESID;
    r.resid_src = nullptr;
    if (fuse && scores != nullptr) {
        r.mode = EPI_RESID_SCORE;
        next_g = score_fin->lnf_g;
        next_b = score_fin->lnf_b;
        r.score_w = score_fin->w_score;
        r.score_b = score_fin->b_score;
        r.score_out = scores;
    }
    r.acc_scale = w.s_2;
    r.bias = w.b2;
    r.ln_gain = next_g;
    r.ln_shift = next_b;
    // FFN down with its LayerNorm or score head accumulates onto the
    // residual (the fused tail's arithmetic, so both give the same bits)
    r.acc_resid = std::is_same_v<Types, Bf16Types> && (r.mode == EPI_RESID_LN || r.mode == EPI_RESID_SCORE);
    ProfScope ps(names[3], s);
    return launch_gemm<TA, T>(h, F, static_cast<const TA*>(w.W2), R, d, F, r, s);
}

static const char* const kEncodeFfnNames[5] = {"encode.gemm_o", "encode.ln2", "encode.gemm_up",
                                               "encode.gemm_down", "encode.oproj_ffn"};
static const char* const kRankFfnNames[5] = {"rank.gemm_o", "rank.ln2", "rank.gemm_up",
                                             "rank.gemm_down", "rank.oproj_ffn"};

template <typename Types>
static upr_status run_encode(const upr_model* m, const typename Types::kv* hist_emb,
                             const upr_segments* hist, const upr_kv_cache* cache,
                             const EncodePlan& p, char* ws, hipStream_t s) {
    using T = typename Types::kv;
    using TA = typename Types::act;
    const upr_config& c = m->cfg;
    const int d = c.d_model, F = c.d_ff, H = c.n_heads, D = c.head_dim;
    const int64_t R = p.rows;
    float* g = reinterpret_cast<float*>(ws + p.off_g);
    TA* a = reinterpret_cast<TA*>(ws + p.off_a);
    T* q = reinterpret_cast<T*>(ws + p.off_q);
    TA* o = reinterpret_cast<TA*>(ws + p.off_o);
    TA* h = reinterpret_cast<TA*>(ws + p.off_h);
    const float qscale = 1.4426950408889634f / std::sqrt((float)D);
    // bf16 models: the first O projection reads the residual from the tokens
    const bool tok_resid = std::is_same_v<Types, Bf16Types>;
    UPR_LAUNCH("encode.init_ln1",
               launch_init_layernorm<T, TA>(hist_emb + p.row0 * d, tok_resid ? nullptr : g, a, R, d,
                                            m->layers[0].ln1_g, m->layers[0].ln1_b, c.ln_eps, s));
    if (p.use_mfma_attn && c.n_layers > 1)
        UPR_LAUNCH("encode.worklist",
                   launch_attn_worklist(hist->offsets_dev, hist->offsets_dev, hist->num_users, H,
                                        p.attn_tile, true, reinterpret_cast<int32_t*>(ws + p.off_work),
                                        p.work_items, hist->offsets_host[0],
                                        hist->offsets_host[hist->num_users], cache->capacity_rows, s));
    for (int l = 0; l < c.n_layers; ++l) {
        const LayerWeights& w = m->layers[l];
        if (l > 0 && !fused_layernorm<Types>(c))
            UPR_LAUNCH("encode.ln1",
                       launch_layernorm<TA>(g, a, R, d, w.ln1_g, w.ln1_b, c.ln_eps, s));
        Epilogue e{};
        e.mode = EPI_QKV_CACHE;
        e.acc_scale = w.s_qkv;
        e.bias = w.bqkv;
        e.out = q;
        e.ldo = d;
        e.col_scale = qscale;
        e.scale_cols = d;
        e.cache_k = plane_ptr(c, cache, l, 0);
        e.cache_v = plane_ptr(c, cache, l, 1);
        e.cache_cap = cache->capacity_rows;
        e.row0 = p.row0;
        e.d_model = d;
        e.head_dim = D;
        UPR_LAUNCH("encode.gemm_qkv",
                   launch_gemm<TA, T>(a, d, static_cast<const TA*>(w.Wqkv), R, 3 * d, d, e, s));
        if (l == c.n_layers - 1) break;     // the cache is complete; nothing reads further
        bool done = false;
        if constexpr (std::is_same_v<Types, Bf16Types>) {
            if (p.use_mfma_attn) {
                UPR_LAUNCH("encode.attn",
                           launch_attn_encode(q, o, p.row0, H, D,
                                              reinterpret_cast<const int32_t*>(ws + p.off_work),
                                              p.work_items, p.attn_tile,
                                              static_cast<const T*>(e.cache_k),
                                              static_cast<const T*>(e.cache_v),
                                              cache->capacity_rows, s));
                done = true;
            }
        }
        if (!done)
            UPR_LAUNCH("encode.attn",
                       launch_attn_encode_simple<T, TA>(q, o, R, p.row0, H, D, hist->offsets_dev,
                                                        hist->num_users,
                                                        static_cast<const T*>(e.cache_k),
                                                        static_cast<const T*>(e.cache_v),
                                                        cache->capacity_rows, s));
        const LayerWeights& wn = m->layers[l + 1];     // l + 1 < n_layers here
        UPR_HIP(launch_ffn_block<Types>(kEncodeFfnNames, c, w, o, a, h, g, R, wn.ln1_g, wn.ln1_b,
                                        tok_resid && l == 0 ? hist_emb + p.row0 * d : nullptr,
                                        nullptr, nullptr, s));
    }
    return UPR_OK;
}

// Outputs of a rank pass: the single score, or the action heads'
// probabilities / utilities.
struct RankOut {
    float* scores = nullptr;
    const upr_heads* heads = nullptr;
    HeadUtility uw{};
    float* probs = nullptr;
    float* util = nullptr;
};

template <typename Types>
static upr_status run_rank(const upr_model* m, const upr_kv_cache* cache,
                           const upr_segments* hist, const typename Types::kv* cand_emb,
                           const upr_segments* cand, const RankOut& out, const RankPlan& p,
                           char* ws, hipStream_t s) {
    using T = typename Types::kv;
    using TA = typename Types::act;
    const upr_config& c = m->cfg;
    const int d = c.d_model, F = c.d_ff, H = c.n_heads, D = c.head_dim;
    const int64_t R = p.rows;
    float* g = reinterpret_cast<float*>(ws + p.off_g);
    TA* a = reinterpret_cast<TA*>(ws + p.off_a);
    T* qkv = reinterpret_cast<T*>(ws + p.off_qkv);
    TA* o = reinterpret_cast<TA*>(ws + p.off_o);
    TA* h = reinterpret_cast<TA*>(ws + p.off_h);
    const float qscale = 1.4426950408889634f / std::sqrt((float)D);
    bool mx_done = false;
    if constexpr (std::is_same_v<Types, Bf16Types>) {
        if (c.dtype == UPR_BF16_MXFP8) {
            const upr_status st = rank_layers_mx(m, cache, hist, cand_emb, cand, p, ws, s);
            if (st != UPR_OK) return st;
            mx_done = true;
        }
    }
    if (!mx_done) {
    // bf16 models: the first O projection reads the residual from the tokens
    const bool tok_resid = std::is_same_v<Types, Bf16Types>;
    UPR_LAUNCH("rank.init_ln1",
               launch_init_layernorm<T, TA>(cand_emb + p.row0 * d, tok_resid ? nullptr : g, a, R, d,
                                            m->layers[0].ln1_g, m->layers[0].ln1_b, c.ln_eps, s));
    if (p.use_mfma_attn)
        UPR_LAUNCH("rank.worklist", launch_attn_worklist(cand->offsets_dev, hist->offsets_dev, cand->num_users, H,
                                     p.attn_tile, false, reinterpret_cast<int32_t*>(ws + p.off_work),
                                     p.work_items, cand->offsets_host[0],
                                     cand->offsets_host[cand->num_users], cache->capacity_rows, s));
    for (int l = 0; l < c.n_layers; ++l) {
        const LayerWeights& w = m->layers[l];
        if (l > 0 && !fused_layernorm<Types>(c))
            UPR_LAUNCH("rank.ln1", launch_layernorm<TA>(g, a, R, d, w.ln1_g, w.ln1_b, c.ln_eps, s));
        Epilogue e{};
        e.mode = EPI_STORE;
        e.acc_scale = w.s_qkv;
        e.bias = w.bqkv;
        e.out = qkv;
        e.ldo = 3 * d;
        e.col_scale = qscale;
        e.scale_cols = d;
        UPR_LAUNCH("rank.gemm_qkv",
                   launch_gemm<TA, T>(a, d, static_cast<const TA*>(w.Wqkv), R, 3 * d, d, e, s));
        const T* ck = static_cast<const T*>(plane_ptr(c, cache, l, 0));
        const T* cv = static_cast<const T*>(plane_ptr(c, cache, l, 1));
        bool done = false;
        if constexpr (std::is_same_v<Types, Bf16Types>) {
            if (p.use_mfma_attn) {
                UPR_LAUNCH("rank.attn", launch_attn_rank(qkv, o, p.row0, H, D,
                                         reinterpret_cast<const int32_t*>(ws + p.off_work),
                                         p.work_items, p.attn_tile, ck, cv, cache->capacity_rows,
                                         s));
                done = true;
            }
        }
        if (!done)
            UPR_LAUNCH("rank.attn", launch_attn_rank_simple<T, TA>(qkv, o, R, p.row0, H, D, cand->offsets_dev,
                                               hist->offsets_dev, cand->num_users, ck, cv,
                                               cache->capacity_rows, s));
        // the next LayerNorm: layer l + 1's LN1, or LN_f before the action heads
        const bool last = l + 1 == c.n_layers;
        const float* ng = !last ? m->layers[l + 1].ln1_g : out.heads ? m->fin.lnf_g : nullptr;
        const float* nb = !last ? m->layers[l + 1].ln1_b : out.heads ? m->fin.lnf_b : nullptr;
        // the score head rides on the last FFN down when the LayerNorms are fused
        float* const fused_scores =
            l + 1 == c.n_layers && !out.heads && fused_layernorm<Types>(c) ? out.scores + p.row0 : nullptr;
        UPR_HIP(launch_ffn_block<Types>(kRankFfnNames, c, w, o, a, h, g, R, ng, nb,
                                        tok_resid && l == 0 ? cand_emb + p.row0 * d : nullptr,
                                        &m->fin, fused_scores, s));
    }
    }  // !mx_done
    if (!out.heads) {
        if (mx_done || !fused_layernorm<Types>(c))
            UPR_LAUNCH("rank.score_head",
                       launch_score_head(g, out.scores + p.row0, R, d, m->fin, c.ln_eps, s));
        return UPR_OK;
    }
    // action heads: z = LN_f(g); hid = gelu(z W1^T + b1) (all heads stacked);
    // per head logit, sigmoid, utility
    const upr_heads* hd = out.heads;
    const int HC = hd->C * hd->Fh;
    if (mx_done || !fused_layernorm<Types>(c))
        UPR_LAUNCH("rank.lnf", launch_layernorm<TA>(g, a, R, d, m->fin.lnf_g, m->fin.lnf_b, c.ln_eps, s));
    Epilogue e{};
    e.mode = EPI_GELU;
    e.acc_scale = hd->s_w1;
    e.bias = hd->b1;
    e.out = h;
    e.ldo = HC;
    UPR_LAUNCH("rank.heads_hidden",
               launch_gemm<TA, T>(a, d, static_cast<const TA*>(hd->W1), R, HC, d, e, s));
    UPR_LAUNCH("rank.heads_out",
               launch_heads_out<TA>(h, HC, R, hd->C, hd->Fh, hd->w2, hd->b2, out.uw,
                                    out.probs ? out.probs + p.row0 * hd->C : nullptr,
                                    out.util ? out.util + p.row0 : nullptr, s));
    return UPR_OK;
}

}  // namespace upr

// ---------------------------------------------------------------------------
// C interface
// ---------------------------------------------------------------------------
extern "C" {

int64_t upr_weights_count(const upr_config* cfg) {
    if (check_config(cfg) != UPR_OK) return -1;
    return weights_count(*cfg);
}

upr_status upr_model_create(const upr_config* cfg, const float* weights_host,
                            int64_t count, upr_model** out) {
    upr_status st = check_config(cfg);
    if (st != UPR_OK) return st;
    if (!weights_host) return fail(UPR_ERR_NULL, "weights_host is NULL");
    if (!out) return fail(UPR_ERR_NULL, "out is NULL");
    const upr_config c = *cfg;
    if (count != weights_count(c))
        return fail(UPR_ERR_WEIGHTS, "weight blob has %lld values, config needs %lld",
                    (long long)count, (long long)weights_count(c));
    const int64_t d = c.d_model, F = c.d_ff;
    // Device image: per layer the four matrices (model dtype), then all
    // vectors (fp32).
    ImageBuilder ib{{}, (upr_dtype)c.dtype};
    auto add_mat = [&](const float* src, int64_t n, float* scale) { return ib.add_mat(src, n, scale); };
    auto add_vec = [&](const float* src, int64_t n) { return ib.add_vec(src, n); };
    struct LayerOff {
        size_t Wqkv, Wo, W1, W2, ln1_g, ln1_b, bqkv, bo, ln2_g, ln2_b, b1, b2;
        size_t WoP = 0, W1p = 0, W2p = 0;   // fragment-major copies for the fused FFN (0: none)
        bool w2_perm = false;
        float s_qkv, s_o, s_1, s_2;
        size_t mx[8];       // fp8 variant: qkv, qkv scales, o, o scales, 1, 1 scales, 2, 2 scales
    };
    const bool mx = c.dtype == UPR_BF16_MXFP8;
    std::vector<LayerOff> lo(c.n_layers);
    const float* p = weights_host;
    std::vector<float> tmp;
    for (int l = 0; l < c.n_layers; ++l) {
        const float* ln1_g = p; p += d;
        const float* ln1_b = p; p += d;
        const float* Wq = p; p += d * d;
        const float* bq = p; p += d;
        const float* Wk = p; p += d * d;
        const float* bk = p; p += d;
        const float* Wv = p; p += d * d;
        const float* bv = p; p += d;
        const float* Wo = p; p += d * d;
        const float* bo = p; p += d;
        const float* ln2_g = p; p += d;
        const float* ln2_b = p; p += d;
        const float* W1 = p; p += F * d;
        const float* b1 = p; p += F;
        const float* W2 = p; p += d * F;
        const float* b2 = p; p += d;
        tmp.assign(Wq, Wq + d * d);
        tmp.insert(tmp.end(), Wk, Wk + d * d);
        tmp.insert(tmp.end(), Wv, Wv + d * d);
        lo[l].Wqkv = add_mat(tmp.data(), 3 * d * d, &lo[l].s_qkv);
        lo[l].Wo = add_mat(Wo, d * d, &lo[l].s_o);
        lo[l].W1 = add_mat(W1, F * d, &lo[l].s_1);
        // Shapes the fused FFN takes: W2's columns in the EPI_GELU_PERM
        // order (so the FFN-up GEMM writes the hidden values in that order,
        // and the unfused pair multiplies exactly the pairs the fused kernel
        // does), and fragment-major copies of W1 and of that W2.
        lo[l].w2_perm = bf16_family(c.dtype) && upr::ffn_fused_supported((int)d, (int)F);
        lo[l].W2 = ib.add_mat(W2, d * F, &lo[l].s_2, lo[l].w2_perm ? F : 0);
        if (lo[l].w2_perm) {
            lo[l].WoP = ib.add_frag(lo[l].Wo, d, d);
            lo[l].W1p = ib.add_frag(lo[l].W1, F, d);
            lo[l].W2p = ib.add_frag(lo[l].W2, d, F);
        }
        if (mx) {
            ib.add_mx(tmp.data(), 3 * d, (int)d, &lo[l].mx[0], &lo[l].mx[1]);
            ib.add_mx(Wo, d, (int)d, &lo[l].mx[2], &lo[l].mx[3]);
            ib.add_mx(W1, F, (int)d, &lo[l].mx[4], &lo[l].mx[5]);
            ib.add_mx(W2, d, (int)F, &lo[l].mx[6], &lo[l].mx[7]);
        }
        lo[l].ln1_g = add_vec(ln1_g, d);
        lo[l].ln1_b = add_vec(ln1_b, d);
        tmp.assign(bq, bq + d);
        tmp.insert(tmp.end(), bk, bk + d);
        tmp.insert(tmp.end(), bv, bv + d);
        lo[l].bqkv = add_vec(tmp.data(), 3 * d);
        lo[l].bo = add_vec(bo, d);
        lo[l].ln2_g = add_vec(ln2_g, d);
        lo[l].ln2_b = add_vec(ln2_b, d);
        lo[l].b1 = add_vec(b1, F);
        lo[l].b2 = add_vec(b2, d);
    }
    const size_t off_lnf_g = add_vec(p, d); p += d;
    const size_t off_lnf_b = add_vec(p, d); p += d;
    const size_t off_ws = add_vec(p, d); p += d;
    const size_t off_bs = add_vec(p, 1); p += 1;

    upr_model* m = new upr_model();
    m->cfg = c;
    st = ib.upload(&m->dev);
    if (st != UPR_OK) {
        delete m;
        return st;
    }
    m->dev_bytes = ib.img.size();
    char* base = static_cast<char*>(m->dev);
    auto fp = [&](size_t off) { return reinterpret_cast<const float*>(base + off); };
    for (int l = 0; l < c.n_layers; ++l) {
        upr::LayerWeights& w = m->layers[l];
        w.Wqkv = base + lo[l].Wqkv;
        w.Wo = base + lo[l].Wo;
        w.W1 = base + lo[l].W1;
        w.W2 = base + lo[l].W2;
        w.WoP = lo[l].WoP ? base + lo[l].WoP : nullptr;
        w.W1p = lo[l].W1p ? base + lo[l].W1p : nullptr;
        w.W2p = lo[l].W2p ? base + lo[l].W2p : nullptr;
        w.w2_perm = lo[l].w2_perm;
        w.s_qkv = lo[l].s_qkv;
        w.s_o = lo[l].s_o;
        w.s_1 = lo[l].s_1;
        w.s_2 = lo[l].s_2;
        w.ln1_g = fp(lo[l].ln1_g);
        w.ln1_b = fp(lo[l].ln1_b);
        w.bqkv = fp(lo[l].bqkv);
        w.bo = fp(lo[l].bo);
        w.ln2_g = fp(lo[l].ln2_g);
        w.ln2_b = fp(lo[l].ln2_b);
        w.b1 = fp(lo[l].b1);
        w.b2 = fp(lo[l].b2);
        auto u8 = [&](size_t off) { return reinterpret_cast<const uint8_t*>(base + off); };
        w.mx_qkv = mx ? u8(lo[l].mx[0]) : nullptr;
        w.mx_qkv_s = mx ? u8(lo[l].mx[1]) : nullptr;
        w.mx_o = mx ? u8(lo[l].mx[2]) : nullptr;
        w.mx_o_s = mx ? u8(lo[l].mx[3]) : nullptr;
        w.mx_1 = mx ? u8(lo[l].mx[4]) : nullptr;
        w.mx_1_s = mx ? u8(lo[l].mx[5]) : nullptr;
        w.mx_2 = mx ? u8(lo[l].mx[6]) : nullptr;
        w.mx_2_s = mx ? u8(lo[l].mx[7]) : nullptr;
    }
    m->fin.lnf_g = fp(off_lnf_g);
    m->fin.lnf_b = fp(off_lnf_b);
    m->fin.w_score = fp(off_ws);
    m->fin.b_score = fp(off_bs);
    *out = m;
    return ok();
}

void upr_model_destroy(upr_model* m) {
    if (!m) return;
    if (m->dev) (void)hipFree(m->dev);
    delete m;
}

size_t upr_kv_cache_bytes(const upr_config* cfg, int64_t capacity_rows) {
    if (check_config(cfg) != UPR_OK || capacity_rows < 0) return 0;
    return (size_t)cfg->n_layers * 2 * cfg->n_heads * (size_t)capacity_rows * cfg->head_dim *
           elem_size(*cfg);
}

int64_t upr_kv_cache_index(const upr_config* cfg, int64_t cap, int32_t layer, int32_t kv,
                           int32_t head, int64_t row, int32_t e) {
    if (check_config(cfg) != UPR_OK) return -1;
    if (layer < 0 || layer >= cfg->n_layers || kv < 0 || kv > 1 || head < 0 ||
        head >= cfg->n_heads || row < 0 || row >= cap || e < 0 || e >= cfg->head_dim)
        return -1;
    return ((((int64_t)layer * 2 + kv) * cfg->n_heads + head) * cap + row) * cfg->head_dim + e;
}

size_t upr_encode_workspace_bytes(const upr_model* m, const upr_segments* hist) {
    if (!m) return 0;
    int64_t first, last;
    if (check_segments(hist, "hist", &first, &last) != UPR_OK) return 0;
    return upr::plan_encode(m->cfg, hist->num_users, hist->offsets_host).bytes;
}

size_t upr_rank_workspace_bytes(const upr_model* m, const upr_segments* hist,
                                const upr_segments* cand) {
    if (!m) return 0;
    int64_t hf, hl, cf, cl;
    if (check_segments(hist, "hist", &hf, &hl) != UPR_OK) return 0;
    if (check_segments(cand, "cand", &cf, &cl) != UPR_OK) return 0;
    if (hist->num_users != cand->num_users) return 0;
    return upr::plan_rank(m->cfg, cand->num_users, cand->offsets_host, hist->offsets_host).bytes;
}

upr_status upr_encode_user(const upr_model* m, const void* hist_emb, const upr_segments* hist,
                           const upr_kv_cache* cache, void* ws, size_t ws_bytes, void* stream) {
    if (!m) return fail(UPR_ERR_NULL, "model is NULL");
    int64_t first, last;
    upr_status st = check_segments(hist, "hist", &first, &last);
    if (st != UPR_OK) return st;
    if (!cache) return fail(UPR_ERR_NULL, "cache is NULL");
    if (last > first && !hist_emb) return fail(UPR_ERR_NULL, "hist_emb is NULL");
    if (last > first && !cache->data) return fail(UPR_ERR_NULL, "cache data is NULL");
    if (cache->capacity_rows < 0 || last > cache->capacity_rows)
        return fail(UPR_ERR_CAPACITY, "history rows end at %lld, cache capacity is %lld",
                    (long long)last, (long long)cache->capacity_rows);
    const upr::EncodePlan p = upr::plan_encode(m->cfg, hist->num_users, hist->offsets_host);
    st = check_workspace(ws, ws_bytes, p.bytes);
    if (st != UPR_OK) return st;
    if (p.rows == 0) return ok();
    clear_pending_error();
    arm_stop_hook();
    hipStream_t s = static_cast<hipStream_t>(stream);
    char* w = static_cast<char*>(ws);
    st = bf16_family(m->cfg.dtype)
             ? upr::run_encode<upr::Bf16Types>(m, static_cast<const bf16*>(hist_emb), hist, cache,
                                               p, w, s)
             : upr::run_encode<upr::F32Types>(m, static_cast<const float*>(hist_emb), hist,
                                              cache, p, w, s);
    return st == UPR_OK ? ok() : st;
}

// upr_rank_candidates, and with `scratch` its no-alloc variant, whose
// workspace is the library's per-GPU scratch array (upr_noalloc.hip).
static upr_status rank_entry(const upr_model* m, const upr_kv_cache* cache,
                             const upr_segments* hist, const void* cand_emb,
                             const upr_segments* cand, float* scores, void* ws,
                             size_t ws_bytes, bool scratch, void* stream) {
    if (!m) return fail(UPR_ERR_NULL, "model is NULL");
    int64_t hf, hl, cf, cl;
    upr_status st = check_segments(hist, "hist", &hf, &hl);
    if (st != UPR_OK) return st;
    st = check_segments(cand, "cand", &cf, &cl);
    if (st != UPR_OK) return st;
    if (hist->num_users != cand->num_users)
        return fail(UPR_ERR_OFFSETS, "hist has %d users, cand has %d", hist->num_users,
                    cand->num_users);
    if (!cache) return fail(UPR_ERR_NULL, "cache is NULL");
    if (cache->capacity_rows < 0 || hl > cache->capacity_rows)
        return fail(UPR_ERR_CAPACITY, "history rows end at %lld, cache capacity is %lld",
                    (long long)hl, (long long)cache->capacity_rows);
    if (cl > cf) {
        if (!cand_emb) return fail(UPR_ERR_NULL, "cand_emb is NULL");
        if (!scores) return fail(UPR_ERR_NULL, "scores is NULL");
        if (hl > hf && !cache->data) return fail(UPR_ERR_NULL, "cache data is NULL");
    }
    const upr::RankPlan p = upr::plan_rank(m->cfg, cand->num_users, cand->offsets_host, hist->offsets_host);
    if (scratch) {
        if (p.bytes > UPR_NOALLOC_SCRATCH_BYTES)
            return fail(UPR_ERR_LIMIT, "the call needs a %zu-byte workspace; the no-alloc scratch "
                        "array holds %zu", p.bytes, (size_t)UPR_NOALLOC_SCRATCH_BYTES);
        if (p.rows == 0) return ok();
        const hipError_t e = upr::noalloc_scratch(&ws);
        if (e != hipSuccess)
            return fail(UPR_ERR_HIP, "scratch array lookup failed: %s", hipGetErrorString(e));
        ws_bytes = UPR_NOALLOC_SCRATCH_BYTES;
    }
    st = check_workspace(ws, ws_bytes, p.bytes);
    if (st != UPR_OK) return st;
    if (p.rows == 0) return ok();
    clear_pending_error();
    arm_stop_hook();
    hipStream_t s = static_cast<hipStream_t>(stream);
    char* w = static_cast<char*>(ws);
    upr::RankOut out;
    out.scores = scores;
    st = bf16_family(m->cfg.dtype)
             ? upr::run_rank<upr::Bf16Types>(m, cache, hist, static_cast<const bf16*>(cand_emb),
                                             cand, out, p, w, s)
             : upr::run_rank<upr::F32Types>(m, cache, hist, static_cast<const float*>(cand_emb),
                                            cand, out, p, w, s);
    return st == UPR_OK ? ok() : st;
}

upr_status upr_rank_candidates(const upr_model* m, const upr_kv_cache* cache,
                               const upr_segments* hist, const void* cand_emb,
                               const upr_segments* cand, float* scores, void* ws,
                               size_t ws_bytes, void* stream) {
    return rank_entry(m, cache, hist, cand_emb, cand, scores, ws, ws_bytes, false, stream);
}

upr_status upr_rank_candidates_noalloc(const upr_model* m, const upr_kv_cache* cache,
                                       const upr_segments* hist, const void* cand_emb,
                                       const upr_segments* cand, float* scores, void* stream) {
    return rank_entry(m, cache, hist, cand_emb, cand, scores, nullptr, 0, true, stream);
}

// ---- per-action heads and utility top-K

static upr_status check_heads_config(const upr_config* cfg, const upr_heads_config* hc) {
    upr_status st = check_config(cfg);
    if (st != UPR_OK) return st;
    if (!hc) return fail(UPR_ERR_NULL, "heads config is NULL");
    if (hc->n_actions < 1 || hc->n_actions > upr::kMaxActions)
        return fail(UPR_ERR_CONFIG, "n_actions %d outside [1, %d]", hc->n_actions, upr::kMaxActions);
    if (hc->hidden < 8 || hc->hidden % 8 != 0 || (int64_t)hc->n_actions * hc->hidden > 8192)
        return fail(UPR_ERR_CONFIG, "hidden %d must be a multiple of 8, >= 8, with n_actions * hidden <= 8192",
                    hc->hidden);
    return UPR_OK;
}

int64_t upr_heads_weights_count(const upr_config* cfg, const upr_heads_config* hc) {
    if (check_heads_config(cfg, hc) != UPR_OK) return -1;
    return (int64_t)hc->n_actions * ((int64_t)hc->hidden * cfg->d_model + 2 * hc->hidden + 1);
}

upr_status upr_heads_create(const upr_model* m, const upr_heads_config* hc,
                            const float* weights_host, int64_t count, upr_heads** out) {
    if (!m) return fail(UPR_ERR_NULL, "model is NULL");
    upr_status st = check_heads_config(&m->cfg, hc);
    if (st != UPR_OK) return st;
    if (!weights_host) return fail(UPR_ERR_NULL, "weights_host is NULL");
    if (!out) return fail(UPR_ERR_NULL, "out is NULL");
    const int64_t need = upr_heads_weights_count(&m->cfg, hc);
    if (count != need)
        return fail(UPR_ERR_WEIGHTS, "heads blob has %lld values, config needs %lld",
                    (long long)count, (long long)need);
    const int64_t d = m->cfg.d_model, C = hc->n_actions, Fh = hc->hidden;
    std::vector<float> W1, b1, w2, b2;
    const float* p = weights_host;
    for (int64_t c = 0; c < C; ++c) {
        W1.insert(W1.end(), p, p + Fh * d); p += Fh * d;
        b1.insert(b1.end(), p, p + Fh); p += Fh;
        w2.insert(w2.end(), p, p + Fh); p += Fh;
        b2.push_back(*p); p += 1;
    }
    ImageBuilder ib{{}, (upr_dtype)m->cfg.dtype};
    upr_heads* hd = new upr_heads();
    const size_t oW1 = ib.add_mat(W1.data(), C * Fh * d, &hd->s_w1);
    const size_t ob1 = ib.add_vec(b1.data(), C * Fh);
    const size_t ow2 = ib.add_vec(w2.data(), C * Fh);
    const size_t ob2 = ib.add_vec(b2.data(), C);
    st = ib.upload(&hd->dev);
    if (st != UPR_OK) {
        delete hd;
        return st;
    }
    char* base = static_cast<char*>(hd->dev);
    hd->cfg = m->cfg;
    hd->C = (int32_t)C;
    hd->Fh = (int32_t)Fh;
    hd->W1 = base + oW1;
    hd->b1 = reinterpret_cast<const float*>(base + ob1);
    hd->w2 = reinterpret_cast<const float*>(base + ow2);
    hd->b2 = reinterpret_cast<const float*>(base + ob2);
    *out = hd;
    return ok();
}

void upr_heads_destroy(upr_heads* hd) {
    if (!hd) return;
    if (hd->dev) (void)hipFree(hd->dev);
    delete hd;
}

static bool same_shape(const upr_config& a, const upr_config& b) {
    return a.d_model == b.d_model && a.n_heads == b.n_heads && a.head_dim == b.head_dim &&
           a.n_layers == b.n_layers && a.d_ff == b.d_ff && a.dtype == b.dtype;
}

size_t upr_rank_actions_workspace_bytes(const upr_model* m, const upr_heads* hd,
                                        const upr_segments* hist, const upr_segments* cand) {
    if (!m || !hd || !same_shape(m->cfg, hd->cfg)) return 0;
    int64_t hf, hl, cf, cl;
    if (check_segments(hist, "hist", &hf, &hl) != UPR_OK) return 0;
    if (check_segments(cand, "cand", &cf, &cl) != UPR_OK) return 0;
    if (hist->num_users != cand->num_users) return 0;
    return upr::plan_rank(m->cfg, cand->num_users, cand->offsets_host, hist->offsets_host,
                          hd->C * hd->Fh).bytes;
}

upr_status upr_rank_actions(const upr_model* m, const upr_heads* hd, const upr_kv_cache* cache,
                            const upr_segments* hist, const void* cand_emb,
                            const upr_segments* cand, const float* utility_weights, float* probs,
                            float* utility, void* ws, size_t ws_bytes, void* stream) {
    if (!m) return fail(UPR_ERR_NULL, "model is NULL");
    if (!hd) return fail(UPR_ERR_NULL, "heads is NULL");
    if (!same_shape(m->cfg, hd->cfg))
        return fail(UPR_ERR_CONFIG, "heads were created for a different model shape");
    int64_t hf, hl, cf, cl;
    upr_status st = check_segments(hist, "hist", &hf, &hl);
    if (st != UPR_OK) return st;
    st = check_segments(cand, "cand", &cf, &cl);
    if (st != UPR_OK) return st;
    if (hist->num_users != cand->num_users)
        return fail(UPR_ERR_OFFSETS, "hist has %d users, cand has %d", hist->num_users,
                    cand->num_users);
    if (!cache) return fail(UPR_ERR_NULL, "cache is NULL");
    if (cache->capacity_rows < 0 || hl > cache->capacity_rows)
        return fail(UPR_ERR_CAPACITY, "history rows end at %lld, cache capacity is %lld",
                    (long long)hl, (long long)cache->capacity_rows);
    if (!utility_weights) return fail(UPR_ERR_NULL, "utility_weights is NULL");
    if (!probs && !utility) return fail(UPR_ERR_NULL, "probs and utility are both NULL");
    if (cl > cf) {
        if (!cand_emb) return fail(UPR_ERR_NULL, "cand_emb is NULL");
        if (hl > hf && !cache->data) return fail(UPR_ERR_NULL, "cache data is NULL");
    }
    const upr::RankPlan p = upr::plan_rank(m->cfg, cand->num_users, cand->offsets_host, hist->offsets_host,
                                           hd->C * hd->Fh);
    st = check_workspace(ws, ws_bytes, p.bytes);
    if (st != UPR_OK) return st;
    if (p.rows == 0) return ok();
    upr::RankOut out;
    out.heads = hd;
    for (int c = 0; c < hd->C; ++c) out.uw.u[c] = utility_weights[c];
    out.probs = probs;
    out.util = utility;
    clear_pending_error();
    arm_stop_hook();
    hipStream_t s = static_cast<hipStream_t>(stream);
    char* w = static_cast<char*>(ws);
    st = bf16_family(m->cfg.dtype)
             ? upr::run_rank<upr::Bf16Types>(m, cache, hist, static_cast<const bf16*>(cand_emb),
                                             cand, out, p, w, s)
             : upr::run_rank<upr::F32Types>(m, cache, hist, static_cast<const float*>(cand_emb),
                                            cand, out, p, w, s);
    return st == UPR_OK ? ok() : st;
}

upr_status upr_topk_by_utility(const float* utility, const upr_segments* cand, int32_t K,
                               int32_t* topk_rows, float* topk_utility, void* stream) {
    static_assert(upr::kTopkMaxCandidates == UPR_TOPK_MAX_CANDIDATES, "limit mismatch");
    int64_t cf, cl;
    upr_status st = check_segments(cand, "cand", &cf, &cl);
    if (st != UPR_OK) return st;
    if (K < 1) return fail(UPR_ERR_LIMIT, "K = %d < 1", K);
    for (int u = 0; u < cand->num_users; ++u) {
        const int32_t k = cand->offsets_host[u + 1] - cand->offsets_host[u];
        if (k > UPR_TOPK_MAX_CANDIDATES)
            return fail(UPR_ERR_LIMIT, "user %d has %d candidates, top-K accepts at most %d", u, k,
                        UPR_TOPK_MAX_CANDIDATES);
    }
    if (cand->num_users == 0) return ok();
    if (!topk_rows) return fail(UPR_ERR_NULL, "topk_rows is NULL");
    if (cl > cf && !utility) return fail(UPR_ERR_NULL, "utility is NULL");
    clear_pending_error();
    hipStream_t s = static_cast<hipStream_t>(stream);
    {
        upr::ProfScope ps("topk", s);
        const hipError_t e = upr::launch_topk(utility, cand->offsets_dev, cand->num_users, K,
                                              topk_rows, topk_utility, cf, cl, s);
        if (e != hipSuccess) return fail(UPR_ERR_HIP, "top-K launch failed: %s", hipGetErrorString(e));
    }
    return ok();
}

// ---- MXFP8 encoding and the scaled fp8 linear map

upr_status upr_mx_quantize_host(const float* x, int64_t rows, int32_t k, uint8_t* codes,
                                uint8_t* scales) {
    if (rows < 0 || k <= 0 || k % 32 != 0)
        return fail(UPR_ERR_LIMIT, "rows %lld / k %d: need rows >= 0 and k a positive multiple of 32",
                    (long long)rows, k);
    if (rows > 0 && (!x || !codes || !scales)) return fail(UPR_ERR_NULL, "x, codes or scales is NULL");
    upr::mx_quantize_host(x, rows, k, codes, scales);
    return ok();
}

upr_status upr_mx_quantize(const void* x, int32_t in_type, int64_t rows, int32_t k, uint8_t* codes,
                           uint8_t* scales, void* stream) {
    if (in_type != UPR_MX_IN_F32 && in_type != UPR_MX_IN_F16 && in_type != UPR_MX_IN_BF16)
        return fail(UPR_ERR_DTYPE, "input type %d is not a upr_mx_input value", in_type);
    if (rows < 0 || k <= 0 || k % 32 != 0)
        return fail(UPR_ERR_LIMIT, "rows %lld / k %d: need rows >= 0 and k a positive multiple of 32",
                    (long long)rows, k);
    if (rows == 0) return ok();
    if (!x || !codes || !scales) return fail(UPR_ERR_NULL, "x, codes or scales is NULL");
    clear_pending_error();
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    {
        upr::ProfScope ps("mx.quantize", s);
        e = in_type == UPR_MX_IN_F32
                ? upr::launch_mx_quantize(static_cast<const float*>(x), rows, k, codes, scales, s)
            : in_type == UPR_MX_IN_F16
                ? upr::launch_mx_quantize(static_cast<const upr::f16*>(x), rows, k, codes, scales, s)
                : upr::launch_mx_quantize(static_cast<const bf16*>(x), rows, k, codes, scales, s);
    }
    if (e != hipSuccess) return fail(UPR_ERR_HIP, "MXFP8 encode launch failed: %s", hipGetErrorString(e));
    return ok();
}

upr_status upr_mx_linear(const uint8_t* a_codes, const uint8_t* a_scales, const uint8_t* w_codes,
                         const uint8_t* w_scales, const float* bias, int64_t M, int32_t N,
                         int32_t K, float* out, void* stream) {
    if (M < 0 || N <= 0 || N % 8 != 0 || K <= 0 || K % 128 != 0)
        return fail(UPR_ERR_LIMIT, "M %lld, N %d, K %d: need M >= 0, N a positive multiple of 8, "
                    "K a positive multiple of 128", (long long)M, N, K);
    if (M == 0) return ok();
    if (!a_codes || !a_scales || !w_codes || !w_scales || !bias || !out)
        return fail(UPR_ERR_NULL, "an operand pointer is NULL");
    upr::Epilogue r{};
    r.mode = upr::EPI_RESID;
    r.acc_scale = 1.0f;
    r.bias = bias;
    r.resid = out;
    r.ldr = N;
    clear_pending_error();
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e;
    {
        upr::ProfScope ps("mx.linear", s);
        e = upr::launch_gemm_mx(a_codes, a_scales, w_codes, w_scales, M, N, K, r, s);
    }
    if (e != hipSuccess) return fail(UPR_ERR_HIP, "MXFP8 GEMM launch failed: %s", hipGetErrorString(e));
    return ok();
}

const char* upr_status_string(int32_t s) {
    switch (s) {
        case UPR_OK: return "ok";
        case UPR_ERR_NULL: return "required pointer is NULL";
        case UPR_ERR_CONFIG: return "unsupported model configuration";
        case UPR_ERR_OFFSETS: return "malformed segment offsets";
        case UPR_ERR_CAPACITY: return "history rows exceed cache capacity";
        case UPR_ERR_WORKSPACE: return "workspace too small or misaligned";
        case UPR_ERR_DTYPE: return "unknown dtype";
        case UPR_ERR_HIP: return "HIP runtime error";
        case UPR_ERR_WEIGHTS: return "weight blob size mismatch";
        case UPR_ERR_LIMIT: return "argument exceeds a documented limit";
        default: return "unknown status";
    }
}

const char* upr_last_error(void) { return g_last_error.c_str(); }

}  // extern "C"
