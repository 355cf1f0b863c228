/*
 * upr.h - C interface of the candidate-ranking library (MI355X / gfx950).
 *
 * The library implements the ranking half of UniPinRec's cross-stage KV-cache
 * sharing (paper Sec. 3, "Overall serving design" and "KV-cache sharing
 * across stages"): a shared transformer encodes each user's action history
 * once and keeps every layer's keys and values; ranking then runs only the
 * candidate tokens through the same transformer, each candidate attending to
 * its user's cached history keys plus its own key and never to another
 * candidate (Sec. 3, "Masked Action Modeling", attention-pattern item), and
 * returns one score per candidate.
 *
 * Conventions shared by every call:
 *   - All functions are extern "C"; no C++ exception crosses this boundary.
 *   - "host" pointers are ordinary CPU memory, "device" pointers are HIP
 *     device memory on the current device.  The caller owns every buffer it
 *     passes; the library never frees or retains them beyond the call (the
 *     kernels it enqueues read/write them until they finish on `stream`).
 *   - `stream` is a hipStream_t passed as void*; NULL means the null stream.
 *     encode/rank enqueue work and return without synchronising.  A fault in
 *     a kernel surfaces at the caller's next synchronisation.
 *   - Arguments are validated on the host before anything is enqueued.  A
 *     validation failure (any status other than UPR_ERR_HIP) means nothing
 *     has been enqueued and no output byte has been written.  UPR_ERR_HIP
 *     reports a failed HIP call or kernel launch; kernels of the same call
 *     enqueued before it may still run and write the call's outputs and
 *     workspace.  A HIP error left pending by the caller's earlier work is
 *     cleared at entry, not reported.  upr_last_error() gives a description
 *     of the last failure (thread-local).
 *   - Row segments: offsets are int32, num_users+1 entries, non-decreasing,
 *     offsets[0] >= 0.  User u owns packed rows offsets[u] .. offsets[u+1]-1.
 *     offsets[0] > 0 is allowed (a call on a sub-range of a shared buffer).
 *     Empty users (equal consecutive offsets) are allowed.
 *     The device copy (offsets_dev) must hold the same values as the host
 *     array while the call's kernels run.  The host array is what the call
 *     validates; kernels that read the device copy check it against the
 *     validated bounds (first and last offset, cache capacity, tile count)
 *     and skip segments that disagree, so a stale device copy
 *     gives meaningless outputs but no access outside the call's buffers.
 *   - A model is immutable after creation and may be used from several host
 *     threads at once; concurrent calls need distinct workspaces and must
 *     not write the same outputs.
 */
#ifndef UPR_H
#define UPR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    UPR_OK = 0,
    UPR_ERR_NULL = 1,       /* a required pointer is NULL                      */
    UPR_ERR_CONFIG = 2,     /* unsupported model shape                         */
    UPR_ERR_OFFSETS = 3,    /* malformed or mismatched segment offsets         */
    UPR_ERR_CAPACITY = 4,   /* history rows exceed the cache capacity          */
    UPR_ERR_WORKSPACE = 5,  /* workspace too small or misaligned               */
    UPR_ERR_DTYPE = 6,      /* unknown arithmetic type                         */
    UPR_ERR_HIP = 7,        /* a HIP runtime call failed                       */
    UPR_ERR_WEIGHTS = 8,    /* weight blob has the wrong number of values      */
    UPR_ERR_LIMIT = 9       /* an argument exceeds a documented limit          */
} upr_status;

typedef enum { UPR_F32 = 0, UPR_BF16 = 1, UPR_BF16_MXFP8 = 2 } upr_dtype;

/* Model shape.  Supported: head_dim in {32, 64}; d_model = n_heads*head_dim,
 * a multiple of 64 and at most 1024; d_ff a multiple of 64 and at most 8192;
 * 1 <= n_layers <= 64.  dtype selects the storage type of tokens and cache
 * and the arithmetic of the model:
 *   UPR_F32:  fp32 throughout.
 *   UPR_BF16: tokens, the K/V cache, queries/keys/values and softmax
 *             probabilities are bf16 (attention contractions are bf16 MFMA);
 *             the operands of the projection GEMMs (LayerNorm outputs,
 *             attention output, FFN hidden, weights) are fp16 (fp16 MFMA,
 *             same peak rate, 3 more significand bits); the residual stream,
 *             normalisation statistics, softmax and every accumulation are
 *             fp32.  Activations entering the projections must stay within
 *             the fp16 range (|x| < 65504).  This is not checked: a value
 *             beyond it becomes an fp16 infinity, and the scores of the rows
 *             it reaches come out non-finite, never silently finite.
 *   UPR_BF16_MXFP8: the UPR_BF16 model (same weight blob, tokens and cache;
 *             encode unchanged) whose ranking layers run their four
 *             projections (Q/K/V, O, FFN up, FFN down) in FP8 (paper Sec. 3,
 *             "FP8 quantization": E4M3 in the forward pass) with OCP
 *             microscaling: every weight row and every projection input row
 *             (LayerNorm outputs, attention output, FFN hidden) is encoded
 *             as E4M3 values with one power-of-two E8M0 scale per 32
 *             consecutive values along the contraction axis (see
 *             upr_mx_quantize_host), and the products accumulate in fp32 on
 *             gfx950's scaled fp8 matrix instructions.  Requires d_model a
 *             multiple of 256 and d_ff a multiple of 128.
 * ln_eps is the LayerNorm epsilon. */
typedef struct {
    int32_t d_model;
    int32_t n_heads;
    int32_t head_dim;
    int32_t n_layers;
    int32_t d_ff;
    int32_t dtype;          /* a upr_dtype value */
    float ln_eps;
} upr_config;

typedef struct upr_model upr_model;     /* opaque */

/* Packed row segments of one call (see the conventions above). */
typedef struct {
    int32_t num_users;
    const int32_t* offsets_host;    /* host, num_users+1 entries              */
    const int32_t* offsets_dev;     /* device, the same num_users+1 values    */
} upr_segments;

/* Packed per-layer K/V cache (device memory, caller-owned).
 * Layout [n_layers][2][n_heads][capacity_rows][head_dim] of the model's dtype:
 * per layer a K plane then a V plane, heads outermost inside a plane, then
 * one row per packed history token (history row r of the encode call is cache
 * row r), then the head's features.  Element (l, kv, h, r, e) sits at
 * upr_kv_cache_index(...).  Each (layer, kv, head, user) block is one
 * contiguous slab of n_u*head_dim elements. */
typedef struct {
    void* data;
    int64_t capacity_rows;
} upr_kv_cache;

/* Number of float values in the weight blob for `cfg`, or -1 if cfg is invalid.
 * Blob order (all float32, linear weights [out, in]), per layer l:
 *   ln1_g[d] ln1_b[d] Wq[d,d] bq[d] Wk[d,d] bk[d] Wv[d,d] bv[d] Wo[d,d] bo[d]
 *   ln2_g[d] ln2_b[d] W1[F,d] b1[F] W2[d,F] b2[d]
 * then lnf_g[d] lnf_b[d] w_score[d] b_score[1]. */
int64_t upr_weights_count(const upr_config* cfg);

/* Create a model: copies the host blob (weights_count floats) to device
 * memory.  For UPR_BF16 every matrix value is rounded to bf16 (nearest, ties
 * to even) -- the model's weights are bf16 -- and stored as fp16 after an
 * exact per-matrix power-of-two scaling (undone in fp32 after each GEMM), so
 * every bf16 weight within 2^29 of its matrix's largest magnitude is kept
 * exactly.  Vectors (gains, shifts, biases, score weights) stay fp32.
 * This is the only call that allocates device memory.  The blob may be freed
 * after return.  *out is set only on UPR_OK. */
upr_status upr_model_create(const upr_config* cfg, const float* weights_host,
                            int64_t weights_count, upr_model** out);

/* Release a model (NULL is ignored).  No call may be using it. */
void upr_model_destroy(upr_model* model);

/* Bytes of a cache with `capacity_rows` rows for cfg (0 if cfg is invalid). */
size_t upr_kv_cache_bytes(const upr_config* cfg, int64_t capacity_rows);

/* Element index of (layer, kv [0 = K, 1 = V], head, row, e) in the cache,
 * computed in int64; -1 if any coordinate is out of range. */
int64_t upr_kv_cache_index(const upr_config* cfg, int64_t capacity_rows, int32_t layer,
                           int32_t kv, int32_t head, int64_t row, int32_t e);

/* Workspace bytes needed by upr_encode_user for `hist` (0 on invalid input). */
size_t upr_encode_workspace_bytes(const upr_model* model, const upr_segments* hist);

/* Workspace bytes needed by upr_rank_candidates (0 on invalid input). */
size_t upr_rank_workspace_bytes(const upr_model* model, const upr_segments* hist,
                                const upr_segments* cand);

/* History encoding (paper Sec. 3, "KV-cache sharing across stages": the
 * O(n^2) history pass whose keys and values ranking reuses).
 * hist_emb: device, [rows, d_model] of the model dtype, row-major, holding the
 * packed history tokens (rows hist->offsets_host[0] .. [num_users]-1 are read).
 * For each user and layer l, the causal transformer (position t attends to
 * positions 0..t of the same user) writes that layer's keys and values of the
 * user's rows into cache plane l.  Only those cache rows are written.
 * ws: device workspace of at least upr_encode_workspace_bytes, 256-byte
 * aligned; its contents are scratch. */
upr_status upr_encode_user(const upr_model* model, const void* hist_emb,
                           const upr_segments* hist, const upr_kv_cache* cache,
                           void* ws, size_t ws_bytes, void* stream);

/* Candidate ranking (paper Sec. 3, "Overall serving design": an incremental
 * forward pass in which only candidate tokens are processed, attending back to
 * the cached history).
 * cand_emb: device, [rows, d_model] of the model dtype; rows
 * cand->offsets_host[0] .. [num_users]-1 are read.  Candidate c of user u
 * attends, at every layer, to the cached keys/values of rows
 * hist->offsets[u] .. hist->offsets[u+1]-1 plus its own key/value, and to no
 * other candidate.  scores: device float32, indexed like cand_emb rows; each
 * row in range receives w . LayerNorm_f(h_c) + b (a raw logit).  The cache is
 * only read, so several rank calls may share one cache.  hist and cand must
 * have the same num_users.  ws: as for encode. */
upr_status upr_rank_candidates(const upr_model* model, const upr_kv_cache* cache,
                               const upr_segments* hist, const void* cand_emb,
                               const upr_segments* cand, float* scores,
                               void* ws, size_t ws_bytes, void* stream);

/* Largest workspace upr_rank_candidates_noalloc can provide (bytes). */
#define UPR_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * ranking as upr_rank_candidates, with the same arguments except the
 * workspace, which comes from a fixed scratch array inside the library
 * (UPR_NOALLOC_SCRATCH_BYTES per GPU, held from the first call on that GPU
 * until the process ends).  Calls needing a larger workspace
 * (upr_rank_workspace_bytes > UPR_NOALLOC_SCRATCH_BYTES; about 5,900
 * candidate rows at d_model 512, d_ff 2048) fail with UPR_ERR_LIMIT before
 * anything is enqueued.  The call allocates nothing (no hipMalloc, hipFree
 * or allocating library routine); its first call on a GPU looks up that
 * GPU's scratch address (UPR_ERR_HIP if the lookup fails).  Every call on one
 * GPU shares that GPU's scratch array, whose contents are the last call's:
 * calls that overlap in time on one GPU (several host threads, or streams
 * that run concurrently) race and must be serialised by the caller.  Nothing
 * in the array needs to start at any particular value.  While the diagnostic
 * profiler (upr_profile_enable) is on, its timing events are created on
 * first use. */
upr_status upr_rank_candidates_noalloc(const upr_model* model, const upr_kv_cache* cache,
                                       const upr_segments* hist, const void* cand_emb,
                                       const upr_segments* cand, float* scores, void* stream);

/* ---------------------------------------------------------------------
 * Cross-process KV-cache pool (paper Sec. 3, "KV-cache sharing across
 * stages": retrieval and ranking run as separate processes; the retrieval
 * process pre-allocates a GPU pool of per-layer K/V slots, exports IPC
 * handles for it to a per-instance file, and the ranking process maps the
 * same allocation and reads the K/V retrieval wrote; slots are reused
 * round-robin).
 * A pool is one device allocation of `slots` caches of capacity_rows rows
 * each, slot-major: slot s is a complete upr_kv_cache (the layout above) at
 * byte offset s * upr_kv_cache_bytes(cfg, capacity_rows), so encode writes
 * a slot and rank reads it in place (no per-request copy).  The allocation
 * is at most UPR_KV_POOL_MAX_BYTES (UPR_ERR_LIMIT otherwise).  The creating
 * process owns the allocation; other processes open it from a handle and
 * must close it before the owner destroys it.  Ordering between processes
 * (encode finished before another process ranks from the slot) is the
 * callers' business, e.g. the owner synchronises its stream before it
 * hands a slot identifier on.
 * --------------------------------------------------------------------- */
typedef struct upr_kv_pool upr_kv_pool;     /* opaque */

#define UPR_KV_POOL_MAX_BYTES (((size_t)2 << 30) - 1)
#define UPR_KV_POOL_MAGIC 0x50525055u       /* "UPRP" */

/* What another process needs to open a pool: plain bytes, fit for a file. */
typedef struct {
    uint32_t magic;             /* UPR_KV_POOL_MAGIC                        */
    int32_t slots;
    int64_t capacity_rows;      /* rows per slot                            */
    uint64_t bytes;             /* size of the allocation                   */
    upr_config cfg;             /* the model shape the slots are laid out for */
    uint8_t ipc[64];            /* hipIpcMemHandle_t of the allocation      */
} upr_kv_pool_handle;

/* Allocate a pool of `slots` >= 1 caches (device memory, contents
 * undefined) on the current device.  *out is set only on UPR_OK. */
upr_status upr_kv_pool_create(const upr_config* cfg, int32_t slots, int64_t capacity_rows,
                              upr_kv_pool** out);

/* The pool's handle (host struct), for upr_kv_pool_open in another process. */
upr_status upr_kv_pool_export(const upr_kv_pool* pool, upr_kv_pool_handle* out);

/* The same handle written to the file `path` (created or replaced whole:
 * written to a temporary name, then renamed). */
upr_status upr_kv_pool_export_file(const upr_kv_pool* pool, const char* path);

/* Map a pool exported by another process (UPR_ERR_CONFIG if the handle is
 * malformed, UPR_ERR_HIP if the mapping fails).  *out is set only on
 * UPR_OK. */
upr_status upr_kv_pool_open(const upr_kv_pool_handle* handle, upr_kv_pool** out);

/* upr_kv_pool_open from a handle file written by upr_kv_pool_export_file. */
upr_status upr_kv_pool_open_file(const char* path, upr_kv_pool** out);

/* The cache of slot `slot` (0 <= slot < slots): data points into the pool
 * (valid until the pool is destroyed), capacity_rows as the pool's. */
upr_status upr_kv_pool_slot(const upr_kv_pool* pool, int32_t slot, upr_kv_cache* out);

/* Next slot of the round-robin order 0, 1, .., slots-1, 0, .. (per pool
 * object, thread-safe); -1 for a NULL pool. */
int32_t upr_kv_pool_next_slot(upr_kv_pool* pool);

/* Shape of the pool: the config, slot count and rows per slot (any output
 * pointer may be NULL). */
upr_status upr_kv_pool_info(const upr_kv_pool* pool, upr_config* cfg, int32_t* slots,
                            int64_t* capacity_rows);

/* Unmap (opened pool) or free (created pool); NULL is ignored.  No call may
 * be using the pool. */
void upr_kv_pool_destroy(upr_kv_pool* pool);

/* ---------------------------------------------------------------------
 * Per-action ranking heads and utility top-K (paper Sec. 3: the ranking
 * objective of Masked Action Modeling gives every action type c = 1..C its
 * own MLP head h_psi_c producing a scalar logit from the transformer's
 * hidden state; the unified L0 + L1 service returns the top K candidates by
 * the heads' utility functions).
 * Readings of the paper fixed here: each head reads z = LayerNorm_f(h) (the
 * model's final LayerNorm, the input of the single score head), has one
 * hidden layer of width `hidden` with tanh-form GELU,
 *   logit_c = w2_c . GELU(W1_c z + b1_c) + b2_c,   p_c = sigmoid(logit_c),
 * and the utility of a candidate is sum_c u_c p_c with caller-given u_c.
 * --------------------------------------------------------------------- */
typedef struct upr_heads upr_heads;     /* opaque */

/* C action heads of width `hidden`.  Supported: 1 <= n_actions <= 8,
 * hidden >= 8, n_actions * hidden a multiple of 8 and at most 8192. */
typedef struct {
    int32_t n_actions;
    int32_t hidden;
} upr_heads_config;

/* Number of float values in a heads blob (-1 if cfg or hc is invalid).
 * Blob order (float32), per head c: W1[hidden, d_model] ([out, in]),
 * b1[hidden], w2[hidden], b2[1]. */
int64_t upr_heads_weights_count(const upr_config* cfg, const upr_heads_config* hc);

/* Create heads for `model` (same device; rounding and storage as the model's
 * weights: bf16 models round every value to bf16 and keep the stacked W1 as
 * fp16 after an exact power-of-two scaling).  Allocates device memory.
 * *out is set only on UPR_OK. */
upr_status upr_heads_create(const upr_model* model, const upr_heads_config* hc,
                            const float* weights_host, int64_t weights_count,
                            upr_heads** out);

/* Release heads (NULL is ignored).  No call may be using them. */
void upr_heads_destroy(upr_heads* heads);

/* Workspace bytes needed by upr_rank_actions (0 on invalid input). */
size_t upr_rank_actions_workspace_bytes(const upr_model* model, const upr_heads* heads,
                                        const upr_segments* hist, const upr_segments* cand);

/* Candidate ranking with the per-action heads: the same forward pass as
 * upr_rank_candidates, then the C heads on LayerNorm_f of each candidate's
 * final hidden state.
 * utility_weights: host float32 [n_actions], the u_c (read during the call).
 * probs: device float32 [rows, n_actions] row-major, indexed like cand_emb
 * rows, receives p_c; may be NULL.  utility: device float32 [rows], indexed
 * like cand_emb rows, receives sum_c u_c p_c; may be NULL (not both NULL).
 * Other arguments as for upr_rank_candidates. */
upr_status upr_rank_actions(const upr_model* model, const upr_heads* heads,
                            const upr_kv_cache* cache, const upr_segments* hist,
                            const void* cand_emb, const upr_segments* cand,
                            const float* utility_weights, float* probs, float* utility,
                            void* ws, size_t ws_bytes, void* stream);

/* Largest candidate count of one user that upr_topk_by_utility accepts. */
#define UPR_TOPK_MAX_CANDIDATES 16384

/* Per-user top K by utility (paper Sec. 3, deployment configurations).
 * utility: device float32, indexed like the candidate rows of `cand` (for
 * example the output of upr_rank_actions).  For each user u, writes row u of
 * topk_rows (device int32 [num_users, K]): the absolute candidate rows of its
 * K highest utilities, highest first; equal utilities keep the lower row
 * first; NaN utilities come after every number; -1 pads rows past the
 * user's candidate count.  topk_utility (device float32 [num_users, K], may
 * be NULL) receives the matching utilities (NaN in padding).  Requires
 * K >= 1 and at most UPR_TOPK_MAX_CANDIDATES candidates per user
 * (UPR_ERR_LIMIT otherwise).  Allocates nothing. */
upr_status upr_topk_by_utility(const float* utility, const upr_segments* cand, int32_t K,
                               int32_t* topk_rows, float* topk_utility, void* stream);

/* ---- MXFP8 encoding (the UPR_BF16_MXFP8 projections' operand format) ----
 * OCP microscaling with E4M3 elements: each row of x [rows, k] (k a positive
 * multiple of 32) is cut into blocks of 32 consecutive values; a block with
 * largest magnitude a gets e = floor(log2 a) - 8 (8 = exponent of E4M3's
 * largest value, 448), at least -127 (-127 also for an all-zero block); its
 * scale byte is e + 127 (E8M0) and each value v becomes the E4M3 code of
 * v / 2^e rounded to the nearest E4M3 value, ties to even, magnitudes above
 * 448 saturated to 448, negative values (also those rounding to zero)
 * keeping the sign bit.  codes is [rows, k] bytes, scales [rows, k / 32]
 * bytes, both row-major.  Input values must be finite. */

/* Host encoding (host pointers, caller-owned).  UPR_ERR_NULL / UPR_ERR_LIMIT
 * (k not a positive multiple of 32, rows < 0). */
upr_status upr_mx_quantize_host(const float* x, int64_t rows, int32_t k, uint8_t* codes,
                                uint8_t* scales);

/* Input element type of upr_mx_quantize. */
typedef enum { UPR_MX_IN_F32 = 0, UPR_MX_IN_F16 = 1, UPR_MX_IN_BF16 = 2 } upr_mx_input;

/* Device encoding on `stream` (device pointers, caller-owned; x of element
 * type in_type, a upr_mx_input value).  Fails (writing nothing) with
 * UPR_ERR_NULL, UPR_ERR_DTYPE or UPR_ERR_LIMIT as the host call.  Allocates
 * nothing. */
upr_status upr_mx_quantize(const void* x, int32_t in_type, int64_t rows, int32_t k,
                           uint8_t* codes, uint8_t* scales, void* stream);

/* out[M, N] += A W^T + bias on the scaled fp8 matrix instructions, A
 * [M, K] and W [N, K] MXFP8 encodings (codes and scales as above, device
 * memory), bias [N] and out [M, N] fp32 (device, row-major, out updated in
 * place).  This is the projection the UPR_BF16_MXFP8 ranking layers run,
 * exposed for testing and for callers with pre-encoded operands.  K a
 * positive multiple of 128, N a positive multiple of 8, M >= 0
 * (UPR_ERR_LIMIT otherwise); NULL pointers give UPR_ERR_NULL.  Allocates
 * nothing. */
upr_status upr_mx_linear(const uint8_t* a_codes, const uint8_t* a_scales, const uint8_t* w_codes,
                         const uint8_t* w_scales, const float* bias, int64_t M, int32_t N,
                         int32_t K, float* out, void* stream);

/* Diagnostics: per-kernel timing with HIP events.  While enabled, encode and
 * rank record a pair of hipEvents on the call's stream around every kernel
 * they launch, labelled with the kernel's name (e.g. "rank.attn").
 * upr_profile_read waits for those events and reports, per name, the number
 * of launches and their summed duration since profiling was last enabled;
 * it returns the number of names (writing at most max_entries to out, which
 * may be NULL).  upr_profile_enable(0/1) discards what was recorded.  The
 * events are created on first use and reused; this path is for measurement,
 * not for serving. */
typedef struct {
    char name[48];
    int64_t launches;
    double total_ms;
} upr_kernel_stat;

upr_status upr_profile_enable(int32_t enable);
int32_t upr_profile_read(upr_kernel_stat* out, int32_t max_entries);

/* Static description of a status code. */
const char* upr_status_string(int32_t status);

/* Description of the last failure on the calling thread ("" if none). */
const char* upr_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* UPR_H */
