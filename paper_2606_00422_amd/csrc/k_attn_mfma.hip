// Attention on the matrix cores for bf16 models with head_dim 64: the
// ranking pass (candidate cross-attention) and the encode pass (causal
// history self-attention) share one kernel.
//
// Ranking (paper Sec. 3: a candidate attends to all of its user's history
// positions and to itself, never to another candidate): for candidate c of
// user u and head h,  o_c = softmax([q_c . K_t]_t<n_u, q_c . k_c) [V; v_c].
// Encode (paper Eq. 2: causal attention over the history, diagonal
// included): for history position i,  o_i = softmax([q_i . K_t]_t<=i) V.
// Queries are pre-scaled by log2(e)/sqrt(D), so the softmax uses exp2.
//
// One workgroup = one work item (user, head, up to 128 candidates or 128
// history rows); four waves of 32 queries (ranking calls over long
// histories: 256 candidates, eight waves, so each K/V stage serves twice the
// queries; calls too small to fill the device: 64 candidates).  The
// user's cached K/V for this layer and head are
// streamed through LDS in 64-key stages (double-buffered, loaded straight
// from global memory into LDS) and shared by all queries of the item.  Per
// 32-key sub-block each wave computes
//   S^T = K Q^T        (v_mfma_f32_16x16x32_bf16, keys x queries),
// so a lane holds 8 logits of ONE query (keys 4g..4g+3 and 16+4g..16+4g+3,
// g = lane/16).  The probabilities, packed to bf16, are directly the B
// operand of
//   O^T += V^T P^T     (e x queries);
// V stays row-major in LDS and the transposing LDS read (ds_read_b64_tr_b16)
// delivers V^T fragments in that same key order.  In the causal pass a wave
// skips sub-blocks that lie entirely after its last query and masks the
// diagonal ones.
//
// Softmax against a fixed reference: each query's reference logit m is its
// own logit q . k_self (ranking: p_self = 1, l = 1, O = v_self to start;
// encode: the diagonal key is one of the streamed keys).  The logit MFMA
// accumulates onto -m, giving s - m directly, and p = 2^(s - m) with no
// running maximum and no rescaling of O: probabilities above 1 are
// accumulated as they are (fp32 sums, bf16 probabilities: relative precision
// does not depend on magnitude), and the normaliser uses the same reference.
// Only overflow can go wrong (a logit about 2^7 above its reference, a range
// no LayerNorm'd model produces); a work item whose sums come out non-finite
// is redone exactly: a first pass finds each query's maximum logit, and the
// second runs against it.  Row sums use v_dot2 over the bf16 probabilities,
// the same values that weight V.
#include "mx.h"
#include "upr_plan.h"

#include <cstdlib>

namespace upr {

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 b8;
typedef __attribute__((ext_vector_type(2))) __bf16 b2;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 b4v;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kD = 64;            // head_dim
constexpr int kKS = 64;           // keys per LDS stage
// 16-query groups per wave: ranking 2 (128 VGPRs, four waves per SIMD: the
// latency of one wave's exponentials and LDS reads hides behind three
// others), or 1 for calls too small to fill the device with 128-candidate
// items (each query's arithmetic is the same either way); the causal pass
// 2 as well (four waves per SIMD; 64 queries per wave, at two waves per
// SIMD, read half the K/V per query but measured 26% slower)
constexpr int kRankQG = 2, kSmallRankQG = 1, kEncodeQG = 2;
static_assert(4 * 16 * kRankQG == kRankAttnTile, "ranking work-list tile must match the kernel");
static_assert(8 * 16 * kRankQG == kLongRankAttnTile, "long-history tile: eight waves of 32 queries");
static_assert(4 * 16 * kSmallRankQG == kSmallRankAttnTile, "small-call tile must match the kernel");
static_assert(4 * 16 * kEncodeQG == kAttnTile, "encode work-list tile must match the kernel");

// LDS layout of a stage: 64 rows (keys) x 128 bytes (64 dims), the eight
// 16-byte chunks of a row XOR-swizzled.  K fragment reads take 16
// consecutive rows at one chunk: key (row / 2) % 8 puts them on distinct bank
// groups.  V transposing reads take 8 consecutive rows x 32 bytes per
// 32-lane pass: key 2 ((row / 2) % 4) keeps the two chunks of a 32-byte pair
// together and puts equal-parity rows on distinct pairs.
__device__ __forceinline__ int key_k(int row) { return (row >> 1) & 7; }
__device__ __forceinline__ int key_v(int row) { return ((row >> 1) & 3) << 1; }

__device__ __forceinline__ float max3(float a, float b, float c) { return fmaxf(a, fmaxf(b, c)); }

// Inf or NaN, tested on the bits (this file is built without NaN semantics).
__device__ __forceinline__ bool nonfinite(float x) {
    return (__float_as_uint(x) & 0x7f800000u) == 0x7f800000u;
}

// 2^x on the transcendental unit (-inf gives 0; 2^128 and above give inf).
__device__ __forceinline__ float fast_exp2(float x) { return __builtin_amdgcn_exp2f(x); }

// Reductions over the four lanes {l, l^16, l^32, l^48} that hold one query:
// v_permlane{16,32}_swap with both operands = v leaves each lane with its own
// value and its xor-partner's, in some order.
__device__ __forceinline__ float pair_max16(float v) {
    const auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float pair_max32(float v) {
    const auto r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return fmaxf(__uint_as_float(r[0]), __uint_as_float(r[1]));
}
__device__ __forceinline__ float quad_sum(float v) {
    auto r = __builtin_amdgcn_permlane16_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    v = __uint_as_float(r[0]) + __uint_as_float(r[1]);
    r = __builtin_amdgcn_permlane32_swap(__float_as_uint(v), __float_as_uint(v), false, false);
    return __uint_as_float(r[0]) + __uint_as_float(r[1]);
}

// CAUSAL = false: ranking; queries are candidate rows of qsrc = q|k|v rows
// (stride 3d, own key and value at +d, +2d).  CAUSAL = true: encode; queries
// are history rows of qsrc = query rows (stride d), own keys in the cache.
// MXO: the output goes out as MXFP8 (codes in `out`, one E8M0 byte per
// 32-value block in `out_scales`), encoded from the fp32 values, for the fp8
// projection variant; else fp16.  kW: waves per workgroup, four, or eight
// for ranking over long histories (256-candidate items, two workgroups per
// CU, so still four waves per SIMD).
template <bool CAUSAL, int kQG, bool MXO = false, int kW = 4>
__global__ __launch_bounds__(64 * kW, kW == 8 ? 2 : (8 / kQG < 4 ? 8 / kQG : 4)) void k_attn_mfma(
    const bf16* __restrict__ qsrc, int64_t qstride, void* __restrict__ out,
    uint8_t* __restrict__ out_scales, int64_t row0, int H, const int4* __restrict__ work,
    const bf16* __restrict__ cache_k, const bf16* __restrict__ cache_v, int64_t cap, int force_exact) {
    // Stages as separate arrays: the compiler can then tell that reads of one
    // stage do not alias the loads filling the other.
    __shared__ __attribute__((aligned(16))) bf16 sK0[kKS * kD];
    __shared__ __attribute__((aligned(16))) bf16 sK1[kKS * kD];
    __shared__ __attribute__((aligned(16))) bf16 sV0[kKS * kD];
    __shared__ __attribute__((aligned(16))) bf16 sV1[kKS * kD];

    constexpr int kQW = 16 * kQG;       // queries per wave
    // the item carries its user's history segment, so nothing here waits on
    // a second dependent load before the first K/V stage can be requested
    const int4 item = work[blockIdx.x];
    const int h = item.w & 0xffff, kc = item.w >> 16;
    if (kc <= 0) return;
    const int64_t c0 = item.z;          // absolute row of the first query
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, l16 = lane & 15;
    const int d = H * kD;
    const int64_t hb = item.x;
    const int n = item.y;
    if (hb < 0 || n < 0 || hb + n > cap) return;   // (never, for an item of the work list)
    // keys streamed: all history (ranking) or positions up to the item's
    // last query (encode); waves past the item's queries only help load
    const int ipos0 = CAUSAL ? (int)(c0 - hb) : 0;
    const int nkeys = CAUSAL ? ipos0 + kc : n;
    // (wave-uniform values made scalar, so the per-wave skips are scalar
    // branches rather than exec-mask updates)
    const bool wave_active = __builtin_amdgcn_readfirstlane((int)(wave * kQW < kc)) != 0;
    const int wave_last = __builtin_amdgcn_readfirstlane(ipos0 + min(wave * kQW + kQW, kc) - 1);
    const int wave_first = __builtin_amdgcn_readfirstlane(ipos0 + wave * kQW);   // encode: first query position

    // ---- history K/V stages, loaded straight into LDS.  Buffer descriptors
    // span the user's n rows, so rows past the history end read as zeros.
    const int nst = (nkeys + kKS - 1) / kKS;
    const __amdgpu_buffer_rsrc_t rsK = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(cache_k + ((int64_t)h * cap + hb) * kD), (short)0, n * kD * 2, 0x00020000);
    const __amdgpu_buffer_rsrc_t rsV = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(cache_v + ((int64_t)h * cap + hb) * kD), (short)0, n * kD * 2, 0x00020000);
    // Each of the kW waves fills kRPW rows of a stage (wave w: rows kRPW w ..)
    // with 8-row loads, two per matrix (four waves) or one (eight); slot s of
    // row r holds logical chunk s ^ key(r).  (Fixed-size arrays: with a
    // template-dependent size the host pass of this compiler drops the
    // kernel's launch stub.)
    constexpr int kRPW = kKS / kW, kLPM = kRPW / 8;
    static_assert(kLPM == 1 || kLPM == 2, "four or eight waves");
    int offK[2], offV[2];
#pragma unroll
    for (int i = 0; i < kLPM; ++i) {
        const int row = kRPW * wave + 8 * i + (lane >> 3), slot = lane & 7;
        offK[i] = row * kD * 2 + ((slot ^ key_k(row)) << 4);
        offV[i] = row * kD * 2 + ((slot ^ key_v(row)) << 4);
    }
    auto issue_loads = [&](bf16* dK, bf16* dV, int st) __attribute__((always_inline)) {
        const int base = st * kKS * kD * 2;
#pragma unroll
        for (int i = 0; i < kLPM; ++i) {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rsK, (__attribute__((address_space(3))) void*)(dK + (kRPW * wave + 8 * i) * kD),
                16, offK[i] + base, 0, 0, 0);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rsV, (__attribute__((address_space(3))) void*)(dV + (kRPW * wave + 8 * i) * kD),
                16, offV[i] + base, 0, 0, 0);
        }
    };

    // The first stage is requested before the queries are loaded, so the two
    // latencies overlap.
    bool first_issued = nst > 0;
    if (first_issued) issue_loads(sK0, sV0, 0);

    // ---- queries of this wave (B operand of S^T), own key/value, initial state
    b8 qf[kQG][2];
    f32x4 negm[kQG];                      // -m of the lane's query, in all four registers
    float l[kQG];                         // lane-partial sums of probabilities
    f32x4 o[kQG][4];                      // O^T: e = 16eb + 4g + r of query l16
    // Loads the queries and starts the softmax against reference
    // max(own logit, mref[qg]) (mref = -inf: the own logit).  Ranking starts
    // from the candidate's own key and value (p_self = 1 against its own
    // logit); encode from nothing (the diagonal key is streamed).
    int qpos[kQG];                        // encode: position of the lane's query
    auto init_state = [&](const float (&mref)[kQG]) __attribute__((always_inline)) {
#pragma unroll
        for (int qg = 0; qg < kQG; ++qg) {
            int qi = wave * kQW + qg * 16 + l16;
            qi = qi < kc ? qi : kc - 1;                  // clamp the ragged tail
            qpos[qg] = ipos0 + qi;
            const bf16* qrow = qsrc + (c0 - row0 + qi) * qstride + h * kD;
            const bf16* krow = CAUSAL ? cache_k + ((int64_t)h * cap + c0 + qi) * kD : qrow + d;
            float s = 0.f;
#pragma unroll
            for (int es = 0; es < 2; ++es) {
                qf[qg][es] = *reinterpret_cast<const b8*>(qrow + es * 32 + 8 * g);
                const b8 kf = *reinterpret_cast<const b8*>(krow + es * 32 + 8 * g);
#pragma unroll
                for (int j = 0; j < 8; ++j) s = fmaf((float)qf[qg][es][j], (float)kf[j], s);
            }
            const float own = quad_sum(s);               // own logit
            const float m0 = fmaxf(own, mref[qg]);
            const float ps = fast_exp2(own - m0);        // 1 unless mref is larger
            negm[qg] = f32x4{-m0, -m0, -m0, -m0};
            if constexpr (CAUSAL) {
                l[qg] = 0.f;
#pragma unroll
                for (int eb = 0; eb < 4; ++eb) o[qg][eb] = f32x4{0.f, 0.f, 0.f, 0.f};
            } else {
                l[qg] = g == 0 ? ps : 0.f;
                const bf16* vrow = qrow + 2 * d;
#pragma unroll
                for (int eb = 0; eb < 4; ++eb) {
                    const bf16* vp = vrow + eb * 16 + 4 * g;
#pragma unroll
                    for (int r = 0; r < 4; ++r) o[qg][eb][r] = ps * (float)vp[r];
                }
            }
        }
    };
    {
        float none[kQG];
#pragma unroll
        for (int qg = 0; qg < kQG; ++qg) none[qg] = -INFINITY;
        init_state(none);
    }

    // One 32-key sub-block (keys kb .. kb+31 of the stage in cK / cV).
    auto sub_block = [&](const bf16* cK, const bf16* cV, int kb, int kabs) __attribute__((always_inline)) {
        if (!wave_active || (CAUSAL && kabs > wave_last)) return;   // nothing to do for this wave
        // S^T - m for 32 keys x 64 queries
        f32x4 s[kQG][2];
        // The MFMA runs of a wave take issue priority over the other wave on
        // its SIMD, whose exponentials then fill the matrix core's gaps.
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            b8 kf[2];
            const int row = kb + t * 16 + l16;
#pragma unroll
            for (int es = 0; es < 2; ++es)
                kf[es] = *reinterpret_cast<const b8*>(&cK[row * kD + (((es * 4 + g) ^ key_k(row)) << 3)]);
#pragma unroll
            for (int qg = 0; qg < kQG; ++qg) {
                f32x4 acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[0], qf[qg][0], negm[qg], 0, 0, 0);
                s[qg][t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[1], qf[qg][1], acc, 0, 0, 0);
            }
        }
        __builtin_amdgcn_s_setprio(0);
        // ranking: mask keys past the history end (last sub-block only);
        // encode: mask keys after the query (diagonal sub-blocks only)
        if (__builtin_expect(CAUSAL ? kabs + 31 > wave_first : kabs + 32 > n, 0)) {
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int key = kabs + t * 16 + 4 * g + r;
#pragma unroll
                    for (int qg = 0; qg < kQG; ++qg)
                        if (CAUSAL ? key > qpos[qg] : key >= n) s[qg][t][r] = -INFINITY;
                }
        }
        b8 pf[kQG];
#pragma unroll
        for (int qg = 0; qg < kQG; ++qg) {
#pragma unroll
            for (int t = 0; t < 2; ++t)
#pragma unroll
                for (int r = 0; r < 4; ++r) pf[qg][t * 4 + r] = (__bf16)fast_exp2(s[qg][t][r]);
            const b2 ones = {(__bf16)1.0f, (__bf16)1.0f};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const b2 pp = {pf[qg][2 * j], pf[qg][2 * j + 1]};
                l[qg] = __builtin_amdgcn_fdot2_f32_bf16(pp, ones, l[qg], false);
            }
        }
        // O^T += V^T P^T.  V^T fragment of e-block eb: lane (g, i) needs
        // V[key(8g + j)][16eb + i]; in each 16-lane group, lane s of a
        // transposing read addresses row 4g + s/4 (+16), dims 16eb + 4(s%4).
        __builtin_amdgcn_s_setprio(1);
#pragma unroll
        for (int eb = 0; eb < 4; ++eb) {
            b8 vf;
#pragma unroll
            for (int hh = 0; hh < 2; ++hh) {
                const int row = kb + 16 * hh + 4 * g + (l16 >> 2);
                const int ch = 2 * eb + ((l16 & 3) >> 1);
                const bf16* p = &cV[row * kD + ((ch ^ key_v(row)) << 3) + ((l16 & 1) << 2)];
                const b4v v4 = __builtin_amdgcn_ds_read_tr16_b64_v4bf16(
                    (__attribute__((address_space(3))) b4v*)(p));
#pragma unroll
                for (int j = 0; j < 4; ++j) vf[4 * hh + j] = v4[j];
            }
#pragma unroll
            for (int qg = 0; qg < kQG; ++qg)
                o[qg][eb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[qg], o[qg][eb], 0, 0, 0);
        }
        __builtin_amdgcn_s_setprio(0);
    };

    auto stage = [&](const bf16* cK, const bf16* cV, bf16* nK, bf16* nV, int st) __attribute__((always_inline)) {
        if (st + 1 < nst) issue_loads(nK, nV, st + 1);
        const int k0 = st * kKS;
        sub_block(cK, cV, 0, k0);
        if (k0 + 32 < nkeys) sub_block(cK, cV, 32, k0 + 32);
        __builtin_amdgcn_s_waitcnt(0x0F70);      // vmcnt(0): next stage landed
        __syncthreads();
    };

    auto run = [&]() __attribute__((always_inline)) {
        if (nst > 0) {
            if (!first_issued) issue_loads(sK0, sV0, 0);    // (the exact redo's second pass)
            first_issued = false;
            __builtin_amdgcn_s_waitcnt(0x0F70);
        }
        __syncthreads();
        int st = 0;
        for (; st + 2 <= nst; st += 2) {
            stage(sK0, sV0, sK1, sV1, st);
            stage(sK1, sV1, sK0, sV0, st + 1);
        }
        if (st < nst) stage(sK0, sV0, sK1, sV1, st);
    };
    run();

    // ---- exact redo (pathological logit ranges only): if a probability or
    // a sum overflowed (a logit more than ~2^7 above its reference), find each
    // query's exact maximum logit over its history first, then run again
    // against it, so no probability exceeds 1.
    bool bad = force_exact != 0;
#pragma unroll
    for (int qg = 0; qg < kQG; ++qg) {
        bad |= nonfinite(l[qg]);
#pragma unroll
        for (int eb = 0; eb < 4; ++eb)
#pragma unroll
            for (int r = 0; r < 4; ++r) bad |= nonfinite(o[qg][eb][r]);
    }
    if (__syncthreads_or(bad)) {
        float mref[kQG];
#pragma unroll
        for (int qg = 0; qg < kQG; ++qg) mref[qg] = -INFINITY;
        for (int st = 0; st < nst; ++st) {
            issue_loads(sK0, sV0, st);
            __builtin_amdgcn_s_waitcnt(0x0F70);
            __syncthreads();
            for (int kb = 0; kb < kKS && st * kKS + kb < nkeys; kb += 16) {
                b8 kf[2];
                const int row = kb + l16;
#pragma unroll
                for (int es = 0; es < 2; ++es)
                    kf[es] = *reinterpret_cast<const b8*>(&sK0[row * kD + (((es * 4 + g) ^ key_k(row)) << 3)]);
#pragma unroll
                for (int qg = 0; qg < kQG; ++qg) {
                    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[0], qf[qg][0], acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[1], qf[qg][1], acc, 0, 0, 0);
                    float mx = -INFINITY;
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int key = st * kKS + kb + 4 * g + r;
                        if (CAUSAL ? key <= qpos[qg] : key < n) mx = fmaxf(mx, acc[r]);
                    }
                    mref[qg] = fmaxf(mref[qg], pair_max32(pair_max16(mx)));
                }
            }
            __syncthreads();
        }
        init_state(mref);
        run();
    }

    // ---- normalise and store (lane holds e = 16eb + 4g + r of query l16)
#pragma unroll
    for (int qg = 0; qg < kQG; ++qg) {
        const int qi = wave * kQW + qg * 16 + l16;
        const float lt = quad_sum(l[qg]);
        const float inv = 1.0f / lt;
        const int64_t orow = c0 - row0 + qi;
        if constexpr (!MXO) {
            if (qi >= kc) continue;
            f16* op = static_cast<f16*>(out) + orow * d + h * kD;
#pragma unroll
            for (int eb = 0; eb < 4; ++eb) {
                typedef __attribute__((ext_vector_type(4))) _Float16 h4;
                h4 v;
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = (f16)keep_f32(o[qg][eb][r] * inv);
                *reinterpret_cast<h4*>(op + eb * 16 + 4 * g) = v;
            }
        } else {
            // MXFP8 encoding of the normalised fp32 values (no narrower
            // intermediate): a head's 64 values are blocks 2h and 2h + 1 of
            // the row (e < 32 and e >= 32, i.e. eb < 2 and eb >= 2), each
            // spread over the query's four lanes.
            float am[2] = {0.f, 0.f};
#pragma unroll
            for (int eb = 0; eb < 4; ++eb)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    o[qg][eb][r] = keep_f32(o[qg][eb][r] * inv);
                    am[eb >> 1] = fmaxf(am[eb >> 1], fabsf(o[qg][eb][r]));
                }
#pragma unroll
            for (int b = 0; b < 2; ++b) am[b] = pair_max32(pair_max16(am[b]));
            if (qi >= kc) continue;
            const int e[2] = {mx_block_exp(am[0]), mx_block_exp(am[1])};
            uint8_t* cp = static_cast<uint8_t*>(out) + orow * d + h * kD;
#pragma unroll
            for (int eb = 0; eb < 4; ++eb) {
                const float sc = mx_inv_scale(e[eb >> 1]);
                *reinterpret_cast<uint32_t*>(cp + eb * 16 + 4 * g) =
                    mx_pack4(o[qg][eb][0] * sc, o[qg][eb][1] * sc, o[qg][eb][2] * sc, o[qg][eb][3] * sc);
            }
            if (g < 2) out_scales[orow * (d / kMxBlock) + h * (kD / kMxBlock) + g] = (uint8_t)(e[g] + 127);
        }
    }
}

// Work list: users ordered by history length (longest first, ties by index)
// when there are at most kSortMax users, else in index order.  Items of user
// u (rank r) occupy H * start_r .. H * (start_r + tiles_u) - 1, item
// H*(start_r + j) + h being tile j of head h (tile tiles_u - 1 - j when
// `reverse`: the causal pass puts a user's costliest, last tiles first), so
// with H = 8 all tiles of one (user, head) share blockIdx % 8 and therefore
// one XCD's L2.  Tiles cover the rows of `coffs` (candidates, or the history
// itself for the causal pass).  An item is (first history row of its user,
// history length, first query row, head | query count << 16).
//
// The offsets are read from device memory, which the caller promises holds
// the host values the call validated.  The kernel checks that promise
// before it writes an item: `coffs` non-decreasing from row_first to
// row_last, `hoffs` non-decreasing within [0, cap], and the tile count equal
// to the one sized on the host.  If any check fails, every item is written
// empty (no queries), so the attention launches touch nothing outside the
// call's buffers (the call's outputs are then meaningless, as the contract
// says for inconsistent offsets).
constexpr int kSortMax = 2048;

__global__ __launch_bounds__(1024) void k_rank_worklist(const int32_t* __restrict__ coffs,
                                                        const int32_t* __restrict__ hoffs, int U,
                                                        int H, int tile, int reverse,
                                                        int4* __restrict__ work, int64_t items,
                                                        int64_t row_first, int64_t row_last,
                                                        int64_t cap) {
    constexpr int kWaves = 1024 / 64;
    __shared__ int s_len[kSortMax];
    __shared__ int s_user[kSortMax];      // user at each rank
    __shared__ int s_scan[1024];          // inclusive scan of tiles over the chunk's ranks
    __shared__ int4 s_seg[1024];          // per rank of the chunk: history start and length, candidate start and count
    __shared__ long long s_wtot[kWaves];
    __shared__ int s_wsum[kWaves];
    __shared__ long long s_carry;
    const int tid = threadIdx.x, lane = tid & 63, wv = tid >> 6;
    {
        bool bad = false;
        long long tiles = 0;
        for (int u = tid; u < U; u += 1024) {
            const int64_t c0 = coffs[u], c1 = coffs[u + 1], h0 = hoffs[u], h1 = hoffs[u + 1];
            bad |= c1 < c0 || h0 < 0 || h1 < h0 || h1 > cap;
            if (c1 >= c0) tiles += (c1 - c0 + tile - 1) / tile;
        }
        if (tid == 0) bad |= coffs[0] != row_first || coffs[U] != row_last;
        // the tile total: wave sums, then thread 0 adds the waves'
#pragma unroll
        for (int off = 32; off > 0; off >>= 1) tiles += __shfl_xor(tiles, off, 64);
        if (lane == 0) s_wtot[wv] = tiles;
        __syncthreads();
        if (tid == 0) {
            long long t = 0;
            for (int w = 0; w < kWaves; ++w) t += s_wtot[w];
            bad |= t > (1ll << 40) || t * H != items;
        }
        if (__syncthreads_or(bad)) {
            for (int64_t i = tid; i < items; i += 1024) work[i] = make_int4(0, 0, 0, 0);
            return;
        }
    }
    const bool sorted = U <= kSortMax;
    if (sorted) {
        for (int u = tid; u < U; u += 1024) s_len[u] = hoffs[u + 1] - hoffs[u];
        __syncthreads();
        for (int u = tid; u < U; u += 1024) {
            const int nu = s_len[u];
            int rank = 0;
            for (int v = 0; v < U; ++v) {
                const int nv = s_len[v];
                rank += (nv > nu) || (nv == nu && v < u);
            }
            s_user[rank] = u;
        }
        __syncthreads();
    }
    if (tid == 0) s_carry = 0;
    __syncthreads();
    // Chunks of 1024 ranks: each thread reads its rank's segments once, the
    // tile counts are scanned (within waves by shuffles, then across the
    // sixteen wave totals), and each thread writes the H items of its tiles,
    // finding a tile's rank by binary search on the scan.
    for (int base = 0; base < U; base += 1024) {
        const int r = base + tid;
        int t = 0;
        int4 seg = make_int4(0, 0, 0, 0);
        if (r < U) {
            const int u = sorted ? s_user[r] : r;
            const int c0 = coffs[u], h0 = hoffs[u];
            seg = make_int4(h0, hoffs[u + 1] - h0, c0, coffs[u + 1] - c0);
            t = (seg.w + tile - 1) / tile;
        }
        s_seg[tid] = seg;
        int v = t;
#pragma unroll
        for (int off = 1; off < 64; off <<= 1) {
            const int y = __shfl_up(v, off, 64);
            if (lane >= off) v += y;
        }
        if (lane == 63) s_wsum[wv] = v;
        __syncthreads();
        for (int w = 0; w < wv; ++w) v += s_wsum[w];
        s_scan[tid] = v;
        __syncthreads();
        const int total = s_scan[1023];                 // tiles of this chunk
        const int nr = min(1024, U - base);             // ranks of this chunk
        for (int x = tid; x < total; x += 1024) {
            int lo = 0, hi = nr - 1;                    // smallest rank with s_scan > x
            while (lo < hi) {
                const int mid = (lo + hi) >> 1;
                if (s_scan[mid] > x) hi = mid; else lo = mid + 1;
            }
            const int4 sg = s_seg[lo];
            const int tr = s_scan[lo] - (lo > 0 ? s_scan[lo - 1] : 0);
            const int j = x - (s_scan[lo] - tr);
            const int tt = reverse ? tr - 1 - j : j;
            const int cnt = min(tile, sg.w - tt * tile);
            const long long idx0 = (long long)H * (s_carry + x);
            for (int hh = 0; hh < H; ++hh)
                if (idx0 + hh < items) work[idx0 + hh] = make_int4(sg.x, sg.y, sg.z + tt * tile, hh | (cnt << 16));
        }
        __syncthreads();
        if (tid == 0) s_carry += total;
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_attn_worklist(const int32_t* row_offsets, const int32_t* hist_offsets, int U,
                                int H, int tile, bool reverse, int32_t* work, int64_t items,
                                int64_t row_first, int64_t row_last, int64_t cap, hipStream_t s) {
    if (items == 0) return hipSuccess;
    k_rank_worklist<<<1, 1024, 0, s>>>(row_offsets, hist_offsets, U, H, tile, reverse ? 1 : 0,
                                       reinterpret_cast<int4*>(work), items, row_first, row_last, cap);
    return hipGetLastError();
}

// UPR_ATTN_EXACT=1 sends every work item through the exact two-pass redo (a
// testing hook for that path).
static int force_exact_flag() {
    const char* e = std::getenv("UPR_ATTN_EXACT");
    return e != nullptr && e[0] == '1';
}

hipError_t launch_attn_rank(const bf16* qkv, f16* o, int64_t row0, int H, int D,
                            const int32_t* work, int64_t items,
                            int tile, const bf16* cache_k, const bf16* cache_v, int64_t cache_cap,
                            hipStream_t s) {
    if (items == 0) return hipSuccess;
    if (D != kD || (tile != kLongRankAttnTile && tile != kRankAttnTile && tile != kSmallRankAttnTile))
        return hipErrorInvalidValue;
    const int4* w = reinterpret_cast<const int4*>(work);
    const int64_t ld = (int64_t)3 * H * kD;
    if (tile == kLongRankAttnTile)
        k_attn_mfma<false, kRankQG, false, 8><<<(unsigned)items, 512, 0, s>>>(
            qkv, ld, o, nullptr, row0, H, w, cache_k, cache_v, cache_cap, force_exact_flag());
    else if (tile == kRankAttnTile)
        k_attn_mfma<false, kRankQG><<<(unsigned)items, 256, 0, s>>>(
            qkv, ld, o, nullptr, row0, H, w, cache_k, cache_v, cache_cap, force_exact_flag());
    else
        k_attn_mfma<false, kSmallRankQG><<<(unsigned)items, 256, 0, s>>>(
            qkv, ld, o, nullptr, row0, H, w, cache_k, cache_v, cache_cap, force_exact_flag());
    return hipGetLastError();
}

hipError_t launch_attn_rank_mx(const bf16* qkv, uint8_t* codes, uint8_t* scales, int64_t row0,
                               int H, int D, const int32_t* work,
                               int64_t items, int tile, const bf16* cache_k, const bf16* cache_v,
                               int64_t cache_cap, hipStream_t s) {
    if (items == 0) return hipSuccess;
    if (D != kD || (tile != kLongRankAttnTile && tile != kRankAttnTile && tile != kSmallRankAttnTile) ||
        scales == nullptr)
        return hipErrorInvalidValue;
    const int4* w = reinterpret_cast<const int4*>(work);
    const int64_t ld = (int64_t)3 * H * kD;
    if (tile == kLongRankAttnTile)
        k_attn_mfma<false, kRankQG, true, 8><<<(unsigned)items, 512, 0, s>>>(
            qkv, ld, codes, scales, row0, H, w, cache_k, cache_v, cache_cap, force_exact_flag());
    else if (tile == kRankAttnTile)
        k_attn_mfma<false, kRankQG, true><<<(unsigned)items, 256, 0, s>>>(
            qkv, ld, codes, scales, row0, H, w, cache_k, cache_v, cache_cap, force_exact_flag());
    else
        k_attn_mfma<false, kSmallRankQG, true><<<(unsigned)items, 256, 0, s>>>(
            qkv, ld, codes, scales, row0, H, w, cache_k, cache_v, cache_cap, force_exact_flag());
    return hipGetLastError();
}

hipError_t launch_attn_encode(const bf16* q, f16* o, int64_t row0, int H, int D,
                              const int32_t* work, int64_t items,
                              int tile, const bf16* cache_k, const bf16* cache_v,
                              int64_t cache_cap, hipStream_t s) {
    if (items == 0) return hipSuccess;
    if (D != kD || tile != kAttnTile) return hipErrorInvalidValue;
    k_attn_mfma<true, kEncodeQG><<<(unsigned)items, 256, 0, s>>>(
        q, (int64_t)H * kD, o, nullptr, row0, H, reinterpret_cast<const int4*>(work), cache_k,
        cache_v, cache_cap, force_exact_flag());
    return hipGetLastError();
}

}  // namespace upr
