// Candidate cross-attention on the matrix cores (bf16, head_dim 64).
//
// For candidate c of user u and head h (paper Sec. 3: a candidate attends to
// all of its user's history positions and to itself, never to another
// candidate):  o_c = softmax([q_c . K_t]_t<n_u, q_c . k_c) [V; v_c],
// with q pre-scaled by log2(e)/sqrt(D) so the softmax uses exp2.
//
// One workgroup = one work item (user, head, up to 256 candidates); four
// waves of 64 candidates.  The user's cached K/V for this layer and head are
// streamed through LDS in 64-key stages (double-buffered) and shared by all
// 256 candidates of the item.  Per 32-key sub-block each wave computes
//   S^T = K Q^T        (v_mfma_f32_16x16x32_bf16, keys x queries),
// so a lane holds 8 logits of ONE query (keys 4g..4g+3 and 16+4g..16+4g+3,
// g = lane/16); the running max / sum of a query need only 2 cross-lane
// steps.  The probabilities, packed to bf16, are directly the B operand of
//   O^T += V^T P^T     (e x queries),
// provided V^T's columns in LDS follow the same key order, which the staging
// transpose writes.  The online softmax starts from the candidate's own
// logit and value (m = s_self, l = 1, O = v_self), then folds in history.
#include "upr_plan.h"

namespace upr {

namespace {

typedef __attribute__((ext_vector_type(8))) __bf16 b8;
typedef __attribute__((ext_vector_type(4))) float f32x4;

constexpr int kD = 64;            // head_dim
constexpr int kQW = 64;           // queries per wave
constexpr int kTQ = 4 * kQW;      // queries per work item
constexpr int kKS = 64;           // keys per LDS stage
static_assert(kTQ == kRankAttnTile, "work-list tile must match the kernel");

// LDS element offset of 16-byte chunk `ch` of 128-byte row `row`, XOR-swizzled.
__device__ __forceinline__ int swz(int row, int ch) { return row * 64 + ((ch ^ (row & 7)) << 3); }

// Column of key kk (0..63 inside a stage) in the transposed V tile: key order
// of the PV B-operand (k-index 8g+j <-> key 4g+j for j<4, 16+4g+(j-4) for j>=4,
// within each 32-key half).
__device__ __forceinline__ int vcol(int kk) {
    const int half = kk >> 5, k = kk & 31;
    const int hi = k >> 4, kr = k & 15;
    return half * 32 + ((kr >> 2) << 3) + (hi << 2) + (kr & 3);
}

__device__ __forceinline__ float max3(float a, float b, float c) { return fmaxf(a, fmaxf(b, c)); }

// 2^x on the transcendental unit.  Softmax arguments are <= 0; results below
// 2^-126 flush to zero, which is what a probability that small contributes.
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



__global__ __launch_bounds__(256, 2) void k_attn_rank(
    const bf16* __restrict__ qkv, f16* __restrict__ out, int64_t row0, int H,
    const int32_t* __restrict__ hist_offsets, const int4* __restrict__ work,
    const bf16* __restrict__ cache_k, const bf16* __restrict__ cache_v, int64_t cap) {
    __shared__ __attribute__((aligned(16))) bf16 sK[2][kKS * kD];
    __shared__ __attribute__((aligned(16))) bf16 sV[2][kD * kKS];   // transposed: [e][key col]

    const int4 item = work[blockIdx.x];
    const int u = item.x, h = item.y, kc = item.w;
    if (kc <= 0) return;
    const int64_t c0 = item.z;          // absolute first candidate row
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, l16 = lane & 15;
    const int d = H * kD;
    const int64_t hb = hist_offsets[u];
    const int n = hist_offsets[u + 1] - hist_offsets[u];
    const bf16* Kh = cache_k + ((int64_t)h * cap + hb) * kD;
    const bf16* Vh = cache_v + ((int64_t)h * cap + hb) * kD;

    // ---- queries of this wave (B operand of S^T), own key/value, initial state
    b8 qf[4][2];
    float m[4], l[4];
    f32x4 o[4][4];
#pragma unroll
    for (int qg = 0; qg < 4; ++qg) {
        int qi = wave * kQW + qg * 16 + l16;
        qi = qi < kc ? qi : kc - 1;                      // clamp the ragged tail
        const bf16* qrow = qkv + (c0 - row0 + qi) * (int64_t)(3 * d) + h * kD;
        const bf16* krow = qrow + d;
        const bf16* vrow = qrow + 2 * d;
        float s = 0.f;
#pragma unroll
        for (int es = 0; es < 2; ++es) {
            qf[qg][es] = *reinterpret_cast<const b8*>(qrow + es * 32 + 8 * g);
            const b8 kf = *reinterpret_cast<const b8*>(krow + es * 32 + 8 * g);
#pragma unroll
            for (int j = 0; j < 8; ++j) s = fmaf((float)qf[qg][es][j], (float)kf[j], s);
        }
        m[qg] = quad_sum(s);                             // own logit
        l[qg] = g == 0 ? 1.f : 0.f;                      // lane-partial sum
#pragma unroll
        for (int eb = 0; eb < 4; ++eb) {
            const bf16* vp = vrow + eb * 16 + 4 * g;
#pragma unroll
            for (int r = 0; r < 4; ++r) o[qg][eb][r] = (float)vp[r];
        }
    }

    // ---- history K/V stages
    const int nst = (n + kKS - 1) / kKS;
    // K staging: thread loads 16-byte chunk (tid&7) of key rows tid>>3 and (tid>>3)+32.
    // V staging: thread loads e-chunk (tid>>5) of keys 2*(tid&31) and 2*(tid&31)+1.
    uint4 rk[2], rv[2];
    auto gload = [&](int st) {
        const int k0 = st * kKS;
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int key = (tid >> 3) + 32 * i;
            rk[i] = k0 + key < n ? *reinterpret_cast<const uint4*>(Kh + (int64_t)(k0 + key) * kD + (tid & 7) * 8)
                                 : make_uint4(0, 0, 0, 0);
            const int vkey = 2 * (tid & 31) + i;
            rv[i] = k0 + vkey < n ? *reinterpret_cast<const uint4*>(Vh + (int64_t)(k0 + vkey) * kD + (tid >> 5) * 8)
                                  : make_uint4(0, 0, 0, 0);
        }
    };
    auto swrite = [&](int buf) {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
            const int key = (tid >> 3) + 32 * i;
            *reinterpret_cast<uint4*>(&sK[buf][swz(key, tid & 7)]) = rk[i];
        }
        // transpose V: (V[k][e], V[k+1][e]) -> one dword at column vcol(k) of row e
        const int kk = 2 * (tid & 31), col = vcol(kk), e0 = (tid >> 5) * 8;
        const uint32_t* a = reinterpret_cast<const uint32_t*>(&rv[0]);
        const uint32_t* b = reinterpret_cast<const uint32_t*>(&rv[1]);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const uint32_t pair = __builtin_amdgcn_perm(b[j >> 1], a[j >> 1],
                                                        (j & 1) ? 0x07060302u : 0x05040100u);
            const int e = e0 + j;
            *reinterpret_cast<uint32_t*>(&sV[buf][swz(e, col >> 3) + (col & 7)]) = pair;
        }
    };

    if (nst > 0) {
        gload(0);
        swrite(0);
    }
    __syncthreads();
    for (int st = 0; st < nst; ++st) {
        const int buf = st & 1;
        if (st + 1 < nst) gload(st + 1);
#pragma unroll
        for (int sub = 0; sub < 2; ++sub) {
            const int kbase = st * kKS + sub * 32;
            if (kbase >= n) break;
            // S^T for 32 keys x 64 queries
            f32x4 s[4][2];
#pragma unroll
            for (int t = 0; t < 2; ++t) {
                b8 kf[2];
#pragma unroll
                for (int es = 0; es < 2; ++es)
                    kf[es] = *reinterpret_cast<const b8*>(&sK[buf][swz(sub * 32 + t * 16 + l16, es * 4 + g)]);
#pragma unroll
                for (int qg = 0; qg < 4; ++qg) {
                    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[0], qf[qg][0], acc, 0, 0, 0);
                    acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(kf[1], qf[qg][1], acc, 0, 0, 0);
                    s[qg][t] = acc;
                }
            }
            // mask keys past the history end (last sub-block only; kept off the
            // steady-state path as an unlikely branch)
            if (__builtin_expect(kbase + 32 > n, 0)) {
#pragma unroll
                for (int t = 0; t < 2; ++t)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const bool dead = kbase + t * 16 + 4 * g + r >= n;
#pragma unroll
                        for (int qg = 0; qg < 4; ++qg)
                            if (dead) s[qg][t][r] = -INFINITY;
                    }
            }
            // online softmax update
            float alpha[4];
            bool grew = false;
            b8 pf[4];
#pragma unroll
            for (int qg = 0; qg < 4; ++qg) {
                float mx = max3(s[qg][0][0], s[qg][0][1], s[qg][0][2]);
                mx = max3(mx, s[qg][0][3], s[qg][1][0]);
                mx = max3(mx, s[qg][1][1], s[qg][1][2]);
                mx = fmaxf(mx, s[qg][1][3]);
                mx = pair_max32(pair_max16(mx));
                const float mn = fmaxf(m[qg], mx);
                grew |= mn > m[qg];
                alpha[qg] = fast_exp2(m[qg] - mn);
                m[qg] = mn;
                float sum = 0.f;
#pragma unroll
                for (int t = 0; t < 2; ++t)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const float p = fast_exp2(s[qg][t][r] - mn);
                        sum += p;
                        pf[qg][t * 4 + r] = (__bf16)p;
                    }
                l[qg] = fmaf(l[qg], alpha[qg], sum);
            }
            if (__any(grew)) {
#pragma unroll
                for (int qg = 0; qg < 4; ++qg)
#pragma unroll
                    for (int eb = 0; eb < 4; ++eb)
#pragma unroll
                        for (int r = 0; r < 4; ++r) o[qg][eb][r] *= alpha[qg];
            }
            // O^T += V^T P^T
#pragma unroll
            for (int eb = 0; eb < 4; ++eb) {
                const b8 vf = *reinterpret_cast<const b8*>(&sV[buf][swz(eb * 16 + l16, sub * 4 + g)]);
#pragma unroll
                for (int qg = 0; qg < 4; ++qg)
                    o[qg][eb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(vf, pf[qg], o[qg][eb], 0, 0, 0);
            }
        }
        if (st + 1 < nst) swrite(buf ^ 1);
        __syncthreads();
    }

    // ---- normalise and store (lane holds e = 16eb + 4g + r of query l16)
#pragma unroll
    for (int qg = 0; qg < 4; ++qg) {
        const int qi = wave * kQW + qg * 16 + l16;
        const float lt = quad_sum(l[qg]);
        if (qi >= kc) continue;
        const float inv = 1.0f / lt;
        f16* orow = out + (c0 - row0 + qi) * (int64_t)d + h * kD;
#pragma unroll
        for (int eb = 0; eb < 4; ++eb) {
            typedef __attribute__((ext_vector_type(4))) _Float16 h4;
            h4 v;
#pragma unroll
            for (int r = 0; r < 4; ++r) v[r] = (f16)keep_f32(o[qg][eb][r] * inv);
            *reinterpret_cast<h4*>(orow + eb * 16 + 4 * g) = v;
        }
    }
}

// Work list: users ordered by history length (longest first, ties by index)
// when there are at most kSortMax users, else in index order.  Items of user
// u (rank r) occupy H * start_r .. H * (start_r + tiles_u) - 1, item
// H*(start_r + t) + h being tile t of head h, so with H = 8 all tiles of one
// (user, head) share blockIdx % 8 and therefore one XCD's L2.
constexpr int kSortMax = 2048;

__global__ __launch_bounds__(1024) void k_rank_worklist(const int32_t* __restrict__ coffs,
                                                        const int32_t* __restrict__ hoffs, int U,
                                                        int H, int tile, int4* __restrict__ work,
                                                        int64_t items) {
    __shared__ int s_len[kSortMax];
    __shared__ int s_tiles[kSortMax];     // tiles of the user at each rank
    __shared__ int s_user[kSortMax];      // user at each rank
    __shared__ int s_scan[1024];
    __shared__ long long s_carry;
    const int tid = threadIdx.x;
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
            s_tiles[rank] = (coffs[u + 1] - coffs[u] + tile - 1) / tile;
        }
        __syncthreads();
    }
    if (tid == 0) s_carry = 0;
    __syncthreads();
    // chunked exclusive scan of tiles in rank order; each rank then writes its items
    for (int base = 0; base < U; base += 1024) {
        const int r = base + tid;
        int u = -1, t = 0;
        if (r < U) {
            u = sorted ? s_user[r] : r;
            t = sorted ? s_tiles[r] : (coffs[r + 1] - coffs[r] + tile - 1) / tile;
        }
        s_scan[tid] = t;
        __syncthreads();
        for (int off = 1; off < 1024; off <<= 1) {
            const int v = tid >= off ? s_scan[tid - off] : 0;
            __syncthreads();
            s_scan[tid] += v;
            __syncthreads();
        }
        const long long start = s_carry + s_scan[tid] - t;
        if (u >= 0) {
            const int k = coffs[u + 1] - coffs[u];
            for (int j = 0; j < t; ++j)
                for (int hh = 0; hh < H; ++hh) {
                    const long long idx = (long long)H * (start + j) + hh;
                    if (idx < items) {
                        const int cnt = min(tile, k - j * tile);
                        work[idx] = make_int4(u, hh, coffs[u] + j * tile, cnt);
                    }
                }
        }
        __syncthreads();
        if (tid == 1023) s_carry += s_scan[1023];
        __syncthreads();
    }
}

}  // namespace

hipError_t launch_rank_worklist(const int32_t* cand_offsets, const int32_t* hist_offsets, int U,
                                int H, int tile, int32_t* work, int64_t items, hipStream_t s) {
    if (items == 0) return hipSuccess;
    k_rank_worklist<<<1, 1024, 0, s>>>(cand_offsets, hist_offsets, U, H, tile,
                                       reinterpret_cast<int4*>(work), items);
    return hipGetLastError();
}

hipError_t launch_attn_rank(const bf16* qkv, f16* o, int64_t row0, int H, int D,
                            const int32_t* cand_offsets, const int32_t* hist_offsets,
                            const int32_t* work, int64_t items, int tile, const bf16* cache_k,
                            const bf16* cache_v, int64_t cache_cap, hipStream_t s) {
    (void)cand_offsets;
    if (items == 0) return hipSuccess;
    if (D != kD || tile != kTQ) return hipErrorInvalidValue;
    k_attn_rank<<<(unsigned)items, 256, 0, s>>>(qkv, o, row0, H, hist_offsets,
                                                reinterpret_cast<const int4*>(work), cache_k,
                                                cache_v, cache_cap);
    return hipGetLastError();
}

}  // namespace upr
