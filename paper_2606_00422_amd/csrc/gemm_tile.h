// Pieces of the projection GEMM shared with the fused FFN kernel (device
// code, header-only): operand types, tile constants, the XCD-aware tile
// order, the LDS swizzle, GELU, fp16/bf16 packing, and the epilogue that
// applies a wave's 128 x 64 (or 32 x 64) accumulator tile to its outputs.
#pragma once

#include "epilogue.h"
#include "mx.h"
#include "upr_plan.h"

namespace upr {

namespace gemm_detail {
typedef __attribute__((ext_vector_type(8))) _Float16 h8;
typedef __attribute__((ext_vector_type(16))) float f32x16;
typedef __attribute__((ext_vector_type(4))) unsigned u32x4;
typedef __attribute__((ext_vector_type(4))) float f32x4;
typedef __attribute__((ext_vector_type(8))) int i32x8;
typedef __attribute__((ext_vector_type(4))) int i32x4;

constexpr int kBK = 64;                            // K-step (fp16 values)
constexpr int kThreads = 512;                      // 8 waves
constexpr int kWN = 64, kTN = kWN / 32;            // per-wave tile columns, 32-column MFMA tiles
constexpr int kCPR = kBK / 8;                      // 16-byte chunks per LDS row (8)
// Block tile by epilogue and height: 2 (M) x 4 (N) waves of (32 TM) x 64,
// i.e. 256 x 256 for TM = 4; the residual update with LayerNorm needs whole
// rows in one workgroup, so it takes (32 TM) x 512 with the eight waves side
// by side along N.  TM = 4 ("tall") for large M; TM = 1 ("short") when tall
// tiles would leave compute units idle: every output element is still the
// same MFMA chain over K in the same order, so results do not depend on the
// choice.  Loads per leading wave per K-step: rows / 32 (a load fills 8 rows,
// four leading waves).
template <int MODE, int TM>
struct Shape {
    static constexpr bool kWide = MODE == EPI_RESID_LN || MODE == EPI_RESID_LN_MX || MODE == EPI_RESID_SCORE;
    static constexpr int kTM = TM, kWM = 32 * TM;
    static constexpr int kBM = kWide ? kWM : 2 * kWM, kBN = kWide ? 512 : 256;
    static constexpr int kWavesN = kWide ? 8 : 4;
    static constexpr int kLoadsA = kBM * kCPR / (kThreads / 2), kLoadsB = kBN * kCPR / (kThreads / 2);
};

// Epilogue staging row strides (elements).  fp32: 272 bytes, so the 16 rows
// written by one 16-lane group of 16-byte stores fall on distinct bank
// groups; 16-bit: 144 bytes, likewise, and rows 8 apart land on disjoint
// halves.
constexpr int kStage32 = 68, kStage16 = 72;
constexpr int kRegionBytes = 16384;                // LDS staging region per wave

__device__ __forceinline__ int xcd_tile(int b, int nb) {
    const int per = nb >> 3, rem = nb & 7;
    const int xcd = b & 7, slot = b >> 3;
    return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

// gfx950's LDS serves a 16-byte access for 16 lanes per pass across 64 banks
// (256 bytes = 2 rows).  Fragment reads take 16 consecutive rows at one
// logical chunk; the chunk is XORed with (row / 2) % 8 so those rows land
// on distinct bank groups.  Element offset of logical chunk `chunk` of row
// `row`:
__device__ __forceinline__ int swz(int row, int chunk) {
    return row * kBK + ((chunk ^ ((row >> 1) & 7)) << 3);
}

// GELU, tanh form, as x * sigmoid(2y) with y = sqrt(2/pi) (x + 0.044715 x^3):
// 0.5 x (1 + tanh(y)) = x / (1 + 2^(-2 log2(e) y)), the exponent folded to
// x (c1 + c2 x^2).
__device__ __forceinline__ float gelu_fast(float x) {
    constexpr float c1 = -2.0f * 1.4426950408889634f * 0.7978845608028654f;
    constexpr float c2 = c1 * 0.044715f;
    const float t = fmaf(c2, x * x, c1);
    return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(x * t));
}

// Two values rounded to bf16 (BF) or fp16, packed low-first (one
// v_cvt_pk_{bf16,f16}_f32, round to nearest even).
template <bool BF>
__device__ __forceinline__ unsigned pack2(float a, float b) {
    typedef __attribute__((ext_vector_type(2))) float f2;
    typedef __attribute__((ext_vector_type(2))) __bf16 bf2;
    typedef __attribute__((ext_vector_type(2))) _Float16 hf2;
    const f2 v = {keep_f32(a), keep_f32(b)};
    if constexpr (BF)
        return __builtin_bit_cast(unsigned, __builtin_convertvector(v, bf2));
    else
        return __builtin_bit_cast(unsigned, __builtin_convertvector(v, hf2));
}

// Epilogue of one wave's 128 x 64 tile (acc in the transposed MFMA layout:
// register r of tile (j, i) holds row 32i + lane%32 and column
// 32j + 8(r/4) + 4(lane/32) + r%4 of the wave tile at (wrow0, wcol0)),
// 32 rows at a time through the wave's own LDS region.
//
// fp32 residual update: the raw accumulators are staged (32 x 272 bytes)
// and come back row-contiguous, lane l holding columns 4(l%16) .. +3 of rows
// 4p + l/16, p = 0..7: the bias is one float4 per lane loaded before the
// first pass, each store covers 256-byte row segments, and the residual
// rows of the next pass are loaded while this one is processed.
//
// 16-bit outputs: scale, bias and the operation are applied in the MFMA
// layout; after conversion lane pairs (l, l+32) exchange halves with
// v_permlane32_swap so each lane holds eight consecutive columns (16 bytes)
// and the staged rows (32 x 144 bytes) are written back as 128-byte
// segments, 16 bytes per lane (narrower stores measured slower).
//
// Residual update with LayerNorm (whole rows in the workgroup, the eight
// waves side by side along N): after a pass's updated rows are stored, each
// wave reduces, per row, the mean and the sum of squared deviations of its
// (up to) 64 columns; the waves exchange them through `lnx` at a workgroup
// barrier, and each combines the eight partials (Chan et al.'s pairwise
// update: M2 = sum M2_w + n_w (mean_w - mean)^2) into the row's mean and
// 1/sqrt(var + eps), then writes LN of its columns.  wn: the wave's column
// block within the tile.
template <int MODE, int kTM>
__device__ __forceinline__ void store_tile(const f32x16 (&acc)[kTN][kTM], char* const region,
                                           int64_t wrow0, int wcol0, int64_t M, int N,
                                           const Epilogue& epi, int lane, float* const lnx, int wn,
                                           float* const scx = nullptr) {
    constexpr int kWM = 32 * kTM;           // rows of the wave tile
    const int lrow = lane & 31, lhalf = lane >> 5;
    const float sc = epi.acc_scale;
    if constexpr (MODE == EPI_RESID || MODE == EPI_RESID_LN || MODE == EPI_RESID_LN_MX ||
                  MODE == EPI_RESID_SCORE) {
        constexpr bool kLN = MODE != EPI_RESID, kLnMx = MODE == EPI_RESID_LN_MX;
        constexpr bool kScore = MODE == EPI_RESID_SCORE;
        const int ch = lane & 15, rsub = lane >> 4;
        const int col = wcol0 + ch * 4;
        const bool col_ok = col < N;                  // N is a multiple of 8
        const float4 bias4 = col_ok ? *reinterpret_cast<const float4*>(epi.bias + col)
                                    : make_float4(0.f, 0.f, 0.f, 0.f);
        float* const st = reinterpret_cast<float*>(region);
        // The wave tile's residual rows through a buffer descriptor whose
        // range ends at row M: rows past the end load zeros and their stores
        // are dropped, so the passes need no branches and the wait before a
        // pass's stores can leave the next pass's loads in flight.  Lanes
        // whose columns lie past N address beyond the range.
        const int64_t rows_valid = M - wrow0 < 0 ? 0 : (M - wrow0 < kWM ? M - wrow0 : kWM);
        const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
            epi.resid + wrow0 * epi.ldr, (short)0, (int)(rows_valid * epi.ldr * 4), 0x00020000);
        const unsigned ldr4 = (unsigned)epi.ldr * 4u;
        const unsigned vo = col_ok ? (unsigned)rsub * ldr4 + (unsigned)col * 4u : 0x80000000u;
        float4 g[2][8];                     // residual rows of passes i (even/odd)
        // bf16 residual source (first layer: the tokens), same rows and
        // columns at half the byte offsets; a lane past N keeps an offset
        // (2^30) beyond the range
        const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<unsigned short*>(static_cast<const unsigned short*>(epi.resid_src)) + wrow0 * epi.ldr,
            (short)0, (int)(rows_valid * epi.ldr * 2), 0x00020000);
        const bool from_src = epi.resid_src != nullptr;
        const bool acc_has_resid = (MODE == EPI_RESID_LN || MODE == EPI_RESID_SCORE) && epi.acc_resid != 0;
        auto load_resid = [&](int i, float4 (&dst)[8]) {
            if (acc_has_resid) return;          // the accumulators carry it
            if (from_src) {
                typedef __attribute__((ext_vector_type(2))) unsigned u32x2;
#pragma unroll
                for (int p = 0; p < 8; ++p) {
                    const u32x2 w = __builtin_bit_cast(
                        u32x2, __builtin_amdgcn_raw_buffer_load_b64(
                                   rsrc, (vo + (unsigned)(i * 32 + p * 4) * ldr4) >> 1, 0, 0));
                    dst[p] = make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u),
                                         __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xffff0000u));
                }
                return;
            }
#pragma unroll
            for (int p = 0; p < 8; ++p)
                dst[p] = __builtin_bit_cast(
                    float4, __builtin_amdgcn_raw_buffer_load_b128(rs, vo + (unsigned)(i * 32 + p * 4) * ldr4, 0, 0));
        };
        float4 ln_g = make_float4(0.f, 0.f, 0.f, 0.f), ln_b = ln_g;
        __amdgpu_buffer_rsrc_t rln = rs, rlns = rs;
        unsigned lnld2 = 0, vln = 0x80000000u, lnsld = 0, vlns = 0x80000000u;
        float4 sw = make_float4(0.f, 0.f, 0.f, 0.f);    // EPI_RESID_SCORE: score weights
        if constexpr (kLN) {
            if (col_ok) {
                ln_g = *reinterpret_cast<const float4*>(epi.ln_gain + col);
                ln_b = *reinterpret_cast<const float4*>(epi.ln_shift + col);
                if constexpr (kScore) sw = *reinterpret_cast<const float4*>(epi.score_w + col);
            }
        }
        if constexpr (kLN && !kScore) {
            // LN output rows through a descriptor ending at row M, like the
            // residual; 16-bit values, or MXFP8 codes (and a second
            // descriptor over the scale bytes), four per lane.
            constexpr int kOB = kLnMx ? 1 : 2;      // bytes per output value
            rln = __builtin_amdgcn_make_buffer_rsrc(static_cast<char*>(epi.ln_out) + wrow0 * epi.ln_ldo * kOB,
                                                    (short)0, (int)(rows_valid * epi.ln_ldo * kOB), 0x00020000);
            lnld2 = (unsigned)epi.ln_ldo * kOB;
            vln = col_ok ? (unsigned)rsub * lnld2 + (unsigned)col * kOB : 0x80000000u;
            if constexpr (kLnMx) {
                const int64_t sld = epi.ln_ldo / kMxBlock;
                rlns = __builtin_amdgcn_make_buffer_rsrc(static_cast<char*>(epi.ln_scales) + wrow0 * sld,
                                                         (short)0, (int)(rows_valid * sld), 0x00020000);
                lnsld = (unsigned)sld;
                vlns = col_ok ? (unsigned)rsub * lnsld + (unsigned)(wcol0 / kMxBlock) : 0x80000000u;
            }
        }
        float4 hv[8];                       // EPI_RESID_LN: the pass's updated rows
        // lnx[buf][row][wave] = (mean_w, M2_w) of the wave's columns for the
        // pass's 32 rows, double-buffered by pass: a buffer is rewritten two
        // passes later, after every wave has passed the barrier that follows
        // its reads.
        auto ln_pass = [&](int i) {
            float2* const X = reinterpret_cast<float2*>(lnx) + (i & 1) * (32 * 8);
            // this wave's valid columns (the tile starts at column 0: N <= 512)
            const int nw = N - wcol0;
            const float cnt = (float)(nw < 0 ? 0 : nw > kWN ? kWN : nw);
            // Row sums over the 16 lanes of a row group, eight rows at once:
            // each exchange halves the rows a lane keeps, so lane ch ends with
            // row ch / 2 (8 exchanges instead of 8 x 4).
            auto rows8_sum = [&](const float (&t)[8]) {
                const bool b3 = ch & 8, b2 = ch & 4, b1 = ch & 2;
                float u[4], v[2];
#pragma unroll
                for (int k = 0; k < 4; ++k)
                    u[k] = (b3 ? t[4 + k] : t[k]) + __shfl_xor(b3 ? t[k] : t[4 + k], 8, 64);
#pragma unroll
                for (int k = 0; k < 2; ++k)
                    v[k] = (b2 ? u[2 + k] : u[k]) + __shfl_xor(b2 ? u[k] : u[2 + k], 4, 64);
                const float w = (b1 ? v[1] : v[0]) + __shfl_xor(b1 ? v[0] : v[1], 2, 64);
                return w + __shfl_xor(w, 1, 64);
            };
            const int gbase = lane & ~15;
            float t[8];
#pragma unroll
            for (int p = 0; p < 8; ++p) t[p] = col_ok ? (hv[p].x + hv[p].y) + (hv[p].z + hv[p].w) : 0.f;
            const float mrow = cnt > 0.f ? rows8_sum(t) / cnt : 0.f;      // mean of row ch / 2
#pragma unroll
            for (int p = 0; p < 8; ++p) {
                const float mw = __shfl(mrow, gbase + 2 * p, 64);
                float q = 0.f;
                if (col_ok) {
                    const float u0 = hv[p].x - mw, u1 = hv[p].y - mw, u2 = hv[p].z - mw, u3 = hv[p].w - mw;
                    q = fmaf(u0, u0, fmaf(u1, u1, fmaf(u2, u2, u3 * u3)));
                }
                t[p] = q;
            }
            const float qrow = rows8_sum(t);
            if ((ch & 1) == 0) X[((ch >> 1) * 4 + rsub) * 8 + wn] = make_float2(mrow, qrow);
            // every wave has written this pass's partials (the empty asm
            // statements keep the compiler from moving LDS accesses across
            // the barrier)
            __builtin_amdgcn_s_waitcnt(0xC07F);
            asm volatile("" ::: "memory");
            __builtin_amdgcn_s_barrier();
            asm volatile("" ::: "memory");
            // lane l (and l + 32) combines row l % 32
            const float4* const xr = reinterpret_cast<const float4*>(X + lrow * 8);
            float mean_w[8], m2_w[8];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const float4 v = xr[k];
                mean_w[2 * k] = v.x; m2_w[2 * k] = v.y; mean_w[2 * k + 1] = v.z; m2_w[2 * k + 1] = v.w;
            }
            float n_w[8], tot = 0.f, sum = 0.f;
#pragma unroll
            for (int w = 0; w < 8; ++w) {
                const int c = N - w * kWN;
                n_w[w] = (float)(c < 0 ? 0 : c > kWN ? kWN : c);
                tot += n_w[w];
                sum = fmaf(n_w[w], mean_w[w], sum);
            }
            const float mu = sum / tot;
            float M2 = 0.f;
#pragma unroll
            for (int w = 0; w < 8; ++w) {
                const float dm = mean_w[w] - mu;
                M2 += fmaf(n_w[w] * dm, dm, m2_w[w]);
            }
            const float rstd = 1.0f / sqrtf(M2 / tot + epi.ln_eps);
            if constexpr (kScore) {
                // per row, this wave's share of LN(row) . w over its four
                // columns per lane, summed over the row group like the
                // statistics; the waves' shares meet in scx at a second
                // workgroup barrier, and lane l < 32 adds the eight of row
                // l in wave order
                float t2[8];
#pragma unroll
                for (int p = 0; p < 8; ++p) {
                    const float mu_p = __shfl(mu, p * 4 + rsub, 64);
                    const float rs_p = __shfl(rstd, p * 4 + rsub, 64);
                    const float4 h = hv[p];
                    float d4 = 0.f;
                    if (col_ok) {
                        d4 = fmaf(fmaf((h.x - mu_p) * rs_p, ln_g.x, ln_b.x), sw.x, d4);
                        d4 = fmaf(fmaf((h.y - mu_p) * rs_p, ln_g.y, ln_b.y), sw.y, d4);
                        d4 = fmaf(fmaf((h.z - mu_p) * rs_p, ln_g.z, ln_b.z), sw.z, d4);
                        d4 = fmaf(fmaf((h.w - mu_p) * rs_p, ln_g.w, ln_b.w), sw.w, d4);
                    }
                    t2[p] = d4;
                }
                const float prow = rows8_sum(t2);
                float* const S = scx + (i & 1) * (32 * 8);
                if ((ch & 1) == 0) S[((ch >> 1) * 4 + rsub) * 8 + wn] = prow;
                __builtin_amdgcn_s_waitcnt(0xC07F);
                asm volatile("" ::: "memory");
                __builtin_amdgcn_s_barrier();
                asm volatile("" ::: "memory");
                const int64_t row = wrow0 + i * 32 + lrow;
                if (wn == 0 && lhalf == 0 && row < M) {
                    const float4 a0 = *reinterpret_cast<const float4*>(S + lrow * 8);
                    const float4 a1 = *reinterpret_cast<const float4*>(S + lrow * 8 + 4);
                    const float sc = ((((((a0.x + a0.y) + a0.z) + a0.w) + a1.x) + a1.y) + a1.z) + a1.w;
                    epi.score_out[row] = sc + *epi.score_b;
                }
                return;
            }
            // LN of this lane's four columns of rows p*4 + rsub
#pragma unroll
            for (int p = 0; p < 8; ++p) {
                const float mu_p = __shfl(mu, p * 4 + rsub, 64);
                const float rs_p = __shfl(rstd, p * 4 + rsub, 64);
                const float4 h = hv[p];
                if constexpr (kLnMx) {
                    // a 32-column block is eight lanes (ch 0-7 or 8-15 of
                    // the row group); its first lane's pair of lanes writes
                    // the wave's two scale bytes
                    float y[4] = {keep_f32(fmaf((h.x - mu_p) * rs_p, ln_g.x, ln_b.x)),
                                  keep_f32(fmaf((h.y - mu_p) * rs_p, ln_g.y, ln_b.y)),
                                  keep_f32(fmaf((h.z - mu_p) * rs_p, ln_g.z, ln_b.z)),
                                  keep_f32(fmaf((h.w - mu_p) * rs_p, ln_g.w, ln_b.w))};
                    if (!col_ok) y[0] = y[1] = y[2] = y[3] = 0.f;
                    float amax = fmaxf(fmaxf(fabsf(y[0]), fabsf(y[1])), fmaxf(fabsf(y[2]), fabsf(y[3])));
                    amax = fmaxf(amax, __shfl_xor(amax, 1, 64));
                    amax = fmaxf(amax, __shfl_xor(amax, 2, 64));
                    amax = fmaxf(amax, __shfl_xor(amax, 4, 64));
                    const int e = mx_block_exp(amax);
                    const float inv = mx_inv_scale(e);
                    __builtin_amdgcn_raw_buffer_store_b32(mx_pack4(y[0] * inv, y[1] * inv, y[2] * inv, y[3] * inv),
                                                          rln, vln + (unsigned)(i * 32 + p * 4) * lnld2, 0, 0);
                    const int e_hi = __shfl_xor(e, 8, 64);
                    if (ch == 0)
                        __builtin_amdgcn_raw_buffer_store_b16(
                            (unsigned short)((e + 127) | ((e_hi + 127) << 8)), rlns,
                            vlns + (unsigned)(i * 32 + p * 4) * lnsld, 0, 0);
                    continue;
                }
                const unsigned lo = pack2<false>(fmaf((h.x - mu_p) * rs_p, ln_g.x, ln_b.x),
                                                 fmaf((h.y - mu_p) * rs_p, ln_g.y, ln_b.y));
                const unsigned hi = pack2<false>(fmaf((h.z - mu_p) * rs_p, ln_g.z, ln_b.z),
                                                 fmaf((h.w - mu_p) * rs_p, ln_g.w, ln_b.w));
                typedef __attribute__((ext_vector_type(2))) unsigned u32x2;
                __builtin_amdgcn_raw_buffer_store_b64(u32x2{lo, hi}, rln,
                                                      vln + (unsigned)(i * 32 + p * 4) * lnld2, 0, 0);
            }
        };
        load_resid(0, g[0]);
#pragma unroll
        for (int i = 0; i < kTM; ++i) {
#pragma unroll
            for (int j = 0; j < kTN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const float4 v = make_float4(acc[j][i][4 * q + 0], acc[j][i][4 * q + 1],
                                                 acc[j][i][4 * q + 2], acc[j][i][4 * q + 3]);
                    *reinterpret_cast<float4*>(st + lrow * kStage32 + j * 32 + 8 * q + 4 * lhalf) = v;
                }
            __builtin_amdgcn_s_waitcnt(0xC07F);
            __builtin_amdgcn_wave_barrier();
            if (i + 1 < kTM) load_resid(i + 1, g[(i + 1) & 1]);
            float4 x[8];
#pragma unroll
            for (int p = 0; p < 8; ++p)
                x[p] = *reinterpret_cast<const float4*>(st + (p * 4 + rsub) * kStage32 + ch * 4);
#pragma unroll
            for (int p = 0; p < 8; ++p) {
                const float4 r = g[i & 1][p];
                const u32x4 o = __builtin_bit_cast(
                    u32x4, acc_has_resid
                               ? make_float4(fmaf(x[p].x, sc, bias4.x), fmaf(x[p].y, sc, bias4.y),
                                             fmaf(x[p].z, sc, bias4.z), fmaf(x[p].w, sc, bias4.w))
                               : make_float4(r.x + fmaf(x[p].x, sc, bias4.x), r.y + fmaf(x[p].y, sc, bias4.y),
                                             r.z + fmaf(x[p].z, sc, bias4.z), r.w + fmaf(x[p].w, sc, bias4.w)));
                if constexpr (!kScore)
                    __builtin_amdgcn_raw_buffer_store_b128(o, rs, vo + (unsigned)(i * 32 + p * 4) * ldr4, 0,
                                                           2 /* nt */);
                if constexpr (kLN) hv[p] = __builtin_bit_cast(float4, o);
            }
            if constexpr (kLN) ln_pass(i);
            __builtin_amdgcn_s_waitcnt(0xC07F);
            __builtin_amdgcn_wave_barrier();
        }
    } else if constexpr (MODE == EPI_GELU_MX) {
        // In the MFMA layout a lane holds, for row 32i + lane%32, sixteen of
        // the 32 columns of block j (8q + 4h .. +3, q = 0..3) and lane l^32
        // the other sixteen: one exchange gives the block maximum.  After
        // encoding, two v_permlane32_swap exchanges give lane l (h = 0) the
        // codes of columns 0-15 and lane l+32 those of 16-31; lanes of h = 0
        // write the row's two scale bytes.  The codes are staged through the
        // wave's LDS region (32 rows x 80 bytes: 16-byte writes of 16
        // consecutive rows fall on distinct bank groups) and written back as
        // the row's whole 64 bytes, 16 rows per store instruction (stores
        // straight from the MFMA layout cover 32 bytes of 32 rows and doubled
        // the HBM write traffic).
        float4 bq[kTN][4];
#pragma unroll
        for (int j = 0; j < kTN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int col = wcol0 + j * 32 + 8 * q + 4 * lhalf;
                bq[j][q] = col < N ? *reinterpret_cast<const float4*>(epi.bias + col)
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
            }
        uint8_t* const codes = static_cast<uint8_t*>(epi.out);
        uint8_t* const scales = static_cast<uint8_t*>(epi.out_scales);
        unsigned char* const stg = reinterpret_cast<unsigned char*>(region);
        constexpr int kStageMx = 80;            // staging row stride (bytes)
        const int64_t lds = epi.ldo / kMxBlock;
        const bool cols_ok = wcol0 < N;                 // N is a multiple of 64
#pragma unroll
        for (int i = 0; i < kTM; ++i) {
            const int64_t row = wrow0 + i * 32 + lrow;
            unsigned sc2 = 0;
#pragma unroll
            for (int j = 0; j < kTN; ++j) {
                float v[16];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    v[4 * q + 0] = gelu_fast(fmaf(acc[j][i][4 * q + 0], sc, bq[j][q].x));
                    v[4 * q + 1] = gelu_fast(fmaf(acc[j][i][4 * q + 1], sc, bq[j][q].y));
                    v[4 * q + 2] = gelu_fast(fmaf(acc[j][i][4 * q + 2], sc, bq[j][q].z));
                    v[4 * q + 3] = gelu_fast(fmaf(acc[j][i][4 * q + 3], sc, bq[j][q].w));
                }
                float amax = 0.f;
#pragma unroll
                for (int r = 0; r < 16; ++r) amax = fmaxf(amax, fabsf(v[r]));
                amax = fmaxf(amax, __shfl_xor(amax, 32, 64));
                const int e = mx_block_exp(amax);
                const float inv = mx_inv_scale(e);
                unsigned u[4];
#pragma unroll
                for (int q = 0; q < 4; ++q)
                    u[q] = mx_pack4(v[4 * q] * inv, v[4 * q + 1] * inv, v[4 * q + 2] * inv,
                                    v[4 * q + 3] * inv);
                const auto r02 = __builtin_amdgcn_permlane32_swap(u[0], u[2], false, false);
                const auto r13 = __builtin_amdgcn_permlane32_swap(u[1], u[3], false, false);
                const u32x4 o = {r02[0], r02[1], r13[0], r13[1]};
                sc2 |= (unsigned)(e + 127) << (8 * j);
                *reinterpret_cast<u32x4*>(stg + lrow * kStageMx + j * 32 + 16 * lhalf) = o;
            }
            if (lhalf == 0 && row < M && cols_ok)
                *reinterpret_cast<unsigned short*>(scales + row * lds + wcol0 / kMxBlock) =
                    (unsigned short)sc2;
            __builtin_amdgcn_s_waitcnt(0xC07F);
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int pp = 0; pp < 2; ++pp) {
                const int r = pp * 16 + (lane >> 2), c = (lane & 3) * 16;
                const u32x4 x = *reinterpret_cast<const u32x4*>(stg + r * kStageMx + c);
                const int64_t grow = wrow0 + i * 32 + r;
                if (grow < M && cols_ok)
                    __builtin_nontemporal_store(x, reinterpret_cast<u32x4*>(codes + grow * epi.ldo + wcol0 + c));
            }
            __builtin_amdgcn_s_waitcnt(0xC07F);
            __builtin_amdgcn_wave_barrier();
        }
    } else {
        // Per run of four columns: multiplier and bias.  EPI_STORE scales
        // columns < scale_cols by col_scale, EPI_QKV_CACHE the query columns
        // (< d_model); both fold the factor into multiplier and bias.
        float4 bq[kTN][4];
        float cq[kTN][4];
#pragma unroll
        for (int j = 0; j < kTN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int col = wcol0 + j * 32 + 8 * q + 4 * lhalf;
                float4 b = col < N ? *reinterpret_cast<const float4*>(epi.bias + col)
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
                float c = sc;
                if constexpr (MODE != EPI_GELU && MODE != EPI_GELU_PERM) {
                    const int lim = MODE == EPI_STORE ? epi.scale_cols : epi.d_model;
                    const float cs = col < lim ? epi.col_scale : 1.0f;
                    c = sc * cs;
                    b = make_float4(b.x * cs, b.y * cs, b.z * cs, b.w * cs);
                }
                bq[j][q] = b;
                cq[j][q] = c;
            }
        constexpr bool kGelu = MODE == EPI_GELU || MODE == EPI_GELU_PERM;
        constexpr bool kBf = !kGelu;
        unsigned short* const st = reinterpret_cast<unsigned short*>(region);
        const int ch = lane & 7, rs = lane >> 3;
        const int col = wcol0 + ch * 8;
        // Staged rows come back as row lr0 + off of the wave tile, lane
        // (ch, rs) holding columns col .. col+7; the destination of row
        // wrow0 + lr0 + off is obase + off * ostride.
        const int lr0 = (rs >> 1) + 8 * (rs & 1);
        const int rows_left = (int)min(M - wrow0 - lr0, (int64_t)kWM);
        unsigned short* obase = static_cast<unsigned short*>(epi.out) + (wrow0 + lr0) * epi.ldo + col;
        int64_t ostride = epi.ldo;
        if constexpr (MODE == EPI_QKV_CACHE) {
            const int d = epi.d_model;
            if (col >= d) {   // 8 columns never straddle a head (head_dim % 8 == 0)
                const int part = col >= 2 * d ? 2 : 1;
                const int c = col - part * d;
                const int h = c / epi.head_dim, e = c - h * epi.head_dim;
                unsigned short* plane = static_cast<unsigned short*>(part == 1 ? epi.cache_k : epi.cache_v);
                obase = plane + ((int64_t)h * epi.cache_cap + (epi.row0 + wrow0 + lr0)) * epi.head_dim + e;
                ostride = epi.head_dim;
            }
        }
#pragma unroll
        for (int i = 0; i < kTM; ++i) {
#pragma unroll
            for (int j = 0; j < kTN; ++j) {
                unsigned pk[4][2];
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    float v[4];
                    v[0] = fmaf(acc[j][i][4 * q + 0], cq[j][q], bq[j][q].x);
                    v[1] = fmaf(acc[j][i][4 * q + 1], cq[j][q], bq[j][q].y);
                    v[2] = fmaf(acc[j][i][4 * q + 2], cq[j][q], bq[j][q].z);
                    v[3] = fmaf(acc[j][i][4 * q + 3], cq[j][q], bq[j][q].w);
                    if constexpr (kGelu) {
#pragma unroll
                        for (int r = 0; r < 4; ++r) v[r] = gelu_fast(v[r]);
                    }
                    pk[q][0] = pack2<kBf>(v[0], v[1]);
                    pk[q][1] = pack2<kBf>(v[2], v[3]);
                }
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    u32x4 o;
                    if constexpr (MODE == EPI_GELU_PERM) {
                        // columns 16c + {4h..4h+3, 8+4h..8+4h+3} are positions
                        // 16c + 8h .. +7 of the permuted order: already the
                        // lane's own 16 bytes
                        o = u32x4{pk[2 * c][0], pk[2 * c][1], pk[2 * c + 1][0], pk[2 * c + 1][1]};
                    } else {
#pragma unroll
                        for (int w = 0; w < 2; ++w) {
                            const auto r = __builtin_amdgcn_permlane32_swap(pk[2 * c][w], pk[2 * c + 1][w],
                                                                            false, false);
                            o[w] = r[0];
                            o[2 + w] = r[1];
                        }
                    }
                    *reinterpret_cast<u32x4*>(st + lrow * kStage16 + j * 32 + 16 * c + 8 * lhalf) = o;
                }
            }
            __builtin_amdgcn_s_waitcnt(0xC07F);
            __builtin_amdgcn_wave_barrier();
#pragma unroll
            for (int p = 0; p < 4; ++p) {
                const int off = i * 32 + 16 * (p >> 1) + 4 * (p & 1);
                const u32x4 o = *reinterpret_cast<const u32x4*>(st + (off - i * 32 + lr0) * kStage16 + ch * 8);
                if (off >= rows_left || col >= N) continue;          // N is a multiple of 8
                __builtin_nontemporal_store(o, reinterpret_cast<u32x4*>(obase + off * ostride));
            }
            __builtin_amdgcn_s_waitcnt(0xC07F);
            __builtin_amdgcn_wave_barrier();
        }
    }
}

// Accumulators of a wave's tile set to resid / acc_scale (Epilogue::
// acc_resid): register r of tile (j, i) takes row wrow0 + 32i + lane%32,
// column wcol0 + 32j + 8(r/4) + 4(lane/32) + r%4, one float4 per run of four
// columns; rows past M read zeros (buffer range), columns past N stay zero.
template <int kTM>
__device__ __forceinline__ void load_acc_resid(f32x16 (&acc)[kTN][kTM], const Epilogue& epi, int64_t wrow0,
                                               int wcol0, int64_t M, int N, int lane) {
    constexpr int kWM = 32 * kTM;
    const int lrow = lane & 31, lhalf = lane >> 5;
    const float inv = 1.0f / epi.acc_scale;     // a power of two: exact
    const int64_t rows_valid = M - wrow0 < 0 ? 0 : (M - wrow0 < kWM ? M - wrow0 : kWM);
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        epi.resid + wrow0 * epi.ldr, (short)0, (int)(rows_valid * epi.ldr * 4), 0x00020000);
#pragma unroll
    for (int j = 0; j < kTN; ++j)
#pragma unroll
        for (int i = 0; i < kTM; ++i)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int col = wcol0 + 32 * j + 8 * q + 4 * lhalf;
                float4 r = make_float4(0.f, 0.f, 0.f, 0.f);
                if (col < N)                           // N is a multiple of 8
                    r = __builtin_bit_cast(float4, __builtin_amdgcn_raw_buffer_load_b128(
                                                       rs, (unsigned)((i * 32 + lrow) * epi.ldr + col) * 4u, 0, 0));
                acc[j][i][4 * q + 0] = r.x * inv;
                acc[j][i][4 * q + 1] = r.y * inv;
                acc[j][i][4 * q + 2] = r.z * inv;
                acc[j][i][4 * q + 3] = r.w * inv;
            }
}

// Compute units of the current device.
inline int device_cus() {
    constexpr int kMaxDevices = 64;
    static int cached[kMaxDevices];              // 0: not yet queried
    int dev = 0, cus = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
    if (cached[dev] == 0) {
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            return 256;
        cached[dev] = cus;
    }
    return cached[dev];
}

}  // namespace gemm_detail

}  // namespace upr
