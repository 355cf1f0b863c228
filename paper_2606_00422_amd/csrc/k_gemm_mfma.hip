// Projection GEMM on the matrix cores: out = A[M,K] W[N,K]^T (+ epilogue),
// A and W fp16 (both K-contiguous), fp32 accumulation with
// v_mfma_f32_32x32x16_f16.
//
// Block tile 256 (rows of A) x 256 (rows of W), K in steps of 64, eight
// waves in a 2 (M) x 4 (N) grid, each owning 128 x 64 outputs = 4 x 2 MFMA
// tiles.  The MFMA computes the transposed tile, C^T = W A^T (W as the
// first operand), so each lane holds runs of four consecutive output
// columns of one row.
//
// Main loop.  A and W tiles go straight from global memory into LDS
// (buffer loads with the LDS bit: no staging registers; rows past the end
// read as zeros), in two stages (three for the short tiles of small calls,
// whose K-loop waits on the load round trip).  LDS rows are 128 bytes (64
// fp16) whose eight 16-byte chunks are XOR-swizzled, so fragment reads are
// bank-conflict free.  The two waves sharing a SIMD (w and w+4) run in
// opposite phases ("ping-pong"): while one reads its operand fragments from
// LDS into registers, the other runs its MFMAs, and they swap at each
// barrier.  Only the four leading waves issue the global loads, one K-step
// ahead (two with three stages).
//
// Epilogue.  Stores straight from the MFMA layout touch 32 rows per
// instruction with 8-16 bytes each and reach about 60% of the bandwidth of
// row-contiguous stores.  Each wave therefore stages its raw accumulators
// through its own LDS region, 32 rows at a time, and applies scale, bias and
// the epilogue operation on the row-contiguous read-back, writing full
// 256-byte (fp32 residual) or 128-byte (16-bit output) row segments.  The
// stores are non-temporal, so the output stream does not evict the operand
// panels that later tiles re-read from L2.
//
// Residual update with LayerNorm (EPI_RESID_LN: the LayerNorm that follows
// the output projection and the FFN down projection).  LayerNorm needs whole
// rows, so this mode takes a 128 x 512 tile (rows of at most 512 values) with
// the eight waves side by side along N, each still 128 x 64.  After a 32-row
// pass of the residual update, each wave reduces per-row mean and squared
// deviations over its columns, the waves exchange them through LDS at a
// workgroup barrier, and each writes the normalized values of its columns as
// fp16: the updated residual is never read back from HBM.  With MXFP8
// operands (EPI_RESID_LN_MX) the LayerNorm is written as MXFP8 (a 32-column
// block is eight lanes of a row group) and the tile is 64 x 512: two
// 128-row stages would leave no LDS for the K-step's scale dwords.
//
// Tile order is XCD-aware: workgroup b runs on XCD b % 8 and the tiles are
// renumbered so each XCD sweeps a contiguous range of (M-panel, N-tile)
// pairs; the N-tiles of one A row-panel then share one L2.
//
// MXFP8 operands (fp8 projection variant).  The same kernel with E4M3 codes:
// a 128-byte LDS row now holds 128 K-values, so one K-step covers twice the
// depth with the same loads, swizzle and LDS traffic, and the MFMA is
// v_mfma_scale_f32_32x32x64_f8f6f4 (twice the fp16 rate).  Its operand
// layout (probed): lane l holds row l % 32; the 32 bytes of lane l are K
// [16h, 16h+16) and [32+16h, 32+16h+16) of the instruction's 64 (h = l / 32),
// and the E8M0 scale lane l supplies applies to 32-value block h of its row
// (bytes 0-15 of lanes l and l+32 form block 0).  So a lane reads LDS chunks
// 4kk + h and 4kk + 2 + h, and takes byte 2kk + h of its row's scale dword
// (the four blocks of the K-step; op_sel picks byte 2kk after a shift by
// 8h).  The scale dwords of a K-step (one per row of A and of W) ride along
// with the tile loads into two small LDS arrays per stage.
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
        auto load_resid = [&](int i, float4 (&dst)[8]) {
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
                    u32x4, make_float4(r.x + fmaf(x[p].x, sc, bias4.x), r.y + fmaf(x[p].y, sc, bias4.y),
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
                if constexpr (MODE != EPI_GELU) {
                    const int lim = MODE == EPI_STORE ? epi.scale_cols : epi.d_model;
                    const float cs = col < lim ? epi.col_scale : 1.0f;
                    c = sc * cs;
                    b = make_float4(b.x * cs, b.y * cs, b.z * cs, b.w * cs);
                }
                bq[j][q] = b;
                cq[j][q] = c;
            }
        constexpr bool kBf = MODE != EPI_GELU;
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
                    if constexpr (MODE == EPI_GELU) {
#pragma unroll
                        for (int r = 0; r < 4; ++r) v[r] = gelu_fast(v[r]);
                    }
                    pk[q][0] = pack2<kBf>(v[0], v[1]);
                    pk[q][1] = pack2<kBf>(v[2], v[3]);
                }
#pragma unroll
                for (int c = 0; c < 2; ++c) {
                    u32x4 o;
#pragma unroll
                    for (int w = 0; w < 2; ++w) {
                        const auto r = __builtin_amdgcn_permlane32_swap(pk[2 * c][w], pk[2 * c + 1][w],
                                                                        false, false);
                        o[w] = r[0];
                        o[2 + w] = r[1];
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

template <int MODE, bool MX, int TM>
__global__ __launch_bounds__(kThreads, 1) void k_gemm_mfma(const void* __restrict__ Av, int64_t lda,
                                                           const void* __restrict__ Wv,
                                                           const uint8_t* __restrict__ As,
                                                           const uint8_t* __restrict__ Ws,
                                                           int64_t M, int N, int K, Epilogue epi) {
    using SH = Shape<MODE, TM>;
    constexpr int kBM = SH::kBM, kBN = SH::kBN, kWavesN = SH::kWavesN;
    constexpr int kLoadsA = SH::kLoadsA, kLoadsB = SH::kLoadsB;
    constexpr int kTM = SH::kTM, kWM = SH::kWM;
    // Two LDS stages as separate arrays: the compiler can then tell that
    // fragment reads of one stage do not alias the loads filling the other.
    // Short 256-wide tiles (small calls: one tile per compute unit, the
    // K-loop waits on each stage's round trip) keep a third stage and load
    // two K-steps ahead.
    constexpr int kStages = (!SH::kWide && TM == 1) ? 3 : 2;
    __shared__ __attribute__((aligned(16))) f16 sA0[kBM * kBK];
    __shared__ __attribute__((aligned(16))) f16 sA1[kBM * kBK];
    __shared__ __attribute__((aligned(16))) f16 sA2[kStages == 3 ? kBM * kBK : 8];
    __shared__ __attribute__((aligned(16))) f16 sB0[kBN * kBK];
    __shared__ __attribute__((aligned(16))) f16 sB1[kBN * kBK];
    __shared__ __attribute__((aligned(16))) f16 sB2[kStages == 3 ? kBN * kBK : 8];
    // MXFP8: the K-step's scale dword of every row of A and of W
    // (at least one 64-row slice each: a slice is one load instruction)
    constexpr int kSA = MX ? (kBM < 64 ? 64 : kBM) : 1, kSB = MX ? kBN : 1;
    __shared__ uint32_t sSA0[kSA], sSA1[kSA], sSB0[kSB], sSB1[kSB];
    __shared__ uint32_t sSA2[kStages == 3 ? kSA : 1], sSB2[kStages == 3 ? kSB : 1];
    // Epilogue staging of short 256-wide tiles (their A stages are too small
    // to hold it): one region per wave, three in each of the W stages
    constexpr int kShortRegion = 32 * kStage32 * 4;
    static_assert(kStages == 2 || SH::kWide || 3 * kShortRegion <= kBN * kBK * 2, "staging fits a stage");
    constexpr int kEB = MX ? 1 : 2;         // bytes per operand value
    const char* const A = static_cast<const char*>(Av);
    const char* const W = static_cast<const char*>(Wv);

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);     // uniform: wave-derived values stay scalar
    const int wm = wave / kWavesN, wn = wave % kWavesN;
    const int tiles_n = (N + kBN - 1) / kBN;
    const int t = xcd_tile(blockIdx.x, gridDim.x);
    const int64_t m0 = (int64_t)(t / tiles_n) * kBM;
    const int n0 = (t % tiles_n) * kBN;
    const bool lead = __builtin_amdgcn_readfirstlane(wave) < 4;

    // Buffer descriptors over this tile's rows of A and W: rows past M (N)
    // fall outside num_records and load as zeros, so tails need no branches.
    const int64_t rows_a = M - m0 < kBM ? M - m0 : kBM;
    const int rows_b = N - n0 < kBN ? N - n0 : kBN;
    const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(A + m0 * lda * kEB), (short)0, (int)(rows_a * lda * kEB), 0x00020000);
    const __amdgpu_buffer_rsrc_t rsB = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(W + (int64_t)n0 * K * kEB), (short)0, (int)((int64_t)rows_b * K * kEB), 0x00020000);

    // Direct global -> LDS loads by the leading waves: a load instruction's
    // 64 lanes fill 64 consecutive 16-byte LDS slots = 8 rows.  Load i of
    // leading wave lw covers rows 8 (lw kL + i) + lane/8; slot s of row r
    // must hold logical chunk s ^ key(r), key(r) = (r / 2) % 8, which for
    // loads 16 rows apart is the same.  So the offsets of a wave's first
    // two loads plus a uniform step of 16 rows address every load (a wave
    // with a single load, kL = 1, uses the first only).  (The step stays in
    // the per-lane offset: the buffer range check that zero-fills rows past
    // the end does not cover the scalar offset.)
    const int lw = wave & 3;
    int voA[2], voB[2];
#pragma unroll
    for (int p = 0; p < 2; ++p) {
        const int ra = (lw * kLoadsA + p) * 8 + (lane >> 3), rb = (lw * kLoadsB + p) * 8 + (lane >> 3);
        voA[p] = (int)(ra * lda * kEB + (((lane & 7) ^ ((ra >> 1) & 7)) << 4));
        voB[p] = rb * K * kEB + (((lane & 7) ^ ((rb >> 1) & 7)) << 4);
    }
    const int rowstepA = (int)(16 * lda * kEB), rowstepB = 16 * K * kEB;
    // MXFP8 scales: leading wave lw loads the dwords of rows 64 (lw + 4 s)
    // .. +63, s = 0, 1, .., of A and of W for a K-step (K/32 bytes per row;
    // dword t = blocks 4t..4t+3)
    const int kblk = K / kMxBlock;
    const __amdgpu_buffer_rsrc_t rsSA = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(MX ? As + m0 * kblk : As), (short)0, MX ? (int)(rows_a * kblk) : 0, 0x00020000);
    const __amdgpu_buffer_rsrc_t rsSB = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(MX ? Ws + (int64_t)n0 * kblk : Ws), (short)0, MX ? (int)((int64_t)rows_b * kblk) : 0,
        0x00020000);
    const int voS = (lw * 64 + lane) * kblk;
    static_assert(kBN % 64 == 0, "whole 64-row slices of W scales");
    auto issue_scales = [&](uint32_t* dSA, uint32_t* dSB, int t) {
        if constexpr (MX) {
            // A: slices starting past kBM rows (short tiles) are not loaded;
            // the slice of a tile under 64 rows reads zeros past the tile's
            // rows into the array's slack
#pragma unroll
            for (int sl = 0; sl * 4 * 64 < kBM; ++sl)
                if ((lw + 4 * sl) * 64 < kBM)
                    __builtin_amdgcn_raw_ptr_buffer_load_lds(
                        rsSA, (__attribute__((address_space(3))) void*)(dSA + (lw + 4 * sl) * 64), 4,
                        voS + 4 * sl * 64 * kblk + 4 * t, 0, 0, 0);
#pragma unroll
            for (int sl = 0; sl * 4 * 64 < kBN; ++sl)
                __builtin_amdgcn_raw_ptr_buffer_load_lds(
                    rsSB, (__attribute__((address_space(3))) void*)(dSB + (lw + 4 * sl) * 64), 4,
                    voS + 4 * sl * 64 * kblk + 4 * t, 0, 0, 0);
        }
    };
    // k0: byte offset of the K-step within a row (128 per step)
    auto issue_loads = [&](f16* dA, f16* dB, int k0) {
        // opaque copies keep the per-load offsets from being hoisted into
        // sixteen live registers
        int rsa = rowstepA, rsb = rowstepB;
        asm volatile("" : "+s"(rsa), "+s"(rsb));
#pragma unroll
        for (int i = 0; i < kLoadsA; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rsA, (__attribute__((address_space(3))) void*)(dA + (lw * kLoadsA + i) * 64 * 8),
                16, voA[i & 1] + (i >> 1) * rsa + k0, 0, 0, 0);
#pragma unroll
        for (int i = 0; i < kLoadsB; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rsB, (__attribute__((address_space(3))) void*)(dB + (lw * kLoadsB + i) * 64 * 8),
                16, voB[i & 1] + (i >> 1) * rsb + k0, 0, 0, 0);
    };

    f32x16 acc[kTN][kTM];
#pragma unroll
    for (int j = 0; j < kTN; ++j)
#pragma unroll
        for (int i = 0; i < kTM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[j][i][r] = 0.f;

    const int lrow = lane & 31, lhalf = lane >> 5;
    // fp16: 16-deep fragments; MXFP8: 64-deep fragments + scale dwords.  Each
    // wave reads all of a K-step's fragments in its read phase: the leading
    // waves refill a stage as soon as the trailing waves' read phase on it
    // has ended.
    h8 a[kBK / 16][kTM], b[kBK / 16][kTN];
    i32x8 am[2][kTM], bm[2][kTN];
    unsigned sa[kTM], sb[kTN];
    // Byte offsets, within a stage, of this lane's first fragment row at
    // logical chunk 2m + lhalf (swz written out: the key (row / 2) % 8 is the
    // same for every row tile of the lane).  Row tiles add constants, which
    // fold into the read instructions.
    int offA[4], offB[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        const int ch = (((2 * m + lhalf) ^ ((lrow >> 1) & 7)) << 4);
        offA[m] = (wm * kWM + lrow) * (kBK * 2) + ch;
        offB[m] = (wn * kWN + lrow) * (kBK * 2) + ch;
    }
    // t-th row tile (32 rows down), K-half kk
    auto frag_mx = [&](const f16* c, const int (&off)[4], int t, int kk) {
        const char* p = reinterpret_cast<const char*>(c) + t * 32 * (kBK * 2);
        i32x8 f;
        f.lo = *reinterpret_cast<const i32x4*>(p + off[2 * kk]);
        f.hi = *reinterpret_cast<const i32x4*>(p + off[2 * kk + 1]);
        return f;
    };
    auto read_frags = [&](const f16* cA, const f16* cB, const uint32_t* cSA, const uint32_t* cSB) {
        if constexpr (MX) {
            // recomputed addresses per step (not hoisted into 24 registers)
            asm volatile("" : "+v"(offA[0]), "+v"(offA[1]), "+v"(offA[2]), "+v"(offA[3]),
                         "+v"(offB[0]), "+v"(offB[1]), "+v"(offB[2]), "+v"(offB[3]));
#pragma unroll
            for (int kk = 0; kk < 2; ++kk) {
#pragma unroll
                for (int i = 0; i < kTM; ++i) am[kk][i] = frag_mx(cA, offA, i, kk);
#pragma unroll
                for (int j = 0; j < kTN; ++j) bm[kk][j] = frag_mx(cB, offB, j, kk);
            }
#pragma unroll
            for (int i = 0; i < kTM; ++i) sa[i] = cSA[wm * kWM + i * 32 + lrow] >> (8 * lhalf);
#pragma unroll
            for (int j = 0; j < kTN; ++j) sb[j] = cSB[wn * kWN + j * 32 + lrow] >> (8 * lhalf);
        } else {
#pragma unroll
            for (int kk = 0; kk < kBK / 16; ++kk) {
                const int ch = kk * 2 + lhalf;
#pragma unroll
                for (int i = 0; i < kTM; ++i)
                    a[kk][i] = *reinterpret_cast<const h8*>(&cA[swz(wm * kWM + i * 32 + lrow, ch)]);
#pragma unroll
                for (int j = 0; j < kTN; ++j)
                    b[kk][j] = *reinterpret_cast<const h8*>(&cB[swz(wn * kWN + j * 32 + lrow, ch)]);
            }
        }
    };
    auto compute = [&]() {
        if constexpr (MX) {
            // op_sel picks byte 2kk of the (per-lane shifted) scale dwords
#pragma unroll
            for (int j = 0; j < kTN; ++j)
#pragma unroll
                for (int i = 0; i < kTM; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                        bm[0][j], am[0][i], acc[j][i], 0, 0, 0, (int)sb[j], 0, (int)sa[i]);
#pragma unroll
            for (int j = 0; j < kTN; ++j)
#pragma unroll
                for (int i = 0; i < kTM; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(
                        bm[1][j], am[1][i], acc[j][i], 0, 0, 2, (int)sb[j], 2, (int)sa[i]);
        } else {
#pragma unroll
            for (int kk = 0; kk < kBK / 16; ++kk)
#pragma unroll
                for (int j = 0; j < kTN; ++j)
#pragma unroll
                    for (int i = 0; i < kTM; ++i)
                        acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(b[kk][j], a[kk][i],
                                                                           acc[j][i], 0, 0, 0);
        }
    };

    // Every wave runs the same read / MFMA sequence; the trailing waves run
    // it one phase late (one extra barrier at the start, the leading waves
    // one at the end).  K-step t sits in stage t & 1.  The leading waves
    // issue step t+1's loads at the start of their step t into the other
    // stage (last read by the trailing waves in the phase just ended) and
    // wait for them at the end of step t, before anyone reads them.
    const int nk = K / (kBK * 2 / kEB);
    auto kstep = [&](const f16* cA, const f16* cB, const uint32_t* cSA, const uint32_t* cSB,
                     f16* nA, f16* nB, uint32_t* nSA, uint32_t* nSB, int t) {
        if (lead && t + 1 < nk) {
            issue_loads(nA, nB, (t + 1) * kBK * 2);
            issue_scales(nSA, nSB, t + 1);
        }
        read_frags(cA, cB, cSA, cSB);
        __builtin_amdgcn_s_waitcnt(0xC07F);     // lgkmcnt(0): fragments in registers
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        compute();
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(0x0F70);     // vmcnt(0): the next stage has landed
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
    };

    if constexpr (kStages == 3) {
        // Step t reads stage t % 3 and its leading waves fill stage
        // (t + 2) % 3, last read in step t - 1 (by the trailing waves before
        // the barrier that ended it); at its end only step t + 1's loads must
        // have landed, so step t + 2's stay in flight.  Leading wave 0 may
        // hold one more load (A's scales) than the count and then waits for
        // it too.
        auto kstep3 = [&](const f16* cA, const f16* cB, const uint32_t* cSA, const uint32_t* cSB,
                          f16* nA, f16* nB, uint32_t* nSA, uint32_t* nSB, int t) {
            if (lead && t + 2 < nk) {
                issue_loads(nA, nB, (t + 2) * kBK * 2);
                issue_scales(nSA, nSB, t + 2);
            }
            read_frags(cA, cB, cSA, cSB);
            __builtin_amdgcn_s_waitcnt(0xC07F);     // lgkmcnt(0): fragments in registers
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
            compute();
            __builtin_amdgcn_sched_barrier(0);
            constexpr int kInFlight = kLoadsA + kLoadsB + (MX ? 1 : 0);
            static_assert(kInFlight < 16, "vmcnt field");
            if (t + 2 < nk)
                __builtin_amdgcn_s_waitcnt(0x0F70 | kInFlight);   // vmcnt(step t+2's loads)
            else
                __builtin_amdgcn_s_waitcnt(0x0F70);               // vmcnt(0)
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
        };
        if (lead) {
            issue_loads(sA0, sB0, 0);
            issue_scales(sSA0, sSB0, 0);
            if (nk > 1) {
                issue_loads(sA1, sB1, kBK * 2);
                issue_scales(sSA1, sSB1, 1);
            }
        }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (!lead) __builtin_amdgcn_s_barrier();
        int kt = 0;
        for (; kt + 3 <= nk; kt += 3) {
            kstep3(sA0, sB0, sSA0, sSB0, sA2, sB2, sSA2, sSB2, kt);
            kstep3(sA1, sB1, sSA1, sSB1, sA0, sB0, sSA0, sSB0, kt + 1);
            kstep3(sA2, sB2, sSA2, sSB2, sA1, sB1, sSA1, sSB1, kt + 2);
        }
        if (kt < nk) kstep3(sA0, sB0, sSA0, sSB0, sA2, sB2, sSA2, sSB2, kt);
        if (kt + 1 < nk) kstep3(sA1, sB1, sSA1, sSB1, sA0, sB0, sSA0, sSB0, kt + 1);
    } else {
        if (lead) {
            issue_loads(sA0, sB0, 0);
            issue_scales(sSA0, sSB0, 0);
        }
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
        if (!lead) __builtin_amdgcn_s_barrier();
        int kt = 0;
        for (; kt + 2 <= nk; kt += 2) {
            kstep(sA0, sB0, sSA0, sSB0, sA1, sB1, sSA1, sSB1, kt);
            kstep(sA1, sB1, sSA1, sSB1, sA0, sB0, sSA0, sSB0, kt + 1);
        }
        if (kt < nk) kstep(sA0, sB0, sSA0, sSB0, sA1, sB1, sSA1, sSB1, kt);
    }
    // Past here every wave has finished its fragment reads (the trailing
    // waves' last reads precede the barrier that ended the leading waves'
    // last step), so the stages are free for the epilogue.

    // ---- epilogue ------------------------------------------------------
    // Register r of transposed tile (j, i) holds output row
    // wm*128 + 32i + lane%32 and column wn*64 + 32j + 8(r/4) + 4(lane/32) + r%4.
    if constexpr (SH::kWide) {
        // The waves exchange row statistics at a workgroup barrier per pass,
        // so the leading waves first take their pending barrier (the
        // trailing waves' last K-step one): all eight enter the epilogue
        // together (letting the leading waves start early measured slower).
        // Staging regions: seven in sB0, one in sB1; the statistics go to sA0.
        if (lead) __builtin_amdgcn_s_barrier();
        constexpr int kRegion = 32 * kStage32 * 4;
        char* const region = wave < 7 ? reinterpret_cast<char*>(sB0) + wave * kRegion
                                      : reinterpret_cast<char*>(sB1);
        // (EPI_RESID_SCORE: the waves' score shares go to sA1)
        store_tile<MODE, kTM>(acc, region, m0 + wm * kWM, n0 + wn * kWN, M, N, epi, lane,
                              reinterpret_cast<float*>(sA0), wn, reinterpret_cast<float*>(sA1));
    } else {
        const int wsel = __builtin_amdgcn_readfirstlane(wave) >> 1;
        f16* const sbase = wsel == 0 ? sA0 : wsel == 1 ? sA1 : wsel == 2 ? sB0 : sB1;
        const int w3 = __builtin_amdgcn_readfirstlane(wave) / 3;
        char* const region =
            kStages == 3 ? reinterpret_cast<char*>(w3 == 0 ? sB0 : w3 == 1 ? sB1 : sB2) +
                               (__builtin_amdgcn_readfirstlane(wave) % 3) * kShortRegion
                         : reinterpret_cast<char*>(sbase) + (wave & 1) * kRegionBytes;
        // Epilogues writing new outputs start only after the trailing
        // waves' last MFMAs (overlapping them measured 4-5% slower); the
        // residual update, which reads as much as it writes, overlaps them.
        constexpr bool kOverlap = MODE == EPI_RESID;
        if (lead && !kOverlap) __builtin_amdgcn_s_barrier();
        store_tile<MODE, kTM>(acc, region, m0 + wm * kWM, n0 + wn * kWN, M, N, epi, lane, nullptr, 0);
        if (lead && kOverlap) __builtin_amdgcn_s_barrier();
    }
}

template <int MODE, int TM>
int64_t tile_count(int64_t M, int N) {
    using SH = Shape<MODE, TM>;
    return ((M + SH::kBM - 1) / SH::kBM) * (int64_t)((N + SH::kBN - 1) / SH::kBN);
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

template <int MODE, bool MX>
hipError_t launch_mode(const void* A, int64_t lda, const void* W, const uint8_t* As,
                       const uint8_t* Ws, int64_t M, int N, int K, const Epilogue& epi,
                       hipStream_t s) {
    // The MXFP8 residual update with LayerNorm takes 64-row tiles: two
    // 128 x 512 stages fill the LDS and leave no room for their scales.
    constexpr int kTall = (MX && Shape<MODE, 4>::kWide) ? 2 : 4;
    const int64_t tall = tile_count<MODE, kTall>(M, N);
    if (tall >= device_cus()) {
        k_gemm_mfma<MODE, MX, kTall><<<(unsigned)tall, kThreads, 0, s>>>(A, lda, W, As, Ws, M, N, K, epi);
    } else {
        const int64_t shorts = tile_count<MODE, 1>(M, N);
        k_gemm_mfma<MODE, MX, 1><<<(unsigned)shorts, kThreads, 0, s>>>(A, lda, W, As, Ws, M, N, K, epi);
    }
    return hipGetLastError();
}

}  // namespace gemm_detail

hipError_t launch_gemm_mfma(const f16* A, int64_t lda, const f16* W, int64_t M, int N, int K,
                            const Epilogue& epi, hipStream_t s) {
    using namespace gemm_detail;
    if (M == 0) return hipSuccess;
    // whole 64-deep K-steps, 16-byte operand loads, 16-byte output chunks
    if (K <= 0 || K % kBK != 0 || lda % 8 != 0 || N % 8 != 0) return hipErrorInvalidValue;
    switch (epi.mode) {
        case EPI_STORE:
            if (epi.ldo % 8 != 0 || epi.scale_cols % 4 != 0) return hipErrorInvalidValue;
            return launch_mode<EPI_STORE, false>(A, lda, W, nullptr, nullptr, M, N, K, epi, s);
        case EPI_GELU:
            if (epi.ldo % 8 != 0) return hipErrorInvalidValue;
            return launch_mode<EPI_GELU, false>(A, lda, W, nullptr, nullptr, M, N, K, epi, s);
        case EPI_RESID:
            if (epi.ldr % 4 != 0) return hipErrorInvalidValue;
            return launch_mode<EPI_RESID, false>(A, lda, W, nullptr, nullptr, M, N, K, epi, s);
        case EPI_RESID_LN:
            static_assert(Shape<EPI_RESID_LN, 4>::kBN == kResidLnMaxN, "tile spans the widest row");
            if (epi.ldr % 4 != 0 || N > kResidLnMaxN || epi.ln_ldo % 4 != 0 ||
                !epi.ln_gain || !epi.ln_shift || !epi.ln_out)
                return hipErrorInvalidValue;
            return launch_mode<EPI_RESID_LN, false>(A, lda, W, nullptr, nullptr, M, N, K, epi, s);
        case EPI_RESID_SCORE:
            if (epi.ldr % 4 != 0 || N > kResidLnMaxN || !epi.ln_gain || !epi.ln_shift ||
                !epi.score_w || !epi.score_b || !epi.score_out)
                return hipErrorInvalidValue;
            return launch_mode<EPI_RESID_SCORE, false>(A, lda, W, nullptr, nullptr, M, N, K, epi, s);
        case EPI_QKV_CACHE:
            if (epi.ldo % 8 != 0 || epi.head_dim % 8 != 0 || epi.d_model % 8 != 0)
                return hipErrorInvalidValue;
            return launch_mode<EPI_QKV_CACHE, false>(A, lda, W, nullptr, nullptr, M, N, K, epi, s);
        default: return hipErrorInvalidValue;
    }
}

hipError_t launch_gemm_mx(const uint8_t* A, const uint8_t* A_scales, const uint8_t* W,
                          const uint8_t* W_scales, int64_t M, int N, int K, const Epilogue& epi,
                          hipStream_t s) {
    using namespace gemm_detail;
    if (M == 0) return hipSuccess;
    // whole 128-deep K-steps over rows of K codes, 16-byte output chunks
    if (K <= 0 || K % 128 != 0 || N % 8 != 0 || !A_scales || !W_scales) return hipErrorInvalidValue;
    switch (epi.mode) {
        case EPI_STORE:
            if (epi.ldo % 8 != 0 || epi.scale_cols % 4 != 0) return hipErrorInvalidValue;
            return launch_mode<EPI_STORE, true>(A, K, W, A_scales, W_scales, M, N, K, epi, s);
        case EPI_RESID:
            if (epi.ldr % 4 != 0) return hipErrorInvalidValue;
            return launch_mode<EPI_RESID, true>(A, K, W, A_scales, W_scales, M, N, K, epi, s);
        case EPI_GELU_MX:
            if (N % 64 != 0 || epi.ldo % 64 != 0 || !epi.out_scales) return hipErrorInvalidValue;
            return launch_mode<EPI_GELU_MX, true>(A, K, W, A_scales, W_scales, M, N, K, epi, s);
        case EPI_RESID_LN_MX:
            // whole 64-column wave blocks (two scale bytes per row and wave)
            if (epi.ldr % 4 != 0 || N > kResidLnMaxN || N % 64 != 0 || epi.ln_ldo % 64 != 0 ||
                epi.ln_ldo < N || !epi.ln_gain || !epi.ln_shift || !epi.ln_out || !epi.ln_scales)
                return hipErrorInvalidValue;
            return launch_mode<EPI_RESID_LN_MX, true>(A, K, W, A_scales, W_scales, M, N, K, epi, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace upr
