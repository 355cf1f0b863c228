// The tail of a layer on the matrix cores, for bf16 models with d <= 512:
//   g[m, :] += o[m, :] Wo^T + bo;   a[m, :] = LN2(g[m, :])
//   g[m, :] += gelu(a[m, :] W1^T + b1) W2^T + b2
// followed by the LayerNorm of the updated rows (the next layer's LN1, or
// LN_f before the action heads) or by the score head, as the projection
// GEMM's whole-row epilogues do.  Neither LN2's output nor the F-wide hidden
// row leaves the compute unit: the unfused sequence (O projection with a
// residual+LN2 epilogue, FFN up with a GELU epilogue, FFN down) writes and
// re-reads R x d + R x F fp16 values through HBM per layer.
//
// One workgroup = 128 rows (TM = 4 row tiles of 32) and the whole output
// row; eight waves.  Calls whose 128-row tiles would leave compute units idle
// run the unfused sequence on short tiles instead (ffn_fused_rows), with the
// same results bit for bit: both feed the matrix cores the same products in
// the same order and round the same sums in the same order.
//  * The tile's rows of the attention output o are loaded into LDS (d/64
//    blocks of [rows x 64], the GEMM's swizzled 128-byte rows).
//  * O projection: the eight waves side by side along the output (64
//    columns each, all rows) accumulate o Wo^T over K = d, transposed as in
//    the GEMM (Wo rows are the MFMA's first operand).  Its epilogue works in
//    the MFMA layout (no LDS staging: the resident rows' LDS is where LN2
//    goes): each lane updates its own residual values, sums them for the
//    row statistics in the same association tree as the GEMM's staged
//    epilogue, and writes LN2 of its columns as fp16 straight into the
//    resident-row layout, where a then stays.  The row statistics meet in
//    the chunk buffer's LDS, free until the first chunk.  The updated
//    residual never goes to HBM: it stays in the accumulators, divided by
//    W2's power-of-two scale, as the FFN down's starting value.
//  * The hidden dimension is walked in chunks of 128.  Up phase: waves in a
//    2 (rows) x 4 (hidden columns) grid compute h = a W1c^T, 64 x 32 each.
//    Bias and GELU are applied in registers and the fp16 values go to the
//    chunk buffer in LDS.  Down phase: as the O projection, the eight waves
//    accumulate h W2c^T into the fp32 tile that the final epilogue consumes.
//  * Weights come straight from global memory (L2) into registers, in a
//    fragment-major layout built at model creation: fragment (t, kk) of a
//    [N, K] matrix is 1 KB, lane l holding row 32t + l % 32 and eight
//    consecutive positions 16kk + 8(l / 32) .. + 7 of K.  Every weight load
//    of a wave is one coalesced 1 KB block, issued 5-8 fragments ahead in
//    one stream (Wo, W1 of chunk 0, then W1 of chunk c with W2 of chunk
//    c - 1); each step's code is kept in program order (scheduling
//    barriers) so that the loads stay ahead and the LDS reads one step
//    ahead.
//  * The hidden index of W2 is stored permuted within each 16-group
//    (kHidPerm: 0-3, 8-11, 4-7, 12-15) so that the up phase's accumulator
//    registers are the down phase's operand chunks as they are: lane
//    (row, half h) of a 32-column tile holds hidden columns 8q + 4h + s
//    (q, s = 0..3), i.e. positions 8h .. 8h + 7 of the permuted order of the
//    16-groups {q = 0, 1} and {q = 2, 3}.  Each lane writes two 16-byte
//    chunks per row tile, no shuffles.
//  * Each wave runs the up phase and GELU of chunk c before the down phase
//    of chunk c - 1 (whose hidden values are in the chunk buffer), then two
//    workgroup barriers: before the buffer is overwritten with chunk c
//    (every wave has finished the down phase) and after it is written.
//    With no barrier between a wave's GELU and its next MFMAs, the two
//    waves of a SIMD drift apart and one's GELU overlaps the other's
//    matrix-core work (1-1.5% faster than the down phase right after the
//    write, bit-identical).
//  * A wave raises its issue priority for each run of MFMAs, so the other
//    wave on its SIMD fills the matrix core's gaps with its loads and GELU.
#include "gemm_tile.h"

namespace upr {

namespace ffn_detail {

using namespace gemm_detail;

constexpr int kFC = 128;              // hidden columns per chunk
constexpr int kMaxD = 512;            // widest row (the tile spans whole rows)
// Weight fragments in flight per wave, by K-blocks of the up phase: as deep
// as the 256 registers of two waves per SIMD allow, and a divisor of the
// fragments per block of the stream (4 KB + 16), so a step's slot depends
// only on its place in its block.
template <int KB>
constexpr int ring_depth() { return KB == 8 ? 6 : KB == 6 ? 5 : 8; }
constexpr int kDownSteps = kFC / 16;  // k-steps of the down phase per chunk (8)

// Epilogue LDS (after the last up phase the resident rows are free):
// eight staging regions, the LayerNorm statistics, the score shares.
constexpr int kEpiRegion = 32 * kStage32 * 4;
constexpr int kEpiBytes = 8 * kEpiRegion + 2 * 32 * 8 * 8 + 2 * 32 * 8 * 4;

template <int TM>
constexpr int smem_bytes() {
    constexpr int main = 32 * TM * kMaxD * 2 + 32 * TM * kFC * 2;
    return main > kEpiBytes ? main : kEpiBytes;
}

// Epilogue of the O projection in the MFMA layout: lane (row 32i + l%32,
// half h) of wave w holds columns 64w + 32j + 8q + 4h + (0..3) of that row
// in acc[j][i][4q .. 4q+3].  Per 32-row pass: g = r + (acc * s + bo), the
// row's mean and squared deviations over the wave's 64 columns, exchanged
// through `lnx` at a workgroup barrier, then LN2 as fp16 into the resident
// rows' LDS (K-block w, the swizzled 128-byte rows).  g itself is not
// stored: acc[j][i] leaves as g * inv2 (inv2 = 1 / FFN down's scale, a power
// of two), the starting value of the FFN down accumulators, so the final
// epilogue's update acc * s2 + b2 completes the residual stream (as the
// unfused FFN-down GEMM does when it loads g into its accumulators).  Association: the staged epilogue sums each run of four columns,
// (x + y) + (z + w), then pairs the runs 32 columns apart, then 16, then 8,
// then 4 (the exchange over its 16 lanes); here the same pairs are in
// registers (j, then q's high bit, then its low bit) and the last is the
// lane pair (l, l + 32), so the sums, and everything after, are the same
// bits.  Rows past M: the residual descriptor ends at row M (loads read
// zeros); their values are finite and never stored.
template <int TM, int KB>
__device__ __forceinline__ void oproj_epilogue(f32x16 (&acc)[kTN][TM], f16* const sA, float* const lnx,
                                               const float* const par, int64_t m0, int64_t M,
                                               const Epilogue& epa, float inv2, int wave, int lane,
                                               bool cols_on) {
    constexpr int kRows = 32 * TM, kD = 64 * KB;
    const int lrow = lane & 31, lhalf = lane >> 5;
    const float sc = epa.acc_scale;
    const int64_t rows_valid = M - m0 < kRows ? M - m0 : kRows;
    const __amdgpu_buffer_rsrc_t rs = __builtin_amdgcn_make_buffer_rsrc(
        epa.resid + m0 * kD, (short)0, (int)(rows_valid * kD * 4), 0x00020000);
    const __amdgpu_buffer_rsrc_t rsrc = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<unsigned short*>(static_cast<const unsigned short*>(epa.resid_src)) + m0 * kD, (short)0,
        (int)(rows_valid * kD * 2), 0x00020000);
    const bool from_src = epa.resid_src != nullptr;
    const float cnt = cols_on ? 64.f : 0.f;
    const int colw = 64 * wave + 4 * lhalf;
    // residual values of pass i (lane's row 32i + l%32); the first pass's
    // are requested before the barrier
    auto load_r = [&](int i, float4 (&dst)[kTN][4]) __attribute__((always_inline)) {
        const unsigned vrow = (unsigned)(i * 32 + lrow) * kD;
#pragma unroll
        for (int j = 0; j < kTN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const unsigned col = (unsigned)(colw + 32 * j + 8 * q);
                if (!cols_on) {
                    dst[j][q] = make_float4(0.f, 0.f, 0.f, 0.f);
                } else if (from_src) {
                    typedef __attribute__((ext_vector_type(2))) unsigned u32x2;
                    const u32x2 w = __builtin_bit_cast(
                        u32x2, __builtin_amdgcn_raw_buffer_load_b64(rsrc, (vrow + col) * 2, 0, 0));
                    dst[j][q] = make_float4(__uint_as_float(w.x << 16), __uint_as_float(w.x & 0xffff0000u),
                                            __uint_as_float(w.y << 16), __uint_as_float(w.y & 0xffff0000u));
                } else {
                    dst[j][q] = __builtin_bit_cast(
                        float4, __builtin_amdgcn_raw_buffer_load_b128(rs, (vrow + col) * 4, 0, 0));
                }
            }
    };
    float4 rb[kTN][4];
    load_r(0, rb);
    // every wave has read its last fragment of o: the resident rows' LDS
    // can take LN2
    __builtin_amdgcn_s_waitcnt(0xC07F);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        if (i > 0) load_r(i, rb);
        float4 (&o)[kTN][4] = rb;
#pragma unroll
        for (int j = 0; j < kTN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int col = colw + 32 * j + 8 * q;
                const float4 r = o[j][q];
                const float4 b = cols_on ? *reinterpret_cast<const float4*>(par + col)
                                         : make_float4(0.f, 0.f, 0.f, 0.f);
                f32x16& a = acc[j][i];
                o[j][q] = make_float4(r.x + fmaf(a[4 * q + 0], sc, b.x), r.y + fmaf(a[4 * q + 1], sc, b.y),
                                      r.z + fmaf(a[4 * q + 2], sc, b.z), r.w + fmaf(a[4 * q + 3], sc, b.w));
                a[4 * q + 0] = o[j][q].x * inv2;
                a[4 * q + 1] = o[j][q].y * inv2;
                a[4 * q + 2] = o[j][q].z * inv2;
                a[4 * q + 3] = o[j][q].w * inv2;
            }
        // the row's sum over the wave's columns, then its squared deviations
        auto tree = [&](const float (&t)[kTN][4]) {
            float u[4];
#pragma unroll
            for (int q = 0; q < 4; ++q) u[q] = t[0][q] + t[1][q];
            const float v0 = u[0] + u[2], v1 = u[1] + u[3];
            const float w = v0 + v1;
            return w + __shfl_xor(w, 32, 64);
        };
        float t[kTN][4];
#pragma unroll
        for (int j = 0; j < kTN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q)
                t[j][q] = cols_on ? (o[j][q].x + o[j][q].y) + (o[j][q].z + o[j][q].w) : 0.f;
        const float mrow = cnt > 0.f ? tree(t) / cnt : 0.f;
#pragma unroll
        for (int j = 0; j < kTN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float sq = 0.f;
                if (cols_on) {
                    const float u0 = o[j][q].x - mrow, u1 = o[j][q].y - mrow, u2 = o[j][q].z - mrow,
                                u3 = o[j][q].w - mrow;
                    sq = fmaf(u0, u0, fmaf(u1, u1, fmaf(u2, u2, u3 * u3)));
                }
                t[j][q] = sq;
            }
        const float qrow = tree(t);
        float2* const X = reinterpret_cast<float2*>(lnx) + (i & 1) * (32 * 8);
        if (lhalf == 0) X[lrow * 8 + wave] = make_float2(mrow, qrow);
        __builtin_amdgcn_s_waitcnt(0xC07F);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
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
            const int c = kD - w * 64;
            n_w[w] = (float)(c < 0 ? 0 : c > 64 ? 64 : c);
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
        const float rstd = 1.0f / sqrtf(M2 / tot + epa.ln_eps);
        if (cols_on) {
            char* const rowp = reinterpret_cast<char*>(sA + wave * kRows * 64) + (i * 32 + lrow) * 128;
            const int key = (lrow >> 1) & 7;
#pragma unroll
            for (int j = 0; j < kTN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int col = colw + 32 * j + 8 * q;
                    const float4 g = *reinterpret_cast<const float4*>(par + kD + col);
                    const float4 b = *reinterpret_cast<const float4*>(par + 2 * kD + col);
                    const float4 h = o[j][q];
                    const unsigned lo = pack2<false>(fmaf((h.x - mu) * rstd, g.x, b.x),
                                                     fmaf((h.y - mu) * rstd, g.y, b.y));
                    const unsigned hi = pack2<false>(fmaf((h.z - mu) * rstd, g.z, b.z),
                                                     fmaf((h.w - mu) * rstd, g.w, b.w));
                    typedef __attribute__((ext_vector_type(2))) unsigned u32x2;
                    *reinterpret_cast<u32x2*>(rowp + (((4 * j + q) ^ key) << 4) + 8 * lhalf) = u32x2{lo, hi};
                }
        }
    }
    // LN2 is in LDS before the up phase reads it
    __builtin_amdgcn_s_waitcnt(0xC07F);
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
}

// KB = d / 64 (K-blocks of the up phase), TM = row tiles of 32.  O: the
// attention output rows (fp16, [M, d]).
template <int MODE, int TM, int KB>
__global__ __launch_bounds__(512, 1) void k_ffn_fused(const f16* __restrict__ O,
                                                      const h8* __restrict__ WoP,
                                                      const h8* __restrict__ W1p,
                                                      const h8* __restrict__ W2p,
                                                      const float* __restrict__ b1, float s1,
                                                      int64_t M, int F, Epilogue epa, Epilogue epi) {
    constexpr int kRows = 32 * TM;
    constexpr int kD = 64 * KB;
    constexpr int kUpSteps = 4 * KB;                   // 16-deep k-steps of the up phase
    constexpr int kSteps = kUpSteps + 2 * kDownSteps;  // weight fragments per chunk (and per block)
    constexpr int kUT = TM >= 2 ? TM / 2 : 1;          // up-phase row tiles per wave
    constexpr int kRing = ring_depth<KB>();
    static_assert(kSteps % kRing == 0 && kRing <= kUpSteps, "ring slots repeat every block");
    __shared__ __attribute__((aligned(16))) char smem[smem_bytes<TM>()];
    f16* const sA = reinterpret_cast<f16*>(smem);                          // [KB][kRows x 64]
    f16* const sH = reinterpret_cast<f16*>(smem + kRows * kMaxD * 2);      // [2][kRows x 64]
    // The O projection epilogue's bias, LN2 gain and LN2 shift ([3][kD]),
    // staged once behind its statistics exchange in the chunk buffer's LDS
    // (free until the first chunk), so that its passes read them from LDS
    // instead of one global round trip per column group and pass.
    constexpr int kLnxBytes = 2 * 32 * 8 * 8;
    static_assert(kLnxBytes + 3 * kMaxD * 4 <= 32 * TM * kFC * 2, "parameters fit in the chunk buffer");
    float* const sPar = reinterpret_cast<float*>(smem + kRows * kMaxD * 2 + kLnxBytes);

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int lrow = lane & 31, lhalf = lane >> 5;
    const int t = xcd_tile(blockIdx.x, gridDim.x);
    const int64_t m0 = (int64_t)t * kRows;
    const int nch = F / kFC;
    const int fsteps = F / 16;

    // up-phase role: rows 64 um .. (TM = 1: 32 rows on waves 0-3), hidden
    // columns 32 un ..
    const int um = TM >= 2 ? wave >> 2 : 0, un = wave & 3;
    const bool up_on = TM >= 2 || wave < 4;
    // down-phase role: output columns 64 wave .. +63
    const bool dn_on = kD == kMaxD || wave * 64 < kD;

    float par[3];
    if (tid < kD) {
        par[0] = epa.bias[tid];
        par[1] = epa.ln_gain[tid];
        par[2] = epa.ln_shift[tid];
    }
    // ---- the tile's rows of o: direct loads into LDS, 8 rows x 128 bytes
    // of one K-block per instruction; rows past M read as zeros.
    {
        const int64_t rows = M - m0 < kRows ? M - m0 : kRows;
        const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<f16*>(O + m0 * kD), (short)0, (int)(rows * kD * 2), 0x00020000);
        const int r8 = lane >> 3, slot = lane & 7;
#pragma unroll
        for (int ins = 0; ins < (kRows / 8) * KB / 8; ++ins) {
            const int g = ins * 8 + wave;                  // instruction index, all waves
            const int kb = g / (kRows / 8), blk = g % (kRows / 8);
            const int row = blk * 8 + r8;
            const int voff = row * kD * 2 + kb * 128 + ((slot ^ ((row >> 1) & 7)) << 4);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rsA, (__attribute__((address_space(3))) void*)(sA + kb * kRows * 64 + blk * 8 * 64), 16,
                voff, 0, 0, 0);
        }
    }

    // ---- weight fragment stream of chunk c: step s < kUpSteps is W1
    // fragment (4c + un, s); then W2 fragments (2 wave + j, 8c + kk') for
    // kk' = 0..7, j = 0, 1.  Buffer loads: the lane's 16 bytes at a fixed
    // offset, the fragment's position as a wave-uniform scalar offset (no
    // per-load address registers); past the end a load reads zeros.
    const __amdgpu_buffer_rsrc_t rsW1 = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<h8*>(W1p), (short)0, (int)((int64_t)F * kD * 2), 0x00020000);
    const __amdgpu_buffer_rsrc_t rsW2 = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<h8*>(W2p), (short)0, (int)((int64_t)F * kD * 2), 0x00020000);
    const int lane_off = lane * 16;
    auto load_w1 = [&](int c, int s) __attribute__((always_inline)) -> u32x4 {
        return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                          rsW1, lane_off, ((4 * c + un) * kUpSteps + s) * 1024, 0));
    };
    auto load_w2 = [&](int c, int q) __attribute__((always_inline)) -> u32x4 {
        const int kkp = q >> 1, j = q & 1;
        return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                          rsW2, lane_off, ((2 * wave + j) * fsteps + 8 * c + kkp) * 1024, 0));
    };
    constexpr int kW2Steps = 2 * kDownSteps;
    // O projection: k-step kk, column tile j of the wave is stream
    // step 2 kk + j < kOSteps, Wo fragment (2 wave + j, kk); those steps
    // come before chunk 0's.  Slots count from the start of chunk 0, so a
    // chunk-0 fragment prefetched during the O projection lands in the slot
    // the chunk loop reads it from.
    constexpr int kOK = 4 * KB;                        // k-steps of the O projection (d / 16)
    constexpr int kOSteps = 2 * kOK;
    static_assert(kOSteps >= kRing, "the O projection fills the ring");
    auto slot_o = [](int s) { return ((s - kOSteps) % kRing + kRing) % kRing; };
    const __amdgpu_buffer_rsrc_t rsWo = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<h8*>(WoP), (short)0, kD * kD * 2, 0x00020000);
    auto load_o = [&](int s) __attribute__((always_inline)) -> u32x4 {
        const int kk = s >> 1, j = s & 1;
        return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                                    rsWo, lane_off, ((2 * wave + j) * kOK + kk) * 1024, 0));
    };
    u32x4 ring[kRing];     // fragments as 32-bit words (16-bit vector phis get split)
#pragma unroll
    for (int s = 0; s < kRing; ++s)
        if (dn_on) ring[slot_o(s)] = load_o(s);

    f32x16 acc[kTN][TM];
#pragma unroll
    for (int j = 0; j < kTN; ++j)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[j][i][r] = 0.f;

    __builtin_amdgcn_s_waitcnt(0x0F70);      // vmcnt(0): the resident rows have landed
    if (tid < kD) {
        sPar[tid] = par[0];
        sPar[kD + tid] = par[1];
        sPar[2 * kD + tid] = par[2];
    }
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");

    // LDS byte offsets of this lane's fragment row at logical chunk 2m +
    // lhalf of a 128-byte row (swz written out; the key is the same for
    // every 32-row tile of the lane)
    int choff[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) choff[m] = (((2 * m + lhalf) ^ ((lrow >> 1) & 7)) << 4);

    // operand fragments from LDS, read one step ahead of their MFMAs
    auto a_frags = [&](int s, h8 (&dst)[kUT]) __attribute__((always_inline)) {
        const char* base = reinterpret_cast<const char*>(sA + (s >> 2) * kRows * 64);
#pragma unroll
        for (int i = 0; i < kUT; ++i)
            dst[i] = *reinterpret_cast<const h8*>(base + (um * 64 + i * 32 + lrow) * 128 + choff[s & 3]);
    };
    // hidden fragment q = kk' TM + i (k-step kk', row tile i)
    auto h_frag = [&](int q) __attribute__((always_inline)) -> h8 {
        const int kkp = q / TM, i = q % TM;
        const char* base = reinterpret_cast<const char*>(sH + (kkp >> 2) * kRows * 64);
        return *reinterpret_cast<const h8*>(base + (i * 32 + lrow) * 128 + choff[kkp & 3]);
    };

    {
        // ---- O projection: acc = o Wo^T, the operand fragments of o
        // rolling through three registers two row tiles ahead of their
        // MFMAs, as in the down phase
        constexpr int kOQ = kOK * TM;
        auto o_frag = [&](int q) __attribute__((always_inline)) -> h8 {
            const int kk = q / TM, i = q % TM;
            const char* base = reinterpret_cast<const char*>(sA + (kk >> 2) * kRows * 64);
            return *reinterpret_cast<const h8*>(base + (i * 32 + lrow) * 128 + choff[kk & 3]);
        };
        auto refill_o = [&](int s) __attribute__((always_inline)) {
            const int sn = s + kRing;
            if (sn < kOSteps) {
                if (dn_on) ring[slot_o(s)] = load_o(sn);
            } else if (up_on) {
                ring[slot_o(s)] = load_w1(0, sn - kOSteps);
            }
        };
        h8 of[3];
        if (dn_on) {
            of[0] = o_frag(0);
            of[1] = o_frag(1);
        }
#pragma unroll
        for (int q = 0; q < kOQ; ++q) {
            const int kk = q / TM, i = q % TM;
            if (dn_on && q + 2 < kOQ) of[(q + 2) % 3] = o_frag(q + 2);
            if (dn_on) {
                __builtin_amdgcn_s_setprio(1);
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(h8, ring[slot_o(2 * kk + j)]), of[q % 3],
                                                                       acc[j][i], 0, 0, 0);
                __builtin_amdgcn_s_setprio(0);
            }
            if (i == TM - 1) {
                refill_o(2 * kk);
                refill_o(2 * kk + 1);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
        // (acc leaves holding the updated residual / FFN down's scale)
        oproj_epilogue<TM, KB>(acc, sA, reinterpret_cast<float*>(sH), sPar, m0, M, epa, 1.0f / epi.acc_scale,
                               wave, lane, dn_on);
    }


    // ---- the weight stream after the O projection, in blocks: block 0 is
    // chunk 0's W1 steps; block c (1 <= c < nch) holds chunk c's W1 steps,
    // then chunk c - 1's W2 steps; the last block is the last chunk's W2
    // steps.  Blocks after the first are kSteps long, a multiple of kRing,
    // so a step's slot follows from its place in its block alone; a consumed
    // slot is refilled with the step kRing later.  Where the next step may
    // lie in either matrix (at a block boundary) the choice is made on the
    // scalar unit, so the ring slots need no branch merges.  Loads past a
    // matrix's end read zeros (W1 past the last chunk; W2 rows of waves
    // without output columns) and are never used.
    auto load_sel = [&](bool w1, int c1, int s1, int c2, int q2) __attribute__((always_inline)) -> u32x4 {
        const int o1 = ((4 * c1 + un) * kUpSteps + s1) * 1024;
        const int o2 = ((2 * wave + (q2 & 1)) * fsteps + 8 * c2 + (q2 >> 1)) * 1024;
        return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(w1 ? rsW1 : rsW2, lane_off,
                                                                               w1 ? o1 : o2, 0));
    };
    // step sp of block c (1 <= c <= nch; block nch is the last one)
    auto fetch = [&](int c, int sp) __attribute__((always_inline)) -> u32x4 {
        // (a step across a block boundary has sp < kRing <= 2 kDownSteps,
        // which in the last block is a W2 step)
        if (sp < kUpSteps) return load_sel(c < nch, c, sp, c - 1, sp);
        return load_w2(c - 1, sp - kUpSteps);
    };
    auto refill_first = [&](int s) __attribute__((always_inline)) {           // block 0
        const int sn = s + kRing;
        ring[s % kRing] = sn < kUpSteps ? load_w1(0, sn) : fetch(1, sn - kUpSteps);
    };
    auto refill_mid = [&](int c, int s) __attribute__((always_inline)) {      // block c
        const int sn = s + kRing;
        ring[(kUpSteps + s) % kRing] = sn < kSteps ? fetch(c, sn) : fetch(c + 1, sn - kSteps);
    };
    auto refill_last = [&](int j) __attribute__((always_inline)) {          // last block
        const int jn = j + kRing;
        ring[(kUpSteps + j) % kRing] = jn < kW2Steps ? load_w2(nch - 1, jn) : load_w1(nch, jn - kW2Steps);
    };

    // The lane's LDS offsets pass through an opaque statement at the start
    // of each phase, so the compiler derives the phase's fragment addresses
    // there instead of keeping every one of them live across the chunk loop.
    auto fresh_offsets = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int m = 0; m < 4; ++m) asm volatile("" : "+v"(choff[m]));
    };
    // ---- up phase: h[kUT tiles][32 hidden] = a W1c^T, its weight steps at
    // slots (base + s) % kRing; then bias, GELU and fp16 into pk.  Each
    // step's code stays in program order (scheduling barriers), so the
    // weight loads remain kRing steps ahead of their use and the LDS reads
    // one step.  The chunk's bias is requested with the first step, ahead
    // of the ring loads that GELU must not wait for.
    unsigned pk[kUT][2][4];
    auto up_gelu = [&](auto base_c, int c, auto&& refill) __attribute__((always_inline)) {
        constexpr int base = decltype(base_c)::value;
        fresh_offsets();
        float4 bq[4];
        f32x16 hacc[kUT];
#pragma unroll
        for (int i = 0; i < kUT; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) hacc[i][r] = 0.f;
        h8 af[2][kUT];
        if (up_on) a_frags(0, af[0]);
#pragma unroll
        for (int s = 0; s < kUpSteps; ++s) {
            if (up_on && s + 1 < kUpSteps) a_frags(s + 1, af[(s + 1) & 1]);
            if (up_on) {
                __builtin_amdgcn_s_setprio(1);
#pragma unroll
                for (int i = 0; i < kUT; ++i)
                    hacc[i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(h8, ring[(base + s) % kRing]), af[s & 1][i],
                                                                     hacc[i], 0, 0, 0);
                __builtin_amdgcn_s_setprio(0);
            }
            refill(s);
            __builtin_amdgcn_sched_barrier(0);
        }
        // lane (row, half h) holds hidden columns 32 un + 8q + 4h + s of its
        // rows; chunk b of a row tile takes q in {2b, 2b + 1}, i.e.
        // down-phase k-step 2 un + b, half h
        if (up_on) {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                bq[q] = *reinterpret_cast<const float4*>(b1 + c * kFC + 32 * un + 8 * q + 4 * lhalf);
#pragma unroll
            for (int i = 0; i < kUT; ++i)
#pragma unroll
                for (int b = 0; b < 2; ++b)
#pragma unroll
                    for (int qq = 0; qq < 2; ++qq) {
                        const int q = 2 * b + qq;
                        const float v0 = gelu_fast(fmaf(hacc[i][4 * q + 0], s1, bq[q].x));
                        const float v1 = gelu_fast(fmaf(hacc[i][4 * q + 1], s1, bq[q].y));
                        const float v2 = gelu_fast(fmaf(hacc[i][4 * q + 2], s1, bq[q].z));
                        const float v3 = gelu_fast(fmaf(hacc[i][4 * q + 3], s1, bq[q].w));
                        pk[i][b][2 * qq] = pack2<false>(v0, v1);
                        pk[i][b][2 * qq + 1] = pack2<false>(v2, v3);
                    }
        }
        __builtin_amdgcn_sched_barrier(0);
    };
    // the chunk's hidden values into the chunk buffer, then a barrier before
    // any wave's down phase reads them
    auto write_h = [&]() __attribute__((always_inline)) {
        if (up_on) {
#pragma unroll
            for (int i = 0; i < kUT; ++i)
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    const int kkp = 2 * un + b;                 // down-phase k-step
                    char* dst = reinterpret_cast<char*>(sH + (kkp >> 2) * kRows * 64) +
                                (um * 64 + i * 32 + lrow) * 128 + choff[kkp & 3];
                    *reinterpret_cast<u32x4*>(dst) = u32x4{pk[i][b][0], pk[i][b][1], pk[i][b][2], pk[i][b][3]};
                }
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);     // lgkmcnt(0): this wave's writes are done
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };
    // ---- down phase: acc += h W2c^T over the chunk's 8 k-steps, W2 step
    // j at slot (base + j) % kRing; the hidden fragments roll through three
    // registers, read two row tiles ahead of their MFMAs
    constexpr int kHQ = kDownSteps * TM;          // hidden fragments per chunk
    auto down_phase = [&](auto base_c, auto&& refill) __attribute__((always_inline)) {
        constexpr int base = decltype(base_c)::value;
        fresh_offsets();
        h8 hf[3];
        if (dn_on) {
            hf[0] = h_frag(0);
            if (kHQ > 1) hf[1] = h_frag(1);
        }
#pragma unroll
        for (int q = 0; q < kHQ; ++q) {
            const int kkp = q / TM, i = q % TM;
            if (dn_on && q + 2 < kHQ) hf[(q + 2) % 3] = h_frag(q + 2);
            const int s0 = 2 * kkp;                     // W2 step of the pair
            if (dn_on) {
                __builtin_amdgcn_s_setprio(1);
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(h8, ring[(base + s0 + j) % kRing]),
                                                                       hf[q % 3], acc[j][i], 0, 0, 0);
                __builtin_amdgcn_s_setprio(0);
            }
            if (i == TM - 1) {
                refill(s0);
                refill(s0 + 1);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };
    // every wave has finished reading the chunk buffer
    auto sync_reads = [&]() __attribute__((always_inline)) {
        __builtin_amdgcn_s_waitcnt(0xC07F);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
    };
    // block 0: chunk 0's up phase and GELU (the chunk buffer is free: the O
    // projection's epilogue finished with it at its last barrier)
    up_gelu(std::integral_constant<int, 0>{}, 0, refill_first);
    write_h();
    // block c: chunk c's up phase and GELU, then chunk c - 1's down phase.
    // With no barrier between GELU and the down phase, a wave that finishes
    // its GELU goes on to its MFMAs while the other wave of its SIMD may
    // still be in GELU, so the matrix core and the vector ALUs overlap.
    for (int c = 1; c < nch; ++c) {
        up_gelu(std::integral_constant<int, kUpSteps>{}, c, [&](int s) { refill_mid(c, s); });
        down_phase(std::integral_constant<int, 2 * kUpSteps>{}, [&](int s) { refill_mid(c, kUpSteps + s); });
        sync_reads();
        write_h();
    }
    down_phase(std::integral_constant<int, kUpSteps>{}, refill_last);

    // ---- epilogue: residual update, then LayerNorm or the score head, on
    // whole rows.  Its staging regions reuse the resident rows' LDS and, for
    // 32-row tiles, the chunk buffer as well: every wave must have finished
    // its last down phase first (waves without output columns get here
    // early).
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    char* const region = smem + wave * kEpiRegion;
    float* const lnx = reinterpret_cast<float*>(smem + 8 * kEpiRegion);
    float* const scx = reinterpret_cast<float*>(smem + 8 * kEpiRegion + 2 * 32 * 8 * 8);
    store_tile<MODE, TM>(acc, region, m0, wave * 64, M, kD, epi, lane, lnx, wave, scx);
}

template <int MODE, int TM>
hipError_t launch_kb(int KB, unsigned grid, const f16* O, const h8* WoP, const h8* W1p, const h8* W2p,
                     const float* b1, float s1, int64_t M, int F, const Epilogue& epa, const Epilogue& epi,
                     hipStream_t s) {
    switch (KB) {
        case 2: k_ffn_fused<MODE, TM, 2><<<grid, 512, 0, s>>>(O, WoP, W1p, W2p, b1, s1, M, F, epa, epi); break;
        case 4: k_ffn_fused<MODE, TM, 4><<<grid, 512, 0, s>>>(O, WoP, W1p, W2p, b1, s1, M, F, epa, epi); break;
        case 6: k_ffn_fused<MODE, TM, 6><<<grid, 512, 0, s>>>(O, WoP, W1p, W2p, b1, s1, M, F, epa, epi); break;
        case 8: k_ffn_fused<MODE, TM, 8><<<grid, 512, 0, s>>>(O, WoP, W1p, W2p, b1, s1, M, F, epa, epi); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int MODE>
hipError_t launch_mode(const f16* O, const h8* WoP, const Epilogue& epa, const h8* W1p, const h8* W2p,
                       const float* b1, float s1, int64_t M, int d, int F, const Epilogue& epi, hipStream_t s) {
    return launch_kb<MODE, 4>(d / 64, (unsigned)((M + 127) / 128), O, WoP, W1p, W2p, b1, s1, M, F, epa, epi, s);
}

}  // namespace ffn_detail

bool ffn_fused_rows(int64_t M) { return (M + 127) / 128 >= gemm_detail::device_cus(); }

bool ffn_fused_supported(int d, int F) {
    return (d == 128 || d == 256 || d == 384 || d == 512) && F > 0 && F % ffn_detail::kFC == 0;
}

hipError_t launch_ffn_fused(const f16* O, const f16* WoP, const Epilogue& epa, const f16* W1p,
                            const f16* W2p, const float* b1, float s1, int64_t M, int d, int F,
                            const Epilogue& epi, hipStream_t s) {
    using namespace ffn_detail;
    if (M == 0) return hipSuccess;
    if (!ffn_fused_supported(d, F) || epi.ldr != d || !epi.ln_gain || !epi.ln_shift)
        return hipErrorInvalidValue;
    if (epa.mode != EPI_RESID_LN || epa.acc_resid || epa.resid != epi.resid || epa.ldr != d || !epa.bias ||
        !epa.ln_gain || !epa.ln_shift || !epi.acc_resid)
        return hipErrorInvalidValue;
    const h8* wo = reinterpret_cast<const h8*>(WoP);
    const h8* w1 = reinterpret_cast<const h8*>(W1p);
    const h8* w2 = reinterpret_cast<const h8*>(W2p);
    switch (epi.mode) {
        case EPI_RESID_LN:
            if (!epi.ln_out || epi.ln_ldo % 4 != 0) return hipErrorInvalidValue;
            return launch_mode<EPI_RESID_LN>(O, wo, epa, w1, w2, b1, s1, M, d, F, epi, s);
        case EPI_RESID_SCORE:
            if (!epi.score_w || !epi.score_b || !epi.score_out) return hipErrorInvalidValue;
            return launch_mode<EPI_RESID_SCORE>(O, wo, epa, w1, w2, b1, s1, M, d, F, epi, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace upr
