// Fused FFN on the matrix cores, for bf16 models with d <= 512:
//   g[m, :] += gelu(a[m, :] W1^T + b1) W2^T + b2
// followed by the LayerNorm of the updated rows (the next layer's LN1, or
// LN_f before the action heads) or by the score head, as the projection
// GEMM's whole-row epilogues do.  The F-wide hidden row never leaves the
// compute unit: the unfused pair (FFN up with a GELU epilogue, FFN down)
// writes and re-reads R x F fp16 values through HBM per layer.
//
// One workgroup = 128 rows (TM = 4 row tiles of 32) and the whole output
// row; eight waves.  Calls whose 128-row tiles would leave compute units idle
// run the unfused pair on short tiles instead (ffn_fused_rows), with the
// same results bit for bit: both feed the matrix cores the same products in
// the same order.
//  * The rows of `a` (the LN2 output) are loaded once into LDS and stay
//    there (d/64 blocks of [rows x 64], the GEMM's swizzled 128-byte rows).
//  * The hidden dimension is walked in chunks of 128.  Up phase: waves in a
//    2 (rows) x 4 (hidden columns) grid compute h = a W1c^T, 64 x 32 each,
//    transposed as in the GEMM (W1 rows are the MFMA's first operand).  Bias
//    and GELU are applied in registers and the fp16 values go to the chunk
//    buffer in LDS.  Down phase: the eight waves side by side along the
//    output (64 columns each, all rows) accumulate h W2c^T into the fp32
//    tile that the epilogue consumes.
//  * Weights come straight from global memory (L2) into registers, in a
//    fragment-major layout built at model creation: fragment (t, kk) of a
//    [N, K] matrix is 1 KB, lane l holding row 32t + l % 32 and eight
//    consecutive positions 16kk + 8(l / 32) .. + 7 of K.  Every weight load
//    of a wave is one coalesced 1 KB block, issued 5-8 fragments ahead; each
//    step's code is kept in program order (scheduling barriers) so that the
//    loads stay ahead and the LDS reads one step ahead.
//  * The hidden index of W2 is stored permuted within each 16-group
//    (kHidPerm: 0-3, 8-11, 4-7, 12-15) so that the up phase's accumulator
//    registers are the down phase's operand chunks as they are: lane
//    (row, half h) of a 32-column tile holds hidden columns 8q + 4h + s
//    (q, s = 0..3), i.e. positions 8h .. 8h + 7 of the permuted order of the
//    16-groups {q = 0, 1} and {q = 2, 3}.  Each lane writes two 16-byte
//    chunks per row tile, no shuffles.
//  * Two workgroup barriers per chunk: before the chunk buffer is
//    overwritten (every wave has finished the previous down phase) and
//    after it is written.
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
// fragments per chunk (4 KB + 16), so a slot refilled with the next chunk's
// fragment is the slot that fragment is read from.
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

// KB = d / 64 (K-blocks of the up phase), TM = row tiles of 32.
template <int MODE, int TM, int KB>
__global__ __launch_bounds__(512, 1) void k_ffn_fused(const f16* __restrict__ A,
                                                      const h8* __restrict__ W1p,
                                                      const h8* __restrict__ W2p,
                                                      const float* __restrict__ b1, float s1,
                                                      int64_t M, int F, Epilogue epi) {
    constexpr int kRows = 32 * TM;
    constexpr int kD = 64 * KB;
    constexpr int kUpSteps = 4 * KB;                   // 16-deep k-steps of the up phase
    constexpr int kSteps = kUpSteps + 2 * kDownSteps;  // weight fragments per chunk
    constexpr int kUT = TM >= 2 ? TM / 2 : 1;          // up-phase row tiles per wave
    constexpr int kRing = ring_depth<KB>();
    static_assert(kSteps % kRing == 0 && kRing <= kUpSteps, "ring slots repeat every chunk");
    __shared__ __attribute__((aligned(16))) char smem[smem_bytes<TM>()];
    f16* const sA = reinterpret_cast<f16*>(smem);                          // [KB][kRows x 64]
    f16* const sH = reinterpret_cast<f16*>(smem + kRows * kMaxD * 2);      // [2][kRows x 64]

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

    // ---- resident rows of a: direct loads into LDS, 8 rows x 128 bytes of
    // one K-block per instruction; rows past M read as zeros.
    {
        const int64_t rows = M - m0 < kRows ? M - m0 : kRows;
        const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<f16*>(A + m0 * kD), (short)0, (int)(rows * kD * 2), 0x00020000);
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
    auto load_frag = [&](int c, int s) __attribute__((always_inline)) -> h8 {
        u32x4 v;
        if (s < kUpSteps) {
            v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                              rsW1, lane_off, ((4 * c + un) * kUpSteps + s) * 1024, 0));
        } else {
            const int q = s - kUpSteps, kkp = q >> 1, j = q & 1;
            v = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                              rsW2, lane_off, ((2 * wave + j) * fsteps + 8 * c + kkp) * 1024, 0));
        }
        return __builtin_bit_cast(h8, v);
    };
    auto active = [&](int s) { return s < kUpSteps ? up_on : dn_on; };
    h8 ring[kRing];
#pragma unroll
    for (int s = 0; s < kRing; ++s)
        if (active(s)) ring[s] = load_frag(0, s);

    f32x16 acc[kTN][TM];
#pragma unroll
    for (int j = 0; j < kTN; ++j)
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[j][i][r] = 0.f;

    __builtin_amdgcn_s_waitcnt(0x0F70);      // vmcnt(0): the resident rows have landed
    asm volatile("" ::: "memory");
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");

    // LDS byte offsets of this lane's fragment row at logical chunk 2m +
    // lhalf of a 128-byte row (swz written out; the key is the same for
    // every 32-row tile of the lane)
    int choff[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) choff[m] = (((2 * m + lhalf) ^ ((lrow >> 1) & 7)) << 4);

    // One weight-stream step: fragment s of chunk c is consumed, and the slot
    // refilled with the fragment kRing steps later (this chunk's or the
    // next one's).
    // (After the last chunk the prefetch still runs: W1 fragments of chunk
    // nch lie past the end of W1p and read as zeros, W2 fragments of chunk
    // nch are the next tile's first ones; either way nothing uses them.)
    auto refill = [&](int c, int s) __attribute__((always_inline)) {
        const int sn = s + kRing;
        if (sn < kSteps) {
            if (active(sn)) ring[s % kRing] = load_frag(c, sn);
        } else if (active(sn - kSteps)) {
            ring[s % kRing] = load_frag(c + 1, sn - kSteps);
        }
    };
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

    for (int c = 0; c < nch; ++c) {
        // ---- up phase: h[kUT tiles][32 hidden] = a W1c^T.  Each step's code
        // stays in program order (scheduling barriers), so the weight loads
        // remain kRing steps ahead of their use and the LDS reads one step.
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
                    hacc[i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ring[s % kRing], af[s & 1][i],
                                                                     hacc[i], 0, 0, 0);
                __builtin_amdgcn_s_setprio(0);
            }
            refill(c, s);
            __builtin_amdgcn_sched_barrier(0);
        }
        // ---- bias, GELU, fp16: lane (row, half h) holds hidden columns
        // 32 un + 8q + 4h + s of its rows; chunk b of a row tile takes q in
        // {2b, 2b + 1}, i.e. down-phase k-step 2 un + b, half h.
        u32x4 hv[kUT][2];
        if (up_on) {
            float4 bq[4];
#pragma unroll
            for (int q = 0; q < 4; ++q)
                bq[q] = *reinterpret_cast<const float4*>(b1 + c * kFC + 32 * un + 8 * q + 4 * lhalf);
#pragma unroll
            for (int i = 0; i < kUT; ++i)
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    unsigned pk[4];
#pragma unroll
                    for (int qq = 0; qq < 2; ++qq) {
                        const int q = 2 * b + qq;
                        const float v0 = gelu_fast(fmaf(hacc[i][4 * q + 0], s1, bq[q].x));
                        const float v1 = gelu_fast(fmaf(hacc[i][4 * q + 1], s1, bq[q].y));
                        const float v2 = gelu_fast(fmaf(hacc[i][4 * q + 2], s1, bq[q].z));
                        const float v3 = gelu_fast(fmaf(hacc[i][4 * q + 3], s1, bq[q].w));
                        pk[2 * qq] = pack2<false>(v0, v1);
                        pk[2 * qq + 1] = pack2<false>(v2, v3);
                    }
                    hv[i][b] = u32x4{pk[0], pk[1], pk[2], pk[3]};
                }
        }
        // every wave has finished reading the previous chunk's buffer
        __builtin_amdgcn_s_waitcnt(0xC07F);
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        if (up_on) {
#pragma unroll
            for (int i = 0; i < kUT; ++i)
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    const int kkp = 2 * un + b;                 // down-phase k-step
                    char* dst = reinterpret_cast<char*>(sH + (kkp >> 2) * kRows * 64) +
                                (um * 64 + i * 32 + lrow) * 128 + choff[kkp & 3];
                    *reinterpret_cast<u32x4*>(dst) = hv[i][b];
                }
        }
        __builtin_amdgcn_s_waitcnt(0xC07F);     // lgkmcnt(0): this wave's writes are done
        asm volatile("" ::: "memory");
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        // ---- down phase: acc += h W2c^T over the chunk's 8 k-steps; the
        // hidden fragments roll through three registers, read two row tiles
        // ahead of their MFMAs
        constexpr int kHQ = kDownSteps * TM;      // hidden fragments per chunk
        h8 hf[3];
        if (dn_on) {
            hf[0] = h_frag(0);
            if (kHQ > 1) hf[1] = h_frag(1);
        }
#pragma unroll
        for (int q = 0; q < kHQ; ++q) {
            const int kkp = q / TM, i = q % TM;
            if (dn_on && q + 2 < kHQ) hf[(q + 2) % 3] = h_frag(q + 2);
            const int s0 = kUpSteps + 2 * kkp;
            if (dn_on) {
                __builtin_amdgcn_s_setprio(1);
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(ring[(s0 + j) % kRing],
                                                                       hf[q % 3], acc[j][i], 0, 0, 0);
                __builtin_amdgcn_s_setprio(0);
            }
            if (i == TM - 1) {
                refill(c, s0);
                refill(c, s0 + 1);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    }

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
hipError_t launch_kb(int KB, unsigned grid, const f16* A, const h8* W1p, const h8* W2p,
                     const float* b1, float s1, int64_t M, int F, const Epilogue& epi, hipStream_t s) {
    switch (KB) {
        case 2: k_ffn_fused<MODE, TM, 2><<<grid, 512, 0, s>>>(A, W1p, W2p, b1, s1, M, F, epi); break;
        case 4: k_ffn_fused<MODE, TM, 4><<<grid, 512, 0, s>>>(A, W1p, W2p, b1, s1, M, F, epi); break;
        case 6: k_ffn_fused<MODE, TM, 6><<<grid, 512, 0, s>>>(A, W1p, W2p, b1, s1, M, F, epi); break;
        case 8: k_ffn_fused<MODE, TM, 8><<<grid, 512, 0, s>>>(A, W1p, W2p, b1, s1, M, F, epi); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

template <int MODE>
hipError_t launch_mode(const f16* A, const h8* W1p, const h8* W2p, const float* b1, float s1,
                       int64_t M, int d, int F, const Epilogue& epi, hipStream_t s) {
    return launch_kb<MODE, 4>(d / 64, (unsigned)((M + 127) / 128), A, W1p, W2p, b1, s1, M, F, epi, s);
}

}  // namespace ffn_detail

bool ffn_fused_rows(int64_t M) { return (M + 127) / 128 >= gemm_detail::device_cus(); }

bool ffn_fused_supported(int d, int F) {
    return (d == 128 || d == 256 || d == 384 || d == 512) && F > 0 && F % ffn_detail::kFC == 0;
}

hipError_t launch_ffn_fused(const f16* A, const f16* W1p, const f16* W2p, const float* b1,
                            float s1, int64_t M, int d, int F, const Epilogue& epi, hipStream_t s) {
    using namespace ffn_detail;
    if (M == 0) return hipSuccess;
    if (!ffn_fused_supported(d, F) || epi.ldr != d || !epi.ln_gain || !epi.ln_shift)
        return hipErrorInvalidValue;
    const h8* w1 = reinterpret_cast<const h8*>(W1p);
    const h8* w2 = reinterpret_cast<const h8*>(W2p);
    switch (epi.mode) {
        case EPI_RESID_LN:
            if (!epi.ln_out || epi.ln_ldo % 4 != 0) return hipErrorInvalidValue;
            return launch_mode<EPI_RESID_LN>(A, w1, w2, b1, s1, M, d, F, epi, s);
        case EPI_RESID_SCORE:
            if (!epi.score_w || !epi.score_b || !epi.score_out) return hipErrorInvalidValue;
            return launch_mode<EPI_RESID_SCORE>(A, w1, w2, b1, s1, M, d, F, epi, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace upr
