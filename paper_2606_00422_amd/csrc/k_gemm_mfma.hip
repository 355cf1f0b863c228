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
#include "gemm_tile.h"

namespace upr {

namespace gemm_detail {

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
    // (FFN down with its LayerNorm: the accumulators start at the residual)
    if constexpr (!MX && (MODE == EPI_RESID_LN || MODE == EPI_RESID_SCORE))
        if (epi.acc_resid) load_acc_resid<kTM>(acc, epi, m0 + wm * kWM, n0 + wn * kWN, M, N, lane);

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
        case EPI_GELU_PERM:
            if (epi.ldo % 16 != 0 || N % 16 != 0) return hipErrorInvalidValue;
            return launch_mode<EPI_GELU_PERM, false>(A, lda, W, nullptr, nullptr, M, N, K, epi, s);
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

// bf16 models: fp16 projection operands on the matrix cores
template <>
hipError_t launch_gemm<f16, bf16>(const f16* A, int64_t lda, const f16* W, int64_t M, int N,
                                  int K, const Epilogue& epi, hipStream_t s) {
    return launch_gemm_mfma(A, lda, W, M, N, K, epi, s);
}

}  // namespace upr
