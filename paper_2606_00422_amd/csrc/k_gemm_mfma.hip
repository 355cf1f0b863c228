// Projection GEMM on the matrix cores: out = A[M,K] W[N,K]^T (+ epilogue),
// A and W fp16 (both K-contiguous), fp32 accumulation with
// v_mfma_f32_32x32x16_f16.
//
// Block tile 256 (rows of A) x 256 (rows of W), K in steps of 64, eight
// waves in a 2 (M) x 4 (N) grid, each owning 128 x 64 outputs = 4 x 2 MFMA
// tiles.  The MFMA computes the transposed tile, C^T = W A^T (W as the
// first operand), so each lane ends up holding four CONSECUTIVE output
// columns of one row: epilogues read/write 16 bytes (fp32 residual) or 8
// bytes (fp16/bf16) per lane instead of scattering 2-byte values.
//
// A and W tiles go straight from global memory into LDS (buffer loads with
// the LDS bit: no staging registers, out-of-range rows read as zeros),
// double-buffered: each K-step reads all its operand fragments from LDS,
// issues the next K-step's loads, then runs its 32 MFMAs while they fly.  LDS rows are 128 bytes (64 fp16) and the
// eight 16-byte chunks of each row are XOR-swizzled so fragment reads are
// bank-conflict free.
//
// Tile order is XCD-aware: workgroup b runs on XCD b % 8 and the tiles are
// renumbered so each XCD sweeps a contiguous range of (M-panel, N-tile)
// pairs; the N-tiles of one A row-panel then share one L2.
#include "epilogue.h"
#include "upr_plan.h"

namespace upr {

namespace gemm_detail {

typedef __attribute__((ext_vector_type(8))) _Float16 h8;
typedef __attribute__((ext_vector_type(4))) _Float16 h4;
typedef __attribute__((ext_vector_type(4))) __bf16 b4;
typedef __attribute__((ext_vector_type(16))) float f32x16;

// Tile shapes.  Big: 256x256, K-step 64, 8 waves of 128x64, one workgroup
// per CU (128 KB LDS).  Wide: 256x128, K-step 32, 4 waves of 128x64, two
// workgroups per CU (48 KB LDS each), so one workgroup's epilogue overlaps
// the other's MFMAs.
template <int BM_, int BN_, int BK_, int WAVES_M_, int WAVES_N_, int MIN_BLOCKS_>
struct Tile {
    static constexpr int BM = BM_, BN = BN_, BK = BK_;
    static constexpr int WAVES_M = WAVES_M_, WAVES_N = WAVES_N_;
    static constexpr int THREADS = 64 * WAVES_M * WAVES_N, MIN_BLOCKS = MIN_BLOCKS_;
    static constexpr int WM = BM / WAVES_M, WN = BN / WAVES_N;     // per-wave tile
    static constexpr int TM = WM / 32, TN = WN / 32;               // 32x32 MFMA tiles
    static constexpr int CPR = BK / 8;                             // 16-byte chunks per LDS row
    static constexpr int RPB = 16 / CPR;                           // rows per 256-byte bank line
    static constexpr int LOADS_A = BM * CPR / THREADS, LOADS_B = BN * CPR / THREADS;
    static_assert(BM * CPR % (THREADS) == 0 && BN * CPR % THREADS == 0, "whole loads per thread");
    static_assert(LOADS_A % 1 == 0 && 64 % CPR == 0, "a wave's load covers whole rows");
};
using TileBig = Tile<256, 256, 64, 2, 4, 1>;
using TileWide = Tile<256, 128, 32, 2, 2, 2>;

__device__ __forceinline__ int xcd_tile(int b, int nb) {
    const int per = nb >> 3, rem = nb & 7;
    const int xcd = b & 7, slot = b >> 3;
    return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

// gfx950's LDS serves a 16-byte access for 16 lanes per pass across 64 banks
// (256 bytes = RPB rows).  Fragment reads take 16 consecutive rows at one
// logical chunk; rows with equal (row % RPB) share bank slots, so the chunk
// is XORed with (row / RPB) % CPR to spread them.  Element offset of logical
// chunk `chunk` of row `row`:
template <class TL>
__device__ __forceinline__ int swz(int row, int chunk) {
    return row * TL::BK + ((chunk ^ ((row / TL::RPB) % TL::CPR)) << 3);
}

// GELU, tanh form, as x * sigmoid(2y) with y = sqrt(2/pi) (x + 0.044715 x^3):
// 0.5 x (1 + tanh(y)) = x / (1 + exp(-2y)).
__device__ __forceinline__ float gelu_fast(float x) {
    const float x2 = x * x;
    const float u = fmaf(0.044715f * x2, x, x);                  // x + 0.044715 x^3
    const float z = -2.0f * 1.4426950408889634f * 0.7978845608028654f * u;
    return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z));
}

template <class TL, int MODE, typename TKV>
__device__ __forceinline__ void gemm_tile(const f16* __restrict__ A, int64_t lda,
                                          const f16* __restrict__ W, int64_t M, int N, int K,
                                          const Epilogue& epi) {
    constexpr int kBM = TL::BM, kBN = TL::BN, kBK = TL::BK;
    constexpr int kWavesN = TL::WAVES_N, kWM = TL::WM, kWN = TL::WN, kTM = TL::TM, kTN = TL::TN;
    constexpr int kCPR = TL::CPR;
    __shared__ __attribute__((aligned(16))) f16 sA[2][kBM * kBK];
    __shared__ __attribute__((aligned(16))) f16 sB[2][kBN * kBK];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / kWavesN, wn = wave % kWavesN;
    const int tiles_n = (N + kBN - 1) / kBN;
    const int t = xcd_tile(blockIdx.x, gridDim.x);
    const int64_t m0 = (int64_t)(t / tiles_n) * kBM;
    const int n0 = (t % tiles_n) * kBN;

    // Buffer descriptors over this tile's rows of A and W: rows past M (N)
    // fall outside num_records and load as zeros, so tails need no branches.
    const int64_t rows_a = M - m0 < kBM ? M - m0 : kBM;
    const int rows_b = N - n0 < kBN ? N - n0 : kBN;
    const __amdgpu_buffer_rsrc_t rsA = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(A + m0 * lda), (short)0, (int)(rows_a * lda * 2), 0x00020000);
    const __amdgpu_buffer_rsrc_t rsB = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(W + (int64_t)n0 * K), (short)0, (int)((int64_t)rows_b * K * 2), 0x00020000);

    // Direct global -> LDS loads: a wave's 64 lanes fill 64 consecutive
    // 16-byte LDS slots.  Slot s of row r must hold logical chunk
    // s ^ key(r), so that is the chunk each lane fetches.
    int offA[TL::LOADS_A], offB[TL::LOADS_B];
#pragma unroll
    for (int i = 0; i < TL::LOADS_A; ++i) {
        const int c = (wave * TL::LOADS_A + i) * 64 + lane;
        const int row = c / kCPR, slot = c % kCPR;
        const int lch = slot ^ ((row / TL::RPB) % kCPR);
        offA[i] = (int)(row * lda * 2 + lch * 16);
    }
#pragma unroll
    for (int i = 0; i < TL::LOADS_B; ++i) {
        const int c = (wave * TL::LOADS_B + i) * 64 + lane;
        const int row = c / kCPR, slot = c % kCPR;
        const int lch = slot ^ ((row / TL::RPB) % kCPR);
        offB[i] = row * K * 2 + lch * 16;
    }
    auto issue_loads = [&](int buf, int k0) {
#pragma unroll
        for (int i = 0; i < TL::LOADS_A; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rsA, (__attribute__((address_space(3))) void*)(&sA[buf][(wave * TL::LOADS_A + i) * 64 * 8]),
                16, offA[i] + k0 * 2, 0, 0, 0);
#pragma unroll
        for (int i = 0; i < TL::LOADS_B; ++i)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rsB, (__attribute__((address_space(3))) void*)(&sB[buf][(wave * TL::LOADS_B + i) * 64 * 8]),
                16, offB[i] + k0 * 2, 0, 0, 0);
    };

    f32x16 acc[kTN][kTM];
#pragma unroll
    for (int j = 0; j < kTN; ++j)
#pragma unroll
        for (int i = 0; i < kTM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[j][i][r] = 0.f;

    const int lrow = lane & 31, lhalf = lane >> 5;
    // One K-step: read all of its operand fragments from LDS buffer `buf`
    // first, then issue the next K-step's loads, then run the MFMAs.  The
    // order matters: the compiler waits for outstanding LDS-DMA loads before
    // any later LDS read (it cannot see that they target the other buffer),
    // so reads issued after the DMA would serialise load and compute.
    auto step = [&](int buf, int next_k0, bool issue_next) {
        h8 a[kBK / 16][kTM], b[kBK / 16][kTN];
#pragma unroll
        for (int kk = 0; kk < kBK / 16; ++kk) {
            const int ch = kk * 2 + lhalf;
#pragma unroll
            for (int i = 0; i < kTM; ++i)
                a[kk][i] = *reinterpret_cast<const h8*>(&sA[buf][swz<TL>(wm * kWM + i * 32 + lrow, ch)]);
#pragma unroll
            for (int j = 0; j < kTN; ++j)
                b[kk][j] = *reinterpret_cast<const h8*>(&sB[buf][swz<TL>(wn * kWN + j * 32 + lrow, ch)]);
        }
        __builtin_amdgcn_sched_barrier(0);
        if (issue_next) issue_loads(buf ^ 1, next_k0);
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int kk = 0; kk < kBK / 16; ++kk)
#pragma unroll
            for (int j = 0; j < kTN; ++j)
#pragma unroll
                for (int i = 0; i < kTM; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(b[kk][j], a[kk][i],
                                                                       acc[j][i], 0, 0, 0);
        // keep the end-of-step wait and barrier behind the MFMAs
        __builtin_amdgcn_sched_barrier(0);
    };

    // K-step j lives in LDS buffer j&1.  Step kt computes from buffer kt&1
    // while the loads of kt+1 fill the other buffer (free: its last readers
    // passed the previous barrier); each wave waits for its own loads before
    // the barrier that publishes the buffer.
    const int nk = K / kBK;
    issue_loads(0, 0);
    __builtin_amdgcn_s_waitcnt(0);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        step(kt & 1, (kt + 1) * kBK, kt + 1 < nk);
        __builtin_amdgcn_s_waitcnt(0);
        __syncthreads();
    }

    // Epilogue.  Register r of transposed tile (j, i) holds output row
    // m0 + wm*128 + 32i + lane%32 and column n0 + wn*64 + 32j + 8(r/4) + 4(lane/32) + r%4.
    // All loads are issued before their uses (bias once per tile, the fp32
    // residual once per row-tile) so their latencies overlap.
    const float* __restrict__ bias_p = epi.bias;
    float4 bq[kTN][4];
#pragma unroll
    for (int j = 0; j < kTN; ++j)
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const int col = n0 + wn * kWN + j * 32 + 8 * q + 4 * lhalf;
            bq[j][q] = col < N ? *reinterpret_cast<const float4*>(bias_p + col)
                               : make_float4(0.f, 0.f, 0.f, 0.f);
        }
    const float sc = epi.acc_scale;
#pragma unroll
    for (int i = 0; i < kTM; ++i) {
        const int64_t row = m0 + wm * kWM + i * 32 + lrow;
        if (row >= M) continue;
        float4 v[kTN][4];
#pragma unroll
        for (int j = 0; j < kTN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                v[j][q].x = fmaf(acc[j][i][4 * q + 0], sc, bq[j][q].x);
                v[j][q].y = fmaf(acc[j][i][4 * q + 1], sc, bq[j][q].y);
                v[j][q].z = fmaf(acc[j][i][4 * q + 2], sc, bq[j][q].z);
                v[j][q].w = fmaf(acc[j][i][4 * q + 3], sc, bq[j][q].w);
            }
        if constexpr (MODE == EPI_RESID) {
            float* __restrict__ rrow = epi.resid + row * epi.ldr;
            float4 g[kTN][4];
#pragma unroll
            for (int j = 0; j < kTN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int col = n0 + wn * kWN + j * 32 + 8 * q + 4 * lhalf;
                    if (col < N) g[j][q] = *reinterpret_cast<const float4*>(rrow + col);
                }
#pragma unroll
            for (int j = 0; j < kTN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int col = n0 + wn * kWN + j * 32 + 8 * q + 4 * lhalf;
                    if (col >= N) continue;
                    float4 o = g[j][q];
                    o.x += v[j][q].x; o.y += v[j][q].y; o.z += v[j][q].z; o.w += v[j][q].w;
                    *reinterpret_cast<float4*>(rrow + col) = o;
                }
        } else {
#pragma unroll
            for (int j = 0; j < kTN; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    const int col = n0 + wn * kWN + j * 32 + 8 * q + 4 * lhalf;
                    if (col >= N) continue;          // N is a multiple of 4
                    const float vv[4] = {v[j][q].x, v[j][q].y, v[j][q].z, v[j][q].w};
                    if constexpr (MODE == EPI_GELU) {
                        h4 o;
#pragma unroll
                        for (int r = 0; r < 4; ++r) o[r] = (f16)keep_f32(gelu_fast(vv[r]));
                        *reinterpret_cast<h4*>(static_cast<f16*>(epi.out) + row * epi.ldo + col) = o;
                    } else if constexpr (MODE == EPI_STORE) {
                        const float cs = col < epi.scale_cols ? epi.col_scale : 1.0f;
                        b4 o;
#pragma unroll
                        for (int r = 0; r < 4; ++r) o[r] = (__bf16)keep_f32(vv[r] * cs);
                        *reinterpret_cast<b4*>(static_cast<bf16*>(epi.out) + row * epi.ldo + col) = o;
                    } else {   // EPI_QKV_CACHE: 4 columns never straddle a head (head_dim % 4 == 0)
                        const int d = epi.d_model;
                        b4 o;
                        bf16* dst;
                        if (col < d) {
#pragma unroll
                            for (int r = 0; r < 4; ++r) o[r] = (__bf16)keep_f32(vv[r] * epi.col_scale);
                            dst = static_cast<bf16*>(epi.out) + row * epi.ldo + col;
                        } else {
                            const int part = col >= 2 * d ? 2 : 1;
                            const int c = col - part * d;
                            const int h = c / epi.head_dim, e = c - h * epi.head_dim;
#pragma unroll
                            for (int r = 0; r < 4; ++r) o[r] = (__bf16)keep_f32(vv[r]);
                            bf16* plane = static_cast<bf16*>(part == 1 ? epi.cache_k : epi.cache_v);
                            dst = plane + ((int64_t)h * epi.cache_cap + (epi.row0 + row)) * epi.head_dim + e;
                        }
                        *reinterpret_cast<b4*>(dst) = o;
                    }
                }
        }
    }
}

template <class TL, int MODE, typename TKV>
__global__ __launch_bounds__(TL::THREADS, TL::MIN_BLOCKS) void k_gemm_mfma(
    const f16* __restrict__ A, int64_t lda, const f16* __restrict__ W, int64_t M, int N, int K,
    Epilogue epi) {
    gemm_tile<TL, MODE, TKV>(A, lda, W, M, N, K, epi);
}

template <class TL, int MODE>
hipError_t launch_mode(const f16* A, int64_t lda, const f16* W, int64_t M, int N, int K,
                       const Epilogue& epi, hipStream_t s) {
    const int64_t tiles = ((M + TL::BM - 1) / TL::BM) * (int64_t)((N + TL::BN - 1) / TL::BN);
    k_gemm_mfma<TL, MODE, bf16><<<(unsigned)tiles, TL::THREADS, 0, s>>>(A, lda, W, M, N, K, epi);
    return hipGetLastError();
}

template <class TL>
hipError_t launch_tile(const f16* A, int64_t lda, const f16* W, int64_t M, int N, int K,
                       const Epilogue& epi, hipStream_t s) {
    switch (epi.mode) {
        case EPI_STORE: return launch_mode<TL, EPI_STORE>(A, lda, W, M, N, K, epi, s);
        case EPI_GELU: return launch_mode<TL, EPI_GELU>(A, lda, W, M, N, K, epi, s);
        case EPI_RESID: return launch_mode<TL, EPI_RESID>(A, lda, W, M, N, K, epi, s);
        case EPI_QKV_CACHE: return launch_mode<TL, EPI_QKV_CACHE>(A, lda, W, M, N, K, epi, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace gemm_detail

using gemm_detail::TileBig;
using gemm_detail::TileWide;
using gemm_detail::launch_tile;

#ifndef GEMM_TILE_CHOICE
#define GEMM_TILE_CHOICE launch_tile<TileBig>
#endif
hipError_t launch_gemm_mfma(const f16* A, int64_t lda, const f16* W, int64_t M, int N, int K,
                            const Epilogue& epi, hipStream_t s) {
    if (M == 0) return hipSuccess;
    if (K % 64 != 0 || lda % 8 != 0 || N % 4 != 0) return hipErrorInvalidValue;
    return GEMM_TILE_CHOICE(A, lda, W, M, N, K, epi, s);
}

}  // namespace upr
