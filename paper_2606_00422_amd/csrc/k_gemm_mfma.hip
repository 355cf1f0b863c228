// Projection GEMM on the matrix cores: out = A[M,K] W[N,K]^T (+ epilogue),
// A and W fp16 (both K-contiguous), fp32 accumulation with
// v_mfma_f32_32x32x16_f16.
//
// Block tile BM x BN, K in steps of 64.  Four waves in a 2x2 grid, each owning
// a (BM/2) x (BN/2) sub-tile of 32x32 MFMA tiles.  A and W tiles are staged
// through LDS, double-buffered: the next K-step is fetched into registers
// while the current one feeds the MFMAs.  LDS rows are 128 bytes (64 fp16);
// the eight 16-byte chunks of row r are stored XOR-swizzled (chunk c at slot
// c ^ (r & 7)), so the 16-byte operand reads of 8 consecutive rows hit 8
// different bank groups.
//
// Tile order is XCD-aware: workgroup b runs on XCD b % 8, and the tiles are
// renumbered so every XCD sweeps a contiguous range of (M-panel, N-tile)
// pairs; the N-tiles of one A row-panel then share one L2.
#include "epilogue.h"
#include "upr_plan.h"

namespace upr {

namespace {

typedef __attribute__((ext_vector_type(8))) _Float16 h8;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int kBK = 64;

__device__ __forceinline__ int xcd_tile(int b, int nb) {
    const int per = nb >> 3, rem = nb & 7;
    const int xcd = b & 7, slot = b >> 3;
    return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

__device__ __forceinline__ int swz(int row, int chunk) { return row * kBK + ((chunk ^ (row & 7)) << 3); }

// GELU, tanh form, written as x * sigmoid(2y) with y = sqrt(2/pi)(x + 0.044715 x^3):
// 0.5 x (1 + tanh(y)) = x / (1 + exp(-2y)).
__device__ __forceinline__ float gelu_fast(float x) {
    const float y2 = -2.0f * 0.7978845608028654f * (x + 0.044715f * x * x * x);
    return x / (1.0f + __expf(y2));
}

template <int BM, int BN, typename TKV>
__global__ __launch_bounds__(256, 2) void k_gemm_mfma(const f16* __restrict__ A, int64_t lda,
                                                      const f16* __restrict__ W, int64_t M, int N,
                                                      int K, Epilogue epi) {
    constexpr int WM = BM / 2, WN = BN / 2;
    constexpr int TM = WM / 32, TN = WN / 32;
    constexpr int CA = BM * 8 / 256, CB = BN * 8 / 256;   // 16-byte chunks per thread
    __shared__ __attribute__((aligned(16))) f16 sA[2][BM * kBK];
    __shared__ __attribute__((aligned(16))) f16 sB[2][BN * kBK];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave >> 1, wn = wave & 1;
    const int tiles_n = (N + BN - 1) / BN;
    const int t = xcd_tile(blockIdx.x, gridDim.x);
    const int64_t m0 = (int64_t)(t / tiles_n) * BM;
    const int n0 = (t % tiles_n) * BN;

    uint4 ra[CA], rb[CB];
    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < CA; ++i) {
            const int c = tid + 256 * i, row = c >> 3, ch = c & 7;
            const int64_t gm = m0 + row;
            ra[i] = gm < M ? *reinterpret_cast<const uint4*>(A + gm * lda + k0 + ch * 8)
                           : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
            const int c = tid + 256 * i, row = c >> 3, ch = c & 7;
            const int gn = n0 + row;
            rb[i] = gn < N ? *reinterpret_cast<const uint4*>(W + (int64_t)gn * K + k0 + ch * 8)
                           : make_uint4(0, 0, 0, 0);
        }
    };
    auto swrite = [&](int buf) {
#pragma unroll
        for (int i = 0; i < CA; ++i) {
            const int c = tid + 256 * i;
            *reinterpret_cast<uint4*>(&sA[buf][swz(c >> 3, c & 7)]) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
            const int c = tid + 256 * i;
            *reinterpret_cast<uint4*>(&sB[buf][swz(c >> 3, c & 7)]) = rb[i];
        }
    };

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    const int nk = K / kBK;
    gload(0);
    swrite(0);
    __syncthreads();
    const int lrow = lane & 31, lhalf = lane >> 5;
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) gload((kt + 1) * kBK);
#pragma unroll
        for (int kk = 0; kk < kBK / 16; ++kk) {
            const int ch = kk * 2 + lhalf;
            h8 a[TM], b[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i)
                a[i] = *reinterpret_cast<const h8*>(&sA[buf][swz(wm * WM + i * 32 + lrow, ch)]);
#pragma unroll
            for (int j = 0; j < TN; ++j)
                b[j] = *reinterpret_cast<const h8*>(&sB[buf][swz(wn * WN + j * 32 + lrow, ch)]);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a[i], b[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) swrite(buf ^ 1);
        __syncthreads();
    }

    // Epilogue.  Accumulator register r of a 32x32 tile holds row
    // 8*(r/4) + 4*(lane/32) + r%4 and column lane%32.
    const int mode = epi.mode;
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = n0 + wn * WN + j * 32 + lrow;
            if (col >= N) continue;
            const float bias = epi.bias[col];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int64_t row = m0 + wm * WM + i * 32 + 8 * (r >> 2) + 4 * lhalf + (r & 3);
                if (row >= M) continue;
                float v = acc[i][j][r] * epi.acc_scale + bias;
                if (mode == EPI_RESID) {
                    epi.resid[row * epi.ldr + col] += v;
                } else if (mode == EPI_GELU) {
                    static_cast<f16*>(epi.out)[row * epi.ldo + col] = (f16)gelu_fast(v);
                } else if (mode == EPI_STORE) {
                    if (col < epi.scale_cols) v *= epi.col_scale;
                    static_cast<TKV*>(epi.out)[row * epi.ldo + col] = (TKV)v;
                } else {
                    epilogue_apply<TKV, f16>(epi, row, col, acc[i][j][r]);
                }
            }
        }
}

template <int BM, int BN>
hipError_t launch_tile(const f16* A, int64_t lda, const f16* W, int64_t M, int N, int K,
                       const Epilogue& epi, hipStream_t s) {
    const int64_t tiles = ((M + BM - 1) / BM) * (int64_t)((N + BN - 1) / BN);
    k_gemm_mfma<BM, BN, bf16><<<(unsigned)tiles, 256, 0, s>>>(A, lda, W, M, N, K, epi);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_mfma(const f16* A, int64_t lda, const f16* W, int64_t M, int N, int K,
                            const Epilogue& epi, hipStream_t s) {
    if (M == 0) return hipSuccess;
    if (K % kBK != 0 || lda % 8 != 0) return hipErrorInvalidValue;
    return launch_tile<128, 128>(A, lda, W, M, N, K, epi, s);
}

}  // namespace upr
