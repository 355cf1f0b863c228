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
// A and W tiles are staged through LDS, double-buffered, with global loads
// issued two K-steps ahead into two register sets, so a load has two K-steps
// of MFMA work (about 2000 cycles per SIMD) to arrive.  LDS rows are 128
// bytes (64 fp16) and the eight 16-byte chunks of each row are XOR-swizzled so
// fragment reads and staging writes are bank-conflict free.
//
// Tile order is XCD-aware: workgroup b runs on XCD b % 8 and the tiles are
// renumbered so each XCD sweeps a contiguous range of (M-panel, N-tile)
// pairs; the N-tiles of one A row-panel then share one L2.
#include <type_traits>

#include "epilogue.h"
#include "upr_plan.h"

namespace upr {

namespace {

typedef __attribute__((ext_vector_type(8))) _Float16 h8;
typedef __attribute__((ext_vector_type(4))) _Float16 h4;
typedef __attribute__((ext_vector_type(4))) __bf16 b4;
typedef __attribute__((ext_vector_type(16))) float f32x16;

constexpr int kBK = 64;
constexpr int kBM = 256, kBN = 256;
constexpr int kWavesM = 2, kWavesN = 4, kThreads = 64 * kWavesM * kWavesN;
constexpr int kWM = kBM / kWavesM, kWN = kBN / kWavesN;    // 128 x 64 per wave
constexpr int kTM = kWM / 32, kTN = kWN / 32;              // 4 x 2 MFMA tiles

__device__ __forceinline__ int xcd_tile(int b, int nb) {
    const int per = nb >> 3, rem = nb & 7;
    const int xcd = b & 7, slot = b >> 3;
    return xcd < rem ? xcd * (per + 1) + slot : rem * (per + 1) + (xcd - rem) * per + slot;
}

// gfx950's LDS serves a 16-byte access for 16 lanes per pass across 64 banks
// (256 bytes); fragment reads take 16 consecutive rows, so the swizzle key is
// (row >> 1) & 7 (rows of equal parity land in the same 128-byte bank half).
__device__ __forceinline__ int swz(int row, int chunk) {
    return row * kBK + ((chunk ^ ((row >> 1) & 7)) << 3);
}

// GELU, tanh form, as x * sigmoid(2y) with y = sqrt(2/pi) (x + 0.044715 x^3):
// 0.5 x (1 + tanh(y)) = x / (1 + exp(-2y)).
__device__ __forceinline__ float gelu_fast(float x) {
    const float x2 = x * x;
    const float u = fmaf(0.044715f * x2, x, x);                  // x + 0.044715 x^3
    const float z = -2.0f * 1.4426950408889634f * 0.7978845608028654f * u;
    return x * __builtin_amdgcn_rcpf(1.0f + __builtin_amdgcn_exp2f(z));
}

template <int MODE, typename TKV>
__global__ __launch_bounds__(kThreads, 1) void k_gemm_mfma(const f16* __restrict__ A, int64_t lda,
                                                           const f16* __restrict__ W, int64_t M,
                                                           int N, int K, Epilogue epi) {
    constexpr int CA = kBM * 8 / kThreads, CB = kBN * 8 / kThreads;   // 16-byte chunks per thread
    __shared__ __attribute__((aligned(16))) f16 sA[2][kBM * kBK];
    __shared__ __attribute__((aligned(16))) f16 sB[2][kBN * kBK];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / kWavesN, wn = wave % kWavesN;
    const int tiles_n = (N + kBN - 1) / kBN;
    const int t = xcd_tile(blockIdx.x, gridDim.x);
    const int64_t m0 = (int64_t)(t / tiles_n) * kBM;
    const int n0 = (t % tiles_n) * kBN;

    uint4 ra[2][CA], rb[2][CB];     // two register sets: K-steps of either parity
    auto gload = [&](int set, int k0) {
#pragma unroll
        for (int i = 0; i < CA; ++i) {
            const int c = tid + kThreads * i, row = c >> 3, ch = c & 7;
            const int64_t gm = m0 + row;
            ra[set][i] = gm < M ? *reinterpret_cast<const uint4*>(A + gm * lda + k0 + ch * 8)
                                : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
            const int c = tid + kThreads * i, row = c >> 3, ch = c & 7;
            const int gn = n0 + row;
            rb[set][i] = gn < N ? *reinterpret_cast<const uint4*>(W + (int64_t)gn * K + k0 + ch * 8)
                                : make_uint4(0, 0, 0, 0);
        }
    };
    auto swrite = [&](int set, int buf) {
#pragma unroll
        for (int i = 0; i < CA; ++i) {
            const int c = tid + kThreads * i;
            *reinterpret_cast<uint4*>(&sA[buf][swz(c >> 3, c & 7)]) = ra[set][i];
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
            const int c = tid + kThreads * i;
            *reinterpret_cast<uint4*>(&sB[buf][swz(c >> 3, c & 7)]) = rb[set][i];
        }
    };

    f32x16 acc[kTN][kTM];
#pragma unroll
    for (int j = 0; j < kTN; ++j)
#pragma unroll
        for (int i = 0; i < kTM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[j][i][r] = 0.f;

    const int lrow = lane & 31, lhalf = lane >> 5;
    auto compute = [&](int buf) {
#pragma unroll
        for (int kk = 0; kk < kBK / 16; ++kk) {
            const int ch = kk * 2 + lhalf;
            h8 a[kTM], b[kTN];
#pragma unroll
            for (int i = 0; i < kTM; ++i)
                a[i] = *reinterpret_cast<const h8*>(&sA[buf][swz(wm * kWM + i * 32 + lrow, ch)]);
#pragma unroll
            for (int j = 0; j < kTN; ++j)
                b[j] = *reinterpret_cast<const h8*>(&sB[buf][swz(wn * kWN + j * 32 + lrow, ch)]);
#pragma unroll
            for (int j = 0; j < kTN; ++j)
#pragma unroll
                for (int i = 0; i < kTM; ++i)
                    acc[j][i] = __builtin_amdgcn_mfma_f32_32x32x16_f16(b[j], a[i], acc[j][i], 0, 0, 0);
        }
    };

    // K-step j lives in register set j&1 and LDS buffer j&1.  Step kt issues
    // the load of kt+2, computes kt, then stores kt+1 (loaded during kt-1).
    const int nk = K / kBK;
    gload(0, 0);
    if (nk > 1) gload(1, kBK);
    swrite(0, 0);
    __syncthreads();
    auto step = [&](int kt, auto par) {
        constexpr int P = decltype(par)::value;          // kt & 1
        if (kt + 2 < nk) gload(P, (kt + 2) * kBK);
        compute(P);
        if (kt + 1 < nk) swrite(P ^ 1, P ^ 1);
        __syncthreads();
    };
    int kt = 0;
    for (; kt + 1 < nk; kt += 2) {
        step(kt, std::integral_constant<int, 0>{});
        step(kt + 1, std::integral_constant<int, 1>{});
    }
    if (kt < nk) step(kt, std::integral_constant<int, 0>{});

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

template <int MODE>
hipError_t launch_mode(const f16* A, int64_t lda, const f16* W, int64_t M, int N, int K,
                       const Epilogue& epi, hipStream_t s) {
    const int64_t tiles = ((M + kBM - 1) / kBM) * (int64_t)((N + kBN - 1) / kBN);
    k_gemm_mfma<MODE, bf16><<<(unsigned)tiles, kThreads, 0, s>>>(A, lda, W, M, N, K, epi);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gemm_mfma(const f16* A, int64_t lda, const f16* W, int64_t M, int N, int K,
                            const Epilogue& epi, hipStream_t s) {
    if (M == 0) return hipSuccess;
    if (K % kBK != 0 || lda % 8 != 0 || N % 4 != 0) return hipErrorInvalidValue;
    switch (epi.mode) {
        case EPI_STORE: return launch_mode<EPI_STORE>(A, lda, W, M, N, K, epi, s);
        case EPI_GELU: return launch_mode<EPI_GELU>(A, lda, W, M, N, K, epi, s);
        case EPI_RESID: return launch_mode<EPI_RESID>(A, lda, W, M, N, K, epi, s);
        case EPI_QKV_CACHE: return launch_mode<EPI_QKV_CACHE>(A, lda, W, M, N, K, epi, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace upr
