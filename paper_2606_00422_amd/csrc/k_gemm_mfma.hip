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
// A and W tiles are staged through LDS, double-buffered: the next K-step is
// fetched into registers while the current one feeds the MFMAs.  LDS rows are
// 128 bytes (64 fp16) and the eight 16-byte chunks of row r are stored
// XOR-swizzled (chunk c at slot c ^ (r & 7)), so the operand reads of 8
// consecutive rows hit 8 different bank groups.
//
// Tile order is XCD-aware: workgroup b runs on XCD b % 8 and the tiles are
// renumbered so each XCD sweeps a contiguous range of (M-panel, N-tile)
// pairs; the N-tiles of one A row-panel then share one L2.
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

__device__ __forceinline__ int swz(int row, int chunk) { return row * kBK + ((chunk ^ (row & 7)) << 3); }

// GELU, tanh form, as x * sigmoid(2y) with y = sqrt(2/pi) (x + 0.044715 x^3):
// 0.5 x (1 + tanh(y)) = x / (1 + exp(-2y)).
__device__ __forceinline__ float gelu_fast(float x) {
    const float z = -2.0f * 1.4426950408889634f * 0.7978845608028654f * (x + 0.044715f * x * x * x);
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

    uint4 ra[CA], rb[CB];
    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < CA; ++i) {
            const int c = tid + kThreads * i, row = c >> 3, ch = c & 7;
            const int64_t gm = m0 + row;
            ra[i] = gm < M ? *reinterpret_cast<const uint4*>(A + gm * lda + k0 + ch * 8)
                           : make_uint4(0, 0, 0, 0);
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
            const int c = tid + kThreads * i, row = c >> 3, ch = c & 7;
            const int gn = n0 + row;
            rb[i] = gn < N ? *reinterpret_cast<const uint4*>(W + (int64_t)gn * K + k0 + ch * 8)
                           : make_uint4(0, 0, 0, 0);
        }
    };
    auto swrite = [&](int buf) {
#pragma unroll
        for (int i = 0; i < CA; ++i) {
            const int c = tid + kThreads * i;
            *reinterpret_cast<uint4*>(&sA[buf][swz(c >> 3, c & 7)]) = ra[i];
        }
#pragma unroll
        for (int i = 0; i < CB; ++i) {
            const int c = tid + kThreads * i;
            *reinterpret_cast<uint4*>(&sB[buf][swz(c >> 3, c & 7)]) = rb[i];
        }
    };

    f32x16 acc[kTN][kTM];
#pragma unroll
    for (int j = 0; j < kTN; ++j)
#pragma unroll
        for (int i = 0; i < kTM; ++i)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[j][i][r] = 0.f;

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
        if (kt + 1 < nk) swrite(buf ^ 1);
        __syncthreads();
    }

    // Epilogue.  Register r of transposed tile (j, i) holds output row
    // m0 + wm*128 + 32i + lane%32 and column n0 + wn*64 + 32j + 8(r/4) + 4(lane/32) + r%4.
#pragma unroll
    for (int i = 0; i < kTM; ++i) {
        const int64_t row = m0 + wm * kWM + i * 32 + lrow;
        if (row >= M) continue;
#pragma unroll
        for (int j = 0; j < kTN; ++j)
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int col = n0 + wn * kWN + j * 32 + 8 * q + 4 * lhalf;
                if (col >= N) continue;          // N is a multiple of 4
                const float4 bias = *reinterpret_cast<const float4*>(epi.bias + col);
                float v[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) v[r] = acc[j][i][4 * q + r] * epi.acc_scale;
                v[0] += bias.x; v[1] += bias.y; v[2] += bias.z; v[3] += bias.w;
                if constexpr (MODE == EPI_RESID) {
                    float4* p = reinterpret_cast<float4*>(epi.resid + row * epi.ldr + col);
                    float4 g = *p;
                    g.x += v[0]; g.y += v[1]; g.z += v[2]; g.w += v[3];
                    *p = g;
                } else if constexpr (MODE == EPI_GELU) {
                    h4 o;
#pragma unroll
                    for (int r = 0; r < 4; ++r) o[r] = (f16)gelu_fast(v[r]);
                    *reinterpret_cast<h4*>(static_cast<f16*>(epi.out) + row * epi.ldo + col) = o;
                } else if constexpr (MODE == EPI_STORE) {
                    const float sc = col < epi.scale_cols ? epi.col_scale : 1.0f;
                    b4 o;
#pragma unroll
                    for (int r = 0; r < 4; ++r) o[r] = (__bf16)(v[r] * sc);
                    *reinterpret_cast<b4*>(static_cast<bf16*>(epi.out) + row * epi.ldo + col) = o;
                } else {   // EPI_QKV_CACHE: 4 columns never straddle a head (head_dim % 4 == 0)
                    const int d = epi.d_model;
                    b4 o;
                    bf16* dst;
                    if (col < d) {
#pragma unroll
                        for (int r = 0; r < 4; ++r) o[r] = (__bf16)(v[r] * epi.col_scale);
                        dst = static_cast<bf16*>(epi.out) + row * epi.ldo + col;
                    } else {
                        const int part = col >= 2 * d ? 2 : 1;
                        const int c = col - part * d;
                        const int h = c / epi.head_dim, e = c - h * epi.head_dim;
#pragma unroll
                        for (int r = 0; r < 4; ++r) o[r] = (__bf16)v[r];
                        bf16* plane = static_cast<bf16*>(part == 1 ? epi.cache_k : epi.cache_v);
                        dst = plane + ((int64_t)h * epi.cache_cap + (epi.row0 + row)) * epi.head_dim + e;
                    }
                    *reinterpret_cast<b4*>(dst) = o;
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
