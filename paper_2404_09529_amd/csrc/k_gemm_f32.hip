// float32 projection GEMM C = A B^T (A [M, K] activations, B [N, K] weights) for float32
// models: 64 x 64 output tiles, K steps of 16 staged through LDS, 4 x 4 outputs per
// thread on FMA units.  Used by the small float32 decoder; bf16 models use the MFMA GEMM.
#include "device.h"
#include "kernels.h"

namespace {

constexpr int TB = 64, TK = 16, NT = 256;

template <int EPI>
__global__ __launch_bounds__(NT) void gemm_f32_kernel(const float* __restrict__ A, int64_t lda,
                                                      const float* __restrict__ B, int64_t ldb,
                                                      float* __restrict__ C, int64_t ldc, int M, int N, int K) {
    __shared__ float sa[TK][TB + 4];
    __shared__ float sb[TK][TB + 4];
    const int tid = threadIdx.x, tx = tid & 15, ty = tid >> 4;
    const int64_t m0 = int64_t(blockIdx.y) * TB;
    const int n0 = blockIdx.x * TB;
    const int r = tid >> 2, kq = (tid & 3) * 4;
    float acc[4][4] = {};
    for (int k0 = 0; k0 < K; k0 += TK) {
        const f32x4 va = m0 + r < M ? *reinterpret_cast<const f32x4*>(A + (m0 + r) * lda + k0 + kq) : f32x4{};
        const f32x4 vb = n0 + r < N ? *reinterpret_cast<const f32x4*>(B + int64_t(n0 + r) * ldb + k0 + kq)
                                    : f32x4{};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            sa[kq + e][r] = va[e];
            sb[kq + e][r] = vb[e];
        }
        __syncthreads();
#pragma unroll
        for (int kk = 0; kk < TK; ++kk) {
            float av[4], bv[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) av[i] = sa[kk][ty + 16 * i];
#pragma unroll
            for (int j = 0; j < 4; ++j) bv[j] = sb[kk][tx + 16 * j];
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[i][j] = fmaf(av[i], bv[j], acc[i][j]);
        }
        __syncthreads();
    }
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int64_t m = m0 + ty + 16 * i;
        if (m >= M) continue;
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int n = n0 + tx + 16 * j;
            if (n >= N) continue;
            if constexpr (EPI == ppk::kResidual)
                C[m * ldc + n] += acc[i][j];
            else
                C[m * ldc + n] = acc[i][j];
        }
    }
}

}  // namespace

namespace ppk {

void gemm_f32(int epi, const float* A, int64_t lda, const float* B, int64_t ldb, float* C, int64_t ldc, int M,
              int N, int K, hipStream_t s) {
    if (M <= 0 || N <= 0) return;
    const dim3 grid((N + TB - 1) / TB, (M + TB - 1) / TB);
    if (epi == kResidual)
        gemm_f32_kernel<kResidual><<<grid, NT, 0, s>>>(A, lda, B, ldb, C, ldc, M, N, K);
    else
        gemm_f32_kernel<kStore><<<grid, NT, 0, s>>>(A, lda, B, ldb, C, ldc, M, N, K);
}

}  // namespace ppk
