// Projection GEMMs of the decoder layer (section 2.1: X W^Q, X W^K, X W^V; the output
// projection and the SwiGLU MLP of the Llama family) on gfx950 matrix cores.
//
// C[M, N] = A[M, K] B[N, K]^T with A the packed activations (bf16, K contiguous) and B a
// weight matrix in [out, in] layout (bf16, K contiguous), float32 accumulation.
//
// Tiling: one 256-thread workgroup (4 wavefronts) per 256 x 256 output tile, K consumed in
// steps of 64.  Each wavefront owns a 128 (N) x 128 (M) sub-tile = 4 x 4 blocks of the
// 32x32x16 bf16 MFMA, 256 accumulator registers.  The weight block is the MFMA's first
// operand, so a lane's accumulators are 4-element runs along N of one activation row:
// the epilogue writes 8-byte (bf16) or 16-byte (float32) runs without a transpose.
//
// Data path per K step: global -> registers (16-byte loads, 8 threads per 128-byte row)
// for step k+1 while the matrix cores consume step k from LDS; LDS is double-buffered
// (2 x 64 KB) so one barrier per step suffices.  LDS rows are 128 bytes = 8 chunks of 16
// bytes; chunk c of row r is stored at c ^ f(r), f(r) = (r ^ r>>3) & 7, which makes the
// fragment reads (32 rows x one chunk per half-wavefront) hit distinct banks whether the
// LDS serves 8 or 16 lanes of a 16-byte read per cycle.
//
// Scheduling: a launch has far more tiles than the 256 CUs.  Workgroups are dealt to the
// 8 XCDs round-robin, so the linear workgroup id is remapped to make each XCD's
// workgroups a contiguous range of tiles, and tiles are ordered in groups of 8 M-tiles
// sweeping N, so the tiles resident on one XCD share activation and weight panels in its
// L2.  M-tiles made only of row-tail padding are skipped (packed batches only carry pads
// at row tails, section 3.1).
#include "device.h"
#include "kernels.h"

namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int NT = 256;
constexpr int CH = BK * 2 / 16;  // 16-byte chunks per LDS row
constexpr int GROUP_M = 8;

struct Stage {
    u32x4 a[BM * CH];
    u32x4 b[BN * CH];
};

__device__ __forceinline__ int swz(int row, int c) { return c ^ ((row ^ (row >> 3)) & 7); }

__device__ __forceinline__ bool tile_active(const int32_t* slot_seg, int capacity, int m0, int M) {
    if (!slot_seg || slot_seg[m0] >= 0) return true;
    // first slot is a row-tail pad: inactive unless another row starts inside the tile
    const int64_t next_row = (int64_t(m0) / capacity + 1) * capacity;
    return next_row < min(m0 + BM, M);
}

template <typename V>
__device__ __forceinline__ bf16x8 as_bf16x8(V v) { return __builtin_bit_cast(bf16x8, v); }

template <int EPI>
__global__ __launch_bounds__(NT) void gemm_bf16_kernel(const bf16* __restrict__ A, int64_t lda,
                                                       const bf16* __restrict__ B, int64_t ldb,
                                                       void* __restrict__ Cv, int64_t ldc, int M, int K,
                                                       const int32_t* __restrict__ slot_seg, int capacity,
                                                       int tiles_m, int tiles_n) {
    __shared__ Stage st[2];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;

    // ---- which tile: XCD-contiguous remap of the workgroup id, then grouped order
    const int total = tiles_m * tiles_n;
    const int g = blockIdx.x;
    const int xcd = g & 7, local = g >> 3;
    const int full = total >> 3, rem = total & 7;
    const int lin = xcd < rem ? xcd * (full + 1) + local : rem * (full + 1) + (xcd - rem) * full + local;
    const int group = lin / (GROUP_M * tiles_n);
    const int first_m = group * GROUP_M;
    const int gsz = min(tiles_m - first_m, GROUP_M);
    const int in_group = lin - group * GROUP_M * tiles_n;
    const int mt = first_m + in_group % gsz;
    const int nt = in_group / gsz;
    const int m0 = mt * BM, n0 = nt * BN;
    if (!tile_active(slot_seg, capacity, m0, M)) return;

    // ---- global staging: thread owns chunk lc of rows lrow + 32 i, i < 8
    const int lrow = tid >> 3, lc = tid & 7;
    const bf16* a_src[8];
    bool a_ok[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const int m = m0 + lrow + 32 * i;
        a_ok[i] = m < M;
        a_src[i] = A + int64_t(a_ok[i] ? m : m0) * lda + lc * 8;
    }
    const bf16* b_src = B + int64_t(n0 + lrow) * ldb + lc * 8;
    const int64_t b_step = 32 * ldb;
    u32x4 ra[8], rb[8];

    auto gload = [&](int k0) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            ra[i] = a_ok[i] ? *reinterpret_cast<const u32x4*>(a_src[i] + k0) : u32x4{0u, 0u, 0u, 0u};
            rb[i] = *reinterpret_cast<const u32x4*>(b_src + i * b_step + k0);
        }
    };
    auto sstore = [&](Stage& s) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const int r = lrow + 32 * i;
            s.a[r * CH + swz(r, lc)] = ra[i];
            s.b[r * CH + swz(r, lc)] = rb[i];
        }
    };

    f32x16 acc[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i)
#pragma unroll
        for (int j = 0; j < 4; ++j) acc[i][j] = f32x16{};

    const int wn = wave >> 1, wm = wave & 1;
    const int fr = lane & 31, fh = lane >> 5;
    const int nk = K / BK;

    gload(0);
    sstore(st[0]);
    __syncthreads();
    for (int kt = 0; kt < nk; ++kt) {
        const Stage& cur = st[kt & 1];
        if (kt + 1 < nk) gload((kt + 1) * BK);
#pragma unroll
        for (int ks = 0; ks < BK / 16; ++ks) {
            bf16x8 bw[4], ba[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r = wn * 128 + i * 32 + fr;
                bw[i] = as_bf16x8(cur.b[r * CH + swz(r, ks * 2 + fh)]);
            }
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                const int r = wm * 128 + j * 32 + fr;
                ba[j] = as_bf16x8(cur.a[r * CH + swz(r, ks * 2 + fh)]);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i)
#pragma unroll
                for (int j = 0; j < 4; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bw[i], ba[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < nk) sstore(st[(kt + 1) & 1]);
        __syncthreads();
    }

    // ---- epilogue: lane holds, for activation row m, runs of 4 consecutive n
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const int m = m0 + wm * 128 + j * 32 + fr;
        if (m >= M) continue;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int nb = n0 + wn * 128 + i * 32;
            const f32x16& c = acc[i][j];
            if constexpr (EPI == ppk::kStore) {
                bf16* C = static_cast<bf16*>(Cv) + int64_t(m) * ldc;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    bf16x4 v;
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = static_cast<bf16>(c[q * 4 + e]);
                    *reinterpret_cast<bf16x4*>(C + nb + q * 8 + fh * 4) = v;
                }
            } else if constexpr (EPI == ppk::kResidual) {
                float* C = static_cast<float*>(Cv) + int64_t(m) * ldc;
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    f32x4* p = reinterpret_cast<f32x4*>(C + nb + q * 8 + fh * 4);
                    f32x4 v = *p;
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] += c[q * 4 + e];
                    *p = v;
                }
            } else {
                // rows nb..nb+15 of this block are gate rows, nb+16..nb+31 the matching up rows
                bf16* C = static_cast<bf16*>(Cv) + int64_t(m) * ldc + nb / 2;
#pragma unroll
                for (int q = 0; q < 2; ++q) {
                    bf16x4 v;
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = static_cast<bf16>(silu(c[q * 4 + e]) * c[(q + 2) * 4 + e]);
                    *reinterpret_cast<bf16x4*>(C + q * 8 + fh * 4) = v;
                }
            }
        }
    }
}

}  // namespace

namespace ppk {

void gemm_bf16(int epi, const void* A, int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc, int M,
               int N, int K, const int32_t* slot_seg, int capacity, hipStream_t s) {
    if (M <= 0) return;
    const int tiles_m = (M + BM - 1) / BM, tiles_n = N / BN;
    const dim3 grid(tiles_m * tiles_n);
    const bf16* a = static_cast<const bf16*>(A);
    const bf16* b = static_cast<const bf16*>(B);
    switch (epi) {
        case kStore:
            gemm_bf16_kernel<kStore><<<grid, NT, 0, s>>>(a, lda, b, ldb, C, ldc, M, K, slot_seg, capacity,
                                                         tiles_m, tiles_n);
            break;
        case kResidual:
            gemm_bf16_kernel<kResidual><<<grid, NT, 0, s>>>(a, lda, b, ldb, C, ldc, M, K, slot_seg, capacity,
                                                            tiles_m, tiles_n);
            break;
        default:
            gemm_bf16_kernel<kSwiGLU><<<grid, NT, 0, s>>>(a, lda, b, ldb, C, ldc, M, K, slot_seg, capacity,
                                                          tiles_m, tiles_n);
            break;
    }
}

}  // namespace ppk
