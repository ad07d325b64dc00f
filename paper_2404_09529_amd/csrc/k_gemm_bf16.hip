// Projection GEMMs of the decoder layer (section 2.1: X W^Q, X W^K, X W^V; the output
// projection and the SwiGLU MLP of the Llama family) on gfx950 matrix cores.
//
// C[M, N] = A[M, K] B[N, K]^T with A the packed activations (bf16, K contiguous) and B a
// weight matrix in [out, in] layout (bf16, K contiguous), float32 accumulation.
//
// Tiling: one 512-thread workgroup (8 wavefronts) per 256 x 256 output tile, K consumed in
// steps of 64.  Each wavefront owns a 128 (N) x 64 (M) sub-tile = 4 x 2 blocks of the
// 32x32x16 bf16 MFMA, 128 accumulator registers.  The weight block is the MFMA's first
// operand, so a lane's accumulators are 4-element runs along N of one activation row:
// the epilogue writes 8-byte (bf16) or 16-byte (float32) runs without a transpose.
//
// Data path: tiles go straight from global memory into LDS (buffer loads with the LDS
// destination, no staging registers), double-buffered (2 x 64 KB).  Eight wavefronts, two
// per SIMD, run a ping-pong schedule: while one wavefront of a SIMD reads a whole K step of
// MFMA fragments from LDS, the other issues its 32 MFMAs back to back, and they swap at
// every barrier.
//
// Epilogues: bf16 store; float32 residual add; SwiGLU over interleaved gate/up blocks; and,
// for the QKV projection, RoPE at the restart positions (section 3.2) applied to the float32
// accumulators, with queries stored to the packed batch and keys and values stored straight
// into the per-prompt caches (the UNPACK of Algorithm 1).
//
// Scheduling: persistent, one workgroup per CU.  Workgroups are dealt to the 8 XCDs
// round-robin, so XCD x runs workgroups x, x + 8, ...; each XCD owns a contiguous block of
// M-tiles ordered in groups of up to 8 M-tiles sweeping N, and its workgroups take that list
// in strides of their count, so the 32 tiles resident on an XCD always form one compact
// block started together, and the tiles sharing an A or B panel read it from the same L2.
// M-tiles made
// only of row-tail padding are skipped (packed batches only carry pads at row tails,
// section 3.1).
#include "device.h"
#include "kernels.h"

namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int NT = 512;                 // 8 wavefronts, 2 per SIMD
constexpr int ROW_B = BK * 2;           // LDS row: 128 bytes = 8 chunks of 16 bytes
constexpr int OP_B = BM * ROW_B;        // one operand tile in LDS (32 KB)
constexpr int STAGE_B = 2 * OP_B;       // A tile then B tile (64 KB); two stages = 128 KB
constexpr int LOADS = BM * ROW_B / 1024 / 4;  // 1 KB direct-to-LDS loads per wavefront per stage (8)
// group 1 waits for one stage with the next stage's LOADS loads still in flight (vmcnt(8))
static_assert(LOADS == 8, "the vmcnt waits of the K loop assume 8 loads per stage request");
constexpr int LDS_BYTES = 2 * STAGE_B;
// Buffer descriptor word 3 for raw (unstructured) 32-bit-offset loads on gfx9-family parts.
constexpr int kRsrcWord3 = 0x00020000;

// LDS swizzle: logical 16-byte chunk c of tile row r is stored at chunk c ^ f(r).  With
// f(r) = (r ^ r>>3) & 7, the 32 rows x one chunk read by a half-wavefront for an MFMA
// fragment hit distinct banks whether the LDS serves 8 or 16 lanes per cycle.
__device__ __forceinline__ int swz(int r) { return (r ^ (r >> 3)) & 7; }

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ bool tile_active(const int32_t* slot_seg, int capacity, int m0, int M) {
    if (!slot_seg || slot_seg[m0] >= 0) return true;
    // first slot is a row-tail pad: inactive unless another row starts inside the tile
    const int64_t next_row = (int64_t(m0) / capacity + 1) * capacity;
    return next_row < min(m0 + BM, M);
}

__device__ __forceinline__ void barrier() {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// Epilogue of one tile: the lane holds, for activation rows m (two, one per j), runs of 4
// consecutive n of four 32-column blocks.
template <int EPI>
__device__ __forceinline__ void epilogue(const f32x16 (&acc)[4][2], void* __restrict__ Cv, int64_t ldc, int M,
                                         int m0, int n0, int wm, int wn, int fr, int fh,
                                         const int32_t* __restrict__ slot_seg, const ppk::QkvOut& qo) {
    if constexpr (EPI == ppk::kQkvRope) {
        // The wavefront's 128 columns are exactly one head (tiles start at multiples of 256),
        // and the rotate-half partners c and c + 64 are accumulator blocks i and i + 2 of the
        // same lane: RoPE is applied to the float32 accumulators before the one rounding.
        const int head = (n0 + wn * 128) >> 7;
        const int kind = head < qo.H ? 0 : (head < qo.H + qo.Hkv ? 1 : 2);   // q, k, v (uniform)
#pragma unroll
        for (int j = 0; j < 2; ++j) {
            const int m = m0 + wm * 64 + j * 32 + fr;
            if (m >= M) continue;
            bf16* dst;
            if (kind == 0) {
                dst = static_cast<bf16*>(qo.q) + int64_t(m) * qo.ldq + head * 128;
            } else {
                const int kv = qo.slot_kv[m];
                if (kv < 0) continue;
                dst = static_cast<bf16*>(kind == 1 ? qo.kc : qo.vc) + int64_t(kv) * qo.ldkv +
                      (head - qo.H - (kind == 2 ? qo.Hkv : 0)) * 128;
            }
            if (kind < 2) {
                const int pos = slot_seg[m] >= 0 ? qo.slot_pos[m] : 0;
                const float2* cs = qo.table + int64_t(pos) * 64 + fh * 4;
#pragma unroll
                for (int i = 0; i < 2; ++i)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        const f32x4 t0 = *reinterpret_cast<const f32x4*>(cs + i * 32 + q * 8);
                        const f32x4 t1 = *reinterpret_cast<const f32x4*>(cs + i * 32 + q * 8 + 2);
                        const float cv[4] = {t0[0], t0[2], t1[0], t1[2]};
                        const float sv[4] = {t0[1], t0[3], t1[1], t1[3]};
                        bf16x4 lo, hi;
#pragma unroll
                        for (int e = 0; e < 4; ++e) {
                            const float a = acc[i][j][q * 4 + e], b = acc[i + 2][j][q * 4 + e];
                            lo[e] = static_cast<bf16>(a * cv[e] - b * sv[e]);
                            hi[e] = static_cast<bf16>(b * cv[e] + a * sv[e]);
                        }
                        *reinterpret_cast<bf16x4*>(dst + i * 32 + q * 8 + fh * 4) = lo;
                        *reinterpret_cast<bf16x4*>(dst + 64 + i * 32 + q * 8 + fh * 4) = hi;
                    }
            } else {
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int q = 0; q < 4; ++q) {
                        bf16x4 v;
#pragma unroll
                        for (int e = 0; e < 4; ++e) v[e] = static_cast<bf16>(acc[i][j][q * 4 + e]);
                        *reinterpret_cast<bf16x4*>(dst + i * 32 + q * 8 + fh * 4) = v;
                    }
            }
        }
        return;
    }
#pragma unroll
    for (int j = 0; j < 2; ++j) {
        const int m = m0 + wm * 64 + j * 32 + fr;
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

template <int EPI>
__global__ __launch_bounds__(NT) void gemm_bf16_kernel(const bf16* __restrict__ A, int64_t lda,
                                                       const bf16* __restrict__ B, int64_t ldb,
                                                       void* __restrict__ Cv, int64_t ldc, int M, int K,
                                                       const int32_t* __restrict__ slot_seg, int capacity,
                                                       int tiles_m, int tiles_n, ppk::QkvOut qo) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: LDS bases and descriptors in SGPRs

    // ---- persistent schedule.  Workgroups are dealt to the 8 XCDs round-robin (XCD = id % 8)
    // and the grid holds one workgroup per CU, so XCD x runs workgroups x, x + 8, ... one per
    // CU.  XCD x owns the contiguous block of M-tiles [x pm, x pm + pm), ordered in groups of
    // at most 8 M-tiles, each group sweeping all N-tiles; its workgroups take that list in
    // strides of their count.  The tiles resident on an XCD at any time are therefore one
    // compact block of the list (about 8 M x 4 N tiles) started together, at the same K step:
    // each 64-wide K slice of an activation or weight panel is fetched into the XCD's L2 once
    // and read there by every tile of the block.  Every XCD sweeps N at the same rate, so the
    // weight panels are also shared through the last-level cache.
    const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3, n_slots = gridDim.x >> 3;
    const int pm = (tiles_m + 7) / 8;
    const int m_begin = xcd * pm, m_cnt = min(pm, tiles_m - m_begin);
    if (m_cnt <= 0) return;
    const int n_groups = (m_cnt + 7) / 8, gm = (m_cnt + n_groups - 1) / n_groups;
    const int n_local = m_cnt * tiles_n;

    // ---- direct global -> LDS loads.  A stage holds the A tile then the B tile, 8 chunks of
    // 16 bytes per row.  Load t of wavefront w fills 1 KB = rows 8 j .. 8 j + 7 of its operand
    // (j = (w % 4) * 8 + t; wavefronts 0-3 load A, 4-7 load B); lane l lands at physical chunk
    // l % 8 of row 8 j + l / 8, so it fetches the logical chunk that the swizzle puts there.
    // Every quad of lanes reads one aligned 64-byte half of a row.  Rows of A past M read as
    // zero (the descriptor ends at row min(M, m0 + 256)); every access is inside its buffer.
    const bool load_b = wave >= 4;
    const int64_t ld = load_b ? ldb : lda;
    int voff[LOADS];
#pragma unroll
    for (int t = 0; t < LOADS; ++t) {
        const int row = 8 * ((wave & 3) * LOADS + t) + lane / 8;
        voff[t] = static_cast<int>(row * ld * 2) + 16 * ((lane & 7) ^ swz(row));
    }
    const int lds_op = load_b ? OP_B : 0;

    // ---- wavefront sub-tile: 128 (N) x 64 (M) = 4 x 2 MFMA blocks of 32 x 32
    const int wn = wave & 1, wm = wave >> 1;
    const int grp = wave >> 2;               // waves w and w + 4 share a SIMD
    const int fr = lane & 31, fh = lane >> 5;

    // fragment addresses.  Row r = base + 32 i + fr of either operand has swizzle
    // f(r) = g ^ 4 (i & 1) with g = ((fr & 7) ^ (fr >> 3)) & 7 (base is a multiple of 64), so
    // the physical chunk of logical chunk 2 ks + fh is (2 (ks ^ 2 (i & 1))) ^ (fh ^ g): four
    // per-lane offsets cover every (ks, i); the block stride (32 rows = 4 KB) is immediate.
    const int gsw = ((fr & 7) ^ (fr >> 3)) & 7;
    const int x = fh ^ gsw;
    int a_lds[4], b_lds[4];
#pragma unroll
    for (int m = 0; m < 4; ++m) {
        a_lds[m] = (wm * 64 + fr) * ROW_B + 16 * ((2 * m) ^ x);
        b_lds[m] = OP_B + (wn * 128 + fr) * ROW_B + 16 * ((2 * m) ^ x);
    }
    const int nk = K / BK;

    for (int local = slot; local < n_local; local += n_slots) {
        const int group = local / (gm * tiles_n), within = local - group * gm * tiles_n;
        const int first = group * gm, gsz = min(m_cnt - first, gm);
        const int mt = m_begin + first + within % gsz;
        const int nt = within / gsz;
        const int m0 = mt * BM, n0 = nt * BN;
        if (!tile_active(slot_seg, capacity, m0, M)) continue;

        const int a_rows = min(M - m0, BM);
        const __amdgpu_buffer_rsrc_t rsrc = load_b
            ? __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(B + int64_t(n0) * ldb), 0,
                                                static_cast<int>(BN * ldb * 2), kRsrcWord3)
            : __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(A + int64_t(m0) * lda), 0,
                                                static_cast<int>(a_rows * lda * 2), kRsrcWord3);
        auto issue_loads = [&](int kt) {
            char* stage = smem + (kt & 1) * STAGE_B + lds_op;
#pragma unroll
            for (int t = 0; t < LOADS; ++t) {
                lds_void* dst = (lds_void*)(stage + ((wave & 3) * LOADS + t) * 1024);   // generic -> LDS
                __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc, dst, 16, voff[t], kt * BK * 2, 0, 0);
            }
        };

        f32x16 acc[4][2];
#pragma unroll
        for (int i = 0; i < 4; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j) acc[i][j] = f32x16{};
        bf16x8 fw[BK / 16][4], fa[BK / 16][2];
        auto read_frags = [&](int kt) {
            const char* stage = smem + (kt & 1) * STAGE_B;
#pragma unroll
            for (int ks = 0; ks < BK / 16; ++ks) {
#pragma unroll
                for (int i = 0; i < 4; ++i)
                    fw[ks][i] = *reinterpret_cast<const bf16x8*>(stage + b_lds[ks ^ (2 * (i & 1))] + i * 32 * ROW_B);
#pragma unroll
                for (int j = 0; j < 2; ++j)
                    fa[ks][j] = *reinterpret_cast<const bf16x8*>(stage + a_lds[ks ^ (2 * (j & 1))] + j * 32 * ROW_B);
            }
        };
        auto mfmas = [&]() {
            __builtin_amdgcn_s_setprio(1);
#pragma unroll
            for (int ks = 0; ks < BK / 16; ++ks)
#pragma unroll
                for (int i = 0; i < 4; ++i)
#pragma unroll
                    for (int j = 0; j < 2; ++j)
                        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(fw[ks][i], fa[ks][j], acc[i][j], 0, 0, 0);
            __builtin_amdgcn_s_setprio(0);
        };

        // ---- ping-pong over K.  Group 0 runs [memory, MFMA] phases; group 1 runs the same
        // one phase later, so on every SIMD one wavefront issues MFMAs while the other reads
        // LDS.  Tile kt+1 is requested in phase 2kt (group 0 in its memory phase, group 1 at
        // the end of its MFMA phase) and waited for at the end of phase 2kt+1; a stage is
        // refilled only after both groups have read it.  Both groups execute 2 nk + 2
        // barriers, and every LDS read of the tile has completed before the last one, so the
        // next tile may refill either stage right after it.
        // Waits never rely on loads retiring in issue order across descriptors: group 0's A
        // loads (rows past M read as zero) are waited for with vmcnt(0); group 1's B loads
        // are all in range, and it keeps only the next stage's LOADS loads in flight.
        issue_loads(0);
        __builtin_amdgcn_s_waitcnt(0);
        barrier();
        if (grp == 0) {
            for (int kt = 0; kt < nk; ++kt) {
                read_frags(kt);
                if (kt + 1 < nk) issue_loads(kt + 1);        // after the LDS reads: they start first
                __builtin_amdgcn_s_waitcnt(0xc07f);          // lgkmcnt(0): fragments in registers
                barrier();
                mfmas();
                __builtin_amdgcn_s_waitcnt(0x0f70);          // vmcnt(0): this group's part of tile kt+1
                barrier();
            }
            barrier();
        } else {
            if (nk > 1) issue_loads(1);
            barrier();
            for (int kt = 0; kt < nk; ++kt) {
                read_frags(kt);
                // Tile kt+2 goes to the stage this group has just finished reading (group 0 read
                // it in phase 2kt), so its loads are issued here, in this group's memory phase:
                // group 0 issues its loads in the other phase, and the CU's single address unit
                // then sees half of a K step's loads in each phase.  They are waited for one
                // iteration later, so they have two phases to land.
                __builtin_amdgcn_s_waitcnt(0xc07f);          // lgkmcnt(0): fragments in registers
                if (kt + 2 < nk) {
                    issue_loads(kt + 2);
                    __builtin_amdgcn_s_waitcnt(0x0f78);      // vmcnt(8): tile kt+1 landed, kt+2 in flight
                } else {
                    __builtin_amdgcn_s_waitcnt(0x0f70);      // vmcnt(0)
                }
                barrier();
                mfmas();
                barrier();
            }
        }
        epilogue<EPI>(acc, Cv, ldc, M, m0, n0, wm, wn, fr, fh, slot_seg, qo);
    }
    __builtin_amdgcn_s_waitcnt(0);   // no load may still be writing LDS when the workgroup ends
}

}  // namespace

namespace ppk {

namespace {

constexpr size_t kLds = LDS_BYTES;

template <int EPI>
void launch(const void* A, int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc, int M, int N, int K,
            const int32_t* slot_seg, int capacity, const QkvOut& qo, hipStream_t s) {
    static bool attr = [] {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_bf16_kernel<EPI>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, kLds);
        return true;
    }();
    (void)attr;
    const int tiles_m = (M + BM - 1) / BM, tiles_n = N / BN;
    // one workgroup per CU (each needs 128 KB of LDS, so a CU holds one), a multiple of 8 so
    // that every XCD runs the same number; never more workgroups than tiles
    static const int n_cu = [] {
        int dev = 0, n = 0;
        (void)hipGetDevice(&dev);
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 8) n = 8;
        return n / 8 * 8;
    }();
    const int per_xcd = ((tiles_m + 7) / 8) * tiles_n;
    const dim3 grid(8 * min(n_cu / 8, per_xcd));
    gemm_bf16_kernel<EPI><<<grid, NT, kLds, s>>>(static_cast<const bf16*>(A), lda, static_cast<const bf16*>(B),
                                                ldb, C, ldc, M, K, slot_seg, capacity, tiles_m, tiles_n, qo);
}

}  // namespace

void gemm_bf16(int epi, const void* A, int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc, int M,
               int N, int K, const int32_t* slot_seg, int capacity, hipStream_t s) {
    if (M <= 0) return;
    const QkvOut none{};
    switch (epi) {
        case kStore: launch<kStore>(A, lda, B, ldb, C, ldc, M, N, K, slot_seg, capacity, none, s); break;
        case kResidual: launch<kResidual>(A, lda, B, ldb, C, ldc, M, N, K, slot_seg, capacity, none, s); break;
        default: launch<kSwiGLU>(A, lda, B, ldb, C, ldc, M, N, K, slot_seg, capacity, none, s); break;
    }
}

void qkv_rope_bf16(const void* A, int64_t lda, const void* B, int64_t ldb, int M, int K, const int32_t* slot_seg,
                   int capacity, const QkvOut& out, hipStream_t s) {
    if (M <= 0) return;
    launch<kQkvRope>(A, lda, B, ldb, nullptr, 0, M, (out.H + 2 * out.Hkv) * 128, K, slot_seg, capacity, out, s);
}

}  // namespace ppk
