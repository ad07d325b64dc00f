// Projection GEMMs of the decoder layer (section 2.1: X W^Q, X W^K, X W^V; the output
// projection and the SwiGLU MLP of the Llama family) on gfx950 matrix cores.
//
// C[M, N] = A[M, K] B[N, K]^T with A the packed activations (bf16, K contiguous) and B a
// weight matrix in [out, in] layout (bf16, K contiguous), float32 accumulation.
//
// Tiling: one 256-thread workgroup (4 wavefronts, one per SIMD) per 256 x 256 output tile,
// K consumed in steps of 64.  Each wavefront owns a 128 (N) x 128 (M) sub-tile = 8 x 8
// blocks of the 16x16x32 bf16 MFMA; its 256 float32 accumulators live in the accumulation
// registers.  (Under the chip's power limit the 16x16x32 form sustains a higher clock than
// 32x32x16 for the same work: it moves half the accumulator bytes per flop.)  The weight
// block is the MFMA's first operand, so a lane's accumulators are 4-element runs along N of
// one activation row.
//
// Data path: operand tiles go straight from global memory into LDS (buffer loads with the
// LDS destination, no staging registers), whole 128-byte row segments per request.  The LDS
// is a ring of 5 slots of 32 KB, each holding one operand (A or B) of one K-step; slots are
// filled in the order A0 B0 A1 B1 ... and freed in pairs when a step has been read, so two
// operand tiles are always in flight while a step is consumed.  The workgroup's tiles form
// one continuous stream of K-steps: the loads cross tile boundaries, and the first steps of
// the next tile land while the epilogue of the current one runs.  A step is two sub-steps of
// 64 MFMAs per wavefront; each sub-step also reads the fragments of the next sub-step from
// LDS and issues one operand tile (8 loads per wavefront), which keeps the CU's address
// unit about half busy at all times.  One barrier per step.
//
// Epilogues: bf16 store; float32 residual add; SwiGLU over interleaved gate/up blocks; and,
// for the QKV projection, RoPE at the restart positions (section 3.2) applied to the float32
// accumulators, with queries stored to the packed batch and keys and values stored straight
// into the per-prompt caches (the UNPACK of Algorithm 1).  bf16 results are staged through
// LDS and stored as whole rows.
//
// Scheduling: persistent, one workgroup per CU.  Workgroups are dealt to the 8 XCDs
// round-robin, so XCD x runs workgroups x, x + 8, ...; each XCD owns a contiguous block of
// M-tiles ordered in groups of up to 8 M-tiles sweeping N, and its workgroups take that list
// in strides of their count, so the 32 tiles resident on an XCD always form one compact
// block, and the tiles sharing an A or B panel read it from the same L2.  The M-tiles are
// the plan's row-tile list: tiles made only of row-tail padding (packed batches carry pads
// only at row tails, section 3.1) are not in it, so they are neither computed nor counted
// when the tiles are split across the XCDs.
#include "device.h"
#include "kernels.h"

namespace {

constexpr int BM = 256, BN = 256, BK = 64;
constexpr int NT = 256;                  // 4 wavefronts, one per SIMD
constexpr int ROW_B = BK * 2;            // LDS row: 128 bytes = 8 chunks of 16 bytes
constexpr int SLOT_B = BM * ROW_B;       // one operand of one K-step (32 KB)
constexpr int NSLOT = 5;                 // the whole 160 KB LDS of a CU
constexpr int LDS_BYTES = NSLOT * SLOT_B;
constexpr int LOADS = SLOT_B / 1024 / 4; // 1 KB loads per wavefront per operand tile (8)
static_assert(LOADS == 8, "the vmcnt wait of the K loop counts 8 loads per operand tile");

// s_waitcnt immediate: vmcnt(n) and lgkmcnt(0), expcnt not waited for (gfx9 encoding:
// vmcnt bits 3:0 and 15:14, expcnt 6:4, lgkmcnt 11:8)
constexpr int wait_vm_lgkm0(int n) { return ((n >> 4) << 14) | (n & 15) | 0x0070; }
// Buffer descriptor word 3 for raw (unstructured) 32-bit-offset loads on gfx9-family parts.
constexpr int kRsrcWord3 = 0x00020000;

// LDS swizzle: logical 16-byte chunk c of tile row r is stored at chunk c ^ f(r), where f's
// bits are r's bits 1, 3 and 2.  An MFMA fragment read (ds_read_b128) fetches chunks
// 4 ks + l / 16 of rows l % 16; the LDS serves it 16 lanes (256 bytes, all 64 banks) per
// cycle, taking lanes i and i + 32 together (lanes 0-7 with 32-39, and so on), which is
// 8 rows x chunks {c, c ^ 2}.  A 128-byte row covers half the banks, so the 16 accesses are
// conflict-free when (r % 2, physical chunk) are distinct: within each parity the four rows
// must give f values in distinct classes {x, x ^ 2}, i.e. distinct (bit 0, bit 2) of f,
// which are r's bits 1 and 2.  (The same f is also conflict-free if the LDS took 16
// consecutive lanes.)  f depends on r % 16 only.
__device__ __forceinline__ int swz(int r) { return ((r >> 1) & 1) | (((r >> 3) & 1) << 1) | (r & 4); }

typedef __attribute__((address_space(3))) void lds_void;

__device__ __forceinline__ void barrier() {
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
}

// The accumulators of activation blocks 2 jp and 2 jp + 1, pinned in the accumulation
// registers at this point: the epilogue then moves them to vector registers a pair of blocks
// at a time instead of all at once (which would need every vector register and spill).  The
// accumulators are dead afterwards.
__device__ __forceinline__ void take_pair(f32x4 (&acc)[8][8], int jp, f32x4 (&c)[8][2]) {
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            asm volatile("" : "+a"(acc[i][2 * jp + h]) : : "memory");
            c[i][h] = acc[i][2 * jp + h];
        }
}

// Staged bf16 output of 32 activation rows: lanes write 8-byte runs in MFMA layout to this
// wavefront's LDS staging area, then read back whole 16-byte chunks of rows and store them
// with each instruction covering complete rows (full cache lines).  Row r's 16-byte chunk c
// sits at chunk c ^ (r % CHUNKS) of the staging row.
template <int CHUNKS>
__device__ __forceinline__ void stage_put(char* stg, int r, int c, int half, bf16x4 v) {
    *reinterpret_cast<bf16x4*>(stg + r * CHUNKS * 16 + ((c ^ (r % CHUNKS)) * 16) + half * 8) = v;
}

// The epilogue of one wavefront sub-tile (activation rows mb.., weight rows nb0..).  In block
// (i, j) lane l holds activation row mb + 16 j + l % 16 and the 4 consecutive weight rows
// nb0 + 16 i + 4 (l / 16) + 0..3.  stg is this wavefront's 8 KB of LDS, free for the duration
// of the epilogue.
template <int EPI>
__device__ __forceinline__ void epilogue(f32x4 (&acc)[8][8], void* __restrict__ Cv, int64_t ldc, int M,
                                         int mb, int nb0, int lane, const ppk::QkvOut& qo, char* stg) {
    const int lr = lane & 15, g = lane >> 4;
    if constexpr (EPI == ppk::kResidual) {
        // C[m][nb0 ..] += this lane's accumulators, one 16-row block j at a time, staged
        // through LDS (16 rows x 128 floats, 512-byte rows) so that C is read and written as
        // whole rows: instruction k covers rows 2 k and 2 k + 1, 16 bytes per lane.  C moves
        // with non-temporal loads and stores (it is touched once per tile; the O projection
        // measured 3% faster, the down projection the same).  The C
        // rows of block j + 1 are requested before block j is stored: vmcnt counts stores and
        // completes in order, so a load issued after a store would wait for the store.
        // Staging row r's 16-byte chunk q sits at q ^ f(r), f = (r0 << 3) | (r1 << 2) | r2
        // (r's low bits): the MFMA-layout writes (rows r, chunks 4 i + g and 4 i + g ^ 2 per
        // pair of lane groups) and the row reads (rows 2 k and 2 k + 1, chunks 0..7 or 8..15
        // per pair) both land on distinct banks.
        auto f = [](int r) { return ((r & 1) << 3) | (((r >> 1) & 1) << 2) | ((r >> 2) & 1); };
        float* C = static_cast<float*>(Cv);
        const int half = lane >> 5, col = nb0 + 4 * (lane & 31);
        f32x4 cbuf[2][8];
        auto load_block = [&](int j, f32x4 (&buf)[8]) {
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int m = min(mb + 16 * j + 2 * k + half, M - 1);   // rows past M: read, not stored
                buf[k] = __builtin_nontemporal_load(reinterpret_cast<const f32x4*>(C + int64_t(m) * ldc + col));
            }
        };
        load_block(0, cbuf[0]);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (j + 1 < 8) load_block(j + 1, cbuf[(j + 1) & 1]);
            f32x4 cj[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                asm volatile("" : "+a"(acc[i][j]) : : "memory");
                cj[i] = acc[i][j];
            }
#pragma unroll
            for (int i = 0; i < 8; ++i)
                *reinterpret_cast<f32x4*>(stg + lr * 512 + (((4 * i + g) ^ f(lr)) * 16)) = cj[i];
            f32x4 v[8];
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int r = 2 * k + half;
                v[k] = *reinterpret_cast<const f32x4*>(stg + r * 512 + (((lane & 31) ^ f(r)) * 16));
            }
#pragma unroll
            for (int k = 0; k < 8; ++k) {
                const int m = mb + 16 * j + 2 * k + half;
                if (m < M)
                    __builtin_nontemporal_store(v[k] + cbuf[j & 1][k], reinterpret_cast<f32x4*>(C + int64_t(m) * ldc + col));
            }
        }
        // Wait for the stores too (and with them, vmcnt being in order, everything before
        // them), once per tile: otherwise the compiler protects the stores' data registers
        // with vmcnt waits inside the next K loop, where they would stall behind the loads.
        __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(0));
        return;
    }
    if constexpr (EPI == ppk::kQkvRope) {
        // The wavefront's 128 columns are exactly one head (tiles start at multiples of 256),
        // and the rotate-half partners c and c + 64 are accumulator blocks i and i + 4 of the
        // same lane: RoPE is applied to the float32 accumulators before the one rounding.
        // One 16-row block j at a time, staged through LDS (16 rows x 256 bytes) and stored
        // as whole rows.  The slot metadata of all 8 of the lane's rows is read first (a slot
        // outside every span has position 0 and no cache row); the cos/sin rows of block j + 1
        // are requested before block j is stored (vmcnt counts stores and completes in order).
        const int head = nb0 >> 7;
        const int kind = head < qo.H ? 0 : (head < qo.H + qo.Hkv ? 1 : 2);   // q, k, v (uniform)
        int drow[8], pos[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int m = mb + 16 * j + lr, mc = min(m, M - 1);
            const int kv = kind > 0 ? qo.slot_kv[mc] : m;
            drow[j] = m < M ? kv : -1;
            pos[j] = qo.slot_pos[mc];
        }
        f32x4 tb[2][8];
        auto load_tab = [&](int j, f32x4 (&t)[8]) {
            const float2* cs = qo.table + int64_t(pos[j]) * 64 + 4 * g;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                t[2 * i] = *reinterpret_cast<const f32x4*>(cs + 16 * i);
                t[2 * i + 1] = *reinterpret_cast<const f32x4*>(cs + 16 * i + 2);
            }
        };
        if (kind < 2) load_tab(0, tb[0]);
        bf16* base = kind == 0 ? static_cast<bf16*>(qo.q) + head * 128
                               : static_cast<bf16*>(kind == 1 ? qo.kc : qo.vc) +
                                     (head - qo.H - (kind == 2 ? qo.Hkv : 0)) * 128;
        const int64_t ld = kind == 0 ? qo.ldq : qo.ldkv;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            if (kind < 2 && j + 1 < 8) load_tab(j + 1, tb[(j + 1) & 1]);
            f32x4 c[8];
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                asm volatile("" : "+a"(acc[i][j]) : : "memory");
                c[i] = acc[i][j];
            }
            if (kind < 2) {
#pragma unroll
                for (int i = 0; i < 4; ++i) {
                    const f32x4 t0 = tb[j & 1][2 * i], t1 = tb[j & 1][2 * i + 1];
                    const float cv[4] = {t0[0], t0[2], t1[0], t1[2]};
                    const float sv[4] = {t0[1], t0[3], t1[1], t1[3]};
                    bf16x4 lo, hi;
#pragma unroll
                    for (int e = 0; e < 4; ++e) {
                        const float x = c[i][e], y = c[i + 4][e];
                        lo[e] = static_cast<bf16>(x * cv[e] - y * sv[e]);
                        hi[e] = static_cast<bf16>(y * cv[e] + x * sv[e]);
                    }
                    stage_put<16>(stg, lr, 2 * i + (g >> 1), g & 1, lo);
                    stage_put<16>(stg, lr, 8 + 2 * i + (g >> 1), g & 1, hi);
                }
            } else {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    bf16x4 v;
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = static_cast<bf16>(c[i][e]);
                    stage_put<16>(stg, lr, 2 * i + (g >> 1), g & 1, v);
                }
            }
            bf16x8 v[4];
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int r = 4 * k + lane / 16, ch = lane % 16;
                v[k] = *reinterpret_cast<const bf16x8*>(stg + r * 256 + ((ch ^ r) * 16));
            }
#pragma unroll
            for (int k = 0; k < 4; ++k) {
                const int r = 4 * k + lane / 16, ch = lane % 16;
                const int d = __shfl(drow[j], r);   // lane r holds row r's destination
                if (d >= 0) *reinterpret_cast<bf16x8*>(base + int64_t(d) * ld + ch * 8) = v[k];
            }
        }
        __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(0));   // as in the residual epilogue
        return;
    }
    // bf16 outputs: 128 columns (16 chunks) per row, or 64 (8 chunks) after SwiGLU
    constexpr int CH = EPI == ppk::kSwiGLU ? 8 : 16;
#pragma unroll
    for (int jp = 0; jp < 4; ++jp) {
        f32x4 c[8][2];
        take_pair(acc, jp, c);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int r = 16 * h + lr;   // row in the staging block
            if constexpr (EPI == ppk::kSwiGLU) {
                // weight rows 32 k .. +15 (block 2 k) are gate rows, 32 k + 16 .. +31 (block
                // 2 k + 1) the matching up rows: output column 16 k + 4 g + e
#pragma unroll
                for (int k = 0; k < 4; ++k) {
                    bf16x4 v;
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = static_cast<bf16>(silu_rcp(c[2 * k][h][e]) * c[2 * k + 1][h][e]);
                    stage_put<CH>(stg, r, 2 * k + (g >> 1), g & 1, v);
                }
            } else {
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    bf16x4 v;
#pragma unroll
                    for (int e = 0; e < 4; ++e) v[e] = static_cast<bf16>(c[i][h][e]);
                    stage_put<CH>(stg, r, 2 * i + (g >> 1), g & 1, v);
                }
            }
        }
        // read back whole rows: instruction k covers rows (64 / CH) k .. of the 32-row block
        constexpr int RPI = 64 / CH;   // rows per instruction
        bf16x8 v[32 / RPI];
#pragma unroll
        for (int k = 0; k < 32 / RPI; ++k) {
            const int r = k * RPI + lane / CH, ch = lane % CH;
            v[k] = *reinterpret_cast<const bf16x8*>(stg + r * CH * 16 + ((ch ^ (r % CH)) * 16));
        }
#pragma unroll
        for (int k = 0; k < 32 / RPI; ++k) {
            const int r = k * RPI + lane / CH, ch = lane % CH;
            const int mr = mb + 32 * jp + r;
            if (mr >= M) continue;
            bf16* C = static_cast<bf16*>(Cv) + int64_t(mr) * ldc + (EPI == ppk::kSwiGLU ? nb0 / 2 : nb0);
            *reinterpret_cast<bf16x8*>(C + ch * 8) = v[k];
        }
    }
    // the staging area is refilled by this wavefront's own loads right after the epilogue
    __builtin_amdgcn_s_waitcnt(0xc07f);   // lgkmcnt(0)
}

template <int EPI>
__global__ __launch_bounds__(NT, 1) void gemm_bf16_kernel(const bf16* __restrict__ A, int64_t lda,
                                                          const bf16* __restrict__ B, int64_t ldb,
                                                          void* __restrict__ Cv, int64_t ldc, int M, int K,
                                                          const int32_t* __restrict__ mtile_m0, int tiles_m,
                                                          int tiles_n, int balanced, ppk::QkvOut qo) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform: LDS bases and descriptors in SGPRs

    // ---- persistent schedule over tiles_m M-tiles (M-tile i starts at row mtile_m0[i], or at
    // row BM i without a list) and tiles_n N-tiles.  Workgroups are dealt to the 8 XCDs
    // round-robin (XCD = id % 8)
    // and the grid holds one workgroup per CU, so XCD x runs workgroups x, x + 8, ... one per
    // CU.  XCD x owns the contiguous block of M-tiles [x pm, x pm + pm), ordered in groups of
    // at most 8 M-tiles, each group sweeping all N-tiles; its workgroups take that list in
    // strides of their count.  The tiles resident on an XCD at any time are therefore one
    // compact block of the list (about 8 M x 4 N tiles) started together, at the same K step:
    // each K slice of an activation or weight panel is fetched into the XCD's L2 once and
    // read there by every tile of the block.  Every XCD sweeps N at the same rate, so the
    // weight panels are also shared through the last-level cache.
    //
    // When tiles_m is not a multiple of 8 that split can leave one XCD a whole round of tiles
    // more than the average; then (balanced != 0) the same group-ordered list is built over
    // all M-tiles and cut into 8 contiguous ranges of equal length instead, one per XCD (a
    // range may start inside a group, so two XCDs can share an activation panel).
    const int xcd = blockIdx.x & 7, slot = blockIdx.x >> 3, n_slots = gridDim.x >> 3;
    int m_begin, m_cnt, g_begin, n_local;
    if (balanced) {
        const int total = tiles_m * tiles_n, per = (total + 7) / 8;
        m_begin = 0;
        m_cnt = tiles_m;
        g_begin = xcd * per;
        n_local = min(per, total - g_begin);
    } else {
        const int pm = (tiles_m + 7) / 8;
        m_begin = xcd * pm;
        m_cnt = min(pm, tiles_m - m_begin);
        g_begin = 0;
        n_local = m_cnt * tiles_n;
    }
    if (m_cnt <= 0 || n_local <= 0) return;
    const int n_groups = (m_cnt + 7) / 8, gm = (m_cnt + n_groups - 1) / n_groups;
    auto tile_m0 = [&](int local) {
        const int gi = g_begin + local;
        const int group = gi / (gm * tiles_n), within = gi - group * gm * tiles_n;
        const int first = group * gm, gsz = min(m_cnt - first, gm);
        const int mt = m_begin + first + within % gsz;
        return mtile_m0 ? mtile_m0[mt] : mt * BM;
    };
    auto tile_n0 = [&](int local) {
        const int gi = g_begin + local;
        const int group = gi / (gm * tiles_n), within = gi - group * gm * tiles_n;
        const int first = group * gm, gsz = min(m_cnt - first, gm);
        return (within / gsz) * BN;
    };
    const int nk = K / BK;

    // ---- direct global -> LDS loads.  Load t (0..7) of wavefront w fills 1 KB = rows
    // 64 w + 8 t .. + 7 of an operand tile; lane l lands at physical chunk l % 8 of row
    // 64 w + 8 t + l / 8 and fetches the logical chunk that the swizzle puts there.  Rows of
    // A past M are read as row M - 1: every load is in range, so loads complete in the order
    // they were issued, and the results of the duplicated rows are never stored.
    const int64_t lda2 = lda * 2, ldb2 = ldb * 2;
    const int lrow = lane >> 3;
    int chunk_off[LOADS], voff_b[LOADS], voff_a[LOADS];
#pragma unroll
    for (int t = 0; t < LOADS; ++t) {
        chunk_off[t] = 16 * ((lane & 7) ^ swz(8 * (t & 1) + lrow));
        voff_b[t] = static_cast<int>((64 * wave + 8 * t + lrow) * ldb2) + chunk_off[t];
    }

    // load cursor: the K-step whose operand tiles are being requested, into slots l_sa (A)
    // and l_sb (B); l_local >= n_local once the stream is exhausted (its loads are then dead:
    // they read nothing and land in slots that are never read again)
    int l_local = slot, l_kt = 0, l_sa = 0, l_sb = 1;
    __amdgpu_buffer_rsrc_t rsrc_a, rsrc_b;
    const __amdgpu_buffer_rsrc_t rsrc_0 = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(A), 0, 0, kRsrcWord3);
    auto set_cursor_tile = [&]() {
        if (l_local < n_local) {
            const int m0 = tile_m0(l_local), n0 = tile_n0(l_local);
            const int a_rows = min(M - m0, BM);
            rsrc_a = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(A + int64_t(m0) * lda), 0,
                                                       static_cast<int>(a_rows * lda2), kRsrcWord3);
            rsrc_b = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(B + int64_t(n0) * ldb), 0,
                                                       static_cast<int>(BN * ldb2), kRsrcWord3);
#pragma unroll
            for (int t = 0; t < LOADS; ++t)
                voff_a[t] = static_cast<int>(min(64 * wave + 8 * t + lrow, a_rows - 1) * lda2) + chunk_off[t];
        } else {
            rsrc_a = rsrc_0;
            rsrc_b = rsrc_0;
        }
    };
    set_cursor_tile();
    auto load_a = [&](int t) {
        char* dst = smem + l_sa * SLOT_B + (wave * LOADS + t) * 1024;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc_a, (lds_void*)dst, 16, voff_a[t], l_kt * BK * 2, 0, 0);
    };
    auto load_b = [&](int t) {
        char* dst = smem + l_sb * SLOT_B + (wave * LOADS + t) * 1024;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rsrc_b, (lds_void*)dst, 16, voff_b[t], l_kt * BK * 2, 0, 0);
    };
    auto advance_cursor = [&]() {
        l_sa = l_sa >= NSLOT - 2 ? l_sa + 2 - NSLOT : l_sa + 2;
        l_sb = l_sb >= NSLOT - 2 ? l_sb + 2 - NSLOT : l_sb + 2;
        if (l_local >= n_local) return;
        if (++l_kt == nk) {
            l_kt = 0;
            l_local += n_slots;
            set_cursor_tile();
        }
    };

    // ---- wavefront sub-tile: 128 (N) x 128 (M) = 8 x 8 MFMA blocks of 16 x 16.  A fragment
    // of block i for sub-step ks: row base + 16 i + l % 16 (base a multiple of 128), logical
    // chunk 4 ks + l / 16 of the step's 128-byte row.  The row's swizzle depends on l % 16
    // only, so one per-lane offset per sub-step covers all blocks; the block stride (16 rows
    // = 2 KB) is immediate.
    const int wn = wave & 1, wm = wave >> 1;
    int a_lds[2], b_lds[2];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
        const int phys = ((4 * ks + (lane >> 4)) ^ swz(lane & 15)) * 16;
        a_lds[ks] = (wm * 128 + (lane & 15)) * ROW_B + phys;
        b_lds[ks] = (wn * 128 + (lane & 15)) * ROW_B + phys;
    }
    struct Frags { bf16x8 w[8], a[8]; };
    // fragment q of sub-step ks of the step held in slots (sa, sb), in the order the MFMAs
    // first need them: w0, a0..a7, w1..w7
    auto read_one = [&](int sa, int sb, int ks, int q, Frags& f) {
        if (q == 0) {
            f.w[0] = *reinterpret_cast<const bf16x8*>(smem + sb * SLOT_B + b_lds[ks]);
        } else if (q < 9) {
            const int j = q - 1;
            f.a[j] = *reinterpret_cast<const bf16x8*>(smem + sa * SLOT_B + a_lds[ks] + j * 16 * ROW_B);
        } else {
            const int i = q - 8;
            f.w[i] = *reinterpret_cast<const bf16x8*>(smem + sb * SLOT_B + b_lds[ks] + i * 16 * ROW_B);
        }
    };

    // ---- the K-step stream.  Step g holds slots 2g % 5 (A) and (2g+1) % 5 (B).  Per step:
    //   sub-step 0: MFMAs (g, 0); read (g, 1); A tile of step g+2 (into the slot of B of g-1)
    //   wait until step g+1 has landed and this wavefront's reads of step g are done; barrier
    //   sub-step 1: MFMAs (g, 1); read (g+1, 0); B tile of step g+2 (into the slot of A of g)
    // The B tile of g+1 was requested right after the previous barrier, one sub-step before
    // the A tile of g+2; at this barrier the loads issued after it are the 8 of the A tile of
    // g+2, so vmcnt(8) (vmcnt(0) when g+2 does not exist) waits for g+1 exactly.
    int c_local = l_local;
    if (c_local >= n_local) return;
    // prologue: steps 0 and 1
#pragma unroll
    for (int p = 0; p < 2; ++p) {
#pragma unroll
        for (int t = 0; t < LOADS; ++t) load_a(t);
#pragma unroll
        for (int t = 0; t < LOADS; ++t) load_b(t);
        advance_cursor();
    }
    __builtin_amdgcn_s_waitcnt(0);
    barrier();
    Frags F0, F1;
    int c_sa = 0, c_sb = 1;
#pragma unroll
    for (int q = 0; q < 16; ++q) read_one(c_sa, c_sb, 0, q, F0);
    while (true) {
        f32x4 acc[8][8];
#pragma unroll
        for (int i = 0; i < 8; ++i)
#pragma unroll
            for (int j = 0; j < 8; ++j) acc[i][j] = f32x4{};
        // One sub-step: the 64 MFMAs on `cur`, with the 16 fragment reads of the next sub-step
        // (into `nxt`) and one load after every eighth MFMA, in a fixed order: the reads and
        // loads issue while the matrix core works.  The first sub-step (A loads) ends at the
        // barrier: its reads go after every third of the first 48 MFMAs, so they have landed
        // by the time the barrier's wait checks them; the second spreads them over all 64.
        auto substep = [&](const Frags& cur, Frags& nxt, int rsa, int rsb, int rks, bool first) {
#pragma unroll
            for (int m = 0; m < 64; ++m) {
                const int i = m >> 3, j = m & 7;
                acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(cur.w[i], cur.a[j], acc[i][j], 0, 0, 0);
                __builtin_amdgcn_sched_barrier(0);
                if (first) {
                    if (m % 3 == 0 && m < 48) read_one(rsa, rsb, rks, m / 3, nxt);
                } else {
                    if ((m & 3) == 0) read_one(rsa, rsb, rks, m >> 2, nxt);
                }
                if ((m & 7) == 2) {
                    if (first) load_a(m >> 3);
                    else load_b(m >> 3);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
        };
        for (int kt = 0; kt < nk; ++kt) {
            const int n_sa = c_sa >= NSLOT - 2 ? c_sa + 2 - NSLOT : c_sa + 2;
            const int n_sb = c_sb >= NSLOT - 2 ? c_sb + 2 - NSLOT : c_sb + 2;
            substep(F0, F1, c_sa, c_sb, 1, true);    // A tile of g+2
            if (l_local < n_local) __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(LOADS));
            else __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(0));
            barrier();
            substep(F1, F0, n_sa, n_sb, 0, false);   // B tile of g+2
            advance_cursor();                        // the cursor moves to step g+3
            c_sa = n_sa;
            c_sb = n_sb;
        }
        // The slot of the last step's B tile is free until the A tile of step g+3 (its next
        // user) is requested in the next step's first sub-step; wavefront w's staging area is
        // exactly the part of it that w's own loads refill.
        const int m0 = tile_m0(c_local), n0 = tile_n0(c_local);
        const int free_slot = c_sb >= 2 ? c_sb - 2 : c_sb + NSLOT - 2;
        epilogue<EPI>(acc, Cv, ldc, M, m0 + wm * 128, n0 + wn * 128, lane, qo,
                      smem + free_slot * SLOT_B + wave * LOADS * 1024);
        c_local += n_slots;
        if (c_local >= n_local) break;
    }
    __builtin_amdgcn_s_waitcnt(0);   // no load may still be writing LDS when the workgroup ends
}

}  // namespace

namespace ppk {

namespace {

constexpr size_t kLds = LDS_BYTES;

template <int EPI>
void launch(const void* A, int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc, int M, int N, int K,
            const int32_t* mtile_m0, int n_mtiles, const QkvOut& qo, hipStream_t s) {
    static bool attr = [] {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&gemm_bf16_kernel<EPI>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, kLds);
        return true;
    }();
    (void)attr;
    const int tiles_m = mtile_m0 ? n_mtiles : (M + BM - 1) / BM, tiles_n = N / BN;
    if (tiles_m <= 0) return;
    // one workgroup per CU (each needs the whole 160 KB LDS), a multiple of 8 so
    // that every XCD runs the same number; never more workgroups than tiles
    static const int n_cu = [] {
        int dev = 0, n = 0;
        (void)hipGetDevice(&dev);
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n < 8) n = 8;
        return n / 8 * 8;
    }();
    // per-XCD tile count of the M-block split and of the balanced one; the balanced split is
    // taken only when it saves a whole round of workgroups
    const int wg_per_xcd = n_cu / 8;
    const int blocked = ((tiles_m + 7) / 8) * tiles_n, even = (tiles_m * tiles_n + 7) / 8;
    const auto rounds = [&](int t) { return (t + wg_per_xcd - 1) / wg_per_xcd; };
    const int balanced = rounds(even) < rounds(blocked) ? 1 : 0;
    const int per_xcd = balanced ? even : blocked;
    const dim3 grid(8 * min(wg_per_xcd, per_xcd));
    gemm_bf16_kernel<EPI><<<grid, NT, kLds, s>>>(static_cast<const bf16*>(A), lda, static_cast<const bf16*>(B),
                                                ldb, C, ldc, M, K, mtile_m0, tiles_m, tiles_n, balanced, qo);
}

}  // namespace

void gemm_bf16(int epi, const void* A, int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc, int M,
               int N, int K, const int32_t* mtile_m0, int n_mtiles, hipStream_t s) {
    if (M <= 0) return;
    const QkvOut none{};
    switch (epi) {
        case kStore: launch<kStore>(A, lda, B, ldb, C, ldc, M, N, K, mtile_m0, n_mtiles, none, s); break;
        case kResidual: launch<kResidual>(A, lda, B, ldb, C, ldc, M, N, K, mtile_m0, n_mtiles, none, s); break;
        default: launch<kSwiGLU>(A, lda, B, ldb, C, ldc, M, N, K, mtile_m0, n_mtiles, none, s); break;
    }
}

void qkv_rope_bf16(const void* A, int64_t lda, const void* B, int64_t ldb, int M, int K, const int32_t* mtile_m0,
                   int n_mtiles, const QkvOut& out, hipStream_t s) {
    if (M <= 0) return;
    launch<kQkvRope>(A, lda, B, ldb, nullptr, 0, M, (out.H + 2 * out.Hkv) * 128, K, mtile_m0, n_mtiles, out, s);
}

}  // namespace ppk
