// The first generated token of every prompt (section 2.3: the time to first token covers
// prefilling the KV cache and generating the first token): the LM head applied to each
// prompt's last hidden row, and the greedy choice, argmax over the vocabulary with the lowest
// id on ties.
//
// Three launches.  (1) The last hidden row of every prompt (row prompt_kv_off[i+1] - 1 of the
// unpacked hidden state) is gathered into a [k_pad, d] matrix in the model's dtype, rows past
// k zero.  (2) One workgroup per 128 vocabulary rows computes their logits for all prompts and
// reduces them to one (max, lowest id) pair per prompt.  The LM head, vocab x d, dominates the
// traffic: it is read from HBM once per pass over the prompts (one pass for up to 128 prompts
// in bf16), so this kernel is HBM-bound on it (2 vocab d bytes), the prompt matrix being
// re-read from L2.  (3) One workgroup per prompt reduces the per-workgroup pairs; the order it
// uses is total, so the result is deterministic.
#include <math.h>

#include <mutex>
#include <vector>

#include "device.h"
#include "kernels.h"
#include "prepack.h"

namespace {

constexpr int VB = 1;    // vocabulary rows per workgroup of the float32 kernel

struct ArgMax {
    float v;
    int32_t i;
};

// a better than b: larger value, or equal value and lower id; NaN never wins
__device__ __forceinline__ bool better(float av, int ai, float bv, int bi) {
    return av > bv || (av == bv && ai < bi);
}

// Workgroup (i, j): prompt i's last hidden row, columns 2048 j .. + 2047, 8 per thread (two
// 16-byte loads); rows k .. k_pad - 1 are zero.  d is a multiple of 8.
template <typename T>
__global__ __launch_bounds__(256) void gather_last_kernel(const float* __restrict__ hidden, const int32_t* __restrict__ off,
                                                         int k, int k_pad, int d, T* __restrict__ out) {
    const int i = blockIdx.x, c = 8 * (blockIdx.y * 256 + threadIdx.x);
    if (i >= k_pad || c >= d) return;
    f32x4 a = {}, b = {};
    if (i < k) {
        const float* h = hidden + int64_t(off[i + 1] - 1) * d + c;
        a = *reinterpret_cast<const f32x4*>(h);
        b = *reinterpret_cast<const f32x4*>(h + 4);
    }
    T* o = out + int64_t(i) * d + c;
    if constexpr (sizeof(T) == 2) {
        bf16x8 v;
#pragma unroll
        for (int x = 0; x < 4; ++x) { v[x] = static_cast<bf16>(a[x]); v[4 + x] = static_cast<bf16>(b[x]); }
        *reinterpret_cast<bf16x8*>(o) = v;
    } else {
        *reinterpret_cast<f32x4*>(o) = a;
        *reinterpret_cast<f32x4*>(o + 4) = b;
    }
}

// Four wavefronts per workgroup of 128 vocabulary rows: wavefront w owns rows
// n0 = 128 b + 32 w .. + 31 (two blocks of 16 on the rows of the 16x16x32 bf16 MFMA) and all
// prompts, 16 MB at a time (MB blocks of 16 on its columns).  K is consumed in chunks of KC
// columns.  A chunk's weight tile (128 rows x 2 KC bytes) and prompt tile (16 MB rows x 2 KC
// bytes) go from global memory straight into LDS, each 1 KB load a set of whole row segments,
// through a ring of NCH chunks: NCH - 1 chunks are in flight while one is consumed.  The LM
// head streams through once per pass of 16 MB prompts; the prompt rows come from L2.  Rows
// past the vocabulary or the prompts are read as the last row (every load in range) and never
// reported.  In block (nb, mb) lane l holds the logits of prompt 16 mb + l % 16 for vocabulary
// rows n0 + 16 nb + 4 (l / 16) + 0..3.
constexpr int LM_ROWS = 128;            // vocabulary rows per workgroup
// Buffer descriptor word 3 for raw (unstructured) 32-bit-offset loads on gfx9-family parts.
constexpr int kRsrcWord3 = 0x00020000;
// s_waitcnt immediate: vmcnt(n) and lgkmcnt(0), expcnt not waited for (gfx9 encoding).
constexpr int wait_vm_lgkm0(int n) { return ((n >> 4) << 14) | (n & 15) | 0x0070; }

typedef __attribute__((address_space(3))) void lds_void;

// LDS swizzles: logical 16-byte chunk c of tile row r sits at c ^ f(r).  A fragment read takes
// chunk 4 s + l / 16 of rows l % 16, and the LDS serves lanes i and i + 32 together: 8 rows x
// chunks {c, c ^ 2}.
// 128-byte rows (KC = 64; a row covers half the banks): f's bits are r's bits 1, 3 and 2, so the
// 16 (r % 2, physical chunk) pairs are distinct.
// 256-byte rows (KC = 128; a row covers all 64 banks): f's bits 0, 2, 3 are r's bits 0, 1, 2, so
// the 8 rows fall in distinct classes {x, x ^ 2} and the 16 physical chunks are distinct.
template <int KC>
__device__ __forceinline__ int lm_swz(int r) {
    if constexpr (KC == 64) return ((r >> 1) & 1) | (((r >> 3) & 1) << 1) | (r & 4);
    else return (r & 1) | (((r >> 1) & 1) << 2) | (((r >> 2) & 1) << 3);
}

template <int MB, int KC, int NCH>
struct LmGeom {
    static constexpr int ROW_B = 2 * KC;                // bytes of a tile row
    static constexpr int CPR = ROW_B / 16;              // 16-byte chunks per row
    static constexpr int RPL = 1024 / ROW_B;            // rows per 1 KB load
    static constexpr int W_B = LM_ROWS * ROW_B;         // weight tile of a chunk
    static constexpr int P_B = 16 * MB * ROW_B;         // prompt tile of a chunk
    static constexpr int CH_B = W_B + P_B;
    static constexpr int W_LD = W_B / 1024 / 4;         // 1 KB loads per wavefront per chunk
    static constexpr int P_LD = P_B / 1024 / 4;
    static constexpr int LDS = NCH * CH_B;
    static_assert(KC == 64 || KC == 128, "tile rows of 128 or 256 bytes");
    static_assert(P_LD >= 1 && LDS + 4 * 16 * MB * 8 <= 160 * 1024, "LDS of one workgroup");
    static_assert((NCH - 2) * (W_LD + P_LD) <= 63, "vmcnt range");
};

// The loads of wavefront `wave` for K columns of chunk c (clamped: always in range) into ring
// slot c % NCH.
template <class G, int NCH>
__device__ __forceinline__ void lm_issue(__amdgpu_buffer_rsrc_t wrs, __amdgpu_buffer_rsrc_t hrs, char* smem, int c,
                                         int n_ch, int wave, const int* woff, const int* poff) {
    const int col_b = min(c, n_ch - 1) * G::ROW_B;
    char* slot = smem + (c % NCH) * G::CH_B;
#pragma unroll
    for (int t = 0; t < G::W_LD; ++t)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(wrs, (lds_void*)(slot + (G::W_LD * wave + t) * 1024), 16, woff[t],
                                                 col_b, 0, 0);
#pragma unroll
    for (int t = 0; t < G::P_LD; ++t)
        __builtin_amdgcn_raw_ptr_buffer_load_lds(hrs, (lds_void*)(slot + G::W_B + (G::P_LD * wave + t) * 1024), 16,
                                                 poff[t], col_b, 0, 0);
}

template <int MB, int KC, int NCH, int WR>
__global__ __launch_bounds__(256, 1) void lm_head_bf16_kernel(const bf16* __restrict__ hl, int k, int k_pad,
                                                              const bf16* __restrict__ W, int V, int d,
                                                              float* __restrict__ logits,
                                                              ArgMax* __restrict__ part) {
    using G = LmGeom<MB, KC, NCH>;
    constexpr int NB = LM_ROWS / WR / 16;   // row blocks of a wavefront
    constexpr int MW = MB * WR / 4;         // prompt blocks of a wavefront
    static_assert(NB * MW * 4 == 8 * MB, "the 4 wavefronts tile 128 rows x 16 MB prompts");
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ ArgMax red[WR][16 * MB];
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int wr = wave % WR, wp = wave / WR;
    const int nb0 = blockIdx.x * LM_ROWS;
    const int n0 = nb0 + wr * 16 * NB;
    const int lr = lane & 15, q4 = lane >> 4, lrow = lane / G::CPR, lchk = lane % G::CPR;
    const int n_ch = d / KC;
    const int last_row = min(V - 1 - nb0, LM_ROWS - 1);   // rows past it (vocabulary end) read it again
    const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16*>(W + int64_t(nb0) * d), 0, (last_row + 1) * d * 2, kRsrcWord3);
    // load t of wavefront w fills rows RPL (W_LD w + t) + l / CPR of the weight tile (rows
    // RPL (P_LD w + t) + l / CPR of the prompt tile); lane l lands at physical chunk l % CPR and
    // fetches the logical chunk that the swizzle puts there
    int woff[G::W_LD];
#pragma unroll
    for (int t = 0; t < G::W_LD; ++t) {
        const int row = G::RPL * (G::W_LD * wave + t) + lrow;
        woff[t] = min(row, last_row) * d * 2 + 16 * (lchk ^ lm_swz<KC>(row));
    }
    const int f_sw = lm_swz<KC>(lr);
    for (int m0 = 0; m0 < k_pad; m0 += 16 * MB) {
        const int nmb = min(MB, (k_pad - m0) / 16);
        const __amdgpu_buffer_rsrc_t hrs = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<bf16*>(hl + int64_t(m0) * d), 0, 16 * nmb * d * 2, kRsrcWord3);
        int poff[G::P_LD];
#pragma unroll
        for (int t = 0; t < G::P_LD; ++t) {
            const int row = G::RPL * (G::P_LD * wave + t) + lrow;
            poff[t] = min(row, 16 * nmb - 1) * d * 2 + 16 * (lchk ^ lm_swz<KC>(row));
        }
        f32x4 acc[NB][MW] = {};
#pragma unroll
        for (int c = 0; c < NCH - 1; ++c) lm_issue<G, NCH>(wrs, hrs, smem, c, n_ch, wave, woff, poff);
        // At the top of chunk c the loads issued after its own are those of chunks c + 1 ..
        // c + NCH - 2: (NCH - 2) chunks of W_LD + P_LD loads per wavefront.
        for (int c = 0; c < n_ch; ++c) {
            __builtin_amdgcn_sched_barrier(0);
            __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0((NCH - 2) * (G::W_LD + G::P_LD)));
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
            // into the slot every wavefront finished at c - 1
            lm_issue<G, NCH>(wrs, hrs, smem, c + NCH - 1, n_ch, wave, woff, poff);
            const char* slot = smem + (c % NCH) * G::CH_B;
#pragma unroll
            for (int st = 0; st < KC / 32; ++st) {
                const int ch = 16 * ((4 * st + q4) ^ f_sw);
                bf16x8 wf[NB], pf[MW];
#pragma unroll
                for (int nb = 0; nb < NB; ++nb)
                    wf[nb] = *reinterpret_cast<const bf16x8*>(slot + (n0 - nb0 + 16 * nb + lr) * G::ROW_B + ch);
#pragma unroll
                for (int mb = 0; mb < MW; ++mb)
                    if (MW * wp + mb < nmb)
                        pf[mb] = *reinterpret_cast<const bf16x8*>(slot + G::W_B + (16 * (MW * wp + mb) + lr) * G::ROW_B + ch);
#pragma unroll
                for (int mb = 0; mb < MW; ++mb) {
                    if (MW * wp + mb >= nmb) break;
#pragma unroll
                    for (int nb = 0; nb < NB; ++nb)
                        acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf[nb], pf[mb], acc[nb][mb], 0, 0, 0);
                }
            }
        }
        // the loads past the last chunk are dead (clamped, never read); none may still be writing
        // LDS when the ring is refilled or the workgroup ends
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(0));
        // logits and each lane's best of its 4 NB vocabulary rows, per prompt block
#pragma unroll
        for (int mb = 0; mb < MW; ++mb) {
            const int gb = MW * wp + mb;
            if (gb >= nmb) break;
            const int m = m0 + 16 * gb + lr;
            float bv = -INFINITY;
            int bi = INT32_MAX;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) {
                const int nbase = n0 + 16 * nb + 4 * q4;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    if (nbase + r >= V) continue;
                    const float v = acc[nb][mb][r];
                    if (logits && m < k) logits[int64_t(m) * V + nbase + r] = v;
                    if (better(v, nbase + r, bv, bi)) { bv = v; bi = nbase + r; }
                }
            }
            // lanes l, l ^ 16, l ^ 32, l ^ 48 hold the same prompt
#pragma unroll
            for (int x = 16; x < 64; x <<= 1) {
                const float ov = __shfl_xor(bv, x);
                const int oi = __shfl_xor(bi, x);
                if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
            }
            if (lane < 16) red[wr][16 * gb + lane] = ArgMax{bv, bi};
        }
        __syncthreads();
        // the WR row groups combined for the 16 MB prompts; prompt m's pairs are contiguous
        if (threadIdx.x < 16 * nmb && m0 + threadIdx.x < k) {
            ArgMax b = red[0][threadIdx.x];
#pragma unroll
            for (int w2 = 1; w2 < WR; ++w2) {
                const ArgMax o = red[w2][threadIdx.x];
                if (better(o.v, o.i, b.v, b.i)) b = o;
            }
            part[int64_t(m0 + threadIdx.x) * gridDim.x + blockIdx.x] = b;
        }
        __syncthreads();
    }
}

// Up to 64 prompts, d a multiple of 512: the same workgroup tile (128 vocabulary rows x 64
// prompts) with the LM head streamed as long row segments.  Chunk (s, rb) of a workgroup is
// 16 vocabulary rows x 512 K columns, one whole 1 KB segment of each row per load; chunks go
// segment-major (s = 0, 1, ..; rb = 0..7 within a segment) through an LDS ring of NW chunks.
// Cache-cold, HBM streams these 1 KB segments markedly faster than 128-byte ones spread over
// 128 rows.  The wavefronts split K instead of rows: wavefront w takes columns 128 w .. + 127 of
// every chunk (4 MFMA K-steps) and accumulates all 8 row blocks x 4 prompt blocks over its
// quarter of K.  The prompt tile of segment s (64 rows x 1 KB) sits in LDS; at the segment's
// first chunk each wavefront moves its quarter into registers (16 fragments), after which the
// tile of segment s + 1 is loaded in its place, a quarter with each of the segment's first 4
// chunks.  At the end the 4 partial sums of each logit are added through LDS in wavefront
// order.
constexpr int SEG_COLS = 512;                 // K columns of a chunk
constexpr int SEG_W_B = 16 * SEG_COLS * 2;    // 16 KB of weights per chunk
constexpr int SEG_P_B = 64 * SEG_COLS * 2;    // 64 KB prompt tile of a segment

// s_waitcnt count at chunk rb of a segment: the loads a wavefront issued after the one of the
// awaited chunk.  Each chunk step issues the chunk NW - 1 ahead (4 loads) and then, at rb < 4, a
// quarter of the next prompt tile (4 loads); chunk rb was issued NW - 1 steps earlier.  Steps
// before the first chunk are the prologue (weights only, the first prompt tile before them),
// which is what rb < 0 reads as (rb 4..7 carry no prompt loads) while NW <= 5.
constexpr int seg_p_loads(int rb) { return ((rb % 8 + 8) % 8) < 4 ? 4 : 0; }
constexpr int seg_wait(int rb, int NW) {
    int n = seg_p_loads(rb - NW + 1);
    for (int j = rb - NW + 2; j <= rb - 1; ++j) n += 4 + seg_p_loads(j);
    return n;
}

static_assert(seg_wait(0, 4) == 8 && seg_wait(1, 4) == 12 && seg_wait(3, 4) == 20 && seg_wait(4, 4) == 20 &&
                  seg_wait(7, 4) == 8 && seg_wait(0, 5) == 12 && seg_wait(4, 5) == 28 && seg_wait(7, 5) == 16,
              "wait counts worked out by hand for rings of 4 and 5 chunks");

// s_waitcnt needs an immediate: rb is a constant of the unrolled chunk loop, so the switch folds.
template <int NW>
__device__ __forceinline__ void seg_waitcnt(int rb) {
    switch (rb) {
        case 0: __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(seg_wait(0, NW))); break;
        case 1: __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(seg_wait(1, NW))); break;
        case 2: __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(seg_wait(2, NW))); break;
        case 3: __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(seg_wait(3, NW))); break;
        case 4: __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(seg_wait(4, NW))); break;
        case 5: __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(seg_wait(5, NW))); break;
        case 6: __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(seg_wait(6, NW))); break;
        default: __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(seg_wait(7, NW))); break;
    }
}

template <int NW>
__global__ __launch_bounds__(256, 1) void lm_head_seg_kernel(const bf16* __restrict__ hl, int k, int k_pad,
                                                             const bf16* __restrict__ W, int V, int d,
                                                             float* __restrict__ logits, ArgMax* __restrict__ part) {
    static_assert(NW >= 2 && NW <= 5, "the prologue reading of seg_wait");
    static_assert(NW * SEG_W_B + SEG_P_B <= 144 * 1024 && 4 * 8 * 4 * 64 * 16 <= NW * SEG_W_B + SEG_P_B, "LDS");
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ ArgMax red[4][64];
    char* const pbuf = smem + NW * SEG_W_B;
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int nb0 = blockIdx.x * LM_ROWS;
    const int lr = lane & 15, q4 = lane >> 4;
    const int n_seg = d / SEG_COLS;
    // workgroups on one XCD (blockIdx.x, + 8, + 16, ...) start their sweep over the K segments
    // at different segments, so that they do not all read the same 1 KB column of their rows
    // at the same moment (from HBM: 59.4 -> 56.5 us for 64 prompts at vocabulary 32000)
    const int rot = (blockIdx.x >> 3) % n_seg;
    const int rows_p = k_pad;                                  // prompt rows present (<= 64)
    const int last_row = min(V - 1 - nb0, LM_ROWS - 1);
    const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16*>(W + int64_t(nb0) * d), 0, (last_row + 1) * d * 2, kRsrcWord3);
    const __amdgpu_buffer_rsrc_t hrs = __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(hl), 0, rows_p * d * 2,
                                                                         kRsrcWord3);
    // 1 KB row segments land with lane l at physical 16-byte chunk l and take the logical chunk
    // l ^ f(r) (lm_swz<128>: within each 256-byte bank window, so fragment reads of 8 rows x
    // chunks {c, c ^ 2} hit 16 distinct bank groups)
    auto w_issue = [&](int g) {       // chunk g (clamped: dead chunks re-read the last) -> slot g % NW
        const int gc = min(g, 8 * n_seg - 1), rb = gc & 7;
        int sg = (gc >> 3) + rot;
        if (sg >= n_seg) sg -= n_seg;
        char* slot = smem + (g % NW) * SEG_W_B;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int r = 4 * wave + t;
            const int soff = min(16 * rb + r, last_row) * d * 2 + sg * SEG_COLS * 2;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(wrs, (lds_void*)(slot + r * 1024), 16,
                                                     16 * (lane ^ lm_swz<128>(r)), soff, 0, 0);
        }
    };
    auto p_issue = [&](int sg, int i) {   // quarter i of the prompt tile of segment sg (clamped)
        int sc = min(sg, n_seg - 1) + rot;
        if (sc >= n_seg) sc -= n_seg;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int r = 16 * wave + 4 * i + t;
            const int soff = min(r, rows_p - 1) * d * 2 + sc * SEG_COLS * 2;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(hrs, (lds_void*)(pbuf + r * 1024), 16,
                                                     16 * (lane ^ lm_swz<128>(r)), soff, 0, 0);
        }
    };
    f32x4 acc[8][4] = {};
    bf16x8 pf[4][4];
#pragma unroll
    for (int i = 0; i < 4; ++i) p_issue(0, i);
#pragma unroll
    for (int g = 0; g < NW - 1; ++g) w_issue(g);
    for (int sg = 0; sg < n_seg; ++sg) {
#pragma unroll
        for (int rb = 0; rb < 8; ++rb) {
            const int g = 8 * sg + rb;
            __builtin_amdgcn_sched_barrier(0);
            seg_waitcnt<NW>(rb);
            __builtin_amdgcn_s_barrier();
            __builtin_amdgcn_sched_barrier(0);
            if (rb == 0) {
                // this wavefront's quarter of the segment's prompt tile into registers; then the
                // buffer is free for the next segment's tile
#pragma unroll
                for (int st = 0; st < 4; ++st)
#pragma unroll
                    for (int mb = 0; mb < 4; ++mb) {
                        const int r = 16 * mb + lr;
                        pf[st][mb] = *reinterpret_cast<const bf16x8*>(
                            pbuf + r * 1024 + 16 * ((16 * wave + 4 * st + q4) ^ lm_swz<128>(r)));
                    }
                __builtin_amdgcn_sched_barrier(0);
                __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(63));
                __builtin_amdgcn_s_barrier();
                __builtin_amdgcn_sched_barrier(0);
            }
            w_issue(g + NW - 1);
            if (rb < 4) p_issue(sg + 1, rb);
            const char* slot = smem + (g % NW) * SEG_W_B;
#pragma unroll
            for (int st = 0; st < 4; ++st) {
                const bf16x8 wf = *reinterpret_cast<const bf16x8*>(
                    slot + lr * 1024 + 16 * ((16 * wave + 4 * st + q4) ^ lm_swz<128>(lr)));
#pragma unroll
                for (int mb = 0; mb < 4; ++mb)
                    acc[rb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf, pf[st][mb], acc[rb][mb], 0, 0, 0);
            }
        }
    }
    // every load (the dead ones past the last chunk included) has landed before LDS is reused
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(0));
    __syncthreads();
    f32x4* part_sum = reinterpret_cast<f32x4*>(smem);      // [wave][rb][mb][lane]
#pragma unroll
    for (int rb = 0; rb < 8; ++rb)
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) part_sum[((wave * 8 + rb) * 4 + mb) * 64 + lane] = acc[rb][mb];
    __syncthreads();
    // wavefront w finishes row blocks 2 w and 2 w + 1: rows nb0 + 32 w + 16 nb + 4 (l / 16) + 0..3
    const int n0 = nb0 + 32 * wave;
    const int nmb = k_pad / 16;
#pragma unroll
    for (int mb = 0; mb < 4; ++mb) {
        if (mb >= nmb) break;
        const int m = 16 * mb + lr;
        float bv = -INFINITY;
        int bi = INT32_MAX;
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) {
            const int rb = 2 * wave + nb;
            f32x4 v = part_sum[((0 * 8 + rb) * 4 + mb) * 64 + lane];
#pragma unroll
            for (int w2 = 1; w2 < 4; ++w2) v += part_sum[((w2 * 8 + rb) * 4 + mb) * 64 + lane];
            const int nbase = n0 + 16 * nb + 4 * q4;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                if (nbase + r >= V) continue;
                if (logits && m < k) logits[int64_t(m) * V + nbase + r] = v[r];
                if (better(v[r], nbase + r, bv, bi)) { bv = v[r]; bi = nbase + r; }
            }
        }
#pragma unroll
        for (int x = 16; x < 64; x <<= 1) {
            const float ov = __shfl_xor(bv, x);
            const int oi = __shfl_xor(bi, x);
            if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
        }
        if (lane < 16) red[wave][16 * mb + lane] = ArgMax{bv, bi};
    }
    __syncthreads();
    if (threadIdx.x < k_pad && threadIdx.x < k) {
        ArgMax b = red[0][threadIdx.x];
#pragma unroll
        for (int w2 = 1; w2 < 4; ++w2) {
            const ArgMax o = red[w2][threadIdx.x];
            if (better(o.v, o.i, b.v, b.i)) b = o;
        }
        part[int64_t(threadIdx.x) * gridDim.x + blockIdx.x] = b;
    }
}

// float32 model: one wavefront per vocabulary row (its lanes split d, the row read once,
// coalesced), every prompt's logit reduced across the wavefront in a fixed order.
__global__ __launch_bounds__(64) void lm_head_f32_kernel(const float* __restrict__ hl, int k, const float* __restrict__ W,
                                                         int V, int d, float* __restrict__ logits,
                                                         ArgMax* __restrict__ part) {
    const int n = blockIdx.x, lane = threadIdx.x;
    const float* w = W + int64_t(n) * d;
    for (int m = 0; m < k; ++m) {
        const float* h = hl + int64_t(m) * d;
        float s = 0.f;
        for (int c = lane; c < d; c += 64) s = fmaf(h[c], w[c], s);
        s = wave_sum(s);
        if (lane == 0) {
            if (logits) logits[int64_t(m) * V + n] = s;
            part[int64_t(m) * V + n] = ArgMax{s, n};   // a NaN logit never wins the final reduction
        }
    }
}

// One workgroup per prompt: thread t takes the per-workgroup pairs t, t + 256, ..., then the
// pairs are combined across the wavefront and across the 4 wavefronts.  "Larger value, then
// lower id" is a total order on the pairs (NaN never enters one), so the result does not
// depend on the order of combination.
__global__ __launch_bounds__(256) void argmax_finalize_kernel(const ArgMax* __restrict__ part, int n_blocks, int k,
                                                              int32_t* __restrict__ tokens) {
    __shared__ ArgMax red[4];
    const int m = blockIdx.x;
    ArgMax b{-INFINITY, INT32_MAX};
    for (int j = threadIdx.x; j < n_blocks; j += blockDim.x) {
        const ArgMax o = part[int64_t(m) * n_blocks + j];
        if (better(o.v, o.i, b.v, b.i)) b = o;
    }
#pragma unroll
    for (int x = 1; x < 64; x <<= 1) {
        const float ov = __shfl_xor(b.v, x);
        const int oi = __shfl_xor(b.i, x);
        if (better(ov, oi, b.v, b.i)) b = ArgMax{ov, oi};
    }
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = b;
    __syncthreads();
    if (threadIdx.x == 0) {
#pragma unroll
        for (int w = 1; w < 4; ++w)
            if (better(red[w].v, red[w].i, b.v, b.i)) b = red[w];
        tokens[m] = b.i == INT32_MAX ? -1 : b.i;   // -1: every logit was NaN
    }
}

template <int MB, int KC, int NCH, int WR>
void lm_head_launch(const bf16* hl, int k, int k_pad, const bf16* W, int V, int d, float* logits, ArgMax* part,
                    int n_blocks, hipStream_t s) {
    constexpr int lds = LmGeom<MB, KC, NCH>::LDS;
    static bool attr = [] {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&lm_head_bf16_kernel<MB, KC, NCH, WR>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, lds);
        return true;
    }();
    (void)attr;
    lm_head_bf16_kernel<MB, KC, NCH, WR><<<n_blocks, 256, lds, s>>>(hl, k, k_pad, W, V, d, logits, part);
}

template <int NW>
void lm_head_seg_launch(const bf16* hl, int k, int k_pad, const bf16* W, int V, int d, float* logits, ArgMax* part,
                        int n_blocks, hipStream_t s) {
    constexpr int lds = NW * SEG_W_B + SEG_P_B;
    static bool attr = [] {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&lm_head_seg_kernel<NW>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, lds);
        return true;
    }();
    (void)attr;
    lm_head_seg_kernel<NW><<<n_blocks, 256, lds, s>>>(hl, k, k_pad, W, V, d, logits, part);
}

}  // namespace

// Workspace of pp_first_token_noalloc: a file-scope array of this code object, one copy per
// GPU, alive until the process ends.  In host code its name is only a stand-in for the device
// symbol: host code passes kernels the device address that hipGetSymbolAddress returns for
// the current GPU (first_token_scratch), never the array itself.
static __device__ __align__(256) char scratch[PP_FIRST_TOKEN_SCRATCH_BYTES];

namespace ppk {

hipError_t first_token_scratch(void** ptr) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return e;
    static std::mutex mu;
    static std::vector<void*> by_device;     // device id -> address of its copy of `scratch`
    std::lock_guard<std::mutex> lock(mu);
    if (dev >= static_cast<int>(by_device.size())) by_device.resize(dev + 1, nullptr);
    if (!by_device[dev]) {
        void* p = nullptr;
        e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess) return e;
        by_device[dev] = p;
    }
    *ptr = by_device[dev];
    return hipSuccess;
}

size_t first_token_workspace(int dtype, int k, int V, int d) {
    const int k_pad = (k + 15) / 16 * 16;
    const size_t e = dtype == PP_BF16 ? 2 : 4;
    const size_t a = (size_t(k_pad) * d * e + 255) / 256 * 256;
    const size_t rows = dtype == PP_BF16 ? LM_ROWS : VB;
    const size_t n_blocks = (size_t(V) + rows - 1) / rows;
    return a + n_blocks * size_t(k) * sizeof(ArgMax);
}

void first_token(int dtype, const float* hidden, const int32_t* prompt_kv_off, int k, const void* lm_head, int V,
                 int d, void* workspace, float* logits, int32_t* tokens, hipStream_t s) {
    const int k_pad = (k + 15) / 16 * 16;
    const size_t e = dtype == PP_BF16 ? 2 : 4;
    char* ws = static_cast<char*>(workspace);
    ArgMax* part = reinterpret_cast<ArgMax*>(ws + (size_t(k_pad) * d * e + 255) / 256 * 256);
    const int n_blocks = (V + (dtype == PP_BF16 ? LM_ROWS : VB) - 1) / (dtype == PP_BF16 ? LM_ROWS : VB);
    const dim3 g_grid(k_pad, (d + 2047) / 2048);
    if (dtype == PP_BF16) {
        bf16* hl = reinterpret_cast<bf16*>(ws);
        gather_last_kernel<bf16><<<g_grid, 256, 0, s>>>(hidden, prompt_kv_off, k, k_pad, d, hl);
        if (k_pad <= 64 && d % SEG_COLS == 0)
            lm_head_seg_launch<4>(hl, k, k_pad, static_cast<const bf16*>(lm_head), V, d, logits, part, n_blocks, s);
        else if (k_pad <= 64)
            lm_head_launch<4, 64, 4, 2>(hl, k, k_pad, static_cast<const bf16*>(lm_head), V, d, logits, part, n_blocks, s);
        else
            lm_head_launch<8, 64, 4, 2>(hl, k, k_pad, static_cast<const bf16*>(lm_head), V, d, logits, part, n_blocks, s);
    } else {
        float* hl = reinterpret_cast<float*>(ws);
        gather_last_kernel<float><<<g_grid, 256, 0, s>>>(hidden, prompt_kv_off, k, k_pad, d, hl);
        lm_head_f32_kernel<<<n_blocks, 64, 0, s>>>(hl, k, static_cast<const float*>(lm_head), V, d, logits, part);
    }
    argmax_finalize_kernel<<<k, 256, 0, s>>>(part, n_blocks, k, tokens);
}

}  // namespace ppk
