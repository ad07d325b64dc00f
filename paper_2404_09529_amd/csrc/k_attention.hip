// Attention under the independent mask (section 3.2): every query attends causally to
// the keys of its own prompt only.  M' is never materialised; the segment table gives
// each query tile its key range directly.
//
// bf16 kernel (head dim 128), one 256-thread workgroup per (query tile, head):
//   * a work-list entry is (segment, q0): queries [q0, q0+128) of one segment, so only keys
//     [0, min(q0+128, len)) of the same segment are ever used -- every tile outside the
//     prompt's diagonal block of M' is skipped by construction;
//   * key tiles of 64 start at the segment's first key, so only the diagonal tile and the
//     span's tail need a predicate, and the arithmetic of a query is the same wherever its
//     prompt sits (packed and padded layouts give identical results);
//   * wavefront w owns queries q0 + 32w .. q0 + 32w + 31; its Q fragments stay in
//     registers for the whole key loop;
//   * keys and values are read from the per-prompt caches that the QKV projection has just
//     written (UNPACK happens before attention, so the packed layout never holds K or V):
//     a segment's keys are contiguous cache rows.  K and V tiles go from there straight into
//     LDS (16-byte direct-to-LDS loads, double-buffered), both row-major [key][d] with
//     XOR-swizzled 16-byte chunks; the swizzle is applied on the global side of each load;
//   * S^T = K Q^T and O^T += V^T P^T run on the 32x32x16 bf16 MFMA; a lane holds one query,
//     so the running max / sum of the online softmax (Milakov and Gimelshein 2018; the
//     tiling of FlashAttention, Dao et al. 2022) are lane-local plus one exchange with the
//     lane 32 away;
//   * software pipeline with K one tile ahead of V: while the matrix cores compute the
//     scores of key tile t + 1, the vector units turn the scores of tile t into bf16
//     probabilities (exp2, row sums with dot2 on the rounded values), then P V of tile t
//     follows; the exchange of row maxima and sums with the lane 32 away is a permlane32
//     swap, so the softmax never waits on LDS;
//   * the V operand of O^T += V^T P^T is read with the transposing LDS read
//     (ds_read_b64_tr_b16), with key rows chosen so that its key order matches the order in
//     which the S^T accumulators hold the probabilities: P feeds the MFMA from registers
//     as is;
//   * the work list keeps each prompt's query tiles together, and the workgroups of one
//     work item (one per query head) are spread so that each XCD serves whole KV heads: the
//     tiles of a prompt that read the same keys and values run at the same time on the same
//     XCD and share its L2.
// float32 kernel: one wavefront per (query slot, head), a plain online-softmax loop over
// the query's keys, used for float32 models.
#include "device.h"
#include "kernels.h"
#include "prepack.h"

namespace {

constexpr int BQ = PP_QTILE;  // queries per workgroup
constexpr int BKV = 64;       // keys per tile
constexpr int HD = 128;       // head dim of the bf16 kernel
constexpr int NT = 256;
constexpr int ROW = HD * 2;                  // LDS bytes per key row (16 chunks of 16 bytes)
constexpr int TILE_B = BKV * ROW;            // one K or V tile: 16 KB
constexpr int STAGE_B = 2 * TILE_B;          // K tile then V tile; two stages = 64 KB
constexpr int LOADS = TILE_B / 1024 / 4;     // 1 KB loads per wavefront per tile (4)
// Buffer descriptor word 3 for raw (unstructured) 32-bit-offset loads on gfx9-family parts.
constexpr int kRsrcWord3 = 0x00020000;

typedef __attribute__((address_space(3))) void lds_void;
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) s16x4 lds_s16x4;

// K rows: chunk c of key row r stored at c ^ (r & 15): the MFMA fragment reads (32 rows x
// one chunk per half-wavefront) hit distinct banks.  V rows: chunk c stored at c ^ vswz(r),
// vswz = 0, 4, 10, 14 for r & 3 = 0..3: the transposing reads (4 consecutive rows x 32 or 64
// bytes per 16 or 32 lanes) hit distinct banks whether the LDS serves 8 or 16 lanes of a
// 16-byte access per cycle.
__device__ __forceinline__ int kswz(int r) { return r & 15; }
__device__ __forceinline__ int vswz(int r) { return (0xEA40 >> (4 * (r & 3))) & 15; }

template <typename V>
__device__ __forceinline__ bf16x8 as_bf16x8(V v) { return __builtin_bit_cast(bf16x8, v); }

__global__ __launch_bounds__(NT, 2) void attn_bf16_kernel(const bf16* __restrict__ q, int64_t ldq,
                                                          const bf16* __restrict__ kc, const bf16* __restrict__ vc,
                                                          int64_t ldkv, bf16* __restrict__ out, int64_t ldo,
                                                          const int32_t* __restrict__ seg_prompt,
                                                          const int32_t* __restrict__ seg_start,
                                                          const int32_t* __restrict__ seg_len,
                                                          const int32_t* __restrict__ prompt_kv_off,
                                                          const int32_t* __restrict__ qtile_seg,
                                                          const int32_t* __restrict__ qtile_q0, int H, int Hkv,
                                                          float scale_log2) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int w = blockIdx.x / H, j = blockIdx.x - (blockIdx.x / H) * H;
    // Workgroups are dealt to the 8 XCDs round-robin (XCD = workgroup id % 8), and work item w
    // takes ids w H .. w H + H - 1.  When the KV heads split evenly over the XCDs, the query
    // heads sharing a KV head are placed on one XCD (id % 8 = j % 8 picks the KV head's XCD),
    // so that its L2 serves their common keys and values; otherwise head j.
    int h = j;
    if (Hkv % 8 == 0) {
        const int G = H / Hkv, x = j & 7, a = j >> 3;
        h = (x + 8 * (a / G)) * G + a % G;
    }
    const int seg = qtile_seg[w], q0 = qtile_q0[w];
    const int a = seg_start[seg], n = seg_len[seg];
    const int prompt = seg_prompt[seg];
    const int kv0 = prompt_kv_off[prompt], plen = prompt_kv_off[prompt + 1] - kv0;
    const int g = h / (H / Hkv);
    const int n_kv = min(q0 + BQ, n);                 // keys [0, n_kv) of the segment
    const int nkt = (n_kv + BKV - 1) / BKV;

    const int fr = lane & 31, fh = lane >> 5;
    const int qi = q0 + wave * 32 + fr;               // this lane's query (offset in the segment)
    const bool q_ok = qi < n;
    const int wq_lo = q0 + wave * 32;

    bf16x8 qf[HD / 16];
    {
        const bf16* qrow = q + int64_t(a + (q_ok ? qi : 0)) * ldq + int64_t(h) * HD + fh * 8;
#pragma unroll
        for (int ks = 0; ks < HD / 16; ++ks)
            qf[ks] = q_ok ? as_bf16x8(*reinterpret_cast<const u32x4*>(qrow + ks * 16)) : bf16x8{};
    }

    // ---- direct-to-LDS loads from the caches.  Key tile kt covers cache rows kv0 + 64 kt ..
    // + 63; its descriptors start at that row and end at row kv0 + min(n_kv, plen), so rows
    // past the prompt (a padded span's tail) and past the keys in use read as zero.  All
    // offsets are in the per-lane part of the address, the part the range check covers.  Load
    // t of wavefront w fills key rows 4 j .. 4 j + 3 of a tile (j = 4 w + t), lane l landing at
    // physical chunk l % 16 of row 4 j + l / 16.
    const int kv_rows = min(n_kv, plen);
    const int row_b = static_cast<int>(ldkv) * 2;
    const int col = g * HD;
    int koff[LOADS], voff[LOADS];
#pragma unroll
    for (int t = 0; t < LOADS; ++t) {
        const int pr = 4 * (wave * LOADS + t) + lane / 16, pc = lane & 15;
        koff[t] = pr * row_b + (col + 8 * (pc ^ kswz(pr))) * 2;
        voff[t] = pr * row_b + (col + 8 * (pc ^ vswz(pr))) * 2;
    }
    // K tile kt goes to the first half of stage kt & 1, V tile kt to its second half.
    auto tile_rsrc = [&](const bf16* base, int kt) {
        const int64_t first = int64_t(kv0) + kt * BKV;
        const int records = max(kv_rows - kt * BKV, 0) * row_b;
        return __builtin_amdgcn_make_buffer_rsrc(const_cast<bf16*>(base + first * ldkv), 0, records, kRsrcWord3);
    };
    auto issue_k = [&](int kt) {
        char* dst = smem + (kt & 1) * STAGE_B;
        const __amdgpu_buffer_rsrc_t r = tile_rsrc(kc, kt);
#pragma unroll
        for (int t = 0; t < LOADS; ++t)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(dst + (wave * LOADS + t) * 1024), 16, koff[t], 0, 0, 0);
    };
    auto issue_v = [&](int kt) {
        char* dst = smem + (kt & 1) * STAGE_B + TILE_B;
        const __amdgpu_buffer_rsrc_t r = tile_rsrc(vc, kt);
#pragma unroll
        for (int t = 0; t < LOADS; ++t)
            __builtin_amdgcn_raw_ptr_buffer_load_lds(r, (lds_void*)(dst + (wave * LOADS + t) * 1024), 16, voff[t], 0, 0, 0);
    };

    // ---- fragment addresses.  K: row b*32 + fr, chunk (2 ks + fh) ^ (fr & 15).  V (transposing
    // read r of sub-step `sub`, d block db): this lane supplies the address of key row
    // sub*16 + 8 r + 4 (grp / 2) + lane16 / 4 and d columns db*32 + 16 (grp % 2) + 4 (lane16 % 4)
    // .. +3, where grp = lane / 16; the lane then receives 4 consecutive keys of one d.
    const int k_lds = fr * ROW;
    const int kx = fh ^ (fr & 15);                    // chunk (2 ks + fh) ^ (fr & 15) = 2 ks ^ kx
    const int l16 = lane & 15, grp16 = lane >> 4;
    const int vrow = 4 * (grp16 >> 1) + (l16 >> 2);   // + sub*16 + 8 r; vrow & 3 = l16 >> 2
    const int vd = 16 * (grp16 & 1) + 4 * (l16 & 3);   // + db*32
    const int vs = vswz(vrow);

    f32x16 o[HD / 32];
#pragma unroll
    for (int db = 0; db < HD / 32; ++db) o[db] = f32x16{};
    float m_i = -1e30f, l_i = 0.f;
    const float lazy = 8.0f / scale_log2;             // 8 in log2 units, as a raw-score margin

    // S^T of key tile kt: s[b][r] is the raw score of key 64 kt + 32 b + 8 (r / 4) + 4 fh + r % 4
    // for this lane's query.  Every wavefront takes part in every key tile: one whose queries
    // all precede the tile sees only masked scores (p = 0, corr = 1) and leaves o and l as
    // they were.
    auto scores = [&](int kt, f32x16 (&s)[2]) {
        const char* kst = smem + (kt & 1) * STAGE_B;
#pragma unroll
        for (int ks = 0; ks < HD / 16; ++ks)
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const bf16x8 kf = *reinterpret_cast<const bf16x8*>(kst + k_lds + b * 32 * ROW + 16 * ((2 * ks) ^ kx));
                s[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], ks == 0 ? f32x16{} : s[b], 0, 0, 0);
            }
    };
    // The mask (only the diagonal tile and the span's tail need it) and the online-softmax
    // reference.  m_i is a per-lane reference maximum, kept unscaled; the scale 1/sqrt(D) (in
    // log2 units) is folded into one FMA per score before the hardware exp2, and masked
    // scores (-inf) give exactly 0.  The reference moves only when a score exceeds it by more
    // than 8 in log2 units, so probabilities stay <= 2^8 and the output accumulators are
    // rescaled only on those rare steps.  The exchange with the lane 32 away (the other half
    // of the same query's keys) is a permlane32 swap: no LDS round trip.
    auto reference = [&](int kt, f32x16 (&s)[2]) {
        const int kb = kt * BKV;
        if (kb + BKV - 1 > wq_lo || kb + BKV > n_kv) {
            // key kb + 4 fh + off is allowed iff off <= lim (key <= qi and key < n_kv)
            const int lim = min(qi, n_kv - 1) - (kb + 4 * fh);
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r)
                    if (32 * b + 8 * (r >> 2) + (r & 3) > lim) s[b][r] = -INFINITY;
        }
        float mx = -INFINITY;
#pragma unroll
        for (int b = 0; b < 2; ++b)
#pragma unroll
            for (int r = 0; r < 16; ++r) mx = fmaxf(mx, s[b][r]);
        const auto mw = __builtin_amdgcn_permlane32_swap(__float_as_uint(mx), __float_as_uint(mx), false, false);
        mx = fmaxf(__uint_as_float(mw[0]), __uint_as_float(mw[1]));
        if (__any(mx > m_i + lazy)) {
            const float m_new = fmaxf(m_i, mx);
            const float corr = __builtin_amdgcn_exp2f((m_i - m_new) * scale_log2);
            l_i *= corr;
#pragma unroll
            for (int db = 0; db < HD / 32; ++db) o[db] *= corr;
            m_i = m_new;
        }
    };
    // P = exp2(scale s - scale m) rounded to bf16, in the order the PV MFMA takes it from
    // registers (sub-step sub = keys 16 sub .. 16 sub + 15); l gains the sum of the rounded
    // probabilities (two per dot2), so the normaliser matches the weights actually applied.
    auto probs = [&](f32x16 (&s)[2], bf16x8 (&pf)[BKV / 16]) {
        const float nm = -m_i * scale_log2;
#pragma unroll
        for (int sub = 0; sub < BKV / 16; ++sub)
#pragma unroll
            for (int e = 0; e < 8; ++e)
                pf[sub][e] = static_cast<bf16>(__builtin_amdgcn_exp2f(fmaf(s[sub >> 1][(sub & 1) * 8 + e], scale_log2, nm)));
        typedef __bf16 bf16x2_t __attribute__((ext_vector_type(2)));
        const bf16x2_t one2 = {static_cast<bf16>(1.0f), static_cast<bf16>(1.0f)};
        float rs0 = 0.f, rs1 = 0.f;
#pragma unroll
        for (int sub = 0; sub < BKV / 16; ++sub)
#pragma unroll
            for (int e = 0; e < 8; e += 4) {
                rs0 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2_t{pf[sub][e], pf[sub][e + 1]}, one2, rs0, false);
                rs1 = __builtin_amdgcn_fdot2_f32_bf16(bf16x2_t{pf[sub][e + 2], pf[sub][e + 3]}, one2, rs1, false);
            }
        float rs = rs0 + rs1;
        const auto rw = __builtin_amdgcn_permlane32_swap(__float_as_uint(rs), __float_as_uint(rs), false, false);
        l_i += __uint_as_float(rw[0]) + __uint_as_float(rw[1]);
    };
    // O^T += V^T P^T for key tile kt.  Transposing read r of sub-step sub, d block db: this lane
    // supplies the address of key row sub*16 + 8 r + vrow and d columns db*32 + vd .. +3 and
    // receives 4 consecutive keys of one d, in the order the S^T accumulators hold P.
    auto pv = [&](int kt, const bf16x8 (&pf)[BKV / 16]) {
        const char* vst = smem + (kt & 1) * STAGE_B + TILE_B;
#pragma unroll
        for (int sub = 0; sub < BKV / 16; ++sub)
#pragma unroll
            for (int db = 0; db < HD / 32; ++db) {
                s16x4 v2[2];
#pragma unroll
                for (int r = 0; r < 2; ++r) {
                    const int row = sub * 16 + 8 * r + vrow;
                    const int d = db * 32 + vd;
                    const char* p = vst + row * ROW + 16 * ((d >> 3) ^ vs) + (d & 7) * 2;
                    v2[r] = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4*)(p));   // generic -> LDS
                }
                const bf16x8 vf = __builtin_bit_cast(bf16x8, __builtin_shufflevector(v2[0], v2[1], 0, 1, 2, 3, 4, 5, 6, 7));
                o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf[sub], o[db], 0, 0, 0);
            }
    };

    // Software pipeline, K one tile ahead of V: step kt computes the scores of tile kt + 1 on
    // the matrix cores while the vector units turn the scores of tile kt into probabilities,
    // then accumulates P V of tile kt.  At the top of step kt this wavefront waits for its own
    // loads of K(kt+1) and V(kt), and the barrier makes everyone's visible and frees the two
    // halves read in step kt - 1 (K(kt) and V(kt-1)); those are refilled with K(kt+2) and
    // V(kt+1).
    auto step = [&](int kt, f32x16 (&sc)[2], f32x16 (&sn)[2]) {
        __builtin_amdgcn_s_waitcnt(0x0f70);            // vmcnt(0)
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        if (kt + 2 < nkt) issue_k(kt + 2);
        if (kt + 1 < nkt) issue_v(kt + 1);
        reference(kt, sc);
        bf16x8 pf[BKV / 16];
        if (kt + 1 < nkt) {
            scores(kt + 1, sn);
            probs(sc, pf);
            // issue order: K fragments two steps ahead of their MFMAs, and up to 12 vector
            // instructions of the softmax after each score MFMA (the softmax then spreads over
            // the first ~8 of them; 4, 6, 8 and 10 measured 1-3% slower on long prompts)
            __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);      // DS reads
#pragma unroll
            for (int i = 0; i < HD / 16; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);  // MFMA
                __builtin_amdgcn_sched_group_barrier(0x002, 12, 0); // VALU
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
                __builtin_amdgcn_sched_group_barrier(0x002, 12, 0);
            }
        } else {
            probs(sc, pf);
        }
        pv(kt, pf);
        // V operands two MFMAs ahead of their use
        __builtin_amdgcn_sched_group_barrier(0x100, 4, 0);
#pragma unroll
        for (int i = 0; i < (BKV / 16) * (HD / 32); ++i) {
            __builtin_amdgcn_sched_group_barrier(0x100, 2, 0);
            __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
        }
    };

    f32x16 sa[2], sb[2];
    issue_k(0);
    issue_v(0);
    if (nkt > 1) issue_k(1);
    __builtin_amdgcn_s_waitcnt(0x0f70);                // vmcnt(0)
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_sched_barrier(0);
    scores(0, sa);
    int kt = 0;
    for (; kt + 1 < nkt; kt += 2) {
        step(kt, sa, sb);
        step(kt + 1, sb, sa);
    }
    if (kt < nkt) step(kt, sa, sb);

    if (!q_ok) return;
    const float inv_l = 1.0f / l_i;
    bf16* orow = out + int64_t(a + qi) * ldo + int64_t(h) * HD + fh * 4;
#pragma unroll
    for (int db = 0; db < HD / 32; ++db)
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
            bf16x4 v;
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] = static_cast<bf16>(o[db][q4 * 4 + e] * inv_l);
            *reinterpret_cast<bf16x4*>(orow + db * 32 + q4 * 8) = v;
        }
}

// ----------------------------------------------------------------------------- float32
__global__ __launch_bounds__(NT) void attn_f32_kernel(const float* __restrict__ q, int64_t ldq,
                                                      const float* __restrict__ kc, const float* __restrict__ vc,
                                                      int64_t ldkv, float* __restrict__ out, int64_t ldo,
                                                      const int32_t* __restrict__ slot_seg,
                                                      const int32_t* __restrict__ seg_prompt,
                                                      const int32_t* __restrict__ seg_start,
                                                      const int32_t* __restrict__ prompt_kv_off, int T, int H,
                                                      int Hkv, int D, float scale) {
    const int lane = threadIdx.x & 63;
    const int64_t wid = int64_t(blockIdx.x) * (NT / kWave) + (threadIdx.x >> 6);
    const int64_t slot = wid / H;
    if (slot >= T) return;
    const int h = static_cast<int>(wid - slot * H);
    const int seg = slot_seg[slot];
    if (seg < 0) return;
    const int qi = static_cast<int>(slot - seg_start[seg]);
    const int prompt = seg_prompt[seg];
    const int64_t kv0 = prompt_kv_off[prompt];
    const int plen = prompt_kv_off[prompt + 1] - static_cast<int>(kv0);
    const int g = h / (H / Hkv);
    const float* qr = q + slot * ldq + int64_t(h) * D;
    float qv[2], acc[2] = {0.f, 0.f};
#pragma unroll
    for (int c = 0; c < 2; ++c) qv[c] = lane + 64 * c < D ? qr[lane + 64 * c] : 0.f;
    float m = -INFINITY, l = 0.f;
    for (int j = 0; j <= qi; ++j) {
        // keys past the prompt (a padded span's tail) are zero: score 0, value 0
        const bool real = j < plen;
        const float* k = kc + (kv0 + j) * ldkv + int64_t(g) * D;
        const float* v = vc + (kv0 + j) * ldkv + int64_t(g) * D;
        float part = 0.f;
#pragma unroll
        for (int c = 0; c < 2; ++c)
            if (real && lane + 64 * c < D) part += qv[c] * k[lane + 64 * c];
        const float sc = wave_sum(part) * scale;
        const float m_new = fmaxf(m, sc);
        const float corr = expf(m - m_new);
        const float p = expf(sc - m_new);
        l = l * corr + p;
#pragma unroll
        for (int c = 0; c < 2; ++c)
            if (lane + 64 * c < D) acc[c] = acc[c] * corr + (real ? p * v[lane + 64 * c] : 0.f);
        m = m_new;
    }
    float* o = out + slot * ldo + int64_t(h) * D;
#pragma unroll
    for (int c = 0; c < 2; ++c)
        if (lane + 64 * c < D) o[lane + 64 * c] = acc[c] / l;
}

}  // namespace

namespace ppk {

void attention_bf16(const void* q, int64_t ldq, const void* kc, const void* vc, int64_t ldkv, void* out,
                    int64_t ldo, const int32_t* seg_prompt, const int32_t* seg_start, const int32_t* seg_len,
                    const int32_t* prompt_kv_off, const int32_t* qtile_seg, const int32_t* qtile_q0, int n_qtiles,
                    int H, int Hkv, hipStream_t s) {
    if (n_qtiles <= 0) return;
    static bool attr = [] {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&attn_bf16_kernel),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, 2 * STAGE_B);
        return true;
    }();
    (void)attr;
    const float scale_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(HD));
    attn_bf16_kernel<<<dim3(n_qtiles * H), NT, 2 * STAGE_B, s>>>(
        static_cast<const bf16*>(q), ldq, static_cast<const bf16*>(kc), static_cast<const bf16*>(vc), ldkv,
        static_cast<bf16*>(out), ldo, seg_prompt, seg_start, seg_len, prompt_kv_off, qtile_seg, qtile_q0, H, Hkv,
        scale_log2);
}

void attention_f32(const float* q, int64_t ldq, const float* kc, const float* vc, int64_t ldkv, float* out,
                   int64_t ldo, const int32_t* slot_seg, const int32_t* seg_prompt, const int32_t* seg_start,
                   const int32_t* prompt_kv_off, int T, int H, int Hkv, int D, hipStream_t s) {
    const int64_t waves = int64_t(T) * H;
    if (waves == 0) return;
    const unsigned blocks = static_cast<unsigned>((waves + NT / kWave - 1) / (NT / kWave));
    attn_f32_kernel<<<blocks, NT, 0, s>>>(q, ldq, kc, vc, ldkv, out, ldo, slot_seg, seg_prompt, seg_start,
                                          prompt_kv_off, T, H, Hkv, D, 1.0f / sqrtf(static_cast<float>(D)));
}

}  // namespace ppk
