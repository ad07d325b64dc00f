// Attention under the independent mask (section 3.2): every query attends causally to
// the keys of its own prompt only.  M' is never materialised; the segment table gives
// each query tile its key range directly.
//
// bf16 kernel (head dim 128), one 256-thread workgroup per (query tile, head):
//   * a work-list entry is (segment, q0): queries [q0, q0+128) of one segment, so keys
//     [0, min(q0+128, len)) of the same segment are the only ones ever loaded -- every
//     tile outside the prompt's diagonal block is skipped by construction, and only the
//     last key tiles (the diagonal) need an in-tile causal predicate;
//   * wavefront w owns queries q0 + 32w .. q0 + 32w + 31; its Q fragments stay in
//     registers for the whole key loop;
//   * key tiles of 64 are staged through LDS, double-buffered: K as [key][d] rows of 256
//     bytes (chunk c of row r stored at c ^ (r & 15)), V transposed to [d][key] rows of
//     128 bytes so that the value product contracts over keys with 16-byte fragment reads;
//   * S^T = K Q^T and O^T += V^T P^T run on the 32x32x16 bf16 MFMA; a lane holds one
//     query, so the running max / sum of the online softmax (Milakov and Gimelshein 2018;
//     the tiling of FlashAttention, Dao et al. 2022) are lane-local plus one exchange with
//     the lane 32 away; probabilities are fed back as bf16 in registers (the key order of
//     the transposed V tile is permuted to match the accumulator layout of S^T);
//   * query heads sharing a KV head (GQA) are adjacent workgroups, so their K/V tiles are
//     read from L2.
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

struct KVTile {
    u32x4 k[BKV * (HD / 8)];   // [64 keys][16 chunks]
    u32x4 vt[HD * (BKV / 8)];  // [128 d][8 chunks]
};

__device__ __forceinline__ int kswz(int row, int c) { return c ^ (row & 15); }
__device__ __forceinline__ int vswz(int row, int c) { return c ^ ((row ^ (row >> 3)) & 7); }
// Position of key j (within a 64-key tile) in a row of the transposed V tile: bits 2 and 3
// swapped, matching which keys a lane's probabilities cover in the S^T accumulator layout.
__device__ __forceinline__ int vperm(int j) { return (j & ~12) | ((j >> 1) & 4) | ((j << 1) & 8); }

template <typename V>
__device__ __forceinline__ bf16x8 as_bf16x8(V v) { return __builtin_bit_cast(bf16x8, v); }

__global__ __launch_bounds__(NT) void attn_bf16_kernel(const bf16* __restrict__ qkv, int64_t ld,
                                                       bf16* __restrict__ out, int64_t ldo,
                                                       const int32_t* __restrict__ seg_start,
                                                       const int32_t* __restrict__ seg_len,
                                                       const int32_t* __restrict__ qtile_seg,
                                                       const int32_t* __restrict__ qtile_q0, int H, int Hkv,
                                                       float scale_log2) {
    __shared__ KVTile sm[2];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int w = blockIdx.x / H, h = blockIdx.x - (blockIdx.x / H) * H;
    const int seg = qtile_seg[w], q0 = qtile_q0[w];
    const int64_t a = seg_start[seg];
    const int n = seg_len[seg];
    const int g = h / (H / Hkv);
    const int n_kv = min(q0 + BQ, n);  // keys [0, n_kv) of the segment
    const int nkt = (n_kv + BKV - 1) / BKV;

    const bf16* Qp = qkv + int64_t(h) * HD;
    const bf16* Kp = qkv + int64_t(H + g) * HD;
    const bf16* Vp = qkv + int64_t(H + Hkv + g) * HD;

    const int fr = lane & 31, fh = lane >> 5;
    const int qi = q0 + wave * 32 + fr;  // this lane's query (offset in the segment)
    const bool q_ok = qi < n;
    const int wq_lo = q0 + wave * 32;
    const int wq_hi = min(wq_lo + 31, n - 1);

    bf16x8 qf[HD / 16];
    {
        const bf16* qrow = Qp + (a + (q_ok ? qi : 0)) * ld + fh * 8;
#pragma unroll
        for (int ks = 0; ks < HD / 16; ++ks)
            qf[ks] = q_ok ? as_bf16x8(*reinterpret_cast<const u32x4*>(qrow + ks * 16)) : bf16x8{};
    }

    u32x4 rk[4], rv[4];
    auto gload = [&](int kt) {
        const int kb = kt * BKV;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int key = kb + (tid >> 4) + 16 * i;
            rk[i] = key < n_kv ? *reinterpret_cast<const u32x4*>(Kp + (a + key) * ld + (tid & 15) * 8)
                               : u32x4{0u, 0u, 0u, 0u};
        }
        const int vkey = kb + (tid & 63);
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int dc = (tid >> 6) + 4 * i;
            rv[i] = vkey < n_kv ? *reinterpret_cast<const u32x4*>(Vp + (a + vkey) * ld + dc * 8)
                                : u32x4{0u, 0u, 0u, 0u};
        }
    };
    auto sstore = [&](KVTile& t) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int row = (tid >> 4) + 16 * i;
            t.k[row * 16 + kswz(row, tid & 15)] = rk[i];
        }
        const int pos = vperm(tid & 63);
        const int pc = pos >> 3, pe = pos & 7;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const int dc = (tid >> 6) + 4 * i;
            const bf16x8 v = as_bf16x8(rv[i]);
#pragma unroll
            for (int e = 0; e < 8; ++e) {
                const int d = dc * 8 + e;
                bf16* rowp = reinterpret_cast<bf16*>(&t.vt[d * 8]);
                rowp[vswz(d, pc) * 8 + pe] = v[e];
            }
        }
    };

    f32x16 o[HD / 32];
#pragma unroll
    for (int db = 0; db < HD / 32; ++db) o[db] = f32x16{};
    float m_i = -1e30f, l_i = 0.f;

    gload(0);
    sstore(sm[0]);
    __syncthreads();
    for (int kt = 0; kt < nkt; ++kt) {
        const KVTile& cur = sm[kt & 1];
        if (kt + 1 < nkt) gload(kt + 1);
        const int kb = kt * BKV;
        if (kb <= wq_hi) {
            f32x16 s[2] = {f32x16{}, f32x16{}};
#pragma unroll
            for (int ks = 0; ks < HD / 16; ++ks) {
#pragma unroll
                for (int b = 0; b < 2; ++b) {
                    const int row = b * 32 + fr;
                    const bf16x8 kf = as_bf16x8(cur.k[row * 16 + kswz(row, ks * 2 + fh)]);
                    s[b] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(kf, qf[ks], s[b], 0, 0, 0);
                }
            }
            const bool need_mask = (kb + BKV - 1 > wq_lo) || (kb + BKV > n_kv);
            float mx = -INFINITY;
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    float v = s[b][r] * scale_log2;
                    if (need_mask) {
                        const int key = kb + b * 32 + 8 * (r >> 2) + 4 * fh + (r & 3);
                        if (key > qi || key >= n_kv) v = -INFINITY;
                    }
                    s[b][r] = v;
                    mx = fmaxf(mx, v);
                }
            mx = fmaxf(mx, __shfl_xor(mx, 32, kWave));
            const float m_new = fmaxf(m_i, mx);
            const float corr = exp2f(m_i - m_new);
            float rs = 0.f;
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const float p = exp2f(s[b][r] - m_new);
                    s[b][r] = p;
                    rs += p;
                }
            rs += __shfl_xor(rs, 32, kWave);
            l_i = l_i * corr + rs;
            m_i = m_new;
#pragma unroll
            for (int db = 0; db < HD / 32; ++db) o[db] *= corr;
#pragma unroll
            for (int sub = 0; sub < BKV / 16; ++sub) {
                bf16x8 pf;
#pragma unroll
                for (int e = 0; e < 8; ++e) pf[e] = static_cast<bf16>(s[sub >> 1][(sub & 1) * 8 + e]);
#pragma unroll
                for (int db = 0; db < HD / 32; ++db) {
                    const int row = db * 32 + fr;
                    const bf16x8 vf = as_bf16x8(cur.vt[row * 8 + vswz(row, sub * 2 + fh)]);
                    o[db] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(vf, pf, o[db], 0, 0, 0);
                }
            }
        }
        if (kt + 1 < nkt) sstore(sm[(kt + 1) & 1]);
        __syncthreads();
    }

    if (!q_ok) return;
    const float inv_l = 1.0f / l_i;
    bf16* orow = out + (a + qi) * ldo + int64_t(h) * HD + fh * 4;
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
__global__ __launch_bounds__(NT) void attn_f32_kernel(const float* __restrict__ qkv, int64_t ld,
                                                      float* __restrict__ out, int64_t ldo,
                                                      const int32_t* __restrict__ slot_seg,
                                                      const int32_t* __restrict__ seg_start, int T, int H,
                                                      int Hkv, int D, float scale) {
    const int lane = threadIdx.x & 63;
    const int64_t wid = int64_t(blockIdx.x) * (NT / kWave) + (threadIdx.x >> 6);
    const int64_t slot = wid / H;
    if (slot >= T) return;
    const int h = static_cast<int>(wid - slot * H);
    const int seg = slot_seg[slot];
    if (seg < 0) return;
    const int64_t a = seg_start[seg];
    const int g = h / (H / Hkv);
    const float* q = qkv + slot * ld + int64_t(h) * D;
    float qv[2], acc[2] = {0.f, 0.f};
#pragma unroll
    for (int c = 0; c < 2; ++c) qv[c] = lane + 64 * c < D ? q[lane + 64 * c] : 0.f;
    float m = -INFINITY, l = 0.f;
    for (int64_t j = a; j <= slot; ++j) {
        const float* k = qkv + j * ld + int64_t(H + g) * D;
        const float* v = qkv + j * ld + int64_t(H + Hkv + g) * D;
        float part = 0.f;
#pragma unroll
        for (int c = 0; c < 2; ++c)
            if (lane + 64 * c < D) part += qv[c] * k[lane + 64 * c];
        const float sc = wave_sum(part) * scale;
        const float m_new = fmaxf(m, sc);
        const float corr = expf(m - m_new);
        const float p = expf(sc - m_new);
        l = l * corr + p;
#pragma unroll
        for (int c = 0; c < 2; ++c)
            if (lane + 64 * c < D) acc[c] = acc[c] * corr + p * v[lane + 64 * c];
        m = m_new;
    }
    float* o = out + slot * ldo + int64_t(h) * D;
#pragma unroll
    for (int c = 0; c < 2; ++c)
        if (lane + 64 * c < D) o[lane + 64 * c] = acc[c] / l;
}

}  // namespace

namespace ppk {

void attention_bf16(const void* qkv, int64_t ld, void* out, int64_t ldo, const int32_t* seg_start,
                    const int32_t* seg_len, const int32_t* qtile_seg, const int32_t* qtile_q0, int n_qtiles, int H,
                    int Hkv, int D, hipStream_t s) {
    if (n_qtiles <= 0) return;
    const float scale_log2 = 1.4426950408889634f / sqrtf(static_cast<float>(D));
    attn_bf16_kernel<<<dim3(n_qtiles * H), NT, 0, s>>>(static_cast<const bf16*>(qkv), ld, static_cast<bf16*>(out),
                                                        ldo, seg_start, seg_len, qtile_seg, qtile_q0, H, Hkv,
                                                        scale_log2);
}

void attention_f32(const float* qkv, int64_t ld, float* out, int64_t ldo, const int32_t* slot_seg,
                   const int32_t* seg_start, int T, int H, int Hkv, int D, hipStream_t s) {
    const int64_t waves = int64_t(T) * H;
    if (waves == 0) return;
    const unsigned blocks = static_cast<unsigned>((waves + NT / kWave - 1) / (NT / kWave));
    attn_f32_kernel<<<blocks, NT, 0, s>>>(qkv, ld, out, ldo, slot_seg, seg_start, T, H, Hkv, D,
                                          1.0f / sqrtf(static_cast<float>(D)));
}

}  // namespace ppk
