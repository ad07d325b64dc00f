// Generation with packed KV caches (section 4.8): the kernels of one decode step that the
// prefill does not already have.  Each step feeds one new token per prompt through the
// decoder (section 2.2: one forward pass per token, earlier keys and values read from the
// cache).
//
// decode_prep_kernel     per prompt: the token's position pos0 + step (restart positions,
//                        section 3.2, continued into generation), cos/sin of that position
//                        for RoPE (evaluated in float64 as in the prefill's table), the
//                        generation-cache row the step appends to, and identity indices.
// decode_attn_kernel     split-key attention of one query row per prompt against that
//                        prompt's keys only: context rows (its prompt tokens, plus masked
//                        padding in the full-batching layout) and the generated rows so far.
//                        A workgroup takes one (prompt, key/value head, chunk of 128 keys)
//                        and all query heads of the group, so every key and value is read
//                        from HBM once per step; it writes the chunk's (max, sum, output).
// decode_combine_kernel  merges a prompt's chunk results in a fixed order (on the paths that
//                        do not merge them in the O projection's staging, below).
// The projections of a decode step have one row per prompt (k <= 64): C[k, N] = A[k, K]
// W[N, K]^T is bound by streaming W from HBM.
// rowpair_gemm_kernel    QKV and gate/up: one workgroup per 32 weight rows whose epilogue
//                        belongs together (rotate-half pairs; gate and up rows of the same
//                        features), K split four ways across its wavefronts and added
//                        through LDS; RoPE with the query store and the key/value append,
//                        or SwiGLU, in the same kernel.
// rowpair_seg_kernel     the same for up to 16 prompts at K = 2048 or 4096, the weights
//                        loaded as whole 1 KB row segments straight into an LDS ring.
// qkv_seg16_kernel       QKV in that style with 16 rows per workgroup (8 dims and their
//                        rotate-half partners) when the 32-row groups outnumber the CUs.
// splitk_seg_kernel      down (N = d) for up to 16 prompts in that style: 32 rows x a K
//                        split per workgroup, float32 partial sums per split.
// skinny_gemm_kernel     O, and down for more prompts (N = d, too few rows for one
//                        workgroup per 32): about 512 pieces of 64 rows x a K split of up to
//                        6 tiles of 128; each workgroup stages its slice of A (k rows, LDS
//                        sized to k) once and each wavefront streams 16 weight rows into the
//                        16x16x32 bf16 MFMA, all its K steps requested up front; float32
//                        partial sums per split.  For O the staged slice is the attention
//                        output, merged there from the chunk results.
// residual_rmsnorm_kernel  adds those partial sums, in split order, to the residual stream
//                        inside the RMSNorm that follows each projection.
// (A single-kernel split-K with the sum done by the last workgroup of a row group was
// measured slower: its cross-workgroup hand-off costs more than the launch it saves.)
//
// The chunks of the context part are counted from the prompt's first key, and the
// generated keys form chunks of their own, so the packed and the full-batching layouts give
// each valid key the same chunk and lane: their results are bit-identical, the padding
// contributing exact zeros.
#include <math.h>

#include <algorithm>

#include "device.h"
#include "kernels.h"
#include "prepack.h"

namespace {

constexpr int CH = ppk::kDecodeChunk;   // keys per chunk: 4 wavefronts x IT iterations x 8 keys
constexpr int IT = CH / 32;
constexpr float kLog2e = 1.4426950408889634f;

__global__ __launch_bounds__(64) void decode_prep_kernel(int k, int step, const int32_t* __restrict__ pos0,
                                                         const int32_t* __restrict__ gen_off, int D, double theta,
                                                         float2* __restrict__ table, int32_t* __restrict__ slot_pos,
                                                         int32_t* __restrict__ slot_kv, int32_t* __restrict__ slot_seg,
                                                         int32_t* __restrict__ ident) {
    const int i = blockIdx.x, j = threadIdx.x;
    if (i >= k) return;
    const int half = D / 2;
    if (j < half) {
        const double inv_freq = pow(theta, -2.0 * j / static_cast<double>(D));
        const double a = static_cast<double>(pos0[i] + step) * inv_freq;
        table[int64_t(i) * half + j] = make_float2(static_cast<float>(cos(a)), static_cast<float>(sin(a)));
    }
    if (j == 0) {
        slot_pos[i] = i;                 // row i of this step's table
        slot_kv[i] = gen_off[i] + step;  // the row this step appends to
        slot_seg[i] = 0;
        ident[i] = i;
        if (i == k - 1) ident[k] = k;
    }
}

template <typename T, int DL>
__device__ __forceinline__ void load_slice(const T* p, float* v) {
#pragma unroll
    for (int e = 0; e < DL; e += 8) load8(p + e, v + e);
}

// A slice of DL elements held as 16-byte pieces -> float.
template <typename T, int DL>
__device__ __forceinline__ void unpack_slice(const u32x4* raw, float* v) {
    if constexpr (sizeof(T) == 2) {
#pragma unroll
        for (int c = 0; c < DL / 8; ++c) {
            const bf16x8 b = __builtin_bit_cast(bf16x8, raw[c]);
#pragma unroll
            for (int e = 0; e < 8; ++e) v[8 * c + e] = static_cast<float>(b[e]);
        }
    } else {
#pragma unroll
        for (int c = 0; c < DL / 4; ++c) {
            const f32x4 f = __builtin_bit_cast(f32x4, raw[c]);
#pragma unroll
            for (int e = 0; e < 4; ++e) v[4 * c + e] = f[e];
        }
    }
}

// (m, l, o) <- merge of two partial softmax results over disjoint key sets (base-2 scores).
template <int DL>
__device__ __forceinline__ void merge(float& m, float& l, float* o, float m2, float l2, const float* o2) {
    const float M = fmaxf(m, m2);
    const float a = M == -INFINITY ? 0.f : exp2f(m - M);
    const float b = M == -INFINITY ? 0.f : exp2f(m2 - M);
    l = l * a + l2 * b;
#pragma unroll
    for (int e = 0; e < DL; ++e) o[e] = o[e] * a + o2[e] * b;
    m = M;
}

// One (prompt i, key/value head g, chunk c) of the decode attention: the chunk's (max, sum,
// output) for the group's R query heads into part.
template <typename T, int D, int R>
__device__ __forceinline__ void decode_attn_chunk(
    const T* __restrict__ q, int64_t ldq, const T* __restrict__ ctx_k, const T* __restrict__ ctx_v,
    const T* __restrict__ gen_k, const T* __restrict__ gen_v, int64_t ldkv, const int32_t* __restrict__ ctx_off,
    const int32_t* __restrict__ ctx_span, const int32_t* __restrict__ ctx_valid, const int32_t* __restrict__ gen_off,
    int step, int Hkv, int n_ctx_chunks, int n_chunks, float* __restrict__ part, int i, int g, int c) {
    constexpr int DL = D / 8;
    constexpr int PS = D + 4;            // floats per partial: o[D], m, l, 2 unused
    __shared__ float red[4][R][D + 2];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int kg = lane >> 3, dl = lane & 7;
    const T* K;
    const T* V;
    int64_t row0;
    int j0, jend, valid;
    if (c < n_ctx_chunks) {
        j0 = c * CH;
        jend = min(j0 + CH, ctx_span[i]);
        valid = ctx_valid[i];
        row0 = ctx_off[i];
        K = ctx_k;
        V = ctx_v;
    } else {
        j0 = (c - n_ctx_chunks) * CH;
        jend = min(j0 + CH, step + 1);
        valid = step + 1;
        row0 = gen_off[i];
        K = gen_k;
        V = gen_v;
    }
    if (j0 >= jend) return;              // generated keys not there yet: no partial, never combined

    // queries of the group's R heads, pre-scaled so that scores are in base 2
    const float scale = kLog2e * rsqrtf(static_cast<float>(D));
    float qf[R][DL];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        load_slice<T, DL>(q + int64_t(i) * ldq + int64_t(g * R + r) * D + dl * DL, qf[r]);
#pragma unroll
        for (int e = 0; e < DL; ++e) qf[r][e] *= scale;
    }
    float m[R], l[R], o[R][DL];
#pragma unroll
    for (int r = 0; r < R; ++r) {
        m[r] = -INFINITY;
        l[r] = 0.f;
#pragma unroll
        for (int e = 0; e < DL; ++e) o[r][e] = 0.f;
    }
    const int64_t col = int64_t(g) * D + dl * DL;
    // every key and value slice of the chunk requested before the first score (rows past
    // the chunk read as its last row, then ignored), so the HBM latency is paid once
    constexpr int NQ = DL * int(sizeof(T)) / 16;      // 16-byte pieces per slice
    u32x4 kraw[IT][NQ], vraw[IT][NQ];
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int j = min(j0 + 8 * IT * w + 8 * it + kg, jend - 1);
        const int64_t off = (row0 + j) * ldkv + col;
#pragma unroll
        for (int c = 0; c < NQ; ++c) {
            kraw[it][c] = *reinterpret_cast<const u32x4*>(K + off + c * (16 / int(sizeof(T))));
            vraw[it][c] = *reinterpret_cast<const u32x4*>(V + off + c * (16 / int(sizeof(T))));
        }
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
#pragma unroll
        for (int c = 0; c < NQ; ++c) asm volatile("" : "+v"(kraw[it][c]), "+v"(vraw[it][c]));
    }
#pragma unroll
    for (int it = 0; it < IT; ++it) {
        const int j = j0 + 8 * IT * w + 8 * it + kg;
        float kf[DL], vf[DL];
        unpack_slice<T, DL>(kraw[it], kf);
        unpack_slice<T, DL>(vraw[it], vf);
        const bool ok = j < jend && j < valid;   // padding of the full-batching layout is read, then masked
#pragma unroll
        for (int r = 0; r < R; ++r) {
            float s = 0.f;
#pragma unroll
            for (int e = 0; e < DL; ++e) s = fmaf(qf[r][e], kf[e], s);
            s += __shfl_xor(s, 1);
            s += __shfl_xor(s, 2);
            s += __shfl_xor(s, 4);
            if (ok) {
                const float mn = fmaxf(m[r], s);
                const float a = exp2f(m[r] - mn);   // m = -inf at the first key: a = 0
                const float p = exp2f(s - mn);
                l[r] = l[r] * a + p;
#pragma unroll
                for (int e = 0; e < DL; ++e) o[r][e] = fmaf(p, vf[e], o[r][e] * a);
                m[r] = mn;
            }
        }
    }
    // merge the 8 key groups of the wavefront (lanes with the same dl), then the 4 wavefronts
#pragma unroll
    for (int x = 8; x < 64; x <<= 1) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
            float o2[DL];
#pragma unroll
            for (int e = 0; e < DL; ++e) o2[e] = __shfl_xor(o[r][e], x);
            const float m2 = __shfl_xor(m[r], x), l2 = __shfl_xor(l[r], x);
            merge<DL>(m[r], l[r], o[r], m2, l2, o2);
        }
    }
    if (kg == 0) {
#pragma unroll
        for (int r = 0; r < R; ++r) {
#pragma unroll
            for (int e = 0; e < DL; ++e) red[w][r][dl * DL + e] = o[r][e];
            if (dl == 0) {
                red[w][r][D] = m[r];
                red[w][r][D + 1] = l[r];
            }
        }
    }
    __syncthreads();
    for (int idx = threadIdx.x; idx < R * D; idx += 256) {
        const int r = idx / D, e = idx % D;
        float mm = red[0][r][D], ll = red[0][r][D + 1], oo = red[0][r][e];
#pragma unroll
        for (int w2 = 1; w2 < 4; ++w2) merge<1>(mm, ll, &oo, red[w2][r][D], red[w2][r][D + 1], &red[w2][r][e]);
        float* pp = part + ((int64_t(i) * (Hkv * R) + g * R + r) * n_chunks + c) * PS;
        pp[e] = oo;
        if (e == 0) {
            pp[D] = mm;
            pp[D + 1] = ll;
        }
    }
    __syncthreads();   // red is reused by the workgroup's next item
}

// The decode attention's work list: first the generated keys' chunks of every prompt
// (k x n_gen_chunks, prompt-major), then each prompt's context chunks, prompt by prompt
// (ceil(ctx_span / CH) each).  Item -> (prompt, chunk index into the partial results); an
// item past the last context chunk -> prompt -1.  The context chunk counts are summed across
// the lanes, 64 prompts at a time (every lane of the wavefront returns the same answer).
__device__ __forceinline__ int2 attn_item(int item, int k, int n_gen_chunks, int n_ctx_chunks,
                                          const int32_t* __restrict__ ctx_span) {
    if (item < k * n_gen_chunks) return make_int2(item / n_gen_chunks, n_ctx_chunks + item % n_gen_chunks);
    const int idx = item - k * n_gen_chunks;
    const int lane = threadIdx.x & 63;
    int base = 0;
    for (int b = 0; b < k; b += 64) {
        const int l = b + lane;
        int p = l < k ? (ctx_span[l] + CH - 1) / CH : 0;
#pragma unroll
        for (int o = 1; o < 64; o <<= 1) {
            const int t = __shfl_up(p, o);
            if (lane >= o) p += t;
        }
        const int total = __shfl(p, 63);
        if (idx < base + total) {
            const int li = __popcll(__ballot(p + base <= idx));   // prompts of this block wholly before
            const int before = li > 0 ? __shfl(p, li - 1) : 0;
            return make_int2(b + li, idx - base - before);
        }
        base += total;
    }
    return make_int2(-1, 0);
}

// Lane l of wavefront w: key group kg = l / 8 (one key per iteration), dimension slice
// dl = l % 8 (D / 8 consecutive elements).  Keys of the chunk: j0 + 8 IT w + 8 it + kg.
// list == 0: workgroup (i Hkv + g, c) takes chunk c of prompt i and key/value head g, every
// prompt n_ctx_chunks + n_gen_chunks of them (those past its keys return at once).
// list != 0: workgroup (g, y) takes the work-list items y, y + gridDim.y, ... of head g (one
// each when the grid holds them all), so only real chunks occupy the CUs: a batch of nine
// 1-token prompts and one of 1000 at the 7B shape, 10.4 -> 10.0 us.  The host takes the list
// when it is shorter; in the full-batching layout it is not, and the lookup would cost each
// workgroup a dependent load (1.3B: 2% of the step).  bf16 with one query head per key/value
// head: four workgroups per CU (at most 128 registers), as the chunks are latency-bound (at
// 129 registers, three per CU, the 7B batch above took 11.6 us); the other forms would spill.
template <typename T, int D, int R>
__global__ __launch_bounds__(256, (R == 1 && sizeof(T) == 2) ? 4 : 1) void decode_attn_kernel(
    const T* __restrict__ q, int64_t ldq, const T* __restrict__ ctx_k, const T* __restrict__ ctx_v,
    const T* __restrict__ gen_k, const T* __restrict__ gen_v, int64_t ldkv, const int32_t* __restrict__ ctx_off,
    const int32_t* __restrict__ ctx_span, const int32_t* __restrict__ ctx_valid, const int32_t* __restrict__ gen_off,
    int step, int k, int Hkv, int n_ctx_chunks, int n_gen_chunks, int list, float* __restrict__ part) {
    const int n_chunks = n_ctx_chunks + n_gen_chunks;
    if (!list) {
        decode_attn_chunk<T, D, R>(q, ldq, ctx_k, ctx_v, gen_k, gen_v, ldkv, ctx_off, ctx_span, ctx_valid, gen_off,
                                   step, Hkv, n_ctx_chunks, n_chunks, part, blockIdx.x / Hkv, blockIdx.x % Hkv,
                                   blockIdx.y);
        return;
    }
    for (int item = blockIdx.y;; item += gridDim.y) {
        const int2 ic = attn_item(item, k, n_gen_chunks, n_ctx_chunks, ctx_span);
        const int i = __builtin_amdgcn_readfirstlane(ic.x), c = __builtin_amdgcn_readfirstlane(ic.y);
        if (i < 0) return;
        decode_attn_chunk<T, D, R>(q, ldq, ctx_k, ctx_v, gen_k, gen_v, ldkv, ctx_off, ctx_span, ctx_valid, gen_off,
                                   step, Hkv, n_ctx_chunks, n_chunks, part, i, blockIdx.x, c);
    }
}

// One wavefront per (prompt, query head): the prompt's context chunks, then its generated
// chunks, merged in that order; out = o / l.
template <typename T, int D>
__global__ __launch_bounds__(256) void decode_combine_kernel(const float* __restrict__ part, int k, int H,
                                                             const int32_t* __restrict__ ctx_span, int step,
                                                             int n_ctx_chunks, int n_chunks, T* __restrict__ out,
                                                             int64_t ldo) {
    constexpr int PS = D + 4;
    constexpr int E = D / 64;            // dimensions per lane
    const int pair = blockIdx.x * 4 + (threadIdx.x >> 6);
    const int lane = threadIdx.x & 63;
    if (pair >= k * H) return;
    const int i = pair / H, h = pair % H;
    const float* base = part + int64_t(pair) * n_chunks * PS;
    float m = -INFINITY, l = 0.f, o[E];
#pragma unroll
    for (int e = 0; e < E; ++e) o[e] = 0.f;
    const int nc = (ctx_span[i] + CH - 1) / CH, ng = (step + 1 + CH - 1) / CH;
    for (int t = 0; t < nc + ng; ++t) {
        const float* pp = base + int64_t(t < nc ? t : n_ctx_chunks + t - nc) * PS;
        float o2[E];
#pragma unroll
        for (int e = 0; e < E; ++e) o2[e] = pp[lane * E + e];
        merge<E>(m, l, o, pp[D], pp[D + 1], o2);
    }
    const float inv = l > 0.f ? 1.f / l : 0.f;
    T* dst = out + int64_t(i) * ldo + int64_t(h) * D + lane * E;
#pragma unroll
    for (int e = 0; e < E; ++e) dst[e] = static_cast<T>(o[e] * inv);
}

// LDS swizzle of a staged A tile (rows of 128 bf16 = 256 bytes): row r's 16-byte chunk q at
// q ^ gsw(r % 8), gsw placing r's bits 0, 1, 2 at bits 0, 2, 3.  A fragment read takes rows
// r..r+15 at chunk 4 s + l / 16; the lanes served together (i and i + 32) then hit 16
// distinct bank groups.
__device__ __forceinline__ int gsw(int r) { return (r & 1) | (((r >> 1) & 1) << 2) | (((r >> 2) & 1) << 3); }

constexpr int SG_ROWS = 64;     // W rows per workgroup, 16 per wavefront
constexpr int SG_TILE = 128;    // K columns per staged A tile
constexpr int SG_MAX_TILES = 6; // A tiles per K split (4: 1.2% slower at the 7B shape; 8: 0.6%)

// part[s][m][n] = sum over the NT K tiles of split s of A[m, :] . W[n, :], m < k <= 16 NMB.
// Lane l of wavefront w reads 8 consecutive K values of W row n_w + l % 16 at offset
// 8 (l / 16) of each 32-wide step, every step of its split requested before the first MFMA,
// and holds, per prompt block mb, the sums of prompt 16 mb + l % 16 for rows
// n_w + 4 (l / 16) + 0..3.  The slice of A (k_pad rows x NT tiles) is staged once in LDS.
template <int NT, int NMB, bool COMB>
__global__ __launch_bounds__(256) void skinny_gemm_kernel(const bf16* __restrict__ A, int64_t lda, int k,
                                                          const bf16* __restrict__ W, int64_t ldw, int N, int K,
                                                          float* __restrict__ part, ppk::AttnChunks ac) {
    extern __shared__ __attribute__((aligned(16))) char lds[];   // NT tiles of 16 NMB rows x 256 bytes
    constexpr int KP = 16 * NMB, TILE_B = KP * 256;
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int lr = lane & 15, q4 = lane >> 4;
    const int g = blockIdx.x, s = blockIdx.y;   // row group, K split
    const int t0 = s * NT;
    const int nt = min(NT, K / SG_TILE - t0);     // the last split may hold fewer tiles
    const int n_w = g * SG_ROWS + 16 * w;
    const bf16* wrow = W + int64_t(n_w + lr) * ldw + int64_t(t0) * SG_TILE + 8 * q4;
    bf16x8 ring[4 * NT];
#pragma unroll
    for (int j = 0; j < 4 * NT; ++j)
        if (j < 4 * nt) ring[j] = *reinterpret_cast<const bf16x8*>(wrow + 32 * j);
    // stage A[0 .. KP) x tiles t0 .. t0 + nt (rows past k read as row k - 1, or zero when
    // merged from chunks; their sums are never stored).
    // COMB: A is the attention output, formed here from the decode attention's chunk results
    // (128 columns = one head per tile): the chunks of prompt r and head t0 + t merged in
    // the fixed order of decode_combine_kernel, divided by the sum, rounded to bf16.
    for (int idx = threadIdx.x; idx < KP * nt * 16; idx += 256) {
        const int r = idx / (nt * 16), q = idx % (nt * 16), t = q / 16, ch = q % 16;
        const int m = min(r, k - 1);
        bf16x8 v{};
        if constexpr (COMB) {
            if (r >= k) {   // padding rows of the tile: their sums are never stored
                *reinterpret_cast<bf16x8*>(lds + t * TILE_B + r * 256 + 16 * (ch ^ gsw(r & 7))) = v;
                continue;
            }
            constexpr int PS = 128 + 4;
            const float* base = ac.part + (int64_t(m) * ac.H + t0 + t) * ac.n_chunks * PS;
            const int nc = (ac.ctx_span[m] + CH - 1) / CH, ng = (ac.step + 1 + CH - 1) / CH;
            float mm = -INFINITY, ll = 0.f, o[8];
#pragma unroll
            for (int e = 0; e < 8; ++e) o[e] = 0.f;
            // chunks merged in order; the loads of 4 chunks are issued together so that a long
            // prompt waits for one L2 round trip per 4 chunks, not per chunk (8: more registers,
            // fewer waves, slower)
            const int n = nc + ng;
            auto chunk = [&](int c) { return base + int64_t(c < nc ? c : ac.n_ctx_chunks + c - nc) * PS; };
            int c = 0;
            for (; c + 4 <= n; c += 4) {
                float o2[4][8], m2[4], l2[4];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    const float* pp = chunk(c + u);
                    load8(pp + ch * 8, o2[u]);
                    m2[u] = pp[128];
                    l2[u] = pp[129];
                }
#pragma unroll
                for (int u = 0; u < 4; ++u) merge<8>(mm, ll, o, m2[u], l2[u], o2[u]);
            }
            for (; c < n; ++c) {
                const float* pp = chunk(c);
                float o2[8];
                load8(pp + ch * 8, o2);
                merge<8>(mm, ll, o, pp[128], pp[129], o2);
            }
            const float inv = ll > 0.f ? 1.f / ll : 0.f;
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = static_cast<bf16>(o[e] * inv);
        } else {
            v = *reinterpret_cast<const bf16x8*>(A + int64_t(m) * lda + int64_t(t0 + t) * SG_TILE + ch * 8);
        }
        *reinterpret_cast<bf16x8*>(lds + t * TILE_B + r * 256 + 16 * (ch ^ gsw(r & 7))) = v;
    }
    // keep every W fragment in flight from the top: the compiler would otherwise sink each
    // load to its MFMA and pay the HBM latency once per step
#pragma unroll
    for (int j = 0; j < 4 * NT; ++j) asm volatile("" : "+v"(ring[j]));
    __syncthreads();
    f32x4 acc[NMB] = {};
    const int fsw = gsw(lr & 7);
#pragma unroll
    for (int j = 0; j < 4 * NT; ++j) {
        if (j < 4 * nt) {
#pragma unroll
            for (int mb = 0; mb < NMB; ++mb) {
                const bf16x8 h = *reinterpret_cast<const bf16x8*>(lds + (j / 4) * TILE_B + (16 * mb + lr) * 256 +
                                                                  16 * ((4 * (j % 4) + q4) ^ fsw));
                acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ring[j], h, acc[mb], 0, 0, 0);
            }
        }
    }
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) {
        const int m = 16 * mb + lr;
        if (m < k) *reinterpret_cast<f32x4*>(part + (int64_t(s) * k + m) * N + n_w + 4 * q4) = acc[mb];
    }
}

// RoPE (query and key heads) and the stores of one prompt m's dims i .. i + 3 (a) and their
// rotate-half partners i + 64 .. + 67 (b) of QKV output head `head`: queries to q, keys and
// values appended to the caches at row slot_kv[m].
__device__ __forceinline__ void qkv_pair_store(int head, int i, int m, const f32x4& a, const f32x4& b,
                                               const ppk::QkvOut& qo) {
    const bool rotate = head < qo.H + qo.Hkv;
    bf16x4 lo, hi;
    if (rotate) {
        const float2* cs = qo.table + int64_t(qo.slot_pos[m]) * 64 + i;
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            const float2 t = cs[e];
            lo[e] = static_cast<bf16>(a[e] * t.x - b[e] * t.y);
            hi[e] = static_cast<bf16>(b[e] * t.x + a[e] * t.y);
        }
    } else {
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            lo[e] = static_cast<bf16>(a[e]);
            hi[e] = static_cast<bf16>(b[e]);
        }
    }
    bf16* dst;
    if (head < qo.H)
        dst = static_cast<bf16*>(qo.q) + int64_t(m) * qo.ldq + head * 128;
    else
        dst = static_cast<bf16*>(rotate ? qo.kc : qo.vc) + int64_t(qo.slot_kv[m]) * qo.ldkv +
              (head - qo.H - (rotate ? 0 : qo.Hkv)) * 128;
    *reinterpret_cast<bf16x4*>(dst + i) = lo;
    *reinterpret_cast<bf16x4*>(dst + i + 64) = hi;
}

// The rowpair epilogue for prompt m and the 4 rows c .. c + 3 of each of the workgroup's two
// 16-row blocks: a = block 0's sums, b = block 1's.
template <int EPI>
__device__ __forceinline__ void rowpair_epilogue(int g, int m, int c, const f32x4& a, const f32x4& b,
                                                 const ppk::DecodeEpi& ep) {
    if (EPI == ppk::kSwiGLU) {       // features 16 g + c .. + 3: gate a, up b
        bf16x4 o;
#pragma unroll
        for (int e = 0; e < 4; ++e) o[e] = static_cast<bf16>(silu(a[e]) * b[e]);
        *reinterpret_cast<bf16x4*>(static_cast<bf16*>(ep.out) + int64_t(m) * ep.ldo + 16 * g + c) = o;
    } else {                         // QKV: dims i .. i + 3 (a) and i + 64 .. (b) of head g / 4
        qkv_pair_store(g >> 2, 16 * (g & 3) + c, m, a, b, ep.qkv);
    }
}

// Decode projections whose epilogue needs two blocks of 16 weight rows together, SwiGLU (the
// 16 gate rows and the 16 up rows of 16 features) and QKV (16 rotate-half pairs c, c + 64 of
// a head): one workgroup per such 32 rows, its 4 wavefronts each taking a quarter of K, the
// quarters added in wavefront order through LDS and the epilogue applied in the same kernel
// (no partial sums leave the workgroup).  Weight and activation fragments are read straight
// from global memory into a ring of RP_RING steps.  Lane l: weight row r_nb + l % 16 and
// prompt 16 mb + l % 16, K offset 8 (l / 16) of each 32-wide step; it ends with block nb's
// rows r_nb + 4 (l / 16) + 0..3 for prompt 16 mb + l % 16.
constexpr int RP_RING = 2;   // 2: 52 VGPRs; 4, 6 and 8 (132 VGPRs) measured 1-3% slower at the 7B shape

template <int EPI, int NMB>
__global__ __launch_bounds__(256) void rowpair_gemm_kernel(const bf16* __restrict__ A, int64_t lda, int k,
                                                           const bf16* __restrict__ W, int64_t ldw, int K,
                                                           ppk::DecodeEpi ep) {
    __shared__ f32x4 red[4][2][NMB][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int lr = lane & 15, q4 = lane >> 4;
    const int g = blockIdx.x;
    int r0[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
        r0[nb] = EPI == ppk::kSwiGLU ? 32 * g + 16 * nb : (g >> 2) * 128 + 64 * nb + 16 * (g & 3);
    const int kq = K / 4, k0 = w * kq, steps = kq / 32;
    const bf16* wp[2];
    const bf16* ap[NMB];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) wp[nb] = W + int64_t(r0[nb] + lr) * ldw + k0 + 8 * q4;
#pragma unroll
    for (int mb = 0; mb < NMB; ++mb) ap[mb] = A + int64_t(min(16 * mb + lr, k - 1)) * lda + k0 + 8 * q4;
    bf16x8 rw[RP_RING][2], ra[RP_RING][NMB];
    auto issue = [&](int u, int j) {
        const int jj = 32 * min(j, steps - 1);
#pragma unroll
        for (int nb = 0; nb < 2; ++nb) rw[u][nb] = *reinterpret_cast<const bf16x8*>(wp[nb] + jj);
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) ra[u][mb] = *reinterpret_cast<const bf16x8*>(ap[mb] + jj);
    };
#pragma unroll
    for (int u = 0; u < RP_RING; ++u) issue(u, u);
    f32x4 acc[2][NMB] = {};
    for (int j0 = 0; j0 < steps; j0 += RP_RING) {
#pragma unroll
        for (int u = 0; u < RP_RING; ++u) {
            if (j0 + u < steps) {
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
#pragma unroll
                    for (int mb = 0; mb < NMB; ++mb)
                        acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(rw[u][nb], ra[u][mb], acc[nb][mb], 0, 0, 0);
            }
            if (j0 + u + RP_RING < steps) issue(u, j0 + u + RP_RING);
        }
    }
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
#pragma unroll
        for (int mb = 0; mb < NMB; ++mb) red[w][nb][mb][lane] = acc[nb][mb];
    __syncthreads();
    for (int it = threadIdx.x; it < NMB * 64; it += 256) {
        const int mb = it / 64, l = it % 64;
        const int m = 16 * mb + (l & 15), c = 4 * (l >> 4);   // prompt, first of 4 rows of each block
        if (m >= k) continue;
        f32x4 a = red[0][0][mb][l], b = red[0][1][mb][l];
#pragma unroll
        for (int w2 = 1; w2 < 4; ++w2) {
            a += red[w2][0][mb][l];
            b += red[w2][1][mb][l];
        }
        rowpair_epilogue<EPI>(g, m, c, a, b, ep);
    }
}

// Buffer descriptor word 3 for raw (unstructured) 32-bit-offset loads on gfx9-family parts.
constexpr int kRsrcWord3 = 0x00020000;
// s_waitcnt immediate: vmcnt(n) and lgkmcnt(0), expcnt not waited for (gfx9 encoding).
constexpr int wait_vm_lgkm0(int n) { return ((n >> 4) << 14) | (n & 15) | 0x0070; }
typedef __attribute__((address_space(3))) void lds_void;

// The rowpair projections for up to 16 prompts with K = 512 NSEG: the same 32 rows per workgroup
// and epilogue, the weights streamed as whole 1 KB row segments.  Chunk (s, nb) = the 16 rows of
// block nb x K columns 512 s .. + 511; each wavefront loads 4 of its rows (one 1 KB load each)
// straight into an LDS ring of NW chunks, which from HBM runs markedly faster than the 64-byte
// pieces of 16 rows that register loads in the MFMA layout request.  Wavefront w takes columns
// 128 w .. + 127 of every chunk (4 K-steps); its quarter of the prompts' rows (4 fragments per
// segment) goes into registers one segment ahead of its use.  The quarters' sums are added
// through LDS in wavefront order, as in rowpair_gemm_kernel.
constexpr int RS_COLS = 512;                    // K columns of a chunk
constexpr int RS_CHUNK_B = 16 * RS_COLS * 2;    // 16 KB

// LDS swizzle of a 1 KB chunk row: 16-byte chunk q of row r at q ^ f(r), f placing r's bits 0, 1,
// 2 at bits 0, 2, 3 (within each 256-byte bank window): a fragment read (rows r..r+15, chunk
// 16 w + 4 s + l / 16; lanes i and i + 32 served together) hits 16 distinct bank groups.
__device__ __forceinline__ int rs_swz(int r) { return (r & 1) | (((r >> 1) & 1) << 2) | (((r >> 2) & 1) << 3); }

template <int EPI, int NSEG, int NW>
__global__ __launch_bounds__(256, 2) void rowpair_seg_kernel(const bf16* __restrict__ A, int64_t lda, int k,
                                                             const bf16* __restrict__ W, int64_t ldw,
                                                             ppk::DecodeEpi ep) {
    static_assert(NW >= 2 && NW * RS_CHUNK_B >= 4 * 2 * 64 * 16, "ring, and room for the reduction");
    constexpr int NCH = 2 * NSEG;               // chunks: segment-major, block nb within a segment
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lr = lane & 15, q4 = lane >> 4;
    const int g = blockIdx.x;
    int r0[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb)
        r0[nb] = EPI == ppk::kSwiGLU ? 32 * g + 16 * nb : (g >> 2) * 128 + 64 * nb + 16 * (g & 3);
    // Consecutive workgroups are dispatched to consecutive XCDs, so the workgroups that share
    // an XCD are g, g + 8, g + 16, ...; each starts its sweep over the K segments at segment
    // (g / 8) mod NSEG.  Without the stagger all the workgroups of an XCD read the same 1 KB
    // column segment at the same moment, and the kernel's time depended on which XCD received
    // workgroup 0, which varies with the hardware queue that serves the stream: 31 to 43 us for
    // the 7B gate/up projection, against 31 us on every queue with it.
    const int rot = (g >> 3) & (NSEG - 1);
    // one descriptor over rows r0[0] .. r0[1] + 15 (80 rows at most)
    const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16*>(W + int64_t(r0[0]) * ldw), 0, static_cast<int>((int64_t(r0[1] - r0[0] + 15) * ldw + RS_COLS * NSEG) * 2),
        kRsrcWord3);
    auto issue = [&](int c) {                   // chunk c (clamped) into slot c % NW
        const int cc = c < NCH ? c : NCH - 1, sg = cc >> 1, nb = cc & 1;
        char* slot = smem + (c % NW) * RS_CHUNK_B;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int r = 4 * w + t;
            const int soff =
                static_cast<int>((int64_t(r0[nb] - r0[0] + r) * ldw + ((sg + rot) & (NSEG - 1)) * RS_COLS) * 2);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(wrs, (lds_void*)(slot + r * 1024), 16, 16 * (lane ^ rs_swz(r)),
                                                     soff, 0, 0);
        }
    };
    // the weight stream starts first; this wavefront's quarter of the prompt rows (rows past
    // k read as row k - 1; never stored) follows one segment at a time: segment 0's now,
    // segment sg + 1's at the first chunk of segment sg, so that its loads complete, in issue
    // order, with the weight chunk the next segment starts on
#pragma unroll
    for (int c = 0; c < NW - 1; ++c) issue(c);
    __builtin_amdgcn_sched_barrier(0);
    const bf16* arow = A + int64_t(min(lr, k - 1)) * lda + 128 * w + 8 * q4;
    bf16x8 pf[NSEG][4];
#pragma unroll
    for (int st = 0; st < 4; ++st) pf[0][st] = *reinterpret_cast<const bf16x8*>(arow + rot * RS_COLS + 32 * st);
    f32x4 acc[2] = {};
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        // chunk c is in when at most the loads of chunks c + 1 .. c + NW - 2 (4 each) are pending
        // (later register loads only make the wait stricter)
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(4 * (NW - 2)));
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        issue(c + NW - 1);                      // into the slot every wavefront finished at c - 1
        const char* slot = smem + (c % NW) * RS_CHUNK_B;
        const int sg = c >> 1, nb = c & 1;
        if (nb == 0 && sg + 1 < NSEG) {
#pragma unroll
            for (int st = 0; st < 4; ++st)
                pf[sg + 1][st] =
                    *reinterpret_cast<const bf16x8*>(arow + ((sg + 1 + rot) & (NSEG - 1)) * RS_COLS + 32 * st);
        }
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            const bf16x8 wf = *reinterpret_cast<const bf16x8*>(slot + lr * 1024 +
                                                               16 * ((16 * w + 4 * st + q4) ^ rs_swz(lr)));
            acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf, pf[sg][st], acc[nb], 0, 0, 0);
        }
    }
    // the clamped loads past the last chunk land before the ring's LDS is reused
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(0));
    __syncthreads();
    f32x4* red = reinterpret_cast<f32x4*>(smem);   // [w][nb][lane]
    red[(w * 2 + 0) * 64 + lane] = acc[0];
    red[(w * 2 + 1) * 64 + lane] = acc[1];
    __syncthreads();
    if (threadIdx.x < 64) {
        const int l = threadIdx.x, m = l & 15, c = 4 * (l >> 4);
        if (m < k) {
            f32x4 a = red[l], b = red[64 + l];
#pragma unroll
            for (int w2 = 1; w2 < 4; ++w2) {
                a += red[(w2 * 2) * 64 + l];
                b += red[(w2 * 2 + 1) * 64 + l];
            }
            rowpair_epilogue<EPI>(g, m, c, a, b, ep);
        }
    }
}

// The QKV projection for up to 16 prompts at K = 512 NSEG with 16 weight rows per workgroup:
// dims i0 .. i0 + 7 of a head (chunk rows 0-7) and their rotate-half partners i0 + 64 ..
// (rows 8-15).  A 7B layer's 384 groups of 32 rows become 768 workgroups, three on every CU,
// where 32-row workgroups left half the CUs with two and half with one and the busier half
// set the time.  One 16-row x 512-column chunk per K segment through the LDS ring and XCD
// stagger of rowpair_seg_kernel; lane l + 32 holds the partners of lane l's rows, exchanged
// by a lane swap before the RoPE.
template <int NSEG, int NW>
__global__ __launch_bounds__(256, 2) void qkv_seg16_kernel(const bf16* __restrict__ A, int64_t lda, int k,
                                                           const bf16* __restrict__ W, int64_t ldw,
                                                           ppk::QkvOut qo) {
    static_assert(NW >= 2 && NW * RS_CHUNK_B >= 4 * 64 * 16, "ring, and room for the reduction");
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lr = lane & 15, q4 = lane >> 4;
    const int g = blockIdx.x;
    const int head = g >> 3, i0 = 8 * (g & 7);
    const int rlo = head * 128 + i0;            // rows rlo .. rlo + 7 and rlo + 64 .. rlo + 71
    const int rot = (g >> 3) & (NSEG - 1);      // see rowpair_seg_kernel
    const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16*>(W + int64_t(rlo) * ldw), 0, static_cast<int>((71 * ldw + RS_COLS * NSEG) * 2), kRsrcWord3);
    auto issue = [&](int c) {                   // segment c (clamped) into slot c % NW
        const int sg = ((c < NSEG ? c : NSEG - 1) + rot) & (NSEG - 1);
        char* slot = smem + (c % NW) * RS_CHUNK_B;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int r = 4 * w + t;
            const int row = r < 8 ? r : 56 + r;     // 64 + (r - 8)
            const int soff = static_cast<int>((int64_t(row) * ldw + sg * RS_COLS) * 2);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(wrs, (lds_void*)(slot + r * 1024), 16, 16 * (lane ^ rs_swz(r)),
                                                     soff, 0, 0);
        }
    };
#pragma unroll
    for (int c = 0; c < NW - 1; ++c) issue(c);
    __builtin_amdgcn_sched_barrier(0);
    const bf16* arow = A + int64_t(min(lr, k - 1)) * lda + 128 * w + 8 * q4;
    bf16x8 pf[NSEG][4];
#pragma unroll
    for (int st = 0; st < 4; ++st) pf[0][st] = *reinterpret_cast<const bf16x8*>(arow + rot * RS_COLS + 32 * st);
    f32x4 acc = {};
#pragma unroll
    for (int c = 0; c < NSEG; ++c) {
        // segment c is in when at most the loads of segments c + 1 .. c + NW - 2 (4 each) are
        // pending (later register loads only make the wait stricter)
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(4 * (NW - 2)));
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        issue(c + NW - 1);                      // into the slot every wavefront finished at c - 1
        const char* slot = smem + (c % NW) * RS_CHUNK_B;
        if (c + 1 < NSEG) {
#pragma unroll
            for (int st = 0; st < 4; ++st)
                pf[c + 1][st] =
                    *reinterpret_cast<const bf16x8*>(arow + ((c + 1 + rot) & (NSEG - 1)) * RS_COLS + 32 * st);
        }
#pragma unroll
        for (int st = 0; st < 4; ++st) {
            const bf16x8 wf = *reinterpret_cast<const bf16x8*>(slot + lr * 1024 +
                                                               16 * ((16 * w + 4 * st + q4) ^ rs_swz(lr)));
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf, pf[c][st], acc, 0, 0, 0);
        }
    }
    // the clamped loads past the last segment land before the ring's LDS is reused
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(0));
    __syncthreads();
    f32x4* red = reinterpret_cast<f32x4*>(smem);   // [w][lane]
    red[w * 64 + lane] = acc;
    __syncthreads();
    if (threadIdx.x < 64) {
        const int l = threadIdx.x, m = l & 15;
        f32x4 a = red[l];
#pragma unroll
        for (int w2 = 1; w2 < 4; ++w2) a += red[w2 * 64 + l];
        f32x4 b;                                // rows 8 + 4 (l / 16) ..: the partners, from lane l + 32
#pragma unroll
        for (int e = 0; e < 4; ++e) b[e] = __shfl_xor(a[e], 32);
        if (l < 32 && m < k) qkv_pair_store(head, i0 + 4 * (l >> 4), m, a, b, qo);
    }
}

template <int NSEG, int NW>
void launch_qkv_seg16(int N, hipStream_t s, const bf16* A, int64_t lda, int k, const bf16* W, int64_t ldw,
                      const ppk::QkvOut& qo) {
    constexpr int lds = NW * RS_CHUNK_B;
    static bool attr = [] {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&qkv_seg16_kernel<NSEG, NW>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, lds);
        return true;
    }();
    (void)attr;
    qkv_seg16_kernel<NSEG, NW><<<N / 16, 256, lds, s>>>(A, lda, k, W, ldw, qo);
}

template <int EPI, int NSEG, int NW>
void launch_rowpair_seg(int N, hipStream_t s, const bf16* A, int64_t lda, int k, const bf16* W, int64_t ldw,
                        const ppk::DecodeEpi& ep) {
    constexpr int lds = NW * RS_CHUNK_B;
    static bool attr = [] {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&rowpair_seg_kernel<EPI, NSEG, NW>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, lds);
        return true;
    }();
    (void)attr;
    rowpair_seg_kernel<EPI, NSEG, NW><<<N / 32, 256, lds, s>>>(A, lda, k, W, ldw, ep);
}

// Whether rowpair_seg_kernel takes the shape: up to 16 prompts, K = 2048 or 4096.  The ring
// depth follows the grid: three workgroups of 48 KB per CU when there are more than 512 of
// them, else two of 64 KB.
template <int EPI>
bool launch_rowpair_seg_for(int N, int K, hipStream_t s, const bf16* A, int64_t lda, int k, const bf16* W,
                            int64_t ldw, const ppk::DecodeEpi& ep) {
    if (k > 16 || (K != 2048 && K != 4096)) return false;
    const bool wide = N / 32 > 512;
    if (K == 4096) {
        if (wide) launch_rowpair_seg<EPI, 8, 3>(N, s, A, lda, k, W, ldw, ep);
        else launch_rowpair_seg<EPI, 8, 4>(N, s, A, lda, k, W, ldw, ep);
    } else {
        if (wide) launch_rowpair_seg<EPI, 4, 3>(N, s, A, lda, k, W, ldw, ep);
        else launch_rowpair_seg<EPI, 4, 4>(N, s, A, lda, k, W, ldw, ep);
    }
    return true;
}

// Split-K projection for up to 16 prompts (the down projection, whose N = d leaves too few
// 32-row groups for one workgroup each), the weights streamed as 1 KB row segments as in
// rowpair_seg_kernel: workgroup (g, s) takes rows 32 g .. + 31 and split s of the K / 512
// segments (splits differ by at most one segment, none holds more than S), two 16-row blocks
// per segment through an LDS ring of NW chunks, and leaves float32 partial sums
// part[s][m][n] for residual_rmsnorm to add in split order.  When K ends in part of a segment
// (K % 512 = 128, 256 or 384), the 16-byte pieces past K of that segment's rows read pieces
// inside it instead and the prompt columns past K are zeros, so those weights add exact
// zeros.  Chunks past a short split's segments re-read its last one (in bounds, never used,
// and just loaded: L2 hits), which keeps 4 loads per chunk step for the fixed wait counts.
template <int S, int NW>
__global__ __launch_bounds__(256, 2) void splitk_seg_kernel(const bf16* __restrict__ A, int64_t lda, int k,
                                                            const bf16* __restrict__ W, int64_t ldw, int N, int K,
                                                            float* __restrict__ part) {
    static_assert(NW >= 2 && NW * RS_CHUNK_B >= 4 * 2 * 64 * 16, "ring, and room for the reduction");
    constexpr int NCH = 2 * S;
    extern __shared__ __attribute__((aligned(16))) char smem[];
    const int lane = threadIdx.x & 63;
    const int w = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lr = lane & 15, q4 = lane >> 4;
    const int g = blockIdx.x, sp = blockIdx.y, splits = gridDim.y;
    const int nseg = (K + RS_COLS - 1) / RS_COLS;
    const int tail = K - (nseg - 1) * RS_COLS;   // columns of the last segment: 128 .. 512
    const int s_lo = sp * nseg / splits, n_here = (sp + 1) * nseg / splits - s_lo;   // 1 .. S
    // the workgroups that share an XCD (consecutive linear ids go to consecutive XCDs) start
    // their sweeps at different segments of the split
    const int rot = ((g + gridDim.x * sp) >> 3) % n_here;
    const int r0 = 32 * g;
    const __amdgpu_buffer_rsrc_t wrs = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<bf16*>(W + int64_t(r0) * ldw), 0, static_cast<int>((31 * ldw + K) * 2), kRsrcWord3);
    auto seg_of = [&](int sl) {               // the segment the split's sl-th chunk pair reads
        if (sl >= n_here) sl = n_here - 1;    // past a short split: its last segment, still in L2
        const int p = sl + rot;
        return s_lo + (p >= n_here ? p - n_here : p);
    };
    auto issue = [&](int c) {                 // chunk c (clamped) into slot c % NW
        const int cc = c < NCH ? c : NCH - 1, sl = cc >> 1, nb = cc & 1;
        const int sg = seg_of(sl);
        const int qv = sg == nseg - 1 ? tail / 8 : 64;   // 16-byte pieces inside K
        char* slot = smem + (c % NW) * RS_CHUNK_B;
#pragma unroll
        for (int t = 0; t < 4; ++t) {
            const int r = 4 * w + t;
            const int soff = static_cast<int>((int64_t(16 * nb + r) * ldw + int64_t(sg) * RS_COLS) * 2);
            const int q = lane ^ rs_swz(r);
            __builtin_amdgcn_raw_ptr_buffer_load_lds(wrs, (lds_void*)(slot + r * 1024), 16, 16 * (q < qv ? q : q & 15),
                                                     soff, 0, 0);
        }
    };
    // this wavefront's quarter of the prompt rows for the split's sl-th segment (rows past k
    // read as row k - 1, never stored; columns past K as zeros)
    const bf16* arow = A + int64_t(min(lr, k - 1)) * lda + 128 * w + 8 * q4;
    auto prompt = [&](int sl, bf16x8* f) {
        const int sg = seg_of(sl);
        const bool past = sl >= n_here || (sg == nseg - 1 && 128 * w >= tail);
#pragma unroll
        for (int st = 0; st < 4; ++st)
            f[st] = past ? bf16x8{} : *reinterpret_cast<const bf16x8*>(arow + int64_t(sg) * RS_COLS + 32 * st);
    };
#pragma unroll
    for (int c = 0; c < NW - 1; ++c) issue(c);
    __builtin_amdgcn_sched_barrier(0);
    bf16x8 pf[S][4];
    prompt(0, pf[0]);
    f32x4 acc[2] = {};
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        // chunk c is in when at most the loads of chunks c + 1 .. c + NW - 2 (4 each) are pending
        // (later register loads only make the wait stricter)
        __builtin_amdgcn_sched_barrier(0);
        __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(4 * (NW - 2)));
        __builtin_amdgcn_s_barrier();
        __builtin_amdgcn_sched_barrier(0);
        issue(c + NW - 1);                    // into the slot every wavefront finished at c - 1
        const char* slot = smem + (c % NW) * RS_CHUNK_B;
        const int sl = c >> 1, nb = c & 1;
        if (nb == 0 && sl + 1 < S) prompt(sl + 1, pf[sl + 1]);
        if (sl < n_here) {
#pragma unroll
            for (int st = 0; st < 4; ++st) {
                const bf16x8 wf = *reinterpret_cast<const bf16x8*>(slot + lr * 1024 +
                                                                   16 * ((16 * w + 4 * st + q4) ^ rs_swz(lr)));
                acc[nb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wf, pf[sl][st], acc[nb], 0, 0, 0);
            }
        }
    }
    // the clamped loads past the last chunk land before the ring's LDS is reused
    __builtin_amdgcn_sched_barrier(0);
    __builtin_amdgcn_s_waitcnt(wait_vm_lgkm0(0));
    __syncthreads();
    f32x4* red = reinterpret_cast<f32x4*>(smem);   // [w][nb][lane]
    red[(w * 2 + 0) * 64 + lane] = acc[0];
    red[(w * 2 + 1) * 64 + lane] = acc[1];
    __syncthreads();
    if (threadIdx.x < 64) {
        const int l = threadIdx.x, m = l & 15, c = 4 * (l >> 4);
        if (m < k) {
            f32x4 a = red[l], b = red[64 + l];
#pragma unroll
            for (int w2 = 1; w2 < 4; ++w2) {
                a += red[(w2 * 2) * 64 + l];
                b += red[(w2 * 2 + 1) * 64 + l];
            }
            float* dst = part + (int64_t(sp) * k + m) * N + r0 + c;
            *reinterpret_cast<f32x4*>(dst) = a;
            *reinterpret_cast<f32x4*>(dst + 16) = b;
        }
    }
}

template <int S, int NW>
void launch_splitk_seg(int N, int splits, hipStream_t s, const bf16* A, int64_t lda, int k, const bf16* W,
                       int64_t ldw, int K, float* part) {
    constexpr int lds = NW * RS_CHUNK_B;
    static bool attr = [] {
        (void)hipFuncSetAttribute(reinterpret_cast<const void*>(&splitk_seg_kernel<S, NW>),
                                  hipFuncAttributeMaxDynamicSharedMemorySize, lds);
        return true;
    }();
    (void)attr;
    splitk_seg_kernel<S, NW><<<dim3(N / 32, splits), 256, lds, s>>>(A, lda, k, W, ldw, N, K, part);
}

// splitk_seg_kernel's split: the most segments per split (4, 2 or 1) that still gives at least
// 256 workgroups (at the 7B shape 4 segments, 768 workgroups, three per CU; at 1.3B 2, 384:
// 1 segment per workgroup and 8 per split were slower there, as were 4-chunk rings); s = 0
// when the kernel does not take the shape (more than 16 prompts, N % 32 or K % 128 not zero).
struct SegSplit {
    int s, splits;
};
SegSplit seg_split(int k, int N, int K) {
    if (k < 1 || k > 16 || N % 32 != 0 || K % 128 != 0 || K <= 0) return SegSplit{0, 0};
    const int nseg = (K + RS_COLS - 1) / RS_COLS, groups = N / 32;
    int s = 4, splits = (nseg + 3) / 4;
    while (s > 1 && groups * splits < 256) {
        s /= 2;
        splits = (nseg + s - 1) / s;
    }
    return SegSplit{s, splits};
}

template <int EPI>
void launch_rowpair(int nmb, int N, hipStream_t s, const bf16* A, int64_t lda, int k, const bf16* W, int64_t ldw,
                    int K, const ppk::DecodeEpi& ep) {
    const dim3 grid(N / 32);
    switch (nmb) {
        case 1: rowpair_gemm_kernel<EPI, 1><<<grid, 256, 0, s>>>(A, lda, k, W, ldw, K, ep); break;
        case 2: rowpair_gemm_kernel<EPI, 2><<<grid, 256, 0, s>>>(A, lda, k, W, ldw, K, ep); break;
        case 3: rowpair_gemm_kernel<EPI, 3><<<grid, 256, 0, s>>>(A, lda, k, W, ldw, K, ep); break;
        default: rowpair_gemm_kernel<EPI, 4><<<grid, 256, 0, s>>>(A, lda, k, W, ldw, K, ep); break;
    }
}

// Residual add of a split-K projection fused with the RMSNorm that follows it, one workgroup
// of d / (4 E) threads per prompt row, 4 E consecutive elements per thread (E = 1 up to
// d = 4096, 2 up to 8192): x[m] += sum over splits of part[.][m], added in split order, stored
// back; then out[m] = x[m] / sqrt(mean(x[m]^2) + eps) * g.  S = 0: no pending projection.
// The kernel is latency-bound (k workgroups, a few KB each), so everything it reads (the row,
// the gains, up to 8 splits' partial sums) is issued before the first wait: one memory round
// trip where S <= 8 rather than one per split.
template <typename TO, int E>
__global__ __launch_bounds__(1024) void residual_rmsnorm_kernel(float* __restrict__ x, const float* __restrict__ part,
                                                                int S, int k, int d, const float* __restrict__ g,
                                                                TO* __restrict__ out, float eps) {
    __shared__ float red[16];
    const int m = blockIdx.x, c = 4 * E * threadIdx.x;
    float* xr = x + int64_t(m) * d + c;
    f32x4 v[E], gg[E];
#pragma unroll
    for (int e = 0; e < E; ++e) {
        v[e] = *reinterpret_cast<const f32x4*>(xr + 4 * e);
        gg[e] = *reinterpret_cast<const f32x4*>(g + c + 4 * e);
    }
    if (S > 0) {
        const float* p = part + int64_t(m) * d + c;
        const int64_t stride = int64_t(k) * d;
        for (int s = 0; s < S; s += 8) {
            f32x4 a[8][E];
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (s + u < S)
#pragma unroll
                    for (int e = 0; e < E; ++e) a[u][e] = *reinterpret_cast<const f32x4*>(p + (s + u) * stride + 4 * e);
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (s + u < S)
#pragma unroll
                    for (int e = 0; e < E; ++e) v[e] += a[u][e];
        }
#pragma unroll
        for (int e = 0; e < E; ++e) *reinterpret_cast<f32x4*>(xr + 4 * e) = v[e];
    }
    float ss = 0.f;
#pragma unroll
    for (int e = 0; e < E; ++e)
#pragma unroll
        for (int i = 0; i < 4; ++i) ss = fmaf(v[e][i], v[e][i], ss);
    ss = wave_sum(ss);
    const int nw = blockDim.x / 64;
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = ss;
    __syncthreads();
    float tot = 0.f;
    for (int i = 0; i < nw; ++i) tot += red[i];
    const float r = rsqrtf(tot / static_cast<float>(d) + eps);
#pragma unroll
    for (int e = 0; e < E; ++e) {
        if constexpr (sizeof(TO) == 2) {
            bf16x4 o;
#pragma unroll
            for (int i = 0; i < 4; ++i) o[i] = static_cast<bf16>(v[e][i] * r * gg[e][i]);
            *reinterpret_cast<bf16x4*>(out + int64_t(m) * d + c + 4 * e) = o;
        } else {
            *reinterpret_cast<f32x4*>(out + int64_t(m) * d + c + 4 * e) = v[e] * r * gg[e];
        }
    }
}

template <int NT, bool COMB>
void launch_skinny_nt(int nmb, dim3 grid, size_t lds, hipStream_t s, const bf16* A, int64_t lda, int k,
                      const bf16* W, int64_t ldw, int N, int K, float* part, const ppk::AttnChunks& ac) {
    // the staged slice of A takes NT x 16 nmb rows x 256 bytes: up to 96 KB, past the 64 KB
    // a launch gets without asking
    static const bool attr = [] {
        auto allow = [](const void* f, int nmb_) {
            (void)hipFuncSetAttribute(f, hipFuncAttributeMaxDynamicSharedMemorySize, NT * 16 * nmb_ * 256);
        };
        allow(reinterpret_cast<const void*>(&skinny_gemm_kernel<NT, 1, COMB>), 1);
        allow(reinterpret_cast<const void*>(&skinny_gemm_kernel<NT, 2, COMB>), 2);
        allow(reinterpret_cast<const void*>(&skinny_gemm_kernel<NT, 3, COMB>), 3);
        allow(reinterpret_cast<const void*>(&skinny_gemm_kernel<NT, 4, COMB>), 4);
        return true;
    }();
    (void)attr;
    switch (nmb) {
        case 1: skinny_gemm_kernel<NT, 1, COMB><<<grid, 256, lds, s>>>(A, lda, k, W, ldw, N, K, part, ac); break;
        case 2: skinny_gemm_kernel<NT, 2, COMB><<<grid, 256, lds, s>>>(A, lda, k, W, ldw, N, K, part, ac); break;
        case 3: skinny_gemm_kernel<NT, 3, COMB><<<grid, 256, lds, s>>>(A, lda, k, W, ldw, N, K, part, ac); break;
        default: skinny_gemm_kernel<NT, 4, COMB><<<grid, 256, lds, s>>>(A, lda, k, W, ldw, N, K, part, ac); break;
    }
}

template <bool COMB>
void launch_skinny(int nt, int nmb, dim3 grid, hipStream_t s, const bf16* A, int64_t lda, int k, const bf16* W,
                   int64_t ldw, int N, int K, float* part, const ppk::AttnChunks& ac) {
    const size_t lds = size_t(nt) * 16 * nmb * 256;
    switch (nt) {
        case 1: launch_skinny_nt<1, COMB>(nmb, grid, lds, s, A, lda, k, W, ldw, N, K, part, ac); break;
        case 2: launch_skinny_nt<2, COMB>(nmb, grid, lds, s, A, lda, k, W, ldw, N, K, part, ac); break;
        case 3: launch_skinny_nt<3, COMB>(nmb, grid, lds, s, A, lda, k, W, ldw, N, K, part, ac); break;
        case 4: launch_skinny_nt<4, COMB>(nmb, grid, lds, s, A, lda, k, W, ldw, N, K, part, ac); break;
        case 5: launch_skinny_nt<5, COMB>(nmb, grid, lds, s, A, lda, k, W, ldw, N, K, part, ac); break;
        default: launch_skinny_nt<6, COMB>(nmb, grid, lds, s, A, lda, k, W, ldw, N, K, part, ac); break;
    }
}

template <typename T, int D, int R>
void launch_attn(const void* q, int64_t ldq, const void* ctx_k, const void* ctx_v, const void* gen_k,
                 const void* gen_v, int64_t ldkv, const ppk::DecodeLayout& Ly, int step, int Hkv, float* part,
                 hipStream_t s) {
    // the work list when it is shorter than every prompt's n_ctx_chunks: one workgroup per item
    // and key/value head (the kernel loops over any items past the grid's 65535 rows)
    const bool list = Ly.n_ctx_items < int64_t(Ly.k) * Ly.n_ctx_chunks;
    const int64_t items = int64_t(Ly.k) * Ly.n_gen_chunks + Ly.n_ctx_items;
    const dim3 grid = list ? dim3(Hkv, static_cast<unsigned>(std::min<int64_t>(items, 65535)))
                           : dim3(Ly.k * Hkv, Ly.n_ctx_chunks + Ly.n_gen_chunks);
    decode_attn_kernel<T, D, R><<<grid, 256, 0, s>>>(
        static_cast<const T*>(q), ldq, static_cast<const T*>(ctx_k), static_cast<const T*>(ctx_v),
        static_cast<const T*>(gen_k), static_cast<const T*>(gen_v), ldkv, Ly.ctx_off, Ly.ctx_span, Ly.ctx_valid,
        Ly.gen_off, step, Ly.k, Hkv, Ly.n_ctx_chunks, Ly.n_gen_chunks, list ? 1 : 0, part);
}

template <typename T, int D>
void attn_by_group(int R, const void* q, int64_t ldq, const void* ctx_k, const void* ctx_v, const void* gen_k,
                   const void* gen_v, int64_t ldkv, const ppk::DecodeLayout& Ly, int step, int Hkv, float* part,
                   hipStream_t s) {
    switch (R) {
        case 1: launch_attn<T, D, 1>(q, ldq, ctx_k, ctx_v, gen_k, gen_v, ldkv, Ly, step, Hkv, part, s); break;
        case 2: launch_attn<T, D, 2>(q, ldq, ctx_k, ctx_v, gen_k, gen_v, ldkv, Ly, step, Hkv, part, s); break;
        case 4: launch_attn<T, D, 4>(q, ldq, ctx_k, ctx_v, gen_k, gen_v, ldkv, Ly, step, Hkv, part, s); break;
        default: launch_attn<T, D, 8>(q, ldq, ctx_k, ctx_v, gen_k, gen_v, ldkv, Ly, step, Hkv, part, s); break;
    }
}

template <typename T>
void attn_dispatch(int D, int R, const void* q, int64_t ldq, const void* ctx_k, const void* ctx_v,
                   const void* gen_k, const void* gen_v, int64_t ldkv, const ppk::DecodeLayout& Ly, int step,
                   int Hkv, float* part, void* out, int64_t ldo, hipStream_t s) {
    const int H = Hkv * R;
    const int blocks = (Ly.k * H + 3) / 4;
    const int nch = Ly.n_ctx_chunks + Ly.n_gen_chunks;
    if (D == 128) {
        attn_by_group<T, 128>(R, q, ldq, ctx_k, ctx_v, gen_k, gen_v, ldkv, Ly, step, Hkv, part, s);
        if (!out) return;   // the consumer merges the chunks itself
        decode_combine_kernel<T, 128><<<blocks, 256, 0, s>>>(part, Ly.k, H, Ly.ctx_span, step, Ly.n_ctx_chunks, nch,
                                                             static_cast<T*>(out), ldo);
    } else {
        attn_by_group<T, 64>(R, q, ldq, ctx_k, ctx_v, gen_k, gen_v, ldkv, Ly, step, Hkv, part, s);
        decode_combine_kernel<T, 64><<<blocks, 256, 0, s>>>(part, Ly.k, H, Ly.ctx_span, step, Ly.n_ctx_chunks, nch,
                                                            static_cast<T*>(out), ldo);
    }
}

}  // namespace

namespace ppk {

void decode_prep(const DecodeLayout& Ly, int step, int D, float theta, float2* table, int32_t* slot_pos,
                 int32_t* slot_kv, int32_t* slot_seg, int32_t* ident, hipStream_t s) {
    decode_prep_kernel<<<Ly.k, 64, 0, s>>>(Ly.k, step, Ly.pos0, Ly.gen_off, D, static_cast<double>(theta), table,
                                           slot_pos, slot_kv, slot_seg, ident);
}

void decode_attention(int dtype, const void* q, int64_t ldq, const void* ctx_k, const void* ctx_v,
                      const void* gen_k, const void* gen_v, int64_t ldkv, const DecodeLayout& Ly, int step, int H,
                      int Hkv, int D, float* part, void* out, int64_t ldo, hipStream_t s) {
    const int R = H / Hkv;
    if (dtype == PP_BF16)
        attn_dispatch<bf16>(D, R, q, ldq, ctx_k, ctx_v, gen_k, gen_v, ldkv, Ly, step, Hkv, part, out, ldo, s);
    else
        attn_dispatch<float>(D, R, q, ldq, ctx_k, ctx_v, gen_k, gen_v, ldkv, Ly, step, Hkv, part, out, ldo, s);
}

SkinnySplit skinny_split(int N, int K) {
    const int tiles = K / SG_TILE, groups = N / SG_ROWS;
    const int target = std::max(1, (512 + groups - 1) / groups);   // about 512 workgroups (1024, 2048: slower)
    const int per = std::min(SG_MAX_TILES, std::max(1, (tiles + target - 1) / target));
    return SkinnySplit{per, (tiles + per - 1) / per};
}

int decode_gemm_splits(int k, int N, int K) {
    const SegSplit ss = seg_split(k, N, K);
    return ss.s ? ss.splits : skinny_split(N, K).splits;
}

bool skinny_ok(int k, int N, int K) { return k >= 1 && k <= 64 && N % SG_ROWS == 0 && K % SG_TILE == 0; }

void residual_rmsnorm(int dtype_out, float* x, const float* part, int S, int k, int d, const float* g, void* out,
                      float eps, hipStream_t s) {
    // whole wavefronts, at most 1024 threads: d % 256 == 0 up to 4096 (4 elements per thread),
    // d % 512 == 0 up to 8192 (8), as residual_rmsnorm_ok checks
    if (d <= 4096) {
        const int threads = d / 4;
        if (dtype_out == PP_BF16)
            residual_rmsnorm_kernel<bf16, 1><<<k, threads, 0, s>>>(x, part, S, k, d, g, static_cast<bf16*>(out), eps);
        else
            residual_rmsnorm_kernel<float, 1><<<k, threads, 0, s>>>(x, part, S, k, d, g, static_cast<float*>(out), eps);
    } else {
        const int threads = d / 8;
        if (dtype_out == PP_BF16)
            residual_rmsnorm_kernel<bf16, 2><<<k, threads, 0, s>>>(x, part, S, k, d, g, static_cast<bf16*>(out), eps);
        else
            residual_rmsnorm_kernel<float, 2><<<k, threads, 0, s>>>(x, part, S, k, d, g, static_cast<float*>(out), eps);
    }
}

bool residual_rmsnorm_ok(int d) { return d > 0 && (d <= 4096 ? d % 256 == 0 : d <= 8192 && d % 512 == 0); }

void decode_gemm(int epi, const void* A, int64_t lda, int k, const void* W, int64_t ldw, int N, int K, float* part,
                 const DecodeEpi& ep, hipStream_t s) {
    const int nmb = (k + 15) / 16;
    const bf16* a = static_cast<const bf16*>(A);
    const bf16* w = static_cast<const bf16*>(W);
    if (epi == kSwiGLU) {
        if (!launch_rowpair_seg_for<kSwiGLU>(N, K, s, a, lda, k, w, ldw, ep))
            launch_rowpair<kSwiGLU>(nmb, N, s, a, lda, k, w, ldw, K, ep);
        return;
    }
    if (epi == kQkvRope) {
        // 16-row workgroups when the 32-row groups outnumber the CUs (7B: 384 groups become 768
        // workgroups, 21.4 -> 20.5 us); with fewer groups (Mistral-7B and 1.3B: 192) the 32-row
        // kernel is faster (16 rows: 2.6% and 3.7% slower steps)
        if (k <= 16 && (K == 2048 || K == 4096) && N / 32 > 256) {
            if (K == 4096) launch_qkv_seg16<8, 3>(N, s, a, lda, k, w, ldw, ep.qkv);
            else launch_qkv_seg16<4, 3>(N, s, a, lda, k, w, ldw, ep.qkv);
            return;
        }
        if (!launch_rowpair_seg_for<kQkvRope>(N, K, s, a, lda, k, w, ldw, ep))
            launch_rowpair<kQkvRope>(nmb, N, s, a, lda, k, w, ldw, K, ep);
        return;
    }
    // kResidual: split-K partial sums, added to the residual stream by residual_rmsnorm
    const SegSplit ss = seg_split(k, N, K);
    switch (ss.s) {
        case 4: return launch_splitk_seg<4, 3>(N, ss.splits, s, a, lda, k, w, ldw, K, part);
        case 2: return launch_splitk_seg<2, 3>(N, ss.splits, s, a, lda, k, w, ldw, K, part);
        case 1: return launch_splitk_seg<1, 3>(N, ss.splits, s, a, lda, k, w, ldw, K, part);
        default: break;   // s = 0: the skinny kernel
    }
    const SkinnySplit sp = skinny_split(N, K);
    const AttnChunks none{};
    launch_skinny<false>(sp.tiles_per_split, nmb, dim3(N / SG_ROWS, sp.splits), s, a, lda, k, w, ldw, N, K, part,
                         none);
}

void decode_gemm_o(int k, const AttnChunks& ac, const void* W, int64_t ldw, int N, int K, float* part,
                   hipStream_t s) {
    const SkinnySplit sp = skinny_split(N, K);
    launch_skinny<true>(sp.tiles_per_split, (k + 15) / 16, dim3(N / SG_ROWS, sp.splits), s, nullptr, 0, k,
                        static_cast<const bf16*>(W), ldw, N, K, part, ac);
}

}  // namespace ppk
