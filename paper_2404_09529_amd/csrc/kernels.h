// Host-side launchers of the gfx950 kernels (one translation unit per kernel family).
// Element types: dtype == PP_F32 -> float, PP_BF16 -> __bf16.  All launches are
// asynchronous on `s`; callers check hipGetLastError once after enqueuing.
#pragma once
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace ppk {

// cos/sin(p * theta^(-2i/D)) for p < P, i < D/2, evaluated in float64, stored float2 [P][D/2].
void rope_table(float2* table, int P, int D, float theta, hipStream_t s);

// x[t] = E[tokens[slot_kv[t]]] (float32), or 0 where slot_kv[t] < 0 or the id is not in [0, vocab).
void embed(int dtype, float* x, const void* E, int vocab, const int32_t* tokens, const int32_t* slot_kv,
           int T, int d, hipStream_t s);

// out[t] = x[t] / sqrt(mean(x[t]^2) + eps) * g, stored in dtype.
void rmsnorm(int dtype, const float* x, const float* g, void* out, int T, int d, float eps, hipStream_t s);

// hidden[slot_kv[t]] = RMSNorm(x[t]) * g (float32) for every slot with slot_kv[t] >= 0.
void rmsnorm_unpack(const float* x, const float* g, float* hidden, const int32_t* slot_kv, int T, int d,
                    float eps, hipStream_t s);

// Rotate-half RoPE, in place, on the first n_heads_rot heads of every row of qkv (row
// stride ld elements) at position slot_pos[t]; rows with slot_seg[t] < 0 are skipped.
void rope_apply(int dtype, void* qkv, int64_t ld, const float2* table, const int32_t* slot_pos,
                const int32_t* slot_seg, int T, int n_heads_rot, int D, hipStream_t s);

// kc[slot_kv[t]] = qkv[t][k_col : k_col+kvw], vc[slot_kv[t]] = qkv[t][k_col+kvw : k_col+2kvw].
void kv_scatter(int dtype, const void* qkv, int64_t ld, int k_col, int kvw, void* kc, void* vc,
                const int32_t* slot_kv, int T, hipStream_t s);

// act[t][f] = SiLU(gu[t][g(f)]) * gu[t][g(f) + 16], g(f) = 32 (f / 16) + f % 16 (float32 path).
void swiglu_f32(const float* gu, float* act, int T, int F, hipStream_t s);

// Epilogues of the projection GEMMs C = A B^T (A [M, K] activations, B [N, K] weights).
enum Epilogue { kStore = 0, kResidual = 1, kSwiGLU = 2, kQkvRope = 3 };

// Destinations of the kQkvRope epilogue.  B is the stacked [Wq; Wk; Wv] with head dim 128;
// q [M, ldq] receives the rotated queries, kc / vc [*, ldkv] the rotated keys and the values
// of every slot with slot_kv >= 0 at row slot_kv.  Rotation angles come from table
// (float2 [positions][64]) at slot_pos (0 for slots outside every span).
struct QkvOut {
    void* q;
    int64_t ldq;
    void* kc;
    void* vc;
    int64_t ldkv;
    const float2* table;
    const int32_t* slot_pos;
    const int32_t* slot_kv;
    int H, Hkv;
};

// bf16 MFMA GEMM.  kStore: C bf16 [M, ldc]; kResidual: C float32 [M, ldc] += A B^T;
// kSwiGLU: B rows interleaved in blocks of 16 (gate, up) and C bf16 [M, ldc] holds
// SiLU(gate) * up.  With mtile_m0 only the n_mtiles 256-row tiles starting at those rows are
// computed (a plan's row-tile list); without it every row.  Requires N % 256 == 0 and
// K % 64 == 0.
void gemm_bf16(int epi, const void* A, int64_t lda, const void* B, int64_t ldb, void* C, int64_t ldc,
               int M, int N, int K, const int32_t* mtile_m0, int n_mtiles, hipStream_t s);

// The QKV projection with RoPE and the cache UNPACK in its epilogue (kQkvRope);
// N = (H + 2 Hkv) * 128; row tiles as gemm_bf16.
void qkv_rope_bf16(const void* A, int64_t lda, const void* B, int64_t ldb, int M, int K,
                   const int32_t* mtile_m0, int n_mtiles, const QkvOut& out, hipStream_t s);

// float32 FMA GEMM (kStore / kResidual).  Requires K % 16 == 0.
void gemm_f32(int epi, const float* A, int64_t lda, const float* B, int64_t ldb, float* C, int64_t ldc,
              int M, int N, int K, hipStream_t s);

// Attention over segments (independent mask): for every query slot of every work-list
// tile, softmax(q k^T / sqrt(D)) v over the keys of its own segment at or before it.
// q [slots, ldq] (H heads of D = 128); keys and values of segment s are rows
// prompt_kv_off[seg_prompt[s]] + j of kc / vc [*, ldkv], zero past the prompt's length.
void attention_bf16(const void* q, int64_t ldq, const void* kc, const void* vc, int64_t ldkv, void* out,
                    int64_t ldo, const int32_t* seg_prompt, const int32_t* seg_start, const int32_t* seg_len,
                    const int32_t* prompt_kv_off, const int32_t* qtile_seg, const int32_t* qtile_q0, int n_qtiles,
                    int H, int Hkv, hipStream_t s);

// float32 attention, one wavefront per (slot, head), same operands; slots outside every
// span are skipped.
void attention_f32(const float* q, int64_t ldq, const float* kc, const float* vc, int64_t ldkv, float* out,
                   int64_t ldo, const int32_t* slot_seg, const int32_t* seg_prompt, const int32_t* seg_start,
                   const int32_t* prompt_kv_off, int T, int H, int Hkv, int D, hipStream_t s);

// First token (greedy) of each of k prompts: logits[m][v] = hidden[prompt_kv_off[m+1]-1] .
// lm_head[v] (hidden row rounded to dtype; float32 accumulation), tokens[m] = argmax over v,
// lowest v on ties, -1 if every logit is NaN.  lm_head [V, d] in dtype; logits [k, V] float32
// or null; workspace of first_token_workspace(dtype, k, V, d) bytes, 256-byte aligned.
// bf16: d % 128 == 0.
size_t first_token_workspace(int dtype, int k, int V, int d);
void first_token(int dtype, const float* hidden, const int32_t* prompt_kv_off, int k, const void* lm_head, int V,
                 int d, void* workspace, float* logits, int32_t* tokens, hipStream_t s);
// The current GPU's copy of the static PP_FIRST_TOKEN_SCRATCH_BYTES workspace of
// pp_first_token_noalloc (its address looked up once per device).
hipError_t first_token_scratch(void** ptr);

// ---------------------------------------------------------------------- generation (decode)
constexpr int kDecodeChunk = 128;   // keys per workgroup of the decode attention

// Device view of a generation layout (pp_gen_dlayout) with the chunk counts of its keys:
// n_ctx_chunks = ceil(max_len / kDecodeChunk), n_gen_chunks = ceil(n_new / kDecodeChunk), and
// n_ctx_items >= the context chunks of all prompts together (the decode attention's grid;
// any it leaves out are taken by a second pass of its workgroups).
struct DecodeLayout {
    int k, n_ctx_chunks, n_gen_chunks, n_ctx_items;
    const int32_t *ctx_off, *ctx_span, *ctx_valid, *pos0, *gen_off;
};

// Per prompt i < k for decode step `step`: table[i] = cos/sin((pos0[i] + step) theta^(-2j/D))
// for j < D/2 (float64, float2 [k][D/2]); slot_pos[i] = i; slot_kv[i] = gen_off[i] + step;
// slot_seg[i] = 0; ident[i] = i for i <= k (k + 1 entries).
void decode_prep(const DecodeLayout& Ly, int step, int D, float theta, float2* table, int32_t* slot_pos,
                 int32_t* slot_kv, int32_t* slot_seg, int32_t* ident, hipStream_t s);

// The decode attention's per-chunk results (k x H x n_chunks x (D + 4) float32: o[D], max,
// sum) and what is needed to merge a prompt's chunks.
struct AttnChunks {
    const float* part;
    const int32_t* ctx_span;
    int step, n_ctx_chunks, n_chunks, H;
};

// One query row per prompt (q [k, ldq], H heads of D) against the prompt's context rows
// ctx_off[i] .. + ctx_span[i] of ctx_k / ctx_v (rows past ctx_valid[i] masked) and its
// generated rows gen_off[i] .. + step of gen_k / gen_v; row stride ldkv; GQA head h reads
// key/value head h / (H / Hkv).  out [k, ldo] = softmax(q k^T / sqrt(D)) v, dtype.
// part: float32 scratch of k * H * (n_ctx_chunks + n_gen_chunks) * (D + 4).  out == NULL:
// the chunk results are left in part for decode_gemm_o to merge.
// D in {64, 128}; H / Hkv in {1, 2, 4, 8}.
void decode_attention(int dtype, const void* q, int64_t ldq, const void* ctx_k, const void* ctx_v,
                      const void* gen_k, const void* gen_v, int64_t ldkv, const DecodeLayout& Ly, int step, int H,
                      int Hkv, int D, float* part, void* out, int64_t ldo, hipStream_t s);

// Destination of a decode-step projection: `out` with row stride `ldo` (kResidual: float32
// x += ..., kSwiGLU: bf16 [k, N/2]), or the QKV outputs (kQkvRope, head dim 128).
struct DecodeEpi {
    void* out;
    int64_t ldo;
    QkvOut qkv;
};

// K split of the skinny GEMM: `splits` pieces of `tiles_per_split` 128-column tiles.
struct SkinnySplit {
    int tiles_per_split, splits;
};
SkinnySplit skinny_split(int N, int K);
// Shapes the skinny GEMM takes: 1 <= k <= 64 rows, N % 64 == 0, K % 128 == 0.
bool skinny_ok(int k, int N, int K);

// The O projection of a decode step (bf16, head dim 128, k <= 64): its activations are the
// attention output, merged from the attention's chunk results while they are staged; float32
// split-K partial sums in part for residual_rmsnorm, as decode_gemm's kResidual.
void decode_gemm_o(int k, const AttnChunks& ac, const void* W, int64_t ldw, int N, int K, float* part,
                   hipStream_t s);

// x[m] += sum of the S splits of part (split order; S = 0: nothing), stored back, then
// out[m] = RMSNorm(x[m]) * g in dtype_out (PP_BF16 or PP_F32); k rows of d <= 4096.
void residual_rmsnorm(int dtype_out, float* x, const float* part, int S, int k, int d, const float* g, void* out,
                      float eps, hipStream_t s);
// Widths residual_rmsnorm takes: d % 256 == 0 up to 4096, d % 512 == 0 up to 8192.
bool residual_rmsnorm_ok(int d);

// bf16 C = A W^T for k <= 64 rows (A [k, lda], W [N, ldw]) with the epilogue `epi`:
// kSwiGLU and kQkvRope in the GEMM kernel itself (N % 32 == 0); kResidual leaves float32
// partial sums in part (decode_gemm_splits(k, N, K) * k * N floats) for residual_rmsnorm to
// add.
void decode_gemm(int epi, const void* A, int64_t lda, int k, const void* W, int64_t ldw, int N, int K, float* part,
                 const DecodeEpi& ep, hipStream_t s);
// The number of K splits decode_gemm's kResidual leaves for k rows of an N x K product.
int decode_gemm_splits(int k, int N, int K);

}  // namespace ppk
