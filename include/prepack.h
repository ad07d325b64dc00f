/*
 * prepack.h -- C ABI of the packed-prefill library for AMD Instinct MI355X (gfx950).
 *
 * Method: Prepacking (Zhao, Israel, Van den Broeck, Grover, 2024).  Prompts of
 * different lengths are bin-packed into fixed-length rows (section 3.1), the
 * decoder runs over the rows with an independent block-diagonal causal mask
 * and positions that restart at every prompt (section 3.2), and the KV cache
 * of every prompt is unpacked into its own contiguous rows (Algorithm 1).
 *
 * Conventions for every call:
 *   - returns a pp_status; PP_OK (0) on success, a negative code otherwise, with
 *     a message for the calling thread available from pp_last_error();
 *   - no exception, abort or exit crosses the ABI;
 *   - the library allocates nothing and keeps no state between calls: every
 *     buffer, host or device, belongs to the caller (one exception: the static
 *     device buffer behind pp_first_token_noalloc);
 *   - "device pointer" means memory of the current HIP device; "host pointer"
 *     means ordinary process memory.
 */
#ifndef PREPACK_H
#define PREPACK_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum pp_status {
    PP_OK = 0,
    PP_ERR_INVALID_ARG = -1,      /* NULL pointer, negative count, length <= 0, bad config      */
    PP_ERR_TOO_LONG = -2,         /* a prompt longer than the row capacity                       */
    PP_ERR_BUFFER_TOO_SMALL = -3, /* a caller buffer (plan arrays, workspace) is too small        */
    PP_ERR_UNSUPPORTED = -4,      /* shape the kernels do not implement (see pp_prefill)          */
    PP_ERR_HIP = -5               /* the HIP runtime reported an error while enqueuing            */
} pp_status;

typedef enum pp_dtype { PP_F32 = 0, PP_BF16 = 1 } pp_dtype;

/* Query-tile length of the attention work list carried in a plan. */
#define PP_QTILE 128

/* Row-tile length (slots) of the projection GEMMs' tile list carried in a plan. */
#define PP_MTILE 256

/* Text for the last non-OK status returned on the calling thread ("" if none). */
const char* pp_last_error(void);

/* Library version string, e.g. "0.1.0 gfx950". */
const char* pp_version(void);

/* ------------------------------------------------------------------------------------------
 * Plan: where every token of the packed batch sits (host memory).
 *
 * The packed batch B of Algorithm 1 is n_rows rows of `capacity` slots; slot t
 * is row t / capacity, column t % capacity.  A segment is one attention span:
 * in a packed plan one prompt, in a padded plan one whole row.  Segments are
 * listed row by row, inside a row in placement order.
 *
 * Caller-owned arrays; the library writes them.  Sizes:
 *   row_seg_ptr   [k + 1]   segments of row r are [row_seg_ptr[r], row_seg_ptr[r+1])
 *   seg_prompt    [k]       prompt index (original order) of each segment
 *   seg_start     [k]       global slot of the segment's first token (row*capacity + column)
 *   seg_len       [k]       attention span length (packed: l_i; padded: max length m)
 *   prompt_kv_off [k + 1]   exclusive prefix sum of lengths in original order: the cache
 *                           rows of prompt i are [prompt_kv_off[i], prompt_kv_off[i+1])
 *   slot_seg      [slot_cap]  segment of each slot, -1 outside every span (row-tail pads)
 *   slot_pos      [slot_cap]  position of each slot inside its span (restart positions,
 *                             section 3.2); 0 outside every span
 *   slot_kv       [slot_cap]  cache row (UNPACK target) of each slot; -1 at every pad slot
 *   qtile_seg     [qtile_cap] attention work list: segment of each query tile
 *   qtile_q0      [qtile_cap] first query (offset inside the segment) of each query tile;
 *                             every (segment, multiple of PP_QTILE below seg_len) appears
 *                             once; the tiles of a segment are consecutive, segments longest
 *                             first (ties: lower segment index), inside a segment the tile
 *                             with the highest first query first
 *   mtile_m0      [mtile_cap] row tiles of the projection GEMMs: the first slot of every
 *                             PP_MTILE-slot tile of the batch (slots t0 .. t0 + PP_MTILE - 1,
 *                             t0 a multiple of PP_MTILE) holding a slot of some span,
 *                             ascending; tiles of row-tail padding alone are left out
 * slot_cap must be >= k * C, qtile_cap >= k * ceil(C / PP_QTILE) and mtile_cap >=
 * ceil(k * C / PP_MTILE), where C is the row capacity actually used (pp_plan_bounds computes
 * all three).
 * ---------------------------------------------------------------------------------------- */
typedef struct pp_plan {
    /* written by pp_pack / pp_pack_padded */
    int32_t k;          /* number of prompts                                         */
    int32_t capacity;   /* slots per row C                                           */
    int32_t n_rows;     /* rows r (r <= k, section 3.1)                              */
    int32_t max_len;    /* m = max l_i                                               */
    int32_t total_len;  /* L = sum l_i                                               */
    int32_t n_qtiles;   /* entries written to qtile_seg / qtile_q0                   */
    int32_t n_mtiles;   /* entries written to mtile_m0                               */
    /* set by the caller */
    int64_t slot_cap;
    int64_t qtile_cap;
    int64_t mtile_cap;
    int32_t* row_seg_ptr;
    int32_t* seg_prompt;
    int32_t* seg_start;
    int32_t* seg_len;
    int32_t* prompt_kv_off;
    int32_t* slot_seg;
    int32_t* slot_pos;
    int32_t* slot_kv;
    int32_t* qtile_seg;
    int32_t* qtile_q0;
    int32_t* mtile_m0;
} pp_plan;

/* Array sizes a plan needs for k prompts in rows of C slots (C = capacity, or the maximum
 * length when capacity is 0 or the plan is padded).  Errors: k < 0, C < 0, NULL outputs. */
pp_status pp_plan_bounds(int32_t k, int32_t C, int64_t* slot_cap, int64_t* qtile_cap, int64_t* mtile_cap);

/* BINPACK + TENSORIZE layout + RESTART-PE + UNPACK map (Algorithm 1; sections 3.1-3.2).
 *
 * First-fit decreasing: prompts in order of decreasing length (ties: lower original index
 * first), each into the lowest-numbered row with enough room, a new row when none has;
 * inside a row prompts sit back to back from column 0 in placement order; pads only at
 * row tails.  capacity == 0 uses the maximum prompt length m as the row size, the
 * paper's choice (section 3.1).
 *
 * lengths: host [k], every l_i >= 1.  k == 0 is valid and yields an empty plan.
 * Errors: PP_ERR_INVALID_ARG (NULL, k < 0, l_i <= 0, capacity < 0),
 *         PP_ERR_TOO_LONG (some l_i > capacity > 0),
 *         PP_ERR_BUFFER_TOO_SMALL (slot_cap / qtile_cap / mtile_cap below pp_plan_bounds).
 * Pure host code, reentrant, O(k log k + k r + r C). */
pp_status pp_pack(const int32_t* lengths, int32_t k, int32_t capacity, pp_plan* plan);

/* Full batching, the paper's baseline (section 4.2): prompt i alone in row i, right-padded
 * to m = max l_i; every row is one causal span of length m (positions 0..m-1); the pad
 * slots carry slot_kv = -1 and are processed but never read back.  Same errors as pp_pack. */
pp_status pp_pack_padded(const int32_t* lengths, int32_t k, pp_plan* plan);

/* ------------------------------------------------------------------------------------------
 * Prefill (Algorithm 1, the model call and UNPACK).
 * ---------------------------------------------------------------------------------------- */

/* Llama-style decoder shape (section 2.1; the paper's appendix model table). */
typedef struct pp_config {
    int32_t n_layers;
    int32_t d_model;    /* d                                                        */
    int32_t n_heads;    /* H query heads                                            */
    int32_t n_kv_heads; /* Hkv key/value heads; query head h reads kv head h/(H/Hkv) */
    int32_t head_dim;   /* D                                                        */
    int32_t ffn_dim;    /* F, SwiGLU width                                          */
    int32_t vocab;
    int32_t dtype;      /* pp_dtype: storage type of weights, activations and cache */
    float rms_eps;
    float rope_theta;
} pp_config;

/* Device pointers; matrices row-major [out_features, in_features].  The per-layer members
 * are host arrays of n_layers device pointers.  Matrix element type = config dtype; norm
 * gains are float32.
 *   embed      [vocab, d]
 *   final_norm [d] float32
 *   attn_norm  [d] float32 per layer
 *   wqkv       [(H + 2 Hkv) D, d]: the rows of Wq, then of Wk, then of Wv
 *   wo         [d, H D]
 *   mlp_norm   [d] float32 per layer
 *   w_gateup   [2F, d]: Wg and Wu interleaved in blocks of 16 rows: rows 32j..32j+15 are
 *              Wg rows 16j..16j+15 and rows 32j+16..32j+31 are Wu rows 16j..16j+15
 *              (F must be a multiple of 16)
 *   w_down     [d, F]                                                                    */
typedef struct pp_weights {
    const void* embed;
    const float* final_norm;
    const float* const* attn_norm;
    const void* const* wqkv;
    const void* const* wo;
    const float* const* mlp_norm;
    const void* const* w_gateup;
    const void* const* w_down;
} pp_weights;

/* A plan copied to device memory: the scalars of pp_plan and device copies of the arrays
 * the kernels read (same meaning and length as in pp_plan; slot arrays hold
 * n_rows * capacity entries, qtile arrays n_qtiles, mtile_m0 n_mtiles).  The scalars are
 * validated on the host; the arrays' contents are trusted to be what pp_pack or
 * pp_pack_padded wrote (the kernels index memory with them). */
typedef struct pp_dplan {
    int32_t k, capacity, n_rows, max_len, total_len, n_qtiles, n_mtiles;
    const int32_t* seg_prompt;
    const int32_t* seg_start;
    const int32_t* seg_len;
    const int32_t* prompt_kv_off;
    const int32_t* slot_seg;
    const int32_t* slot_pos;
    const int32_t* slot_kv;
    const int32_t* qtile_seg;
    const int32_t* qtile_q0;
    const int32_t* mtile_m0;
} pp_dplan;

/* Bytes of device workspace pp_prefill needs for this config and plan.
 * Errors: PP_ERR_INVALID_ARG, PP_ERR_UNSUPPORTED (as pp_prefill). */
pp_status pp_prefill_workspace_size(const pp_config* cfg, const pp_dplan* plan, size_t* bytes);

/* Prefill every prompt of the plan: embed the tokens into the packed batch, run every
 * decoder layer over it with the independent mask (attention restricted to each segment,
 * causal inside it; section 3.2) and restart RoPE positions, and unpack.
 *
 *   tokens    device int32 [total_len], all prompts back to back in original order; an id
 *             outside [0, vocab) embeds as a zero vector
 *   workspace device, >= pp_prefill_workspace_size bytes, 256-byte aligned
 *   hidden    device float32 [total_len, d]: final RMSNorm output of every real token,
 *             in original prompt order (row prompt_kv_off[i] + j = token j of prompt i)
 *   k_cache, v_cache  device, config dtype, [n_layers][total_len][Hkv * D]: per layer the
 *             post-RoPE keys and the values of every real token, same row order
 *   stream    a hipStream_t (NULL = the default stream)
 *
 * Numerics: bf16 storage of weights, normalised activations, q/k/v, attention output
 * and SwiGLU product; float32 accumulation, softmax, RoPE and residual stream; float32
 * throughout for PP_F32.
 * Asynchronous: returns once the work is enqueued on `stream`; errors of the kernels
 * themselves surface at the caller's next synchronisation.  All arguments are validated
 * before anything is enqueued.  Reentrant for distinct workspaces and outputs.
 * Errors: PP_ERR_INVALID_ARG (NULL pointer, inconsistent plan or config),
 *         PP_ERR_BUFFER_TOO_SMALL (workspace), PP_ERR_UNSUPPORTED (H not a multiple of Hkv;
 *         bf16: head_dim != 128, d % 256, F % 128 or (H + 2 Hkv) D % 256 non-zero;
 *         f32: head_dim not 64 or 128, d, F or H D not a multiple of 16),
 *         PP_ERR_HIP (launch failure). */
pp_status pp_prefill(const pp_config* cfg, const pp_weights* w, const pp_dplan* plan,
                     const int32_t* tokens, void* workspace, size_t workspace_bytes,
                     float* hidden, void* k_cache, void* v_cache, void* stream);

/* ------------------------------------------------------------------------------------------
 * Single steps of pp_prefill.  Each enqueues exactly the kernel pp_prefill uses for that
 * step, on caller device buffers, for callers that assemble their own layer loop and for
 * step-by-step verification.  Same conventions: validated before enqueuing, asynchronous.
 * `rows` buffers are row-major with the stated row length; `plan` is a device plan.
 * ---------------------------------------------------------------------------------------- */

typedef enum pp_epilogue {
    PP_EPI_STORE = 0,     /* C = A B^T, stored in dtype                                        */
    PP_EPI_RESIDUAL = 1,  /* C += A B^T, C float32                                              */
    PP_EPI_SWIGLU = 2     /* B = w_gateup layout; C [M, N/2] = SiLU(A Wg^T) * (A Wu^T), dtype    */
} pp_epilogue;

/* TENSORIZE: x[t] = embed[tokens[slot_kv[t]]] as float32 for the plan's n_rows*capacity
 * slots; 0 at pad slots and for token ids outside [0, vocab).  embed [vocab, d] in dtype,
 * x [n_rows*capacity, d] float32, d % 8 == 0. */
pp_status pp_embed(int32_t dtype, const void* embed, int32_t vocab, int32_t d, const int32_t* tokens,
                   const pp_dplan* plan, float* x, void* stream);

/* RMSNorm (the Llama family's normalisation): out[r] = x[r] / sqrt(mean(x[r]^2) + eps) * gain,
 * x [rows, d] float32, gain [d] float32, out [rows, d] in dtype.  d % 4 == 0. */
pp_status pp_rmsnorm(int32_t dtype, const float* x, const float* gain, int32_t rows, int32_t d, float eps,
                     void* out, void* stream);

/* Projection GEMM C = A B^T: A [M, K] (row stride lda), B [N, K] (row stride ldb), both dtype,
 * float32 accumulation; C per epilogue (row stride ldc).  bf16: N % 256 == 0, K % 64 == 0;
 * f32: K % 16 == 0 and no PP_EPI_SWIGLU.  plan may be NULL; when given (bf16 only, and then
 * M must be n_rows * capacity), only the plan's row tiles (mtile_m0) are computed, as in
 * pp_prefill: rows of C in tiles of row-tail padding alone are left unwritten. */
pp_status pp_gemm(int32_t dtype, int32_t epilogue, const void* A, int64_t lda, const void* B, int64_t ldb,
                  void* C, int64_t ldc, int32_t M, int32_t N, int32_t K, const pp_dplan* plan, void* stream);

/* QKV projection with RESTART-PE and the KV-cache UNPACK fused into its epilogue (bf16 only;
 * the float32 path uses pp_gemm + pp_rope + pp_kv_scatter): [q | k | v] = xn wqkv^T with
 * float32 accumulation; q and k rotated (rotate-half RoPE) at each slot's restart position;
 * q stored to q_out [n_rows*capacity, H D]; k and v stored straight into the layer's caches
 * k_cache, v_cache [total_len, Hkv D] at row slot_kv[t] for every real slot t.
 * xn [n_rows*capacity, d] bf16; wqkv [(H+2Hkv) D, d] bf16; table: device scratch of
 * max_len * D/2 float2, filled by this call (cos/sin of position * theta^(-2i/D) in float64). */
pp_status pp_qkv_projection(const pp_config* cfg, const pp_dplan* plan, const void* xn, const void* wqkv,
                            void* table, void* q_out, void* k_cache, void* v_cache, void* stream);

/* RESTART-PE (section 3.2): rotate-half RoPE in place on the query and key heads of
 * qkv [n_rows*capacity, (H+2Hkv)D] at each slot's restart position slot_pos; slots outside
 * every span are left alone.  table: device scratch of max_len * D/2 float2 (8 bytes each),
 * filled by this call with cos/sin of position * theta^(-2i/D) evaluated in float64. */
pp_status pp_rope(const pp_config* cfg, const pp_dplan* plan, void* qkv, void* table, void* stream);

/* UNPACK (Algorithm 1) of one layer's cache: k_cache[slot_kv[t]] and v_cache[slot_kv[t]]
 * ([total_len, Hkv D] each, dtype) from the K and V parts of qkv, for every real slot t. */
pp_status pp_kv_scatter(const pp_config* cfg, const pp_dplan* plan, const void* qkv, void* k_cache,
                        void* v_cache, void* stream);

/* Attention under the independent mask M' (section 3.2): for every slot of every segment,
 * softmax(q k^T / sqrt(D)) v over the keys of the same segment at or before it.
 * q: post-RoPE queries, row t at q + t * ldq (elements), H D per row, one row per slot;
 * k_cache, v_cache: the layer's caches [total_len, Hkv D] (post-RoPE keys), keys of segment s
 * at rows prompt_kv_off[seg_prompt[s]] + j; a key of a span that is no prompt token (full
 * batching's padding) is read as zero.  out [n_rows*capacity, H D]; rows of slots outside
 * every span are not written.  All in dtype. */
pp_status pp_attention(const pp_config* cfg, const pp_dplan* plan, const void* q, int64_t ldq,
                       const void* k_cache, const void* v_cache, void* out, void* stream);

/* Final RMSNorm fused with the hidden-state UNPACK: hidden[slot_kv[t]] = RMSNorm(x[t]) * gain
 * for every real slot; x [n_rows*capacity, d] float32, hidden [total_len, d] float32. */
pp_status pp_final_norm_unpack(const float* x, const float* gain, int32_t d, float eps, const pp_dplan* plan,
                               float* hidden, void* stream);

/* ------------------------------------------------------------------------------------------
 * First token (section 2.3: the time to first token is the time to prefill the KV cache and
 * generate the first token; section 4.3 adds the unpacking, which pp_prefill already did).
 * ---------------------------------------------------------------------------------------- */

/* Bytes of device workspace pp_first_token needs for this config and plan.
 * Errors: PP_ERR_INVALID_ARG, PP_ERR_UNSUPPORTED (as pp_prefill). */
pp_status pp_first_token_workspace_size(const pp_config* cfg, const pp_dplan* plan, size_t* bytes);

/* Greedy first token of every prompt of the plan: for prompt i (original order), its last
 * token's hidden row h_i = hidden[prompt_kv_off[i+1] - 1], the logits h_i . lm_head[v] for
 * every v < vocab, and tokens[i] = the v of maximal logit, the lowest v on ties (-1 if every
 * logit is NaN; NaN logits are never chosen).
 *
 *   hidden    device float32 [total_len, d]: pp_prefill's output
 *   lm_head   device [vocab, d] in the config dtype, row-major ([out, in])
 *   workspace device, >= pp_first_token_workspace_size bytes, 256-byte aligned
 *   logits    device float32 [k, vocab], or NULL when not wanted
 *   tokens    device int32 [k]
 *   stream    a hipStream_t (NULL = the default stream)
 *
 * Numerics: PP_BF16 rounds h_i to bf16 (as every projection input of the bf16 model) and
 * accumulates in float32; PP_F32 is float32 throughout.  The argmax is taken on the float32
 * logits.  Asynchronous; validated before enqueuing; deterministic.
 * Errors: PP_ERR_INVALID_ARG (NULL pointer, misaligned workspace, inconsistent plan or
 *         config), PP_ERR_BUFFER_TOO_SMALL (workspace), PP_ERR_UNSUPPORTED (as pp_prefill),
 *         PP_ERR_HIP (launch failure). */
pp_status pp_first_token(const pp_config* cfg, const pp_dplan* plan, const float* hidden, const void* lm_head,
                         void* workspace, size_t workspace_bytes, float* logits, int32_t* tokens, void* stream);

/* Bytes of the library-owned device buffer behind pp_first_token_noalloc (per GPU). */
#define PP_FIRST_TOKEN_SCRATCH_BYTES (16u << 20)

/* pp_first_token for callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the same kernels and the
 * same results, with the workspace taken from a static device buffer of
 * PP_FIRST_TOKEN_SCRATCH_BYTES that the library holds on every GPU it runs on until the
 * process ends.  The call allocates nothing (no hipMalloc, no hipFree); the caller still
 * passes hidden, lm_head, logits and tokens.
 *
 *   Limit: pp_first_token_workspace_size(cfg, plan) <= PP_FIRST_TOKEN_SCRATCH_BYTES, else
 *          PP_ERR_BUFFER_TOO_SMALL before anything is enqueued.  bf16 needs about
 *          k (2 d + 8 vocab / 128) bytes: e.g. 512 prompts at d = 8192 with a 128,256-token
 *          vocabulary; float32 about k (4 d + 8 vocab): e.g. 64 prompts with vocab 32,000
 *          do not fit.
 *   Sharing: every call on a GPU uses that GPU's one buffer; calls that overlap on one GPU
 *          (concurrent streams, or threads with the same device) race on it and must be
 *          serialised by the caller.  No part of the buffer needs to start at any value:
 *          every byte a call reads was written earlier in the same call.
 *   Set-up: the first call on a device looks up that device's buffer address (no allocation,
 *          no stream work); a caller that captures a graph can make one call before capture.
 * Errors: as pp_first_token, with PP_ERR_BUFFER_TOO_SMALL for the limit above and PP_ERR_HIP
 *         when the buffer's address cannot be obtained. */
pp_status pp_first_token_noalloc(const pp_config* cfg, const pp_dplan* plan, const float* hidden,
                                 const void* lm_head, float* logits, int32_t* tokens, void* stream);

/* ------------------------------------------------------------------------------------------
 * Generation with packed KV caches (section 4.8: the caches of a batch are packed for
 * generation instead of padded to the longest prompt; section 2.2: one forward pass per new
 * token, the keys and values of earlier tokens read from the cache).  Greedy decoding: each
 * step feeds one token per prompt and chooses the next as pp_first_token does.
 * ---------------------------------------------------------------------------------------- */

/* Where the keys and values of each prompt live during generation.  At decode step s
 * (0 <= s < n_new) prompt i's keys are, in this order, the ctx_span[i] rows of the context
 * cache from row ctx_off[i] (the first ctx_valid[i] of them its prompt tokens, the rest
 * full batching's padding, read and masked), then rows gen_off[i] .. gen_off[i] + s of the
 * generation cache, the last of which step s writes.  The token fed at step s sits at
 * position pos0[i] + s (each prompt's own positions continue; section 3.2).
 *
 *   packed (padded == 0): the context cache is pp_prefill's per-prompt cache (ctx_off[i] =
 *          l_0 + .. + l_{i-1}, ctx_span = ctx_valid = l_i, ctx_rows = total length); the
 *          generation cache holds n_new rows per prompt (gen_off[i] = i n_new,
 *          gen_rows = k n_new).  Nothing is padded.
 *   padded (padded == 1): full batching: one cache of k rows of m + n_new slots (m = the
 *          longest prompt), prompt i at row i (m + n_new), its padding up to m read and
 *          masked, its generated tokens from slot m on (ctx_span = m, ctx_valid = l_i,
 *          gen_off[i] = i (m + n_new) + m, ctx_rows = gen_rows = k (m + n_new)): context and
 *          generation cache are then the same buffer.
 * pos0[i] = l_i in both.  max_len = m.  The five arrays are [k] int32, caller-owned. */
typedef struct pp_gen_layout {
    int32_t k, n_new, padded, max_len;
    int64_t ctx_rows, gen_rows;        /* rows per layer of the context / generation caches */
    int32_t *ctx_off, *ctx_span, *ctx_valid, *pos0, *gen_off;
} pp_gen_layout;

/* The same layout with its five arrays in device memory: what the decode calls read. */
typedef struct pp_gen_dlayout {
    int32_t k, n_new, padded, max_len;
    int64_t ctx_rows, gen_rows;
    const int32_t *ctx_off, *ctx_span, *ctx_valid, *pos0, *gen_off;
} pp_gen_dlayout;

/* Fill `layout` (its arrays allocated by the caller, [k] each) for prompts of the given
 * lengths, room for n_new generated tokens each, packed (padded == 0) or full batching.
 * Pure host code, reentrant.
 * Errors: PP_ERR_INVALID_ARG (k <= 0, a length <= 0, n_new <= 0, padded not 0/1, NULL array,
 *         more than 2^31 - 1 rows). */
pp_status pp_gen_layout_make(const int32_t* lengths, int32_t k, int32_t n_new, int32_t padded,
                             pp_gen_layout* layout);

/* Bytes of device workspace pp_decode_step and pp_generate need for this config and layout.
 * Errors: as pp_decode_step's argument checks. */
pp_status pp_decode_workspace_size(const pp_config* cfg, const pp_gen_dlayout* layout, size_t* bytes);

/* Decode step `step` for every prompt: embed tokens_in[i] (the token chosen before: the
 * first token of pp_first_token at step 0), run the decoder on that one row per prompt at
 * position pos0[i] + step (RoPE, attention over the prompt's own keys only, MLP), append its
 * key and value to the generation cache at row gen_off[i] + step of every layer, apply the
 * final norm and the LM head, and choose tokens_out[i] greedily (as pp_first_token: the
 * lowest id of maximal logit, -1 if every logit is NaN).
 *
 *   tokens_in, tokens_out  device int32 [k]
 *   lm_head   device [vocab, d] in the config dtype
 *   ctx_k, ctx_v  device [n_layers][ctx_rows][Hkv D] in dtype: read only
 *   gen_k, gen_v  device [n_layers][gen_rows][Hkv D] in dtype: rows gen_off[i] + step are
 *             written, earlier generated rows read (in the padded layout the same buffers
 *             as ctx_k, ctx_v)
 *   workspace device, >= pp_decode_workspace_size bytes, 256-byte aligned
 *   logits    device float32 [k, vocab], or NULL
 *   stream    a hipStream_t (NULL = the default stream)
 *
 * Numerics as pp_prefill (bf16 storage of weights, activations, q/k/v and caches; float32
 * accumulation, softmax and residual stream), and as pp_first_token for the choice.  The
 * packed and the full-batching layouts give bit-identical results.  Asynchronous; validated
 * before enqueuing; the layout's device arrays are trusted to be what pp_gen_layout_make
 * wrote.
 * Errors: PP_ERR_INVALID_ARG (NULL pointer, step outside [0, n_new), inconsistent layout,
 *         misaligned workspace), PP_ERR_BUFFER_TOO_SMALL (workspace), PP_ERR_UNSUPPORTED
 *         (as pp_prefill, and H / Hkv not in {1, 2, 4, 8}), PP_ERR_HIP (launch failure). */
pp_status pp_decode_step(const pp_config* cfg, const pp_weights* w, const pp_gen_dlayout* layout, int32_t step,
                         const int32_t* tokens_in, const void* lm_head, const void* ctx_k, const void* ctx_v,
                         void* gen_k, void* gen_v, void* workspace, size_t workspace_bytes, float* logits,
                         int32_t* tokens_out, void* stream);

/* n_steps <= n_new decode steps back to back on `stream`, with no host synchronisation:
 * step s consumes tokens[s - 1] (tokens_first at s = 0) and writes tokens[s]; tokens is
 * device int32 [n_steps][k].  Same buffers and errors as pp_decode_step. */
pp_status pp_generate(const pp_config* cfg, const pp_weights* w, const pp_gen_dlayout* layout, int32_t n_steps,
                      const int32_t* tokens_first, const void* lm_head, const void* ctx_k, const void* ctx_v,
                      void* gen_k, void* gen_v, void* workspace, size_t workspace_bytes, int32_t* tokens,
                      void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PREPACK_H */
