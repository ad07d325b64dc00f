// Generation with packed KV caches (section 4.8): the cache layouts and the decode step.
//
// Host side only.  pp_gen_layout_make places every prompt's keys and values (packed: the
// prefill's per-prompt cache plus n_new rows per prompt; full batching: k rows of
// m + n_new slots).  pp_decode_step validates everything, carves the caller's workspace and
// enqueues, without host synchronisation:
//
//   decode_prep (positions, RoPE rows, append rows); embed of the k fed tokens
//   per layer: rmsnorm -> QKV projection with RoPE and the append to the generation cache
//              (bf16: the prefill's fused epilogue; float32: GEMM, RoPE, scatter) ->
//              split-key decode attention + combine -> O GEMM (+residual) -> rmsnorm ->
//              gate/up GEMM with SwiGLU -> down GEMM (+residual); with the split-K GEMMs
//              the residual adds of O and down happen in the norm that follows each
//   final rmsnorm (float32) -> LM head and greedy choice (the first-token kernels, one
//   row per prompt).
// The projections: for bf16 steps of up to 64 prompts, weight-streaming GEMMs for one row
// per prompt (QKV and gate/up with their epilogues in the kernel; O and down as split-K
// partial sums that the next norm adds); otherwise the prefill's GEMM kernels with M = k.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdint>

#include "kernels.h"
#include "prepack.h"
#include "status.h"

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }
size_t elem_size(int dtype) { return dtype == PP_BF16 ? 2 : 4; }

struct Layout {
    size_t x = 0, xn = 0, q = 0, attn = 0, act = 0, gu = 0, h = 0, part = 0, table = 0, ints = 0, ft = 0, gpart = 0,
           total = 0;
};

// The projections of a decode step as (N, K).
struct Proj {
    int N, K;
};
void projections(const pp_config* c, Proj (&p)[4]) {
    const int d = c->d_model, hd = c->n_heads * c->head_dim;
    p[0] = {(c->n_heads + 2 * c->n_kv_heads) * c->head_dim, d};   // QKV
    p[1] = {d, hd};                                               // O
    p[2] = {2 * c->ffn_dim, d};                                   // gate/up
    p[3] = {d, c->ffn_dim};                                       // down
}

// bf16 steps of up to 64 prompts take the skinny GEMM for every projection when the fused
// residual norm takes the width (d <= 8192).
bool use_skinny(const pp_config* c, int k) {
    if (c->dtype != PP_BF16 || !ppk::residual_rmsnorm_ok(c->d_model)) return false;
    Proj p[4];
    projections(c, p);
    for (const Proj& q : p)
        if (!ppk::skinny_ok(k, q.N, q.K)) return false;
    return true;
}

int chunks(int n) { return (n + ppk::kDecodeChunk - 1) / ppk::kDecodeChunk; }

Layout layout_of(const pp_config* c, const pp_gen_dlayout* g) {
    const size_t k = g->k, e = elem_size(c->dtype);
    const size_t d = c->d_model, F = c->ffn_dim, D = c->head_dim;
    const size_t qkv_w = size_t(c->n_heads + 2 * c->n_kv_heads) * D, hd = size_t(c->n_heads) * D;
    const size_t nch = size_t(chunks(g->max_len) + chunks(g->n_new));
    Layout L;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += align_up(bytes);
        return at;
    };
    L.x = take(k * d * 4);
    L.xn = take(k * d * e);
    L.q = take(c->dtype == PP_BF16 ? k * hd * 2 : k * qkv_w * 4);   // bf16: rotated queries only
    L.attn = take(k * hd * e);
    L.act = take(k * F * e);
    L.gu = take(c->dtype == PP_F32 ? k * 2 * F * 4 : 0);
    L.h = take(k * d * 4);
    L.part = take(k * size_t(c->n_heads) * nch * (D + 4) * 4);
    L.table = take(k * (D / 2) * sizeof(float2));
    L.ints = take((4 * k + 1) * sizeof(int32_t));
    L.ft = take(ppk::first_token_workspace(c->dtype, g->k, c->vocab, c->d_model));
    size_t gpart = 0;
    if (use_skinny(c, g->k)) {
        Proj p[4];
        projections(c, p);
        // O and down leave split-K partial sums
        gpart = std::max(size_t(ppk::skinny_split(p[1].N, p[1].K).splits) * k * p[1].N * 4,
                         size_t(ppk::decode_gemm_splits(g->k, p[3].N, p[3].K)) * k * p[3].N * 4);
    }
    L.gpart = take(gpart);
    L.total = off;
    return L;
}

pp_status validate_layout(const pp_config* c, const pp_gen_dlayout* g) {
    if (!g) return pp::fail(PP_ERR_INVALID_ARG, "layout is NULL");
    if (g->k <= 0 || g->n_new <= 0 || g->max_len <= 0 || (g->padded != 0 && g->padded != 1))
        return pp::fail(PP_ERR_INVALID_ARG, "layout k %d, n_new %d, max_len %d, padded %d", g->k, g->n_new,
                        g->max_len, g->padded);
    if (g->ctx_rows <= 0 || g->gen_rows < int64_t(g->k) * g->n_new || g->ctx_rows > INT32_MAX ||
        g->gen_rows > INT32_MAX)
        return pp::fail(PP_ERR_INVALID_ARG, "layout rows: ctx %lld, gen %lld", (long long)g->ctx_rows,
                        (long long)g->gen_rows);
    if (!g->ctx_off || !g->ctx_span || !g->ctx_valid || !g->pos0 || !g->gen_off)
        return pp::fail(PP_ERR_INVALID_ARG, "a device layout array is NULL");
    const int R = c->n_heads / c->n_kv_heads;
    if (R != 1 && R != 2 && R != 4 && R != 8)
        return pp::fail(PP_ERR_UNSUPPORTED, "decode attention needs n_heads / n_kv_heads in {1, 2, 4, 8} (%d)", R);
    return PP_OK;
}

pp_status check_buffers(const pp_config* c, const pp_gen_dlayout* g, const void* lm_head, const void* ctx_k,
                        const void* ctx_v, const void* gen_k, const void* gen_v, const void* workspace,
                        size_t workspace_bytes) {
    if (!lm_head || !ctx_k || !ctx_v || !gen_k || !gen_v)
        return pp::fail(PP_ERR_INVALID_ARG, "lm_head and the four caches must be non-NULL");
    if (!workspace) return pp::fail(PP_ERR_INVALID_ARG, "workspace is NULL");
    if (reinterpret_cast<uintptr_t>(workspace) % kAlign)
        return pp::fail(PP_ERR_INVALID_ARG, "workspace is not %zu-byte aligned", kAlign);
    const size_t need = layout_of(c, g).total;
    if (workspace_bytes < need)
        return pp::fail(PP_ERR_BUFFER_TOO_SMALL, "workspace of %zu bytes < %zu needed", workspace_bytes, need);
    return PP_OK;
}

pp_status check_all(const pp_config* cfg, const pp_weights* w, const pp_gen_dlayout* g) {
    if (pp_status st = pp::validate_config(cfg)) return st;
    if (pp_status st = pp::validate_weights(cfg, w)) return st;
    return validate_layout(cfg, g);
}

// Enqueue one decode step (arguments already validated).
void enqueue_step(const pp_config* cfg, const pp_weights* w, const pp_gen_dlayout* g, int step,
                  const int32_t* tokens_in, const void* lm_head, const void* ctx_k, const void* ctx_v, void* gen_k,
                  void* gen_v, void* workspace, float* logits, int32_t* tokens_out, hipStream_t s) {
    const Layout L = layout_of(cfg, g);
    const int dt = cfg->dtype;
    const bool bf = dt == PP_BF16;
    const int k = g->k;
    const int d = cfg->d_model, H = cfg->n_heads, Hkv = cfg->n_kv_heads, D = cfg->head_dim, F = cfg->ffn_dim;
    const int qkv_w = (H + 2 * Hkv) * D, hd = H * D, kvw = Hkv * D;
    const float eps = cfg->rms_eps;
    const size_t e = elem_size(dt);

    char* ws = static_cast<char*>(workspace);
    float* x = reinterpret_cast<float*>(ws + L.x);
    void* xn = ws + L.xn;
    void* q = ws + L.q;
    void* attn = ws + L.attn;
    void* act = ws + L.act;
    float* gu = reinterpret_cast<float*>(ws + L.gu);
    float* h = reinterpret_cast<float*>(ws + L.h);
    float* part = reinterpret_cast<float*>(ws + L.part);
    float2* table = reinterpret_cast<float2*>(ws + L.table);
    int32_t* slot_pos = reinterpret_cast<int32_t*>(ws + L.ints);
    int32_t* slot_kv = slot_pos + k;
    int32_t* slot_seg = slot_kv + k;
    int32_t* ident = slot_seg + k;        // k + 1 entries
    const size_t ctx_layer = size_t(g->ctx_rows) * kvw * e, gen_layer = size_t(g->gen_rows) * kvw * e;
    // the prompts' context chunks together: at most ceil(ctx_rows / chunk) + k, as every prompt's
    // span lies in its own ctx_rows (and at most k x the longest prompt's)
    const int n_ctx_items = static_cast<int>(std::min<int64_t>(int64_t(k) * chunks(g->max_len),
                                                               (g->ctx_rows + ppk::kDecodeChunk - 1) / ppk::kDecodeChunk + k));
    const ppk::DecodeLayout Ly{k, chunks(g->max_len), chunks(g->n_new), n_ctx_items, g->ctx_off, g->ctx_span,
                               g->ctx_valid, g->pos0, g->gen_off};
    const bool skinny = use_skinny(cfg, k);
    float* gpart = reinterpret_cast<float*>(ws + L.gpart);

    // the split-K residual projections (O, down) leave their partial sums in gpart; the next
    // norm adds them to x (pending = their split count) before normalising
    int pending = 0;
    auto norm = [&](const float* gain, void* out, int out_dtype) {
        if (skinny)
            ppk::residual_rmsnorm(out_dtype, x, gpart, pending, k, d, gain, out, eps, s);
        else
            ppk::rmsnorm(out_dtype, x, gain, out, k, d, eps, s);
        pending = 0;
    };
    ppk::decode_prep(Ly, step, D, cfg->rope_theta, table, slot_pos, slot_kv, slot_seg, ident, s);
    ppk::embed(dt, x, w->embed, cfg->vocab, tokens_in, ident, k, d, s);
    for (int l = 0; l < cfg->n_layers; ++l) {
        const void* ck = static_cast<const char*>(ctx_k) + l * ctx_layer;
        const void* cv = static_cast<const char*>(ctx_v) + l * ctx_layer;
        void* gk = static_cast<char*>(gen_k) + l * gen_layer;
        void* gv = static_cast<char*>(gen_v) + l * gen_layer;
        norm(w->attn_norm[l], xn, dt);
        if (skinny) {
            const ppk::QkvOut qo{q, hd, gk, gv, kvw, table, slot_pos, slot_kv, H, Hkv};
            ppk::decode_gemm(ppk::kQkvRope, xn, d, k, w->wqkv[l], d, qkv_w, d, gpart,
                             ppk::DecodeEpi{nullptr, 0, qo}, s);
            ppk::decode_attention(dt, q, hd, ck, cv, gk, gv, kvw, Ly, step, H, Hkv, D, part, nullptr, hd, s);
            const ppk::AttnChunks ac{part, g->ctx_span, step, Ly.n_ctx_chunks, Ly.n_ctx_chunks + Ly.n_gen_chunks, H};
            ppk::decode_gemm_o(k, ac, w->wo[l], hd, d, hd, gpart, s);
            pending = ppk::skinny_split(d, hd).splits;
        } else if (bf) {
            const ppk::QkvOut qo{q, hd, gk, gv, kvw, table, slot_pos, slot_kv, H, Hkv};
            ppk::qkv_rope_bf16(xn, d, w->wqkv[l], d, k, d, nullptr, 0, qo, s);
            ppk::decode_attention(dt, q, hd, ck, cv, gk, gv, kvw, Ly, step, H, Hkv, D, part, attn, hd, s);
            ppk::gemm_bf16(ppk::kResidual, attn, hd, w->wo[l], hd, x, d, k, d, hd, nullptr, 0, s);
        } else {
            float* qkv32 = static_cast<float*>(q);
            ppk::gemm_f32(ppk::kStore, static_cast<const float*>(xn), d, static_cast<const float*>(w->wqkv[l]), d,
                          qkv32, qkv_w, k, qkv_w, d, s);
            ppk::rope_apply(dt, q, qkv_w, table, slot_pos, slot_seg, k, H + Hkv, D, s);
            ppk::kv_scatter(dt, q, qkv_w, hd, kvw, gk, gv, slot_kv, k, s);
            ppk::decode_attention(dt, q, qkv_w, ck, cv, gk, gv, kvw, Ly, step, H, Hkv, D, part, attn, hd, s);
            ppk::gemm_f32(ppk::kResidual, static_cast<const float*>(attn), hd, static_cast<const float*>(w->wo[l]),
                          hd, x, d, k, d, hd, s);
        }
        norm(w->mlp_norm[l], xn, dt);
        if (skinny) {
            const ppk::QkvOut none{};
            ppk::decode_gemm(ppk::kSwiGLU, xn, d, k, w->w_gateup[l], d, 2 * F, d, gpart,
                             ppk::DecodeEpi{act, F, none}, s);
            ppk::decode_gemm(ppk::kResidual, act, F, k, w->w_down[l], F, d, F, gpart,
                             ppk::DecodeEpi{x, d, none}, s);
            pending = ppk::decode_gemm_splits(k, d, F);
        } else if (bf) {
            ppk::gemm_bf16(ppk::kSwiGLU, xn, d, w->w_gateup[l], d, act, F, k, 2 * F, d, nullptr, 0, s);
            ppk::gemm_bf16(ppk::kResidual, act, F, w->w_down[l], F, x, d, k, d, F, nullptr, 0, s);
        } else {
            ppk::gemm_f32(ppk::kStore, static_cast<const float*>(xn), d, static_cast<const float*>(w->w_gateup[l]), d,
                          gu, 2 * F, k, 2 * F, d, s);
            ppk::swiglu_f32(gu, static_cast<float*>(act), k, F, s);
            ppk::gemm_f32(ppk::kResidual, static_cast<const float*>(act), F, static_cast<const float*>(w->w_down[l]),
                          F, x, d, k, d, F, s);
        }
    }
    norm(w->final_norm, h, PP_F32);
    ppk::first_token(dt, h, ident, k, lm_head, cfg->vocab, d, ws + L.ft, logits, tokens_out, s);
}

}  // namespace

extern "C" pp_status pp_gen_layout_make(const int32_t* lengths, int32_t k, int32_t n_new, int32_t padded,
                                        pp_gen_layout* layout) {
    pp::clear_error();
    if (!lengths || !layout) return pp::fail(PP_ERR_INVALID_ARG, "lengths and layout must be non-NULL");
    if (k <= 0 || n_new <= 0 || (padded != 0 && padded != 1))
        return pp::fail(PP_ERR_INVALID_ARG, "k %d, n_new %d, padded %d", k, n_new, padded);
    if (!layout->ctx_off || !layout->ctx_span || !layout->ctx_valid || !layout->pos0 || !layout->gen_off)
        return pp::fail(PP_ERR_INVALID_ARG, "a layout array is NULL");
    int64_t total = 0;
    int32_t m = 0;
    for (int32_t i = 0; i < k; ++i) {
        if (lengths[i] <= 0) return pp::fail(PP_ERR_INVALID_ARG, "length %d of prompt %d", lengths[i], i);
        total += lengths[i];
        m = std::max(m, lengths[i]);
    }
    const int64_t row = int64_t(m) + n_new;
    const int64_t ctx_rows = padded ? int64_t(k) * row : total;
    const int64_t gen_rows = padded ? int64_t(k) * row : int64_t(k) * n_new;
    if (ctx_rows > INT32_MAX || gen_rows > INT32_MAX)
        return pp::fail(PP_ERR_INVALID_ARG, "%lld cache rows exceed the int32 row index", (long long)gen_rows);
    int64_t off = 0;
    for (int32_t i = 0; i < k; ++i) {
        layout->ctx_off[i] = static_cast<int32_t>(padded ? int64_t(i) * row : off);
        layout->ctx_span[i] = padded ? m : lengths[i];
        layout->ctx_valid[i] = lengths[i];
        layout->pos0[i] = lengths[i];
        layout->gen_off[i] = static_cast<int32_t>(padded ? int64_t(i) * row + m : int64_t(i) * n_new);
        off += lengths[i];
    }
    layout->k = k;
    layout->n_new = n_new;
    layout->padded = padded;
    layout->max_len = m;
    layout->ctx_rows = ctx_rows;
    layout->gen_rows = gen_rows;
    return PP_OK;
}

extern "C" pp_status pp_decode_workspace_size(const pp_config* cfg, const pp_gen_dlayout* layout, size_t* bytes) {
    pp::clear_error();
    if (pp_status st = pp::validate_config(cfg)) return st;
    if (pp_status st = validate_layout(cfg, layout)) return st;
    if (!bytes) return pp::fail(PP_ERR_INVALID_ARG, "bytes is NULL");
    *bytes = layout_of(cfg, layout).total;
    return PP_OK;
}

extern "C" pp_status pp_decode_step(const pp_config* cfg, const pp_weights* w, const pp_gen_dlayout* layout,
                                    int32_t step, const int32_t* tokens_in, const void* lm_head, const void* ctx_k,
                                    const void* ctx_v, void* gen_k, void* gen_v, void* workspace,
                                    size_t workspace_bytes, float* logits, int32_t* tokens_out, void* stream) {
    pp::clear_error();
    if (pp_status st = check_all(cfg, w, layout)) return st;
    if (step < 0 || step >= layout->n_new)
        return pp::fail(PP_ERR_INVALID_ARG, "step %d outside [0, n_new = %d)", step, layout->n_new);
    if (!tokens_in || !tokens_out) return pp::fail(PP_ERR_INVALID_ARG, "tokens_in and tokens_out must be non-NULL");
    if (pp_status st = check_buffers(cfg, layout, lm_head, ctx_k, ctx_v, gen_k, gen_v, workspace, workspace_bytes))
        return st;
    (void)hipGetLastError();
    enqueue_step(cfg, w, layout, step, tokens_in, lm_head, ctx_k, ctx_v, gen_k, gen_v, workspace, logits, tokens_out,
                 static_cast<hipStream_t>(stream));
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return pp::fail(PP_ERR_HIP, "decode step launch failed: %s", hipGetErrorString(err));
    return PP_OK;
}

extern "C" pp_status pp_generate(const pp_config* cfg, const pp_weights* w, const pp_gen_dlayout* layout,
                                 int32_t n_steps, const int32_t* tokens_first, const void* lm_head, const void* ctx_k,
                                 const void* ctx_v, void* gen_k, void* gen_v, void* workspace,
                                 size_t workspace_bytes, int32_t* tokens, void* stream) {
    pp::clear_error();
    if (pp_status st = check_all(cfg, w, layout)) return st;
    if (n_steps < 0 || n_steps > layout->n_new)
        return pp::fail(PP_ERR_INVALID_ARG, "n_steps %d outside [0, n_new = %d]", n_steps, layout->n_new);
    if (n_steps == 0) return PP_OK;
    if (!tokens_first || !tokens) return pp::fail(PP_ERR_INVALID_ARG, "tokens_first and tokens must be non-NULL");
    if (pp_status st = check_buffers(cfg, layout, lm_head, ctx_k, ctx_v, gen_k, gen_v, workspace, workspace_bytes))
        return st;
    (void)hipGetLastError();
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int k = layout->k;
    for (int t = 0; t < n_steps; ++t)
        enqueue_step(cfg, w, layout, t, t == 0 ? tokens_first : tokens + int64_t(t - 1) * k, lm_head, ctx_k, ctx_v,
                     gen_k, gen_v, workspace, nullptr, tokens + int64_t(t) * k, s);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return pp::fail(PP_ERR_HIP, "generate launch failed: %s", hipGetErrorString(err));
    return PP_OK;
}
