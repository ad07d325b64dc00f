// pp_prefill: the model call and UNPACK of Algorithm 1 over a packed batch.
//
// Host side only: validates every argument, carves the caller's workspace, and enqueues
// the kernel sequence on the caller's stream without any host synchronisation:
//
//   rope_table; embed (TENSORIZE through the slot map)
//   per layer: rmsnorm -> QKV projection with RoPE at restart positions and the KV UNPACK
//              fused into its epilogue (bf16; float32 runs GEMM, RoPE and scatter as three
//              launches) -> attention under the independent mask, keys and values read
//              from the caches -> O GEMM (+residual) -> rmsnorm -> gate/up GEMM with
//              SwiGLU -> down GEMM (+residual)
//   final rmsnorm fused with the hidden-state UNPACK.
#include <hip/hip_runtime.h>

#include <cstdint>

#include "kernels.h"
#include "prepack.h"
#include "status.h"

namespace {

constexpr size_t kAlign = 256;
size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

struct Layout {
    size_t x = 0, xn = 0, qkv = 0, attn = 0, act = 0, gu = 0, table = 0, total = 0;
};

size_t elem_size(int dtype) { return dtype == PP_BF16 ? 2 : 4; }

// The attention kernel addresses one prompt's cache rows through a 32-bit buffer range.
pp_status validate_attention_span(const pp_config* c, const pp_dplan* p) {
    const int64_t kvw = int64_t(c->n_kv_heads) * c->head_dim;
    if (c->dtype == PP_BF16 && (int64_t(p->max_len) + 2 * 64) * kvw * 2 > INT32_MAX)
        return pp::fail(PP_ERR_UNSUPPORTED, "max_len %d too long for the attention kernel at this width",
                        p->max_len);
    return PP_OK;
}

pp_status validate_plan(const pp_dplan* p) {
    if (!p) return pp::fail(PP_ERR_INVALID_ARG, "plan is NULL");
    if (p->k < 0 || p->capacity < 0 || p->n_rows < 0 || p->max_len < 0 || p->total_len < 0 || p->n_qtiles < 0 ||
        p->n_mtiles < 0)
        return pp::fail(PP_ERR_INVALID_ARG, "plan scalars must be non-negative");
    if (int64_t(p->n_rows) * p->capacity > INT32_MAX)
        return pp::fail(PP_ERR_INVALID_ARG, "n_rows * capacity overflows int32");
    const int64_t T = int64_t(p->n_rows) * p->capacity;
    if (p->total_len > T || p->max_len > p->capacity || int64_t(p->n_mtiles) * PP_MTILE >= T + PP_MTILE ||
        (p->total_len > 0 && (p->n_qtiles == 0 || p->n_mtiles == 0 || p->max_len == 0)))
        return pp::fail(PP_ERR_INVALID_ARG, "inconsistent plan (total_len %d, rows %d x %d, max_len %d)",
                        p->total_len, p->n_rows, p->capacity, p->max_len);
    if (p->total_len > 0 && (!p->seg_prompt || !p->seg_start || !p->seg_len || !p->prompt_kv_off ||
                             !p->slot_seg || !p->slot_pos || !p->slot_kv || !p->qtile_seg || !p->qtile_q0 ||
                             !p->mtile_m0))
        return pp::fail(PP_ERR_INVALID_ARG, "a device plan array is NULL");
    return PP_OK;
}

Layout layout_of(const pp_config* c, const pp_dplan* p) {
    const size_t T = size_t(p->n_rows) * p->capacity;
    const size_t e = elem_size(c->dtype);
    const size_t d = c->d_model, F = c->ffn_dim;
    const size_t qkv_w = size_t(c->n_heads + 2 * c->n_kv_heads) * c->head_dim;
    const size_t hd = size_t(c->n_heads) * c->head_dim;
    Layout L;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        const size_t at = off;
        off += align_up(bytes);
        return at;
    };
    L.x = take(T * d * 4);
    L.xn = take(T * d * e);
    L.qkv = take(c->dtype == PP_BF16 ? T * hd * 2 : T * qkv_w * 4);   // bf16: queries only
    L.attn = take(T * hd * e);
    L.act = take(T * F * e);
    L.gu = take(c->dtype == PP_F32 ? T * 2 * F * 4 : 0);
    L.table = take(size_t(p->max_len) * (c->head_dim / 2) * sizeof(float2));
    L.total = off;
    return L;
}

}  // namespace

namespace pp {

pp_status validate_config(const pp_config* c) {
    if (!c) return pp::fail(PP_ERR_INVALID_ARG, "config is NULL");
    if (c->n_layers <= 0 || c->d_model <= 0 || c->n_heads <= 0 || c->n_kv_heads <= 0 || c->head_dim <= 0 ||
        c->ffn_dim <= 0 || c->vocab <= 0)
        return pp::fail(PP_ERR_INVALID_ARG, "config sizes must be positive");
    if (c->dtype != PP_F32 && c->dtype != PP_BF16) return pp::fail(PP_ERR_INVALID_ARG, "unknown dtype %d", c->dtype);
    if (!(c->rms_eps >= 0.f) || !(c->rope_theta > 0.f))
        return pp::fail(PP_ERR_INVALID_ARG, "rms_eps must be >= 0 and rope_theta > 0");
    if (c->n_heads % c->n_kv_heads)
        return pp::fail(PP_ERR_UNSUPPORTED, "n_heads %d is not a multiple of n_kv_heads %d", c->n_heads,
                        c->n_kv_heads);
    if (c->head_dim != 64 && c->head_dim != 128)
        return pp::fail(PP_ERR_UNSUPPORTED, "head_dim %d (supported: 64, 128)", c->head_dim);
    const int64_t qkv_w = int64_t(c->n_heads + 2 * c->n_kv_heads) * c->head_dim;
    const int64_t hd = int64_t(c->n_heads) * c->head_dim;
    if (c->dtype == PP_BF16) {
        if (c->head_dim != 128) return pp::fail(PP_ERR_UNSUPPORTED, "bf16 attention needs head_dim 128");
        if (c->d_model % 256 || c->ffn_dim % 128 || qkv_w % 256 || hd % 64)
            return pp::fail(PP_ERR_UNSUPPORTED,
                            "bf16 GEMM tiles need d %% 256 == 0, F %% 128 == 0, (H+2Hkv)D %% 256 == 0 "
                            "(d=%d F=%d (H+2Hkv)D=%lld)",
                            c->d_model, c->ffn_dim, (long long)qkv_w);
    } else {
        if (c->d_model % 16 || c->ffn_dim % 16 || hd % 16)
            return pp::fail(PP_ERR_UNSUPPORTED, "f32 path needs d, F and H*D multiples of 16");
    }
    return PP_OK;
}

pp_status validate_weights(const pp_config* c, const pp_weights* w) {
    if (!w) return pp::fail(PP_ERR_INVALID_ARG, "weights is NULL");
    if (!w->embed || !w->final_norm || !w->attn_norm || !w->wqkv || !w->wo || !w->mlp_norm || !w->w_gateup ||
        !w->w_down)
        return pp::fail(PP_ERR_INVALID_ARG, "a weight pointer is NULL");
    for (int l = 0; l < c->n_layers; ++l)
        if (!w->attn_norm[l] || !w->wqkv[l] || !w->wo[l] || !w->mlp_norm[l] || !w->w_gateup[l] || !w->w_down[l])
            return pp::fail(PP_ERR_INVALID_ARG, "a weight pointer of layer %d is NULL", l);
    return PP_OK;
}

}  // namespace pp

using pp::validate_config;
using pp::validate_weights;

extern "C" pp_status pp_prefill_workspace_size(const pp_config* cfg, const pp_dplan* plan, size_t* bytes) {
    pp::clear_error();
    if (pp_status st = validate_config(cfg)) return st;
    if (pp_status st = validate_plan(plan)) return st;
    if (pp_status st = validate_attention_span(cfg, plan)) return st;
    if (!bytes) return pp::fail(PP_ERR_INVALID_ARG, "bytes is NULL");
    *bytes = layout_of(cfg, plan).total;
    return PP_OK;
}

extern "C" pp_status pp_prefill(const pp_config* cfg, const pp_weights* w, const pp_dplan* plan,
                                const int32_t* tokens, void* workspace, size_t workspace_bytes, float* hidden,
                                void* k_cache, void* v_cache, void* stream) {
    pp::clear_error();
    if (pp_status st = validate_config(cfg)) return st;
    if (pp_status st = validate_plan(plan)) return st;
    if (pp_status st = validate_attention_span(cfg, plan)) return st;
    if (pp_status st = validate_weights(cfg, w)) return st;
    if (plan->total_len == 0) return PP_OK;
    if (!tokens || !hidden || !k_cache || !v_cache)
        return pp::fail(PP_ERR_INVALID_ARG, "tokens, hidden, k_cache and v_cache must be non-NULL");
    const Layout L = layout_of(cfg, plan);
    if (!workspace) return pp::fail(PP_ERR_INVALID_ARG, "workspace is NULL");
    if (reinterpret_cast<uintptr_t>(workspace) % kAlign)
        return pp::fail(PP_ERR_INVALID_ARG, "workspace is not %zu-byte aligned", kAlign);
    if (workspace_bytes < L.total)
        return pp::fail(PP_ERR_BUFFER_TOO_SMALL, "workspace of %zu bytes < %zu needed", workspace_bytes, L.total);

    hipStream_t s = static_cast<hipStream_t>(stream);
    (void)hipGetLastError();  // report only errors raised by the launches below

    const int dt = cfg->dtype;
    const bool bf = dt == PP_BF16;
    const int T = plan->n_rows * plan->capacity;
    const int d = cfg->d_model, H = cfg->n_heads, Hkv = cfg->n_kv_heads, D = cfg->head_dim, F = cfg->ffn_dim;
    const int qkv_w = (H + 2 * Hkv) * D, hd = H * D, kvw = Hkv * D;
    const float eps = cfg->rms_eps;
    const size_t e = elem_size(dt);

    char* ws = static_cast<char*>(workspace);
    float* x = reinterpret_cast<float*>(ws + L.x);
    void* xn = ws + L.xn;
    void* qkv = ws + L.qkv;
    void* attn = ws + L.attn;
    void* act = ws + L.act;
    float* gu = reinterpret_cast<float*>(ws + L.gu);
    float2* table = reinterpret_cast<float2*>(ws + L.table);
    const size_t cache_layer_bytes = size_t(plan->total_len) * kvw * e;

    ppk::rope_table(table, plan->max_len, D, cfg->rope_theta, s);
    ppk::embed(dt, x, w->embed, cfg->vocab, tokens, plan->slot_kv, T, d, s);
    for (int l = 0; l < cfg->n_layers; ++l) {
        void* kc = static_cast<char*>(k_cache) + l * cache_layer_bytes;
        void* vc = static_cast<char*>(v_cache) + l * cache_layer_bytes;
        ppk::rmsnorm(dt, x, w->attn_norm[l], xn, T, d, eps, s);
        if (bf) {
            const ppk::QkvOut qo{qkv, hd, kc, vc, kvw, table, plan->slot_pos, plan->slot_kv, H, Hkv};
            ppk::qkv_rope_bf16(xn, d, w->wqkv[l], d, T, d, plan->mtile_m0, plan->n_mtiles, qo, s);
            ppk::attention_bf16(qkv, hd, kc, vc, kvw, attn, hd, plan->seg_prompt, plan->seg_start, plan->seg_len,
                                plan->prompt_kv_off, plan->qtile_seg, plan->qtile_q0, plan->n_qtiles, H, Hkv, s);
            ppk::gemm_bf16(ppk::kResidual, attn, hd, w->wo[l], hd, x, d, T, d, hd, plan->mtile_m0, plan->n_mtiles, s);
        } else {
            float* qkv32 = static_cast<float*>(qkv);
            ppk::gemm_f32(ppk::kStore, static_cast<const float*>(xn), d, static_cast<const float*>(w->wqkv[l]), d,
                          qkv32, qkv_w, T, qkv_w, d, s);
            ppk::rope_apply(dt, qkv, qkv_w, table, plan->slot_pos, plan->slot_seg, T, H + Hkv, D, s);
            ppk::kv_scatter(dt, qkv, qkv_w, hd, kvw, kc, vc, plan->slot_kv, T, s);
            ppk::attention_f32(qkv32, qkv_w, static_cast<const float*>(kc), static_cast<const float*>(vc), kvw,
                               static_cast<float*>(attn), hd, plan->slot_seg, plan->seg_prompt, plan->seg_start,
                               plan->prompt_kv_off, T, H, Hkv, D, s);
            ppk::gemm_f32(ppk::kResidual, static_cast<const float*>(attn), hd, static_cast<const float*>(w->wo[l]),
                          hd, x, d, T, d, hd, s);
        }
        ppk::rmsnorm(dt, x, w->mlp_norm[l], xn, T, d, eps, s);
        if (bf) {
            ppk::gemm_bf16(ppk::kSwiGLU, xn, d, w->w_gateup[l], d, act, F, T, 2 * F, d, plan->mtile_m0, plan->n_mtiles,
                           s);
            ppk::gemm_bf16(ppk::kResidual, act, F, w->w_down[l], F, x, d, T, d, F, plan->mtile_m0, plan->n_mtiles, s);
        } else {
            ppk::gemm_f32(ppk::kStore, static_cast<const float*>(xn), d, static_cast<const float*>(w->w_gateup[l]), d,
                          gu, 2 * F, T, 2 * F, d, s);
            ppk::swiglu_f32(gu, static_cast<float*>(act), T, F, s);
            ppk::gemm_f32(ppk::kResidual, static_cast<const float*>(act), F, static_cast<const float*>(w->w_down[l]),
                          F, x, d, T, d, F, s);
        }
    }
    ppk::rmsnorm_unpack(x, w->final_norm, hidden, plan->slot_kv, T, d, eps, s);

    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return pp::fail(PP_ERR_HIP, "kernel launch failed: %s", hipGetErrorString(err));
    return PP_OK;
}

// ------------------------------------------------------------------------------------------
// Single steps (the same launches pp_prefill makes).
// ------------------------------------------------------------------------------------------
namespace {

pp_status finish(const char* what) {
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return pp::fail(PP_ERR_HIP, "%s launch failed: %s", what, hipGetErrorString(err));
    return PP_OK;
}

bool bad_dtype(int32_t dt) { return dt != PP_F32 && dt != PP_BF16; }

}  // namespace

extern "C" pp_status pp_embed(int32_t dtype, const void* embed, int32_t vocab, int32_t d, const int32_t* tokens,
                              const pp_dplan* plan, float* x, void* stream) {
    pp::clear_error();
    if (bad_dtype(dtype)) return pp::fail(PP_ERR_INVALID_ARG, "unknown dtype %d", dtype);
    if (pp_status st = validate_plan(plan)) return st;
    if (d <= 0 || d % 8) return pp::fail(PP_ERR_UNSUPPORTED, "d = %d must be a positive multiple of 8", d);
    if (vocab <= 0) return pp::fail(PP_ERR_INVALID_ARG, "vocab = %d must be positive", vocab);
    const int T = plan->n_rows * plan->capacity;
    if (T == 0) return PP_OK;
    if (!embed || !tokens || !x) return pp::fail(PP_ERR_INVALID_ARG, "NULL buffer");
    (void)hipGetLastError();
    ppk::embed(dtype, x, embed, vocab, tokens, plan->slot_kv, T, d, static_cast<hipStream_t>(stream));
    return finish("embed");
}

extern "C" pp_status pp_rmsnorm(int32_t dtype, const float* x, const float* gain, int32_t rows, int32_t d,
                                float eps, void* out, void* stream) {
    pp::clear_error();
    if (bad_dtype(dtype)) return pp::fail(PP_ERR_INVALID_ARG, "unknown dtype %d", dtype);
    if (rows < 0 || d <= 0 || d % 4) return pp::fail(PP_ERR_INVALID_ARG, "rows %d, d %d (d %% 4 == 0)", rows, d);
    if (!(eps >= 0.f)) return pp::fail(PP_ERR_INVALID_ARG, "eps must be >= 0");
    if (rows == 0) return PP_OK;
    if (!x || !gain || !out) return pp::fail(PP_ERR_INVALID_ARG, "NULL buffer");
    (void)hipGetLastError();
    ppk::rmsnorm(dtype, x, gain, out, rows, d, eps, static_cast<hipStream_t>(stream));
    return finish("rmsnorm");
}

extern "C" pp_status pp_gemm(int32_t dtype, int32_t epilogue, const void* A, int64_t lda, const void* B,
                             int64_t ldb, void* C, int64_t ldc, int32_t M, int32_t N, int32_t K,
                             const pp_dplan* plan, void* stream) {
    pp::clear_error();
    if (bad_dtype(dtype)) return pp::fail(PP_ERR_INVALID_ARG, "unknown dtype %d", dtype);
    if (epilogue < PP_EPI_STORE || epilogue > PP_EPI_SWIGLU)
        return pp::fail(PP_ERR_INVALID_ARG, "unknown epilogue %d", epilogue);
    if (M < 0 || N <= 0 || K <= 0) return pp::fail(PP_ERR_INVALID_ARG, "M %d, N %d, K %d", M, N, K);
    const int64_t out_cols = epilogue == PP_EPI_SWIGLU ? N / 2 : N;
    if (lda < K || ldb < K || ldc < out_cols)
        return pp::fail(PP_ERR_INVALID_ARG, "leading dimensions too small (lda %lld ldb %lld ldc %lld)",
                        (long long)lda, (long long)ldb, (long long)ldc);
    if (dtype == PP_BF16) {
        if (N % 256 || K % 64 || lda % 8 || ldb % 8 || ldc % 4)
            return pp::fail(PP_ERR_UNSUPPORTED, "bf16 GEMM needs N %% 256 == 0, K %% 64 == 0, lda/ldb %% 8 == 0, "
                            "ldc %% 4 == 0 (N %d K %d)", N, K);
    } else {
        if (epilogue == PP_EPI_SWIGLU) return pp::fail(PP_ERR_UNSUPPORTED, "f32 GEMM has no SwiGLU epilogue");
        if (K % 16 || lda % 4 || ldb % 4) return pp::fail(PP_ERR_UNSUPPORTED, "f32 GEMM needs K %% 16 == 0");
    }
    if (plan) {
        if (pp_status st = validate_plan(plan)) return st;
        if (dtype != PP_BF16) return pp::fail(PP_ERR_UNSUPPORTED, "row-tile skipping is a bf16 GEMM feature");
        if (int64_t(M) != int64_t(plan->n_rows) * plan->capacity)
            return pp::fail(PP_ERR_INVALID_ARG, "M %d != n_rows * capacity of the plan", M);
        if (M > 0 && !plan->mtile_m0) return pp::fail(PP_ERR_INVALID_ARG, "plan mtile_m0 is NULL");
    }
    if (M == 0) return PP_OK;
    if (!A || !B || !C) return pp::fail(PP_ERR_INVALID_ARG, "NULL buffer");
    (void)hipGetLastError();
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (dtype == PP_BF16)
        ppk::gemm_bf16(epilogue, A, lda, B, ldb, C, ldc, M, N, K, plan ? plan->mtile_m0 : nullptr,
                       plan ? plan->n_mtiles : 0, s);
    else
        ppk::gemm_f32(epilogue, static_cast<const float*>(A), lda, static_cast<const float*>(B), ldb,
                      static_cast<float*>(C), ldc, M, N, K, s);
    return finish("gemm");
}

extern "C" pp_status pp_qkv_projection(const pp_config* cfg, const pp_dplan* plan, const void* xn,
                                       const void* wqkv, void* table, void* q_out, void* k_cache, void* v_cache,
                                       void* stream) {
    pp::clear_error();
    if (pp_status st = validate_config(cfg)) return st;
    if (cfg->dtype != PP_BF16)
        return pp::fail(PP_ERR_UNSUPPORTED, "the fused QKV projection is bf16 only (float32: pp_gemm, pp_rope, "
                        "pp_kv_scatter)");
    if (pp_status st = validate_plan(plan)) return st;
    const int T = plan->n_rows * plan->capacity;
    if (T == 0 || plan->total_len == 0) return PP_OK;
    if (!xn || !wqkv || !table || !q_out || !k_cache || !v_cache)
        return pp::fail(PP_ERR_INVALID_ARG, "NULL buffer");
    (void)hipGetLastError();
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int H = cfg->n_heads, Hkv = cfg->n_kv_heads, D = cfg->head_dim, d = cfg->d_model;
    float2* tab = static_cast<float2*>(table);
    ppk::rope_table(tab, plan->max_len, D, cfg->rope_theta, s);
    const ppk::QkvOut qo{q_out, int64_t(H) * D, k_cache, v_cache, int64_t(Hkv) * D, tab, plan->slot_pos,
                         plan->slot_kv, H, Hkv};
    ppk::qkv_rope_bf16(xn, d, wqkv, d, T, d, plan->mtile_m0, plan->n_mtiles, qo, s);
    return finish("qkv_projection");
}

extern "C" pp_status pp_rope(const pp_config* cfg, const pp_dplan* plan, void* qkv, void* table, void* stream) {
    pp::clear_error();
    if (pp_status st = validate_config(cfg)) return st;
    if (pp_status st = validate_plan(plan)) return st;
    const int T = plan->n_rows * plan->capacity;
    if (T == 0) return PP_OK;
    if (!qkv || !table) return pp::fail(PP_ERR_INVALID_ARG, "NULL buffer");
    (void)hipGetLastError();
    hipStream_t s = static_cast<hipStream_t>(stream);
    const int qkv_w = (cfg->n_heads + 2 * cfg->n_kv_heads) * cfg->head_dim;
    float2* tab = static_cast<float2*>(table);
    ppk::rope_table(tab, plan->max_len, cfg->head_dim, cfg->rope_theta, s);
    ppk::rope_apply(cfg->dtype, qkv, qkv_w, tab, plan->slot_pos, plan->slot_seg, T,
                    cfg->n_heads + cfg->n_kv_heads, cfg->head_dim, s);
    return finish("rope");
}

extern "C" pp_status pp_kv_scatter(const pp_config* cfg, const pp_dplan* plan, const void* qkv, void* k_cache,
                                   void* v_cache, void* stream) {
    pp::clear_error();
    if (pp_status st = validate_config(cfg)) return st;
    if (pp_status st = validate_plan(plan)) return st;
    const int T = plan->n_rows * plan->capacity;
    if (T == 0 || plan->total_len == 0) return PP_OK;
    if (!qkv || !k_cache || !v_cache) return pp::fail(PP_ERR_INVALID_ARG, "NULL buffer");
    (void)hipGetLastError();
    const int H = cfg->n_heads, Hkv = cfg->n_kv_heads, D = cfg->head_dim;
    ppk::kv_scatter(cfg->dtype, qkv, (H + 2 * Hkv) * D, H * D, Hkv * D, k_cache, v_cache, plan->slot_kv, T,
                    static_cast<hipStream_t>(stream));
    return finish("kv_scatter");
}

extern "C" pp_status pp_attention(const pp_config* cfg, const pp_dplan* plan, const void* q, int64_t ldq,
                                  const void* k_cache, const void* v_cache, void* out, void* stream) {
    pp::clear_error();
    if (pp_status st = validate_config(cfg)) return st;
    if (pp_status st = validate_plan(plan)) return st;
    if (pp_status st = validate_attention_span(cfg, plan)) return st;
    const int H = cfg->n_heads, Hkv = cfg->n_kv_heads, D = cfg->head_dim;
    if (ldq < int64_t(H) * D) return pp::fail(PP_ERR_INVALID_ARG, "ldq %lld < H*D", (long long)ldq);
    if (cfg->dtype == PP_BF16 && ldq % 8) return pp::fail(PP_ERR_UNSUPPORTED, "bf16 attention needs ldq %% 8 == 0");
    const int T = plan->n_rows * plan->capacity;
    if (T == 0 || plan->total_len == 0) return PP_OK;
    if (!q || !k_cache || !v_cache || !out) return pp::fail(PP_ERR_INVALID_ARG, "NULL buffer");
    (void)hipGetLastError();
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (cfg->dtype == PP_BF16)
        ppk::attention_bf16(q, ldq, k_cache, v_cache, int64_t(Hkv) * D, out, int64_t(H) * D, plan->seg_prompt,
                            plan->seg_start, plan->seg_len, plan->prompt_kv_off, plan->qtile_seg, plan->qtile_q0,
                            plan->n_qtiles, H, Hkv, s);
    else
        ppk::attention_f32(static_cast<const float*>(q), ldq, static_cast<const float*>(k_cache),
                           static_cast<const float*>(v_cache), int64_t(Hkv) * D, static_cast<float*>(out),
                           int64_t(H) * D, plan->slot_seg, plan->seg_prompt, plan->seg_start, plan->prompt_kv_off,
                           T, H, Hkv, D, s);
    return finish("attention");
}

extern "C" pp_status pp_final_norm_unpack(const float* x, const float* gain, int32_t d, float eps,
                                          const pp_dplan* plan, float* hidden, void* stream) {
    pp::clear_error();
    if (pp_status st = validate_plan(plan)) return st;
    if (d <= 0 || d % 4) return pp::fail(PP_ERR_INVALID_ARG, "d = %d must be a positive multiple of 4", d);
    if (!(eps >= 0.f)) return pp::fail(PP_ERR_INVALID_ARG, "eps must be >= 0");
    const int T = plan->n_rows * plan->capacity;
    if (T == 0 || plan->total_len == 0) return PP_OK;
    if (!x || !gain || !hidden) return pp::fail(PP_ERR_INVALID_ARG, "NULL buffer");
    (void)hipGetLastError();
    ppk::rmsnorm_unpack(x, gain, hidden, plan->slot_kv, T, d, eps, static_cast<hipStream_t>(stream));
    return finish("final_norm_unpack");
}

extern "C" pp_status pp_first_token_workspace_size(const pp_config* cfg, const pp_dplan* plan, size_t* bytes) {
    pp::clear_error();
    if (pp_status st = validate_config(cfg)) return st;
    if (pp_status st = validate_plan(plan)) return st;
    if (!bytes) return pp::fail(PP_ERR_INVALID_ARG, "bytes is NULL");
    *bytes = plan->k > 0 ? ppk::first_token_workspace(cfg->dtype, plan->k, cfg->vocab, cfg->d_model) : 0;
    return PP_OK;
}

namespace {

// The checks pp_first_token and pp_first_token_noalloc share; *need = workspace bytes.
pp_status check_first_token(const pp_config* cfg, const pp_dplan* plan, const float* hidden, const void* lm_head,
                            const int32_t* tokens, size_t* need) {
    if (pp_status st = validate_config(cfg)) return st;
    if (pp_status st = validate_plan(plan)) return st;
    *need = 0;
    if (plan->k == 0) return PP_OK;
    if (plan->total_len < plan->k)
        return pp::fail(PP_ERR_INVALID_ARG, "plan has %d prompts but %d tokens", plan->k, plan->total_len);
    if (!plan->prompt_kv_off) return pp::fail(PP_ERR_INVALID_ARG, "prompt_kv_off is NULL");
    if (!hidden || !lm_head || !tokens) return pp::fail(PP_ERR_INVALID_ARG, "NULL buffer");
    *need = ppk::first_token_workspace(cfg->dtype, plan->k, cfg->vocab, cfg->d_model);
    return PP_OK;
}

}  // namespace

extern "C" pp_status pp_first_token(const pp_config* cfg, const pp_dplan* plan, const float* hidden,
                                    const void* lm_head, void* workspace, size_t workspace_bytes, float* logits,
                                    int32_t* tokens, void* stream) {
    pp::clear_error();
    size_t need = 0;
    if (pp_status st = check_first_token(cfg, plan, hidden, lm_head, tokens, &need)) return st;
    if (plan->k == 0) return PP_OK;
    if (!workspace) return pp::fail(PP_ERR_INVALID_ARG, "NULL buffer");
    if (reinterpret_cast<uintptr_t>(workspace) % kAlign)
        return pp::fail(PP_ERR_INVALID_ARG, "workspace is not %zu-byte aligned", kAlign);
    if (workspace_bytes < need)
        return pp::fail(PP_ERR_BUFFER_TOO_SMALL, "workspace of %zu bytes < %zu needed", workspace_bytes, need);
    (void)hipGetLastError();
    ppk::first_token(cfg->dtype, hidden, plan->prompt_kv_off, plan->k, lm_head, cfg->vocab, cfg->d_model, workspace,
                     logits, tokens, static_cast<hipStream_t>(stream));
    return finish("first_token");
}

extern "C" pp_status pp_first_token_noalloc(const pp_config* cfg, const pp_dplan* plan, const float* hidden,
                                            const void* lm_head, float* logits, int32_t* tokens, void* stream) {
    pp::clear_error();
    size_t need = 0;
    if (pp_status st = check_first_token(cfg, plan, hidden, lm_head, tokens, &need)) return st;
    if (plan->k == 0) return PP_OK;
    if (need > PP_FIRST_TOKEN_SCRATCH_BYTES)
        return pp::fail(PP_ERR_BUFFER_TOO_SMALL,
                        "%d prompts with vocab %d and d %d need %zu bytes of workspace, more than the %u bytes "
                        "of pp_first_token_noalloc's static buffer (use pp_first_token)",
                        plan->k, cfg->vocab, cfg->d_model, need, PP_FIRST_TOKEN_SCRATCH_BYTES);
    void* ws = nullptr;
    const hipError_t e = ppk::first_token_scratch(&ws);
    if (e != hipSuccess)
        return pp::fail(PP_ERR_HIP, "address of the static first-token buffer: %s", hipGetErrorString(e));
    (void)hipGetLastError();
    ppk::first_token(cfg->dtype, hidden, plan->prompt_kv_off, plan->k, lm_head, cfg->vocab, cfg->d_model, ws, logits,
                     tokens, static_cast<hipStream_t>(stream));
    return finish("first_token_noalloc");
}
