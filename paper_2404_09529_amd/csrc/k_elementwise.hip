// HBM-bound kernels of the packed prefill: TENSORIZE (embedding gather into the packed
// batch), RMSNorm, restart-position RoPE (section 3.2), the KV-cache UNPACK scatter
// (Algorithm 1) and the final norm fused with the hidden-state unpack.
//
// Every kernel walks rows of the packed batch with one 64-wide wavefront per row (or per
// contiguous 8-element chunk), so each wavefront touches whole 16-byte-aligned runs and
// the loads/stores are fully coalesced.
#include "device.h"
#include "kernels.h"
#include "prepack.h"

namespace {

constexpr int kBlock = 256;
constexpr int kRowsPerBlock = kBlock / kWave;

template <typename T>
T* at(void* p) { return static_cast<T*>(p); }

// ------------------------------------------------------------------------------- RoPE table
__global__ void rope_table_kernel(float2* __restrict__ table, int64_t n, int half, int D, double theta) {
    const int64_t idx = int64_t(blockIdx.x) * blockDim.x + threadIdx.x;
    if (idx >= n) return;
    const int64_t p = idx / half;
    const int i = static_cast<int>(idx % half);
    const double inv_freq = pow(theta, -2.0 * i / static_cast<double>(D));
    const double a = static_cast<double>(p) * inv_freq;
    table[idx] = make_float2(static_cast<float>(cos(a)), static_cast<float>(sin(a)));
}

// ------------------------------------------------------------------------------- embedding
// NC > 0: d == NC * 512 (8 elements per lane per chunk); every load of the row is issued
// before the first store, so a wavefront has the whole row in flight.  NC == 0: any d that
// is a multiple of 8, one chunk at a time.
template <typename TE, int NC>
__global__ __launch_bounds__(kBlock) void embed_kernel(float* __restrict__ x, const TE* __restrict__ E,
                                                       const int32_t* __restrict__ tokens,
                                                       const int32_t* __restrict__ slot_kv, int T, int d,
                                                       int vocab) {
    const int lane = threadIdx.x % kWave;
    const int64_t row = int64_t(blockIdx.x) * kRowsPerBlock + threadIdx.x / kWave;
    if (row >= T) return;
    float* xr = x + row * d;
    const int kv = slot_kv[row];
    const int tok = kv < 0 ? -1 : tokens[kv];
    if (tok < 0 || tok >= vocab) {  // pad slot, or a token id outside the vocabulary
        float z[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) z[i] = 0.f;
        for (int c = lane * 8; c < d; c += kWave * 8) store8(xr + c, z);
        return;
    }
    const TE* er = E + int64_t(tok) * d;
    if constexpr (NC > 0) {
        float v[NC][8];
#pragma unroll
        for (int c = 0; c < NC; ++c) load8(er + c * 512 + lane * 8, v[c]);
#pragma unroll
        for (int c = 0; c < NC; ++c) store8(xr + c * 512 + lane * 8, v[c]);
    } else {
        float v[8];
        for (int c = lane * 8; c < d; c += kWave * 8) {
            load8(er + c, v);
            store8(xr + c, v);
        }
    }
}

template <typename TE>
void embed_dispatch(float* x, const TE* E, int vocab, const int32_t* tokens, const int32_t* slot_kv, int T, int d,
                    hipStream_t s) {
    const dim3 grid((T + kRowsPerBlock - 1) / kRowsPerBlock);
    const int nc = d % 512 == 0 ? d / 512 : 0;
#define PP_EMB(NC) embed_kernel<TE, NC><<<grid, kBlock, 0, s>>>(x, E, tokens, slot_kv, T, d, vocab)
    switch (nc) {
        case 2: PP_EMB(2); break;
        case 4: PP_EMB(4); break;
        case 8: PP_EMB(8); break;
        case 16: PP_EMB(16); break;
        default: PP_EMB(0); break;
    }
#undef PP_EMB
}

// ------------------------------------------------------------------------------- RMSNorm
__device__ __forceinline__ void store4(float* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }
__device__ __forceinline__ void store4(bf16* p, f32x4 v) {
    bf16x4 b;
#pragma unroll
    for (int i = 0; i < 4; ++i) b[i] = static_cast<bf16>(v[i]);
    *reinterpret_cast<bf16x4*>(p) = b;
}

// NC > 0: d == NC * 256, the row is held in registers (one read of x).  NC == 0: any d that
// is a multiple of 4, two passes over the row.
template <typename TO, int NC, bool UNPACK>
__global__ __launch_bounds__(kBlock) void rmsnorm_kernel(const float* __restrict__ x, const float* __restrict__ g,
                                                         TO* __restrict__ out,
                                                         const int32_t* __restrict__ slot_kv, int T, int d,
                                                         float eps) {
    const int lane = threadIdx.x % kWave;
    const int64_t row = int64_t(blockIdx.x) * kRowsPerBlock + threadIdx.x / kWave;
    if (row >= T) return;
    int64_t dst = row;
    if (UNPACK) {
        const int kv = slot_kv[row];
        if (kv < 0) return;
        dst = kv;
    }
    const float* xr = x + row * d;
    TO* yr = out + dst * d;
    float ss = 0.f;
    if constexpr (NC > 0) {
        f32x4 v[NC];
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            v[c] = *reinterpret_cast<const f32x4*>(xr + c * 256 + lane * 4);
            ss += v[c][0] * v[c][0] + v[c][1] * v[c][1] + v[c][2] * v[c][2] + v[c][3] * v[c][3];
        }
        ss = wave_sum(ss);
        const float scale = rsqrtf(ss / static_cast<float>(d) + eps);
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const f32x4 gg = *reinterpret_cast<const f32x4*>(g + c * 256 + lane * 4);
            store4(yr + c * 256 + lane * 4, v[c] * scale * gg);
        }
    } else {
        for (int c = lane * 4; c < d; c += 256) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(xr + c);
            ss += v[0] * v[0] + v[1] * v[1] + v[2] * v[2] + v[3] * v[3];
        }
        ss = wave_sum(ss);
        const float scale = rsqrtf(ss / static_cast<float>(d) + eps);
        for (int c = lane * 4; c < d; c += 256) {
            const f32x4 v = *reinterpret_cast<const f32x4*>(xr + c);
            const f32x4 gg = *reinterpret_cast<const f32x4*>(g + c);
            store4(yr + c, v * scale * gg);
        }
    }
}

template <typename TO, bool UNPACK>
void rmsnorm_dispatch(const float* x, const float* g, TO* out, const int32_t* slot_kv, int T, int d, float eps,
                      hipStream_t s) {
    const dim3 grid((T + kRowsPerBlock - 1) / kRowsPerBlock);
    const int nc = (d % 256 == 0) ? d / 256 : 0;
#define PP_RMS(NC) rmsnorm_kernel<TO, NC, UNPACK><<<grid, kBlock, 0, s>>>(x, g, out, slot_kv, T, d, eps)
    switch (nc) {
        case 1: PP_RMS(1); break;
        case 2: PP_RMS(2); break;
        case 4: PP_RMS(4); break;
        case 8: PP_RMS(8); break;
        case 16: PP_RMS(16); break;
        case 32: PP_RMS(32); break;
        default: PP_RMS(0); break;
    }
#undef PP_RMS
}

// ------------------------------------------------------------------------------- RoPE
// One thread per (slot, head, run of 8 rotation pairs): reads x[i..i+8) and
// x[i+D/2..i+D/2+8), rotates pair (x_j, x_{j+D/2}) by the angle of pair j at the slot's
// restart position, in float32, and writes back in place.
template <typename T>
__global__ __launch_bounds__(kBlock) void rope_kernel(T* __restrict__ qkv, int64_t ld, const float2* __restrict__ table,
                                                      const int32_t* __restrict__ slot_pos,
                                                      const int32_t* __restrict__ slot_seg, int T_, int nh, int D) {
    const int runs = D / 16;
    const int64_t per_slot = int64_t(nh) * runs;
    const int64_t idx = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    const int64_t slot = idx / per_slot;
    if (slot >= T_) return;
    if (slot_seg[slot] < 0) return;
    const int r = static_cast<int>(idx % per_slot);
    const int head = r / runs, run = r % runs;
    const int half = D / 2;
    T* base = qkv + slot * ld + int64_t(head) * D + run * 8;
    const float2* cs = table + int64_t(slot_pos[slot]) * half + run * 8;
    float a[8], b[8], na[8], nb[8];
    load8(base, a);
    load8(base + half, b);
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        const float2 t = cs[i];
        na[i] = a[i] * t.x - b[i] * t.y;
        nb[i] = b[i] * t.x + a[i] * t.y;
    }
    store8(base, na);
    store8(base + half, nb);
}

// ------------------------------------------------------------------------------- UNPACK
template <typename T>
__global__ __launch_bounds__(kBlock) void kv_scatter_kernel(const T* __restrict__ qkv, int64_t ld, int k_col,
                                                            int kvw, T* __restrict__ kc, T* __restrict__ vc,
                                                            const int32_t* __restrict__ slot_kv, int T_) {
    const int runs = 2 * kvw / 8;
    const int64_t idx = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    const int64_t slot = idx / runs;
    if (slot >= T_) return;
    const int kv = slot_kv[slot];
    if (kv < 0) return;
    const int e = static_cast<int>(idx % runs) * 8;
    const T* src = qkv + slot * ld + k_col + e;
    T* dst = e < kvw ? kc + int64_t(kv) * kvw + e : vc + int64_t(kv) * kvw + (e - kvw);
    float v[8];
    load8(src, v);
    store8(dst, v);
}

__global__ __launch_bounds__(kBlock) void swiglu_f32_kernel(const float* __restrict__ gu, float* __restrict__ act,
                                                            int T_, int F) {
    const int64_t idx = int64_t(blockIdx.x) * kBlock + threadIdx.x;
    if (idx >= int64_t(T_) * F) return;
    const int64_t t = idx / F;
    const int f = static_cast<int>(idx % F);
    const int64_t gi = t * 2 * F + 32 * (f / 16) + f % 16;
    act[idx] = silu(gu[gi]) * gu[gi + 16];
}

unsigned blocks_for(int64_t n) { return static_cast<unsigned>((n + kBlock - 1) / kBlock); }

}  // namespace

namespace ppk {

void rope_table(float2* table, int P, int D, float theta, hipStream_t s) {
    const int64_t n = int64_t(P) * (D / 2);
    if (n == 0) return;
    rope_table_kernel<<<blocks_for(n), kBlock, 0, s>>>(table, n, D / 2, D, static_cast<double>(theta));
}

void embed(int dtype, float* x, const void* E, int vocab, const int32_t* tokens, const int32_t* slot_kv, int T,
           int d, hipStream_t s) {
    if (dtype == PP_BF16)
        embed_dispatch(x, static_cast<const bf16*>(E), vocab, tokens, slot_kv, T, d, s);
    else
        embed_dispatch(x, static_cast<const float*>(E), vocab, tokens, slot_kv, T, d, s);
}

void rmsnorm(int dtype, const float* x, const float* g, void* out, int T, int d, float eps, hipStream_t s) {
    if (dtype == PP_BF16)
        rmsnorm_dispatch<bf16, false>(x, g, at<bf16>(out), nullptr, T, d, eps, s);
    else
        rmsnorm_dispatch<float, false>(x, g, at<float>(out), nullptr, T, d, eps, s);
}

void rmsnorm_unpack(const float* x, const float* g, float* hidden, const int32_t* slot_kv, int T, int d, float eps,
                    hipStream_t s) {
    rmsnorm_dispatch<float, true>(x, g, hidden, slot_kv, T, d, eps, s);
}

void rope_apply(int dtype, void* qkv, int64_t ld, const float2* table, const int32_t* slot_pos,
                const int32_t* slot_seg, int T, int n_heads_rot, int D, hipStream_t s) {
    const int64_t n = int64_t(T) * n_heads_rot * (D / 16);
    if (dtype == PP_BF16)
        rope_kernel<bf16><<<blocks_for(n), kBlock, 0, s>>>(at<bf16>(qkv), ld, table, slot_pos, slot_seg, T,
                                                           n_heads_rot, D);
    else
        rope_kernel<float><<<blocks_for(n), kBlock, 0, s>>>(at<float>(qkv), ld, table, slot_pos, slot_seg, T,
                                                            n_heads_rot, D);
}

void kv_scatter(int dtype, const void* qkv, int64_t ld, int k_col, int kvw, void* kc, void* vc,
                const int32_t* slot_kv, int T, hipStream_t s) {
    const int64_t n = int64_t(T) * (2 * kvw / 8);
    if (dtype == PP_BF16)
        kv_scatter_kernel<bf16><<<blocks_for(n), kBlock, 0, s>>>(static_cast<const bf16*>(qkv), ld, k_col, kvw,
                                                                 at<bf16>(kc), at<bf16>(vc), slot_kv, T);
    else
        kv_scatter_kernel<float><<<blocks_for(n), kBlock, 0, s>>>(static_cast<const float*>(qkv), ld, k_col, kvw,
                                                                  at<float>(kc), at<float>(vc), slot_kv, T);
}

void swiglu_f32(const float* gu, float* act, int T, int F, hipStream_t s) {
    const int64_t n = int64_t(T) * F;
    if (n == 0) return;
    swiglu_f32_kernel<<<blocks_for(n), kBlock, 0, s>>>(gu, act, T, F);
}

}  // namespace ppk
