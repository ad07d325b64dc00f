// The first generated token of every prompt (section 2.3: the time to first token covers
// prefilling the KV cache and generating the first token): the LM head applied to each
// prompt's last hidden row, and the greedy choice, argmax over the vocabulary with the lowest
// id on ties.
//
// Three launches.  (1) The last hidden row of every prompt (row prompt_kv_off[i+1] - 1 of the
// unpacked hidden state) is gathered into a [k_pad, d] matrix in the model's dtype, rows past
// k zero.  (2) One workgroup per 64 vocabulary rows computes their logits for all prompts and
// reduces them to one (max, lowest id) pair per prompt.  The LM head, vocab x d, is read from
// HBM exactly once and dominates the traffic: this kernel is HBM-bound on it (2 vocab d bytes
// in bf16), the prompt matrix being re-read from L2.  (3) One thread per prompt reduces the
// per-workgroup pairs in workgroup order, so the result is deterministic.
#include <math.h>

#include "device.h"
#include "kernels.h"
#include "prepack.h"

namespace {

constexpr int VB = 64;   // vocabulary rows per workgroup (4 wavefronts x 16)

struct ArgMax {
    float v;
    int32_t i;
};

// a better than b: larger value, or equal value and lower id; NaN never wins
__device__ __forceinline__ bool better(float av, int ai, float bv, int bi) {
    return av > bv || (av == bv && ai < bi);
}

template <typename T>
__global__ __launch_bounds__(256) void gather_last_kernel(const float* __restrict__ hidden, const int32_t* __restrict__ off,
                                                         int k, int k_pad, int d, T* __restrict__ out) {
    const int i = blockIdx.x;
    if (i >= k_pad) return;
    T* o = out + int64_t(i) * d;
    if (i >= k) {
        for (int c = threadIdx.x; c < d; c += blockDim.x) o[c] = static_cast<T>(0.f);
        return;
    }
    const float* h = hidden + int64_t(off[i + 1] - 1) * d;
    for (int c = threadIdx.x; c < d; c += blockDim.x) o[c] = static_cast<T>(h[c]);
}

// Wavefront w of workgroup b owns vocabulary rows n0 = 64 b + 16 w .. + 15 as the first
// operand of the 16x16x32 bf16 MFMA (weight rows on the MFMA's rows) and all prompts, 64 at a
// time (4 blocks of 16), as the second.  Fragments come straight from global memory: lane l
// reads 8 consecutive K values of row l % 16 at K offset 8 (l / 16), so four lanes cover 64
// contiguous bytes of a row.  Rows past the vocabulary are read as the last row and never
// reported.  In block mb lane l holds the logits of prompt 16 mb + l % 16 for vocabulary rows
// n0 + 4 (l / 16) + 0..3.
__global__ __launch_bounds__(256) void lm_head_bf16_kernel(const bf16* __restrict__ hl, int k, int k_pad,
                                                           const bf16* __restrict__ W, int V, int d,
                                                           float* __restrict__ logits, ArgMax* __restrict__ part) {
    __shared__ ArgMax red[4][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n0 = blockIdx.x * VB + wave * 16;
    const int lr = lane & 15, kq = 8 * (lane >> 4);
    const bf16* wrow = W + int64_t(min(n0 + lr, V - 1)) * d + kq;
    for (int m0 = 0; m0 < k_pad; m0 += 64) {
        const int nmb = min(4, (k_pad - m0) / 16);
        f32x4 acc[4] = {};
        const bf16* hrow = hl + int64_t(m0 + lr) * d + kq;
        for (int kk = 0; kk < d; kk += 128) {
            // the 4 weight fragments of this 128-wide slice first: they come from HBM
            bf16x8 w[4];
#pragma unroll
            for (int s = 0; s < 4; ++s) w[s] = *reinterpret_cast<const bf16x8*>(wrow + kk + 32 * s);
#pragma unroll
            for (int s = 0; s < 4; ++s)
#pragma unroll
                for (int mb = 0; mb < 4; ++mb)
                    if (mb < nmb) {
                        const bf16x8 h = *reinterpret_cast<const bf16x8*>(hrow + int64_t(16 * mb) * d + kk + 32 * s);
                        acc[mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(w[s], h, acc[mb], 0, 0, 0);
                    }
        }
        // logits and the lane's best of its 4 vocabulary rows, per prompt block
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
            if (mb >= nmb) break;
            const int m = m0 + 16 * mb + lr;
            const int nb = n0 + 4 * (lane >> 4);
            float bv = -INFINITY;
            int bi = INT32_MAX;
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                if (nb + r >= V) continue;
                const float v = acc[mb][r];
                if (logits && m < k) logits[int64_t(m) * V + nb + r] = v;
                if (better(v, nb + r, bv, bi)) { bv = v; bi = nb + r; }
            }
            // lanes l, l ^ 16, l ^ 32, l ^ 48 hold the same prompt
#pragma unroll
            for (int x = 16; x < 64; x <<= 1) {
                const float ov = __shfl_xor(bv, x);
                const int oi = __shfl_xor(bi, x);
                if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
            }
            if (lane < 16) red[wave][16 * mb + lane] = ArgMax{bv, bi};
        }
        __syncthreads();
        // wavefront 0 combines the 4 wavefronts' rows (ascending ids) for the 64 prompts
        if (wave == 0 && lane < 16 * nmb && m0 + lane < k) {
            ArgMax b = red[0][lane];
#pragma unroll
            for (int w2 = 1; w2 < 4; ++w2) {
                const ArgMax o = red[w2][lane];
                if (better(o.v, o.i, b.v, b.i)) b = o;
            }
            part[int64_t(blockIdx.x) * k + m0 + lane] = b;
        }
        __syncthreads();
    }
}

// float32 model: one thread per vocabulary row, prompts one after another.
__global__ __launch_bounds__(VB) void lm_head_f32_kernel(const float* __restrict__ hl, int k, const float* __restrict__ W,
                                                         int V, int d, float* __restrict__ logits,
                                                         ArgMax* __restrict__ part) {
    const int n = blockIdx.x * VB + threadIdx.x;
    const float* w = W + int64_t(min(n, V - 1)) * d;
    for (int m = 0; m < k; ++m) {
        const float* h = hl + int64_t(m) * d;
        float s = 0.f;
        for (int c = 0; c < d; ++c) s = fmaf(h[c], w[c], s);
        float bv = -INFINITY;
        int bi = INT32_MAX;
        if (n < V) {
            if (logits) logits[int64_t(m) * V + n] = s;
            bv = s;
            bi = n;
        }
#pragma unroll
        for (int x = 1; x < 64; x <<= 1) {
            const float ov = __shfl_xor(bv, x);
            const int oi = __shfl_xor(bi, x);
            if (better(ov, oi, bv, bi)) { bv = ov; bi = oi; }
        }
        if (threadIdx.x == 0) part[int64_t(blockIdx.x) * k + m] = ArgMax{bv, bi};
    }
}

__global__ __launch_bounds__(256) void argmax_finalize_kernel(const ArgMax* __restrict__ part, int n_blocks, int k,
                                                              int32_t* __restrict__ tokens) {
    const int m = blockIdx.x * blockDim.x + threadIdx.x;
    if (m >= k) return;
    ArgMax b{-INFINITY, INT32_MAX};
    for (int j = 0; j < n_blocks; ++j) {
        const ArgMax o = part[int64_t(j) * k + m];
        if (better(o.v, o.i, b.v, b.i)) b = o;
    }
    tokens[m] = b.i == INT32_MAX ? -1 : b.i;   // -1: every logit was NaN
}

}  // namespace

namespace ppk {

size_t first_token_workspace(int dtype, int k, int V, int d) {
    const int k_pad = (k + 15) / 16 * 16;
    const size_t e = dtype == PP_BF16 ? 2 : 4;
    const size_t a = (size_t(k_pad) * d * e + 255) / 256 * 256;
    const size_t n_blocks = (size_t(V) + VB - 1) / VB;
    return a + n_blocks * size_t(k) * sizeof(ArgMax);
}

void first_token(int dtype, const float* hidden, const int32_t* prompt_kv_off, int k, const void* lm_head, int V,
                 int d, void* workspace, float* logits, int32_t* tokens, hipStream_t s) {
    const int k_pad = (k + 15) / 16 * 16;
    const size_t e = dtype == PP_BF16 ? 2 : 4;
    char* ws = static_cast<char*>(workspace);
    ArgMax* part = reinterpret_cast<ArgMax*>(ws + (size_t(k_pad) * d * e + 255) / 256 * 256);
    const int n_blocks = (V + VB - 1) / VB;
    if (dtype == PP_BF16) {
        bf16* hl = reinterpret_cast<bf16*>(ws);
        gather_last_kernel<bf16><<<k_pad, 256, 0, s>>>(hidden, prompt_kv_off, k, k_pad, d, hl);
        lm_head_bf16_kernel<<<n_blocks, 256, 0, s>>>(hl, k, k_pad, static_cast<const bf16*>(lm_head), V, d, logits,
                                                     part);
    } else {
        float* hl = reinterpret_cast<float*>(ws);
        gather_last_kernel<float><<<k_pad, 256, 0, s>>>(hidden, prompt_kv_off, k, k_pad, d, hl);
        lm_head_f32_kernel<<<n_blocks, VB, 0, s>>>(hl, k, static_cast<const float*>(lm_head), V, d, logits, part);
    }
    argmax_finalize_kernel<<<(k + 255) / 256, 256, 0, s>>>(part, n_blocks, k, tokens);
}

}  // namespace ppk
