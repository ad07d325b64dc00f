// The first generated token of every prompt (section 2.3: the time to first token covers
// prefilling the KV cache and generating the first token): the LM head applied to each
// prompt's last hidden row, and the greedy choice, argmax over the vocabulary with the lowest
// id on ties.
//
// Three launches.  (1) The last hidden row of every prompt (row prompt_kv_off[i+1] - 1 of the
// unpacked hidden state) is gathered into a [k_pad, d] matrix in the model's dtype, rows past
// k zero.  (2) One workgroup per 128 vocabulary rows computes their logits for all prompts and
// reduces them to one (max, lowest id) pair per prompt.  The LM head, vocab x d, is read from
// HBM exactly once and dominates the traffic: this kernel is HBM-bound on it (2 vocab d bytes
// in bf16), the prompt matrix being re-read from L2.  (3) One workgroup per prompt reduces the
// per-workgroup pairs; the order it uses is total, so the result is deterministic.
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

// Wavefront w of workgroup b owns vocabulary rows n0 = 128 b + 32 w .. + 31 (two blocks of
// 16 on the rows of the 16x16x32 bf16 MFMA) and all prompts, 64 at a time (4 blocks of 16 on
// its columns).  The weight rows stream from HBM straight into registers: lane l reads 8
// consecutive K values of row l % 16 at K offset 8 (l / 16) of a 32-wide step, and the
// fragments of step t + 8 are requested while step t is computed (a ring of 8 steps, 16 KB
// per wavefront in flight).  Rows past the vocabulary are read as the last row and never
// reported.  The prompt rows are shared by the 4 wavefronts through LDS, 128 K columns at a
// time, double-buffered: each 128-column tile is read from L2 once per workgroup.  In block
// (nb, mb) lane l holds the logits of prompt 16 mb + l % 16 for vocabulary rows
// n0 + 16 nb + 4 (l / 16) + 0..3.
constexpr int LM_ROWS = 128;        // vocabulary rows per workgroup
constexpr int HT = 128;             // K columns per LDS tile of prompt rows
constexpr int HT_B = 64 * HT * 2;   // one tile: 64 prompt rows x 256 bytes

// LDS swizzle of the prompt tile: row r's 16-byte chunk q sits at q ^ g(r), g built from r's
// bits 0, 1, 2 placed at bits 0, 2, 3.  A fragment read serves lanes i and i + 32 together:
// rows r..r+7 at chunks q and q ^ 2; a 256-byte row spans all 64 banks, so those 16 accesses
// are conflict-free when the g(r) fall in distinct classes {x, x ^ 2}, which this g does.
__device__ __forceinline__ int gsw(int r) { return (r & 1) | (((r >> 1) & 1) << 2) | (((r >> 2) & 1) << 3); }

__global__ __launch_bounds__(256) void lm_head_bf16_kernel(const bf16* __restrict__ hl, int k, int k_pad,
                                                           const bf16* __restrict__ W, int V, int d,
                                                           float* __restrict__ logits, ArgMax* __restrict__ part) {
    __shared__ __attribute__((aligned(16))) char tile[2][HT_B];
    __shared__ ArgMax red[4][64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n0 = blockIdx.x * LM_ROWS + wave * 32;
    const int lr = lane & 15, q4 = lane >> 4;
    const bf16* wrow[2];
#pragma unroll
    for (int nb = 0; nb < 2; ++nb) wrow[nb] = W + int64_t(min(n0 + 16 * nb + lr, V - 1)) * d + 8 * q4;
    const int S = d / 32;               // K steps of 32; d % 256 == 0, so S % 8 == 0
    const int n_tiles = d / HT;
    // prompt-tile loads: load t (0..3) of wavefront w covers rows 4 (4 w + t) + l / 16, chunk l % 16
    int h_row[4], h_lds[4];
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        h_row[t] = 4 * (4 * wave + t) + q4;
        h_lds[t] = h_row[t] * 256 + 16 * (lr ^ gsw(h_row[t] & 7));
    }
    // fragment reads: row 16 mb + lr, chunk 4 s + q4 (s = step within the tile)
    const int f_base = lr * 256;
    const int f_sw = gsw(lr & 7);
    for (int m0 = 0; m0 < k_pad; m0 += 64) {
        const int nmb = min(4, (k_pad - m0) / 16);
        bf16x8 hreg[4];
        auto load_tile = [&](int c) {   // prompt rows m0.., K columns c*HT.. (clamped: always in range)
            const int cc = min(c, n_tiles - 1);
#pragma unroll
            for (int t = 0; t < 4; ++t) {
                const int row = min(m0 + h_row[t], k_pad - 1);
                hreg[t] = *reinterpret_cast<const bf16x8*>(hl + int64_t(row) * d + cc * HT + lr * 8);
            }
        };
        auto store_tile = [&](int buf) {
#pragma unroll
            for (int t = 0; t < 4; ++t) *reinterpret_cast<bf16x8*>(tile[buf] + h_lds[t]) = hreg[t];
        };
        bf16x8 ring[8][2];
        auto load_w = [&](int u, int t) {   // weight fragments of step t (clamped) into ring slot u
            const int tt = min(t, S - 1);
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) ring[u][nb] = *reinterpret_cast<const bf16x8*>(wrow[nb] + 32 * tt);
        };
        f32x4 acc[2][4] = {};
        auto step = [&](int u, int buf, int s) {   // compute ring slot u with tile buf, step s of it
#pragma unroll
            for (int mb = 0; mb < 4; ++mb) {
                if (mb >= nmb) break;
                const bf16x8 h = *reinterpret_cast<const bf16x8*>(
                    tile[buf] + f_base + 16 * mb * 256 + 16 * ((4 * s + q4) ^ f_sw));
#pragma unroll
                for (int nb = 0; nb < 2; ++nb)
                    acc[nb][mb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(ring[u][nb], h, acc[nb][mb], 0, 0, 0);
            }
        };
        load_tile(0);
        store_tile(0);
#pragma unroll
        for (int u = 0; u < 8; ++u) load_w(u, u);
        __syncthreads();
        for (int t0 = 0; t0 < S; t0 += 8) {
            const int c = t0 / 4;   // tiles c (buffer 0) and c + 1 (buffer 1)
            load_tile(c + 1);
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                step(u, 0, u);
                load_w(u, t0 + 8 + u);
            }
            store_tile(1);
            __syncthreads();
            load_tile(c + 2);
#pragma unroll
            for (int u = 4; u < 8; ++u) {
                step(u, 1, u - 4);
                load_w(u, t0 + 8 + u);
            }
            store_tile(0);
            __syncthreads();
        }
        // logits and each lane's best of its 8 vocabulary rows, per prompt block
#pragma unroll
        for (int mb = 0; mb < 4; ++mb) {
            if (mb >= nmb) break;
            const int m = m0 + 16 * mb + lr;
            float bv = -INFINITY;
            int bi = INT32_MAX;
#pragma unroll
            for (int nb = 0; nb < 2; ++nb) {
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
            if (lane < 16) red[wave][16 * mb + lane] = ArgMax{bv, bi};
        }
        __syncthreads();
        // wavefront 0 combines the 4 wavefronts' rows for the 64 prompts
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
            part[int64_t(n) * k + m] = ArgMax{s, n};   // a NaN logit never wins the final reduction
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
        const ArgMax o = part[int64_t(j) * k + m];
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
    if (dtype == PP_BF16) {
        bf16* hl = reinterpret_cast<bf16*>(ws);
        gather_last_kernel<bf16><<<k_pad, 256, 0, s>>>(hidden, prompt_kv_off, k, k_pad, d, hl);
        lm_head_bf16_kernel<<<n_blocks, 256, 0, s>>>(hl, k, k_pad, static_cast<const bf16*>(lm_head), V, d, logits,
                                                     part);
    } else {
        float* hl = reinterpret_cast<float*>(ws);
        gather_last_kernel<float><<<k_pad, 256, 0, s>>>(hidden, prompt_kv_off, k, k_pad, d, hl);
        lm_head_f32_kernel<<<n_blocks, 64, 0, s>>>(hl, k, static_cast<const float*>(lm_head), V, d, logits, part);
    }
    argmax_finalize_kernel<<<k, 256, 0, s>>>(part, n_blocks, k, tokens);
}

}  // namespace ppk
