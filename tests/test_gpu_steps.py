"""Per-step parity on the GPU: every kernel of the packed prefill, called through its C-ABI
entry point on seeded inputs, against the oracle's step on the same inputs.

Bars: integer / copy steps bit-exact; every bf16-stored output within one bf16 ulp of the
correctly rounded float64 result (a larger gap would be a real error, not rounding), plus
the absolute bar of 2e-2 max / 2e-3 mean for outputs of unit scale; float32 outputs to
float32 accumulation accuracy."""
import numpy as np
import pytest
import torch

from oracle import decoder as D, ffd
from paper_2404_09529_amd import prepack as pp

from .gpu_util import (bf16_dev, check_bar, f32_dev, host64, i32_dev, rand_bf16, report, require_gpu,
                       within_ulps)

pytestmark = pytest.mark.gpu

BAR_MAX, BAR_MEAN = 2e-2, 2e-3


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _cfg(H=32, Hkv=32, d=4096, F=11008, dtype=pp.PP_BF16, D_=128, theta=10000.0):
    return pp.PPConfig(n_layers=1, d_model=d, n_heads=H, n_kv_heads=Hkv, head_dim=D_, ffn_dim=F, vocab=1000,
                       dtype=dtype, rms_eps=1e-5, rope_theta=theta)


# ----------------------------------------------------------------------------- GEMM
@pytest.mark.parametrize("M,N,K", [(300, 12288, 4096), (1, 4096, 11008), (256, 4096, 4096), (513, 6144, 2048),
                                   (700, 2048, 5504)])
def test_gemm_bf16_store(M, N, K):
    rng = np.random.default_rng([M, N, K])
    A, B = rand_bf16(rng, (M, K)), rand_bf16(rng, (N, K), 0.02)
    C = torch.empty((M, N), dtype=torch.bfloat16, device="cuda")
    pp.pp_gemm(pp.PP_BF16, pp.PP_EPI_STORE, bf16_dev(A), K, bf16_dev(B), K, C, N, M, N, K)
    ref = A.astype(np.float64) @ B.astype(np.float64).T
    got = host64(C)
    assert within_ulps(got, ref, 1.0, 1e-6) <= 1.0
    check_bar(f"gemm store {M}x{N}x{K}", got, ref)


@pytest.mark.parametrize("M,N,K", [(384, 4096, 4096), (129, 4096, 11008)])
def test_gemm_bf16_residual(M, N, K):
    rng = np.random.default_rng([M, N, K, 1])
    A, B = rand_bf16(rng, (M, K)), rand_bf16(rng, (N, K), 0.02)
    C0 = rng.standard_normal((M, N)).astype(np.float32)
    C = f32_dev(C0)
    pp.pp_gemm(pp.PP_BF16, pp.PP_EPI_RESIDUAL, bf16_dev(A), K, bf16_dev(B), K, C, N, M, N, K)
    ref = C0.astype(np.float64) + A.astype(np.float64) @ B.astype(np.float64).T
    mx, _ = report(f"gemm residual {M}x{N}x{K}", host64(C), ref)
    assert mx <= 2e-4


@pytest.mark.parametrize("M,F,K", [(300, 11008, 4096), (65, 5504, 2048)])
def test_gemm_bf16_swiglu(M, F, K):
    rng = np.random.default_rng([M, F, K, 2])
    A = rand_bf16(rng, (M, K))
    Wg, Wu = rand_bf16(rng, (F, K), 0.02), rand_bf16(rng, (F, K), 0.02)
    W = pp.interleave_gate_up(bf16_dev(Wg), bf16_dev(Wu)).contiguous()
    C = torch.empty((M, F), dtype=torch.bfloat16, device="cuda")
    pp.pp_gemm(pp.PP_BF16, pp.PP_EPI_SWIGLU, bf16_dev(A), K, W, K, C, F, M, 2 * F, K)
    A64 = A.astype(np.float64)
    ref = D.silu(A64 @ Wg.astype(np.float64).T) * (A64 @ Wu.astype(np.float64).T)
    got = host64(C)
    assert within_ulps(got, ref, 1.0, 1e-5) <= 1.0
    check_bar(f"gemm swiglu {M}x{F}x{K}", got, ref)


@pytest.mark.parametrize("epi", [pp.PP_EPI_STORE, pp.PP_EPI_RESIDUAL])
def test_gemm_bf16_plan_row_tiles(epi):
    """With a plan, the GEMM computes exactly the plan's row tiles: every slot of a prompt is
    correct, and rows of tiles made of row-tail padding alone keep what they held."""
    plan = pp.pp_pack([700, 700, 700, 600, 600, 600, 300], 1024)   # pad-only tiles mid-batch
    T, N, K = plan.n_slots, 4096, 2048
    assert plan.n_mtiles < T // 256                            # some tiles are padding only
    rng = np.random.default_rng([T, epi])
    A, B = rand_bf16(rng, (T, K)), rand_bf16(rng, (N, K), 0.02)
    if epi == pp.PP_EPI_STORE:
        C = torch.full((T, N), float("nan"), dtype=torch.bfloat16, device="cuda")
        base = None
    else:
        base = rng.standard_normal((T, N)).astype(np.float32)
        C = f32_dev(base)
    pp.pp_gemm(pp.PP_BF16, epi, bf16_dev(A), K, bf16_dev(B), K, C, N, T, N, K, pp.DevicePlan(plan))
    got = host64(C)
    covered = np.zeros(T, dtype=bool)
    for m0 in plan.mtile_m0:
        covered[m0:m0 + 256] = True
    assert covered[plan.slot_seg >= 0].all()
    rows = np.nonzero(covered)[0]
    ref = A[rows].astype(np.float64) @ B.astype(np.float64).T
    if epi == pp.PP_EPI_STORE:
        assert within_ulps(got[rows], ref, 1.0, 1e-6) <= 1.0
        assert np.isnan(got[~covered]).all()
    else:
        ref += base[rows]
        assert D.errors(got[rows], ref)[0] <= 2e-4
        assert np.array_equal(got[~covered], base[~covered].astype(np.float64))


def test_gemm_f32():
    rng = np.random.default_rng(7)
    M, N, K = 77, 1376, 688
    A = rng.standard_normal((M, K)).astype(np.float32)
    B = (rng.standard_normal((N, K)) * 0.02).astype(np.float32)
    C = torch.empty((M, N), dtype=torch.float32, device="cuda")
    pp.pp_gemm(pp.PP_F32, pp.PP_EPI_STORE, f32_dev(A), K, f32_dev(B), K, C, N, M, N, K)
    mx, _ = report("gemm f32", host64(C), A.astype(np.float64) @ B.astype(np.float64).T)
    assert mx <= 1e-4


# ----------------------------------------------------------------------------- attention
ATTN_CASES = [
    # lengths, capacity, H, Hkv  (segments shorter / longer than a tile, ragged tails, rows with pads)
    ([1, 5, 64, 127, 128, 129, 300, 700], 1024, 32, 32),
    ([40, 200, 513, 1, 1000], 1024, 32, 8),
    ([2048], 2048, 16, 16),
    ([31, 32, 33, 95, 96, 97, 160, 191, 192, 193], 1024, 16, 4),   # around each wavefront's 32 queries
]


def _attn_inputs(plan, rng, H, Hkv, Dh, scale, dtype):
    """Queries per slot and per-prompt caches, as the QKV projection leaves them."""
    mk = (lambda shape: rand_bf16(rng, shape, scale)) if dtype == pp.PP_BF16 else \
        (lambda shape: (rng.standard_normal(shape) * scale).astype(np.float32))
    return mk((plan.n_slots, H * Dh)), mk((plan.total_len, Hkv * Dh)), mk((plan.total_len, Hkv * Dh))


def _attn_ref(plan, q, kc, vc, H, Hkv, Dh=128):
    """Per segment: causal attention over its prompt's cache rows, zero keys past the prompt."""
    ref = np.zeros((plan.n_slots, H * Dh))
    for s in range(len(plan.seg_start)):
        a, n, p = int(plan.seg_start[s]), int(plan.seg_len[s]), int(plan.seg_prompt[s])
        k0, k1 = int(plan.prompt_kv_off[p]), int(plan.prompt_kv_off[p + 1])
        k = np.zeros((n, Hkv * Dh))
        v = np.zeros((n, Hkv * Dh))
        k[:k1 - k0], v[:k1 - k0] = kc[k0:k1], vc[k0:k1]
        qs = q[a:a + n].astype(np.float64).reshape(n, H, Dh)
        ref[a:a + n] = D.attention(qs, k.reshape(n, Hkv, Dh), v.reshape(n, Hkv, Dh), D.causal(n)).reshape(n, H * Dh)
    return ref


@pytest.mark.parametrize("lengths,cap,H,Hkv", ATTN_CASES)
@pytest.mark.parametrize("padded", [False, True])
def test_attention_bf16(lengths, cap, H, Hkv, padded):
    plan = pp.pp_pack_padded(lengths) if padded else pp.pp_pack(lengths, cap)
    rng = np.random.default_rng(len(lengths) * 131 + cap)
    q, kc, vc = _attn_inputs(plan, rng, H, Hkv, 128, 1.3, pp.PP_BF16)
    out = torch.full((plan.n_slots, H * 128), float("nan"), dtype=torch.bfloat16, device="cuda")
    pp.pp_attention(_cfg(H, Hkv), pp.DevicePlan(plan), bf16_dev(q), H * 128, bf16_dev(kc), bf16_dev(vc), out)
    got = host64(out)
    ref = _attn_ref(plan, q, kc, vc, H, Hkv)
    span = plan.slot_seg >= 0
    assert np.all(np.isfinite(got[span]))
    assert np.all(np.isnan(got[~span]))      # rows outside every span are never written
    real = plan.slot_kv >= 0
    check_bar(f"attention {lengths} H{H}/{Hkv} padded={padded}", got[real], ref[real])


@pytest.mark.parametrize("n,H,Hkv", [(32768, 16, 16), (8192, 32, 8)])
def test_attention_bf16_maximum_length(n, H, Hkv):
    """One segment of the longest prompt a workload holds (a row of 32,768 slots for the 1.3B
    shape; 8,192 with GQA 32/8): sampled query rows, each against the oracle's attention over
    all of its keys, first and last rows and every tile boundary around them included."""
    lengths = [n]
    plan = pp.pp_pack(lengths, n)
    rng = np.random.default_rng([n, H, Hkv])
    q, kc, vc = _attn_inputs(plan, rng, H, Hkv, 128, 1.3, pp.PP_BF16)
    out = torch.empty((plan.n_slots, H * 128), dtype=torch.bfloat16, device="cuda")
    pp.pp_attention(_cfg(H, Hkv, d=H * 128), pp.DevicePlan(plan), bf16_dev(q), H * 128, bf16_dev(kc), bf16_dev(vc),
                    out)
    got = host64(out)
    rows = set(rng.choice(n, size=40, replace=False).tolist()) | {0, 1, 63, 64, 127, 128, n - 129, n - 128, n - 1}
    rows = np.array(sorted(rows))
    ref = np.zeros((len(rows), H * 128))
    for r_i, t in enumerate(rows):
        # query t against its keys 0..t (the causal row of the segment), one query at a time
        qs = q[t].astype(np.float64).reshape(1, H, 128)
        ks = kc[:t + 1].astype(np.float64).reshape(t + 1, Hkv, 128)
        vs = vc[:t + 1].astype(np.float64).reshape(t + 1, Hkv, 128)
        ref[r_i] = D.attention(qs, ks, vs, np.ones((1, t + 1), dtype=bool)).reshape(H * 128)
    assert np.all(np.isfinite(got))
    check_bar(f"attention one segment of {n} H{H}/{Hkv}", got[rows], ref)


def test_attention_bf16_strided_queries():
    """Queries read from a wider row (ldq > H D), e.g. straight out of a fused QKV buffer."""
    lengths, H, Hkv = [77, 300, 5], 16, 4
    plan = pp.pp_pack(lengths, 512)
    rng = np.random.default_rng(12)
    q, kc, vc = _attn_inputs(plan, rng, H, Hkv, 128, 1.0, pp.PP_BF16)
    wide = np.zeros((plan.n_slots, (H + 2 * Hkv) * 128), dtype=np.float32)
    wide[:, :H * 128] = q
    out = torch.zeros((plan.n_slots, H * 128), dtype=torch.bfloat16, device="cuda")
    pp.pp_attention(_cfg(H, Hkv), pp.DevicePlan(plan), bf16_dev(wide), wide.shape[1], bf16_dev(kc), bf16_dev(vc),
                    out)
    real = plan.slot_kv >= 0
    check_bar("attention strided q", host64(out)[real], _attn_ref(plan, q, kc, vc, H, Hkv)[real])


@pytest.mark.parametrize("padded", [False, True])
def test_attention_f32(padded):
    lengths, H, Hkv, Dh = [7, 1, 30, 64], 4, 2, 64
    plan = pp.pp_pack_padded(lengths) if padded else pp.pp_pack(lengths, 64)
    rng = np.random.default_rng(11)
    q, kc, vc = _attn_inputs(plan, rng, H, Hkv, Dh, 1.0, pp.PP_F32)
    out = torch.zeros((plan.n_slots, H * Dh), dtype=torch.float32, device="cuda")
    pp.pp_attention(_cfg(H, Hkv, d=256, F=688, dtype=pp.PP_F32, D_=Dh), pp.DevicePlan(plan), f32_dev(q), H * Dh,
                    f32_dev(kc), f32_dev(vc), out)
    ref = _attn_ref(plan, q, kc, vc, H, Hkv, Dh)
    real = plan.slot_kv >= 0
    mx, _ = report(f"attention f32 padded={padded}", host64(out)[real], ref[real])
    assert mx <= 1e-5


# ----------------------------------------------------------------------------- fused QKV projection
QKV_CASES = [
    # lengths, capacity (None: full batching), H, Hkv, d, theta
    ([1, 5, 64, 127, 128, 129, 300, 700], 1024, 32, 32, 4096, 10000.0),
    ([40, 200, 513, 1, 1000], 1024, 32, 8, 4096, 500000.0),
    ([33, 250, 7], None, 16, 16, 2048, 10000.0),
    ([32768], 32768, 16, 16, 2048, 10000.0),          # 1.3B shape, positions up to 32,767
    ([8192, 17], 8192, 32, 8, 4096, 500000.0),        # Llama-3-8B shape, GQA 32/8, up to 8,191
]


def _sample_real_slots(plan, rng, full_upto=4096):
    """Every real slot of a small plan; for a large one, every segment's first and last slot,
    both sides of every 256-slot GEMM tile boundary, and 2000 random real slots."""
    real = np.nonzero(plan.slot_kv >= 0)[0]
    if len(real) <= full_upto:
        return real
    pick = set(rng.choice(real, size=2000, replace=False).tolist())
    for a, n in zip(plan.seg_start.tolist(), plan.seg_len.tolist()):
        pick |= {a, a + n - 1}
    for b in range(256, plan.n_slots, 256):
        pick |= {b - 1, b}
    pick = np.array(sorted(pick), dtype=np.int64)
    return pick[plan.slot_kv[pick] >= 0]


@pytest.mark.parametrize("lengths,cap,H,Hkv,d,theta", QKV_CASES)
def test_qkv_projection_fused(lengths, cap, H, Hkv, d, theta):
    """Q, K, V projections, RoPE at restart positions and the cache UNPACK, against the
    oracle's separate steps in float64 (on sampled slots of the long cases, including every
    GEMM tile boundary and each prompt's last position)."""
    plan = pp.pp_pack_padded(lengths) if cap is None else pp.pp_pack(lengths, cap)
    rng = np.random.default_rng([len(lengths), d, H, Hkv])
    Dh, T = 128, plan.n_slots
    xn = rand_bf16(rng, (T, d))
    W = rand_bf16(rng, ((H + 2 * Hkv) * Dh, d), 0.02)
    q = torch.full((T, H * Dh), float("nan"), dtype=torch.bfloat16, device="cuda")
    kc = torch.full((plan.total_len, Hkv * Dh), float("nan"), dtype=torch.bfloat16, device="cuda")
    vc = torch.full_like(kc, float("nan"))
    table = torch.empty(plan.max_len * 64 * 2, dtype=torch.float32, device="cuda")
    pp.pp_qkv_projection(_cfg(H, Hkv, d=d, theta=theta), pp.DevicePlan(plan), bf16_dev(xn), bf16_dev(W), table,
                         q, kc, vc)
    torch.cuda.synchronize()
    assert bool(torch.isfinite(kc.float()).all()) and bool(torch.isfinite(vc.float()).all())  # every row written
    real = _sample_real_slots(plan, rng)
    print(f"[parity] qkv {lengths[:4]} H{H}/{Hkv}: {len(real)} sampled slots, positions up to "
          f"{int(plan.slot_pos[real].max())}", flush=True)
    proj = xn[real].astype(np.float64) @ W.astype(np.float64).T
    cos, sin = D.rope_cos_sin(plan.slot_pos[real], Dh, theta)
    n = len(real)
    rq = D.rope(proj[:, :H * Dh].reshape(n, H, Dh), cos, sin).reshape(n, H * Dh)
    rk = D.rope(proj[:, H * Dh:(H + Hkv) * Dh].reshape(n, Hkv, Dh), cos, sin).reshape(n, Hkv * Dh)
    rv = proj[:, (H + Hkv) * Dh:]
    kv_rows = torch.from_numpy(plan.slot_kv[real].astype(np.int64)).cuda()
    got_q = host64(q[torch.from_numpy(real).cuda()])
    got_k, got_v = host64(kc[kv_rows]), host64(vc[kv_rows])
    for name, got, ref in (("q", got_q, rq), ("k", got_k, rk), ("v", got_v, rv)):
        assert within_ulps(got, ref, 1.0, 1e-5) <= 1.0, name
        check_bar(f"qkv projection {name} {lengths[:4]} H{H}/{Hkv}", got, ref)
    # restart: every prompt's first key sits at position 0, where RoPE is the identity
    first_slots = plan.seg_start[plan.seg_len > 0].astype(np.int64)
    assert np.all(plan.slot_pos[first_slots] == 0)
    k0 = xn[first_slots].astype(np.float64) @ W[H * Dh:(H + Hkv) * Dh].astype(np.float64).T
    got_k0 = host64(kc[torch.from_numpy(plan.slot_kv[first_slots].astype(np.int64)).cuda()])
    assert within_ulps(got_k0, k0, 1.0, 1e-5) <= 1.0


# ----------------------------------------------------------------------------- RoPE
@pytest.mark.parametrize("lengths,cap,H,Hkv,theta", [([3, 100, 700, 1], 1024, 32, 32, 10000.0),
                                                     ([8192, 17], 8192, 32, 8, 500000.0),
                                                     ([32768], 32768, 16, 16, 10000.0)])
def test_rope_restart_positions(lengths, cap, H, Hkv, theta):
    plan = pp.pp_pack(lengths, cap)
    rng = np.random.default_rng(cap + H)
    W = (H + 2 * Hkv) * 128
    x = rand_bf16(rng, (plan.n_slots, W), 1.3)
    t = bf16_dev(x)
    table = torch.empty(plan.max_len * 64 * 2, dtype=torch.float32, device="cuda")
    pp.pp_rope(_cfg(H, Hkv, theta=theta), pp.DevicePlan(plan), t, table)
    got = host64(t)
    # sample slots, always including every segment's first and last slot
    idx = set(rng.choice(plan.n_slots, size=min(plan.n_slots, 1500), replace=False).tolist())
    for a, n in zip(plan.seg_start, plan.seg_len):
        idx |= {int(a), int(a + n - 1)}
    idx = np.array(sorted(idx))
    real = idx[plan.slot_seg[idx] >= 0]
    pad = idx[plan.slot_seg[idx] < 0]
    cos, sin = D.rope_cos_sin(plan.slot_pos[real], 128, theta)
    nr = (H + Hkv) * 128
    ref = D.rope(x[real, :nr].astype(np.float64).reshape(len(real), H + Hkv, 128), cos, sin).reshape(len(real), nr)
    assert within_ulps(got[real, :nr], ref, 1.0, 1e-6) <= 1.0
    assert np.array_equal(got[real, nr:], x[real, nr:])          # V untouched
    assert np.array_equal(got[pad], x[pad])                      # pads untouched
    first = plan.seg_start.astype(np.int64)
    assert np.array_equal(got[first, :nr], x[first, :nr])        # restart: position 0 is the identity


# ----------------------------------------------------------------------------- norms, embedding, unpack
@pytest.mark.parametrize("d,dtype", [(4096, pp.PP_BF16), (2048, pp.PP_BF16), (256, pp.PP_F32), (4096, pp.PP_F32)])
def test_rmsnorm(d, dtype):
    rng = np.random.default_rng(d + dtype)
    rows = 333
    x = (rng.standard_normal((rows, d)) * 3).astype(np.float32)
    g = (1 + 0.1 * rng.standard_normal(d)).astype(np.float32)
    out = torch.empty((rows, d), dtype=torch.bfloat16 if dtype == pp.PP_BF16 else torch.float32, device="cuda")
    pp.pp_rmsnorm(dtype, f32_dev(x), f32_dev(g), rows, d, 1e-5, out)
    ref = D.rms_norm(x.astype(np.float64), g.astype(np.float64), 1e-5)
    got = host64(out)
    if dtype == pp.PP_BF16:
        assert within_ulps(got, ref, 1.0, 1e-6) <= 1.0
    else:
        assert report(f"rmsnorm f32 d{d}", got, ref)[0] <= 2e-5


@pytest.mark.parametrize("dtype", [pp.PP_BF16, pp.PP_F32])
@pytest.mark.parametrize("d", [256, 1024, 2048, 4096])         # generic loop; 2, 4, 8 chunks of 512
def test_embed_gather_bit_exact(dtype, d):
    rng = np.random.default_rng(5)
    V = 1000
    lengths = [5, 17, 1, 40]
    plan = pp.pp_pack(lengths, 64)
    E = rand_bf16(rng, (V, d), 0.02) if dtype == pp.PP_BF16 else rng.standard_normal((V, d)).astype(np.float32)
    toks = rng.integers(0, V, sum(lengths)).astype(np.int32)
    toks[3] = V + 5                          # out of range -> zero row (include/prepack.h)
    toks[9] = -3                             # negative: also a zero row
    Ed = bf16_dev(E) if dtype == pp.PP_BF16 else f32_dev(E)
    x = torch.full((plan.n_slots, d), float("nan"), dtype=torch.float32, device="cuda")
    pp.pp_embed(dtype, Ed, V, d, i32_dev(toks), pp.DevicePlan(plan), x)
    got = host64(x)
    want = np.zeros((plan.n_slots, d))
    real = plan.slot_kv >= 0
    ids = toks[plan.slot_kv[real]]
    ok = (ids >= 0) & (ids < V)
    rows = np.nonzero(real)[0]
    want[rows[ok]] = E[ids[ok]]
    assert np.array_equal(got, want)


def test_kv_scatter_bit_exact():
    rng = np.random.default_rng(6)
    H, Hkv = 32, 8
    lengths = [300, 7, 129, 1]
    plan = pp.pp_pack(lengths, 512)
    W = (H + 2 * Hkv) * 128
    qkv = rand_bf16(rng, (plan.n_slots, W))
    L, kvw = plan.total_len, Hkv * 128
    kc = torch.full((L, kvw), float("nan"), dtype=torch.bfloat16, device="cuda")
    vc = torch.full((L, kvw), float("nan"), dtype=torch.bfloat16, device="cuda")
    pp.pp_kv_scatter(_cfg(H, Hkv), pp.DevicePlan(plan), bf16_dev(qkv), kc, vc)
    real = plan.slot_kv >= 0
    want_k = np.zeros((L, kvw))
    want_v = np.zeros((L, kvw))
    want_k[plan.slot_kv[real]] = qkv[real, H * 128:(H + Hkv) * 128]
    want_v[plan.slot_kv[real]] = qkv[real, (H + Hkv) * 128:]
    assert np.array_equal(host64(kc), want_k)
    assert np.array_equal(host64(vc), want_v)


def test_final_norm_unpack():
    rng = np.random.default_rng(8)
    d = 4096
    lengths = [33, 1, 200, 90]
    plan = pp.pp_pack(lengths, 256)
    x = (rng.standard_normal((plan.n_slots, d)) * 2).astype(np.float32)
    g = (1 + 0.1 * rng.standard_normal(d)).astype(np.float32)
    hidden = torch.full((plan.total_len, d), float("nan"), dtype=torch.float32, device="cuda")
    pp.pp_final_norm_unpack(f32_dev(x), f32_dev(g), d, 1e-5, pp.DevicePlan(plan), hidden)
    real = plan.slot_kv >= 0
    want = np.zeros((plan.total_len, d))
    want[plan.slot_kv[real]] = D.rms_norm(x[real].astype(np.float64), g.astype(np.float64), 1e-5)
    assert report("final norm unpack", host64(hidden), want)[0] <= 2e-5
