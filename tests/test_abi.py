"""The C ABI on the CPU: the library loads, exports every declared entry point, packs
bit-exactly like the oracle, and rejects bad arguments before enqueuing anything.
No GPU work is launched here."""
import ctypes
import json
import os
import re

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import ffd
from paper_2404_09529_amd import prepack as pp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
# the plan fields the paper defines (Algorithm 1; sections 3.1 and 3.2), compared bit for bit
# with the oracle; the attention work list is a scheduling choice of the library, checked by
# its own invariants (_check_work_list)
FIELDS = ("row_seg_ptr", "seg_prompt", "seg_start", "seg_len", "prompt_kv_off", "slot_seg", "slot_pos",
          "slot_kv")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(pp.LIB_PATH):
        pytest.fail("libprepack.so is not built (python -m paper_2404_09529_amd.build)")
    return pp.lib()


def declared_functions():
    text = open(os.path.join(ROOT, "include", "prepack.h")).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(pp_[a-z_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(L):
    names = declared_functions()
    assert {"pp_pack", "pp_pack_padded", "pp_prefill", "pp_prefill_workspace_size"} <= set(names)
    for n in names:
        assert hasattr(L, n), n


def test_struct_layouts_match_header():
    assert ctypes.sizeof(pp.PPPlan) == 8 * 4 + 3 * 8 + 11 * 8     # 7 int32 + padding to 8 bytes
    assert ctypes.sizeof(pp.PPConfig) == 10 * 4
    assert ctypes.sizeof(pp.PPDPlan) == 8 * 4 + 10 * 8
    assert ctypes.sizeof(pp.PPWeights) == 8 * 8


def test_version(L):
    assert "gfx950" in pp.pp_version()


def _check_work_list(plan):
    """The attention work list as include/prepack.h states it: every (segment, multiple of
    PP_QTILE below the segment's length) exactly once; a segment's tiles consecutive, segments
    longest first (ties by index), inside a segment the highest first query first."""
    got = list(zip(plan.qtile_seg.tolist(), plan.qtile_q0.tolist()))
    assert sorted(got) == sorted((s, q0) for s in range(plan.k) for q0 in range(0, int(plan.seg_len[s]), pp.PP_QTILE))
    segs = sorted(range(plan.k), key=lambda s: (-int(plan.seg_len[s]), s))
    want = [(s, q0) for s in segs for q0 in reversed(range(0, int(plan.seg_len[s]), pp.PP_QTILE))]
    assert got == want
    # GEMM row tiles: exactly the PP_MTILE-slot tiles holding a slot of some span, ascending
    want_m = [t0 for t0 in range(0, plan.n_slots, pp.PP_MTILE) if (plan.slot_seg[t0:t0 + pp.PP_MTILE] >= 0).any()]
    assert plan.mtile_m0.tolist() == want_m


def _same(plan, ref):
    for s in ("k", "capacity", "n_rows", "max_len", "total_len"):
        assert getattr(plan, s) == getattr(ref, s), s
    for f in FIELDS:
        assert np.array_equal(getattr(plan, f), getattr(ref, f)), f
    _check_work_list(plan)


def test_golden_examples(L, golden_dir):
    with open(os.path.join(golden_dir, "ffd_examples.json")) as f:
        for ex in json.load(f)["examples"]:
            p = pp.pp_pack(ex["lengths"], ex["capacity"])
            assert p.seg_start.tolist() == ex["seg_start"]
            assert p.slot_kv.tolist() == ex["slot_kv"]
            assert p.slot_pos.tolist() == ex["slot_pos"]
            assert p.prompt_kv_off.tolist() == ex["prompt_kv_off"]
            bins = [p.seg_prompt[p.row_seg_ptr[r]:p.row_seg_ptr[r + 1]].tolist() for r in range(p.n_rows)]
            assert bins == ex["bins"]


@settings(max_examples=300, deadline=None)
@given(st.lists(st.integers(1, 300), min_size=1, max_size=60), st.integers(0, 200), st.booleans())
def test_pack_bit_exact_vs_oracle(L, lengths, extra, default_capacity):
    C = 0 if default_capacity else max(lengths) + extra
    _same(pp.pp_pack(lengths, C), ffd.pack(lengths, C))


@settings(max_examples=100, deadline=None)
@given(st.lists(st.integers(1, 200), min_size=1, max_size=40))
def test_pack_padded_bit_exact_vs_oracle(L, lengths):
    _same(pp.pp_pack_padded(lengths), ffd.pack_padded(lengths))


@pytest.mark.parametrize("wid", [1, 2, 3, 4, 5])
def test_pack_bit_exact_on_workload_lengths(L, wid):
    from paper_2404_09529_amd import workloads as W
    wl = W.workload(wid)
    for seed in range(3):
        lengths = W.draw_lengths(wl, seed)
        _same(pp.pp_pack(lengths, wl.capacity), ffd.pack(lengths, wl.capacity))
        assert pp.pp_pack(lengths, wl.capacity).n_rows == ffd.pack(lengths, wl.capacity).n_rows


def test_empty_batch(L):
    p = pp.pp_pack([], 64)
    assert p.n_rows == 0 and p.total_len == 0 and p.n_qtiles == 0
    p = pp.pp_pack_padded([])
    assert p.n_rows == 0


def test_errors(L):
    with pytest.raises(pp.PrepackError) as e:
        pp.pp_pack([3, 0, 2], 8)
    assert e.value.code == pp.PP_ERR_INVALID_ARG and "length 0" in pp.pp_last_error()
    with pytest.raises(pp.PrepackError) as e:
        pp.pp_pack([3, -1], 8)
    assert e.value.code == pp.PP_ERR_INVALID_ARG
    with pytest.raises(pp.PrepackError) as e:
        pp.pp_pack([3, 9, 2], 8)
    assert e.value.code == pp.PP_ERR_TOO_LONG
    with pytest.raises(pp.PrepackError) as e:
        pp.pp_pack([3, 2], -4)
    assert e.value.code == pp.PP_ERR_INVALID_ARG
    with pytest.raises(pp.PrepackError) as e:
        pp.pp_pack([3, 2, 4], 8, slot_cap=23)
    assert e.value.code == pp.PP_ERR_BUFFER_TOO_SMALL
    with pytest.raises(pp.PrepackError) as e:
        pp.pp_pack_padded([3, 2, 4], qtile_cap=2)
    assert e.value.code == pp.PP_ERR_BUFFER_TOO_SMALL
    # a successful call clears the message
    pp.pp_pack([1], 4)
    assert pp.pp_last_error() == ""
    # NULL plan
    lengths = (ctypes.c_int32 * 2)(3, 4)
    assert pp.lib().pp_pack(lengths, 2, 8, None) == pp.PP_ERR_INVALID_ARG
    assert pp.lib().pp_plan_bounds(-1, 4, None, None, None) == pp.PP_ERR_INVALID_ARG
    with pytest.raises(pp.PrepackError) as e:
        pp.pp_pack([300, 200, 300], 512, mtile_cap=2)            # needs ceil(3 * 512 / 256) = 6
    assert e.value.code == pp.PP_ERR_BUFFER_TOO_SMALL


def _cfg(**kw):
    base = dict(n_layers=1, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128, ffn_dim=14336, vocab=1000,
                dtype=pp.PP_BF16, rms_eps=1e-5, rope_theta=5e5)
    base.update(kw)
    return pp.PPConfig(**base)


def _dplan(**kw):
    base = dict(k=2, capacity=256, n_rows=2, max_len=200, total_len=300, n_qtiles=3, n_mtiles=2,
                **{n: 0x1000 for n in ("seg_prompt", "seg_start", "seg_len", "prompt_kv_off", "slot_seg",
                                       "slot_pos", "slot_kv", "qtile_seg", "qtile_q0", "mtile_m0")})
    base.update(kw)
    return pp.PPDPlan(**base)


def _ws(cfg, dp):
    n = ctypes.c_size_t()
    st_ = pp.lib().pp_prefill_workspace_size(ctypes.byref(cfg), ctypes.byref(dp), ctypes.byref(n))
    return st_, n.value


def test_workspace_size_and_config_validation(L):
    st_, n = _ws(_cfg(), _dplan())
    assert st_ == pp.PP_OK
    T = 512
    # x (f32), xn, q (bf16 keeps only the queries: keys and values go straight to the caches),
    # attention output, SwiGLU activations, RoPE table
    want = T * 4096 * 4 + T * 4096 * 2 + T * 4096 * 2 + T * 4096 * 2 + T * 14336 * 2 + 200 * 64 * 8
    assert want <= n <= want + 8 * 256
    assert _ws(_cfg(head_dim=96), _dplan())[0] == pp.PP_ERR_UNSUPPORTED
    assert _ws(_cfg(n_kv_heads=5), _dplan())[0] == pp.PP_ERR_UNSUPPORTED
    assert _ws(_cfg(head_dim=64, n_heads=64, n_kv_heads=16), _dplan())[0] == pp.PP_ERR_UNSUPPORTED  # bf16 needs D=128
    assert _ws(_cfg(d_model=1000), _dplan())[0] == pp.PP_ERR_UNSUPPORTED
    assert _ws(_cfg(ffn_dim=5500), _dplan())[0] == pp.PP_ERR_UNSUPPORTED
    assert _ws(_cfg(dtype=7), _dplan())[0] == pp.PP_ERR_INVALID_ARG
    assert _ws(_cfg(n_layers=0), _dplan())[0] == pp.PP_ERR_INVALID_ARG
    assert _ws(_cfg(dtype=pp.PP_F32, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, ffn_dim=688),
               _dplan())[0] == pp.PP_OK
    assert _ws(_cfg(), _dplan(total_len=600))[0] == pp.PP_ERR_INVALID_ARG        # more tokens than slots (512)
    assert _ws(_cfg(), _dplan(max_len=300))[0] == pp.PP_ERR_INVALID_ARG          # longer than a row
    assert _ws(_cfg(), _dplan(slot_kv=0))[0] == pp.PP_ERR_INVALID_ARG            # NULL device array
    assert _ws(_cfg(), _dplan(prompt_kv_off=0))[0] == pp.PP_ERR_INVALID_ARG
    assert _ws(_cfg(), _dplan(seg_prompt=0))[0] == pp.PP_ERR_INVALID_ARG
    assert _ws(_cfg(), _dplan(mtile_m0=0))[0] == pp.PP_ERR_INVALID_ARG
    assert _ws(_cfg(), _dplan(n_mtiles=0))[0] == pp.PP_ERR_INVALID_ARG            # tokens but no row tile
    assert _ws(_cfg(), _dplan(n_mtiles=3))[0] == pp.PP_ERR_INVALID_ARG            # more tiles than 512 slots hold


def _weights(n_layers):
    arr = (ctypes.c_void_p * n_layers)(*([0x2000] * n_layers))
    vp = ctypes.POINTER(ctypes.c_void_p)
    w = pp.PPWeights(embed=0x2000, final_norm=0x2000,
                     **{k: ctypes.cast(arr, vp) for k in ("attn_norm", "wqkv", "wo", "mlp_norm", "w_gateup",
                                                          "w_down")})
    return w, arr


def test_prefill_rejects_before_enqueue(L):
    """Every check of pp_prefill runs on the host before a launch, so these never touch a GPU."""
    cfg, dp = _cfg(), _dplan()
    w, keep = _weights(1)
    f = pp.lib().pp_prefill
    _, need = _ws(cfg, dp)
    args = lambda ws, nbytes, hid=0x3000: (ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(dp), 0x4000, ws,
                                           nbytes, hid, 0x5000, 0x6000, None)
    assert f(*args(0x10000, need - 1)) == pp.PP_ERR_BUFFER_TOO_SMALL
    assert f(*args(0x10000 + 8, need)) == pp.PP_ERR_INVALID_ARG        # misaligned workspace
    assert f(*args(None, need)) == pp.PP_ERR_INVALID_ARG
    assert f(*args(0x10000, need, hid=None)) == pp.PP_ERR_INVALID_ARG
    assert f(ctypes.byref(cfg), None, ctypes.byref(dp), 0x4000, 0x10000, need, 0x3000, 0x5000, 0x6000,
             None) == pp.PP_ERR_INVALID_ARG
    bad = (ctypes.c_void_p * 1)(None)
    w.wo = ctypes.cast(bad, ctypes.POINTER(ctypes.c_void_p))
    assert f(*args(0x10000, need)) == pp.PP_ERR_INVALID_ARG
    assert "layer 0" in pp.pp_last_error()
    # an empty plan is a no-op that succeeds without touching any pointer
    empty = _dplan(k=0, n_rows=0, capacity=0, max_len=0, total_len=0, n_qtiles=0, n_mtiles=0)
    w2, keep2 = _weights(1)
    assert f(ctypes.byref(cfg), ctypes.byref(w2), ctypes.byref(empty), None, None, 0, None, None, None,
             None) == pp.PP_OK


def test_step_entry_points_reject_before_enqueue(L):
    """Host-side argument checks of the fused QKV projection and of attention."""
    cfg, dp = _cfg(), _dplan()
    f32 = _cfg(dtype=pp.PP_F32, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, ffn_dim=688)
    q = L.pp_qkv_projection
    assert q(ctypes.byref(f32), ctypes.byref(dp), 1, 1, 1, 1, 1, 1, None) == pp.PP_ERR_UNSUPPORTED
    assert q(ctypes.byref(cfg), ctypes.byref(dp), None, 1, 1, 1, 1, 1, None) == pp.PP_ERR_INVALID_ARG
    assert q(ctypes.byref(cfg), None, 1, 1, 1, 1, 1, 1, None) == pp.PP_ERR_INVALID_ARG
    a = L.pp_attention
    assert a(ctypes.byref(cfg), ctypes.byref(dp), 0x1000, 4000, 1, 1, 1, None) == pp.PP_ERR_INVALID_ARG  # ldq < H D
    assert a(ctypes.byref(cfg), ctypes.byref(dp), 0x1000, 4100, 1, 1, 1, None) == pp.PP_ERR_UNSUPPORTED  # ldq % 8
    assert a(ctypes.byref(cfg), ctypes.byref(dp), None, 4096, 1, 1, 1, None) == pp.PP_ERR_INVALID_ARG
    # a prompt too long for the kernel's 32-bit cache addressing is refused up front
    huge = _dplan(capacity=1100000, n_rows=1, max_len=1100000, total_len=300)   # x 8 KV heads x 256 B > 2 GiB
    assert a(ctypes.byref(cfg), ctypes.byref(huge), 0x1000, 4096, 1, 1, 1, None) == pp.PP_ERR_UNSUPPORTED


def test_gemm_rejects_unsupported_shapes_before_enqueue(L):
    """bf16 GEMM tiling limits are checked on the host (no launch, no GPU needed)."""
    g = L.pp_gemm
    ok = dict(A=0x1000, lda=4096, B=0x2000, ldb=4096, C=0x3000, ldc=4096, M=256, N=4096, K=4096)
    def call(**kw):
        a = {**ok, **kw}
        return g(pp.PP_BF16, pp.PP_EPI_STORE, a["A"], a["lda"], a["B"], a["ldb"], a["C"], a["ldc"], a["M"], a["N"],
                 a["K"], None, None)
    assert call(N=4000) == pp.PP_ERR_UNSUPPORTED          # N % 256
    assert call(K=4000, lda=4000, ldb=4000) == pp.PP_ERR_UNSUPPORTED   # K % 64
    assert call(lda=100) == pp.PP_ERR_INVALID_ARG          # lda < K
    assert call(M=0) == pp.PP_OK                           # empty: nothing to do
    assert g(pp.PP_BF16, 7, 0x1000, 4096, 0x2000, 4096, 0x3000, 4096, 256, 4096, 4096, None, None) == pp.PP_ERR_INVALID_ARG


def test_first_token_workspace_and_rejections(L):
    """Workspace size of the first-token step, and its host-side argument checks."""
    cfg, dp = _cfg(vocab=32000), _dplan()
    n = ctypes.c_size_t()
    assert L.pp_first_token_workspace_size(ctypes.byref(cfg), ctypes.byref(dp), ctypes.byref(n)) == pp.PP_OK
    # k = 2 prompts padded to 16 rows of d bf16, then one (float, int32) pair per 128-row
    # vocabulary block and prompt
    assert n.value == 16 * 4096 * 2 + 250 * 2 * 8
    ws = n.value
    f = L.pp_first_token
    ok = dict(h=0x1000, w=0x2000, ws=0x10000, nb=ws, lg=None, tok=0x3000)
    def call(c=cfg, p=dp, **kw):
        a = {**ok, **kw}
        return f(ctypes.byref(c), ctypes.byref(p), a["h"], a["w"], a["ws"], a["nb"], a["lg"], a["tok"], None)
    assert call(h=None) == pp.PP_ERR_INVALID_ARG
    assert call(w=None) == pp.PP_ERR_INVALID_ARG
    assert call(tok=None) == pp.PP_ERR_INVALID_ARG
    assert call(ws=0x10010) == pp.PP_ERR_INVALID_ARG              # not 256-byte aligned
    assert call(nb=ws - 1) == pp.PP_ERR_BUFFER_TOO_SMALL
    assert call(p=_dplan(total_len=1)) == pp.PP_ERR_INVALID_ARG   # fewer tokens than prompts
    assert call(c=_cfg(vocab=0)) == pp.PP_ERR_INVALID_ARG
    assert call(p=_dplan(k=0, total_len=0)) == pp.PP_OK            # no prompt: nothing to do


def test_first_token_noalloc_rejections(L):
    """The allocation-free first token: the same argument checks, and a plan whose workspace
    exceeds the static buffer rejected before anything is enqueued (no GPU touched)."""
    f = L.pp_first_token_noalloc
    cfg, dp = _cfg(vocab=32000), _dplan()
    def call(c=cfg, p=dp, h=0x1000, w=0x2000, tok=0x3000):
        return f(ctypes.byref(c), ctypes.byref(p), h, w, None, tok, None)
    assert call(h=None) == pp.PP_ERR_INVALID_ARG
    assert call(w=None) == pp.PP_ERR_INVALID_ARG
    assert call(tok=None) == pp.PP_ERR_INVALID_ARG
    assert call(p=_dplan(total_len=1)) == pp.PP_ERR_INVALID_ARG
    assert call(p=_dplan(k=0, total_len=0)) == pp.PP_OK
    # float32 keeps one (value, id) pair per vocabulary row and prompt: 2,000,000 x 2 x 8 bytes
    big = _cfg(dtype=pp.PP_F32, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64, ffn_dim=688, vocab=2_000_000)
    n = ctypes.c_size_t()
    assert L.pp_first_token_workspace_size(ctypes.byref(big), ctypes.byref(dp), ctypes.byref(n)) == pp.PP_OK
    assert n.value > pp.PP_FIRST_TOKEN_SCRATCH_BYTES
    assert call(c=big) == pp.PP_ERR_BUFFER_TOO_SMALL
    assert "static buffer" in pp.pp_last_error()
    # a header constant the binding mirrors
    text = open(os.path.join(ROOT, "include", "prepack.h")).read()
    assert re.search(r"#define PP_FIRST_TOKEN_SCRATCH_BYTES \(16u << 20\)", text)
    assert pp.PP_FIRST_TOKEN_SCRATCH_BYTES == 16 << 20


# ----------------------------------------------------------------------------- generation
def test_gen_layout_packed_and_padded_by_hand(L):
    """pp_gen_layout_make on lengths 3, 1, 5 with room for 4 new tokens."""
    p = pp.pp_gen_layout_make([3, 1, 5], 4)
    assert (p.k, p.n_new, p.padded, p.max_len, p.ctx_rows, p.gen_rows) == (3, 4, False, 5, 9, 12)
    assert p.ctx_off.tolist() == [0, 3, 4] and p.ctx_span.tolist() == [3, 1, 5]
    assert p.ctx_valid.tolist() == [3, 1, 5] and p.pos0.tolist() == [3, 1, 5] and p.gen_off.tolist() == [0, 4, 8]
    f = pp.pp_gen_layout_make([3, 1, 5], 4, padded=True)
    assert (f.ctx_rows, f.gen_rows, f.max_len) == (27, 27, 5)   # 3 rows of 5 + 4 slots
    assert f.ctx_off.tolist() == [0, 9, 18] and f.ctx_span.tolist() == [5, 5, 5]
    assert f.ctx_valid.tolist() == [3, 1, 5] and f.gen_off.tolist() == [5, 14, 23]


@settings(max_examples=60, deadline=None)
@given(st.lists(st.integers(1, 300), min_size=1, max_size=40), st.integers(1, 64), st.booleans())
def test_gen_layout_rows_are_disjoint_and_in_range(lengths, n_new, padded):
    """Every key row any decode step reads or writes lies inside its cache, and no two prompts
    (nor a prompt's context and generated rows in the padded layout) share a row."""
    g = pp.pp_gen_layout_make(lengths, n_new, padded)
    used_ctx, used_gen = set(), set()
    for i, l in enumerate(lengths):
        ctx = set(range(g.ctx_off[i], g.ctx_off[i] + g.ctx_span[i]))
        gen = set(range(g.gen_off[i], g.gen_off[i] + n_new))
        assert g.ctx_valid[i] == l and g.pos0[i] == l and g.ctx_span[i] >= l
        assert min(ctx) >= 0 and max(ctx) < g.ctx_rows and min(gen) >= 0 and max(gen) < g.gen_rows
        assert not (ctx & used_ctx) and not (gen & used_gen)
        if padded:
            assert not (ctx & gen) and not (gen & used_ctx) and not (ctx & used_gen)
        used_ctx |= ctx
        used_gen |= gen
    if not padded:   # packed: the context is exactly the prefill's compact cache, nothing padded
        assert g.ctx_rows == sum(lengths) and len(used_ctx) == sum(lengths) and g.gen_rows == len(lengths) * n_new


def test_gen_layout_rejections(L):
    with pytest.raises(pp.PrepackError):
        pp.pp_gen_layout_make([3, 0], 4)
    with pytest.raises(pp.PrepackError):
        pp.pp_gen_layout_make([3], 0)
    with pytest.raises(pp.PrepackError):
        pp.pp_gen_layout_make([], 4)
    with pytest.raises(pp.PrepackError):
        pp.pp_gen_layout_make([1 << 20] * 3000, 4, padded=True)   # more rows than an int32 index


def _glayout(**kw):
    base = dict(k=3, n_new=8, padded=0, max_len=300, ctx_rows=500, gen_rows=24,
                **{n: 0x1000 for n in ("ctx_off", "ctx_span", "ctx_valid", "pos0", "gen_off")})
    base.update(kw)
    return pp.PPGenDLayout(**base)


def test_decode_workspace_and_rejections(L):
    """Workspace size of the decode step and every host-side check of pp_decode_step and
    pp_generate: they return before any launch, so no GPU is needed."""
    cfg, gl = _cfg(vocab=32000), _glayout()
    n = ctypes.c_size_t()
    assert L.pp_decode_workspace_size(ctypes.byref(cfg), ctypes.byref(gl), ctypes.byref(n)) == pp.PP_OK
    k, d, H, D, F = 3, 4096, 32, 128, 14336
    chunks = 3 + 1                                          # ceil(300 / 128) context + 1 generated
    # split-K partial sums of the O and down projections (one row per prompt); the larger one
    # sets the size.  O: about 512 workgroups of 64 rows x up to 6 tiles of 128 columns.
    def splits(N, K):
        tiles, groups = K // 128, N // 64
        target = max(1, -(-512 // groups))
        per = min(6, max(1, -(-tiles // target)))
        return -(-tiles // per)
    # down, up to 16 prompts: the K / 512 segments in splits of at most 4, 2 or 1 (the most
    # that still gives 256 workgroups of 32 rows), near-equal in size
    def seg_splits(N, K):
        nseg, groups = -(-K // 512), N // 32
        for s in (4, 2):
            if groups * -(-nseg // s) >= 256:
                return -(-nseg // s)
        return nseg
    proj = [(48 * 128, d), (d, H * D), (2 * F, d), (d, F)]
    gpart = max(splits(*proj[1]) * k * proj[1][0] * 4, seg_splits(*proj[3]) * k * proj[3][0] * 4)
    want = (k * d * 4 + k * d * 2 + k * H * D * 2 + k * H * D * 2 + k * F * 2 + k * d * 4
            + k * H * chunks * (D + 4) * 4 + k * 64 * 8 + (4 * k + 1) * 4 + 16 * d * 2 + 250 * k * 8
            + gpart)
    assert want <= n.value <= want + 14 * 256
    ws = n.value
    bad = lambda **kw: L.pp_decode_workspace_size(ctypes.byref(cfg), ctypes.byref(_glayout(**kw)),
                                                  ctypes.byref(n))
    assert bad(k=0) == pp.PP_ERR_INVALID_ARG
    assert bad(n_new=0) == pp.PP_ERR_INVALID_ARG
    assert bad(padded=2) == pp.PP_ERR_INVALID_ARG
    assert bad(gen_rows=23) == pp.PP_ERR_INVALID_ARG         # fewer than k * n_new rows
    assert bad(gen_off=0) == pp.PP_ERR_INVALID_ARG           # NULL device array
    odd = _cfg(n_heads=24, n_kv_heads=8, vocab=32000)        # 3 query heads per key/value head
    assert L.pp_decode_workspace_size(ctypes.byref(odd), ctypes.byref(gl), ctypes.byref(n)) == pp.PP_ERR_UNSUPPORTED
    w, keep = _weights(1)
    f = L.pp_decode_step
    ok = dict(step=0, tin=0x3000, lm=0x4000, ck=0x5000, cv=0x6000, gk=0x7000, gv=0x8000, ws=0x10000, nb=ws,
              tout=0x9000)
    def call(c=cfg, g=gl, **kw):
        a = {**ok, **kw}
        return f(ctypes.byref(c), ctypes.byref(w), ctypes.byref(g), a["step"], a["tin"], a["lm"], a["ck"], a["cv"],
                 a["gk"], a["gv"], a["ws"], a["nb"], None, a["tout"], None)
    assert call(step=8) == pp.PP_ERR_INVALID_ARG             # step outside [0, n_new)
    assert call(step=-1) == pp.PP_ERR_INVALID_ARG
    assert call(tin=None) == pp.PP_ERR_INVALID_ARG
    assert call(tout=None) == pp.PP_ERR_INVALID_ARG
    assert call(gk=None) == pp.PP_ERR_INVALID_ARG
    assert call(lm=None) == pp.PP_ERR_INVALID_ARG
    assert call(ws=0x10008) == pp.PP_ERR_INVALID_ARG         # misaligned workspace
    assert call(nb=ws - 1) == pp.PP_ERR_BUFFER_TOO_SMALL
    assert call(c=_cfg(head_dim=96, vocab=32000)) == pp.PP_ERR_UNSUPPORTED
    g = L.pp_generate
    gen = lambda steps, **kw: g(ctypes.byref(cfg), ctypes.byref(w), ctypes.byref(gl), steps, 0x3000, 0x4000,
                                0x5000, 0x6000, 0x7000, 0x8000, kw.get("ws", 0x10000), kw.get("nb", ws), 0x9000,
                                None)
    assert gen(9) == pp.PP_ERR_INVALID_ARG                   # more steps than the caches hold
    assert gen(-1) == pp.PP_ERR_INVALID_ARG
    assert gen(0) == pp.PP_OK                                # nothing to do
    assert gen(4, nb=ws - 256) == pp.PP_ERR_BUFFER_TOO_SMALL
