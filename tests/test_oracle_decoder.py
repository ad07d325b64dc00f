"""Pins for the decoder oracle (oracle/decoder.py).  CPU only.

Each pin is something other than the oracle itself: Hugging Face's Llama code,
torch's textbook causal attention, closed forms, invariants, and the
exactness claim of section 3.3 (packed, padded and per-prompt prefill agree).
"""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

from oracle import decoder as D, ffd
from paper_2404_09529_amd import workloads as W

from . import hf_llama

TINY = dict(d_model=64, n_heads=4, n_kv_heads=4, head_dim=16, ffn_dim=96, vocab=50)
TINY_GQA = dict(d_model=64, n_heads=8, n_kv_heads=2, head_dim=16, ffn_dim=80, vocab=60)


def _case(lengths, n_layers=2, seed=0, **shape):
    return W.make_case(1, seed, n_layers=n_layers, lengths=lengths, random_gains=True, **shape)


def _scatter(plan, rows, per_slot):
    out = np.zeros((plan.total_len,) + per_slot.shape[1:], dtype=per_slot.dtype)
    real = plan.slot_kv >= 0
    out[plan.slot_kv[real]] = per_slot[real]
    return out


# ----------------------------------------------------------------------------- vs Hugging Face
@pytest.mark.parametrize("shape", [TINY, TINY_GQA], ids=["mha", "gqa"])
def test_per_prompt_matches_hugging_face(shape):
    c = _case([7, 1, 12, 4], **shape)
    sh = D.Shape.of(c.shape)
    model = hf_llama.build(c.shape, c.weights)
    ref = D.prefill_per_prompt(c.lengths, c.tokens, c.weights, sh)
    off = np.concatenate([[0], np.cumsum(c.lengths)])
    for i in range(len(c.lengths)):
        a, b = off[i], off[i + 1]
        h, ks, vs = hf_llama.run(model, c.tokens[None, a:b])
        # HF forms RoPE angles in float32, hence the 1e-5 bound rather than 1e-12
        assert D.errors(h[0], ref.hidden[a:b])[0] < 1e-5
        for l in range(sh.n_layers):
            assert D.errors(ks[l][0], ref.k[l][a:b])[0] < 1e-5
            assert D.errors(vs[l][0], ref.v[l][a:b])[0] < 1e-5


@pytest.mark.parametrize("shape", [TINY, TINY_GQA], ids=["mha", "gqa"])
def test_packed_rows_match_hugging_face_with_the_independent_mask(shape):
    """Section 3.2 implemented the way the paper did it (a custom mask and position ids
    handed to a Hugging Face model), compared with the oracle's per-prompt result."""
    c = _case([5, 3, 7, 2, 9, 1], **shape)
    sh = D.Shape.of(c.shape)
    plan = ffd.pack(c.lengths, 12)
    assert plan.n_rows < len(c.lengths)
    C = plan.capacity
    ids = np.zeros(plan.n_slots, dtype=np.int64)
    real = plan.slot_kv >= 0
    ids[real] = c.tokens[plan.slot_kv[real]]
    masks = np.stack([ffd.independent_mask(plan, r) for r in range(plan.n_rows)])
    h, ks, vs = hf_llama.run(hf_llama.build(c.shape, c.weights), ids.reshape(plan.n_rows, C),
                             hf_llama.additive_mask(masks), plan.slot_pos.reshape(plan.n_rows, C))
    ref = D.prefill_per_prompt(c.lengths, c.tokens, c.weights, sh)
    assert D.errors(_scatter(plan, None, h.reshape(plan.n_slots, -1)), ref.hidden)[0] < 1e-5
    for l in range(sh.n_layers):
        assert D.errors(_scatter(plan, None, ks[l].reshape(plan.n_slots, -1)), ref.k[l])[0] < 1e-5
        assert D.errors(_scatter(plan, None, vs[l].reshape(plan.n_slots, -1)), ref.v[l])[0] < 1e-5


def test_padded_batch_matches_hugging_face_full_batching():
    """Section 4.2's baseline: right padding plus a key-padding attention mask."""
    c = _case([6, 2, 9], **TINY_GQA)
    sh = D.Shape.of(c.shape)
    m = int(c.lengths.max())
    off = np.concatenate([[0], np.cumsum(c.lengths)])
    ids = np.zeros((len(c.lengths), m), dtype=np.int64)
    keep = np.zeros((len(c.lengths), m), dtype=np.int64)
    for i, l in enumerate(c.lengths):
        ids[i, :l] = c.tokens[off[i]:off[i + 1]]
        keep[i, :l] = 1
    h, ks, _ = hf_llama.run(hf_llama.build(c.shape, c.weights), ids, torch.from_numpy(keep))
    ours = D.prefill_padded(c.lengths, c.tokens, c.weights, sh)
    for i, l in enumerate(c.lengths):
        assert D.errors(h[i, :l], ours.hidden[off[i]:off[i + 1]])[0] < 1e-5
        assert D.errors(ks[1][i, :l], ours.k[1][off[i]:off[i + 1]])[0] < 1e-5


# ----------------------------------------------------------------------------- exactness (section 3.3)
@pytest.mark.parametrize("capacity", [0, 16, 40])
def test_three_modes_agree(capacity):
    c = _case([9, 3, 14, 1, 6, 6, 2], **TINY_GQA)
    sh = D.Shape.of(c.shape)
    plan = ffd.pack(c.lengths, capacity)
    a = D.prefill_per_prompt(c.lengths, c.tokens, c.weights, sh)
    b = D.prefill_packed_dense(plan, c.tokens, c.weights, sh)
    p = D.prefill_padded(c.lengths, c.tokens, c.weights, sh, pad_token=7)
    for x, y in [(a, b), (a, p)]:
        assert D.errors(x.hidden, y.hidden)[0] < 1e-12
        for l in range(sh.n_layers):
            assert D.errors(x.k[l], y.k[l])[0] < 1e-12
            assert D.errors(x.v[l], y.v[l])[0] < 1e-12


def test_packed_prompts_do_not_see_each_other():
    c = _case([6, 5, 4], n_layers=1, **TINY)
    sh = D.Shape.of(c.shape)
    plan = ffd.pack(c.lengths, 16)
    assert plan.n_rows == 1
    base = D.prefill_packed_dense(plan, c.tokens, c.weights, sh)
    toks = c.tokens.copy()
    toks[6:11] = (toks[6:11] + 1) % 50          # change prompt 1 only
    other = D.prefill_packed_dense(plan, toks, c.weights, sh)
    same = np.r_[0:6, 11:15]
    assert np.array_equal(base.hidden[same], other.hidden[same])
    assert not np.allclose(base.hidden[6:11], other.hidden[6:11])


def test_float32_oracle_close_to_float64():
    c = _case([7, 12, 3], **TINY_GQA)
    sh = D.Shape.of(c.shape)
    a = D.prefill_per_prompt(c.lengths, c.tokens, c.weights, sh)
    b = D.prefill_per_prompt(c.lengths, c.tokens, c.weights, sh, dtype=np.float32)
    assert D.errors(a.hidden, b.hidden)[0] < 1e-4


# ----------------------------------------------------------------------------- single steps
def test_attention_matches_torch_causal_sdpa():
    rng = np.random.default_rng(1)
    n, H, Hkv, Dh = 23, 8, 2, 16
    q, k, v = (rng.standard_normal((n, h, Dh)) for h in (H, Hkv, Hkv))
    ours = D.attention(q, k, v, D.causal(n))
    t = lambda x: torch.from_numpy(x).permute(1, 0, 2)[None]
    ref = F.scaled_dot_product_attention(t(q), t(k), t(v), is_causal=True, enable_gqa=True)
    assert np.abs(ours - ref[0].permute(1, 0, 2).numpy()).max() < 1e-12


def test_attention_special_cases():
    rng = np.random.default_rng(2)
    q, k, v = (rng.standard_normal((1, 2, 8)) for _ in range(3))
    # a one-token prompt attends only to itself: the output is its own V, exactly
    assert np.array_equal(D.attention(q, k, v, D.causal(1)), v)
    # a query with no allowed key gets 0
    o = D.attention(q, k, v, np.zeros((1, 1), dtype=bool))
    assert np.array_equal(o, np.zeros_like(o))
    # equal keys: uniform average of the visible values
    n = 5
    q = rng.standard_normal((n, 1, 8))
    k = np.repeat(rng.standard_normal((1, 1, 8)), n, axis=0)
    v = rng.standard_normal((n, 1, 8))
    o = D.attention(q, k, v, D.causal(n))
    for i in range(n):
        assert np.allclose(o[i, 0], v[: i + 1, 0].mean(axis=0), atol=1e-14)


def test_rope_properties():
    rng = np.random.default_rng(3)
    Dh, theta = 16, 10000.0
    x = rng.standard_normal((1, 3, Dh))
    c0, s0 = D.rope_cos_sin(np.array([0]), Dh, theta)
    assert np.array_equal(D.rope(x, c0, s0), x)             # position 0 is the identity
    pos = np.array([0, 1, 5, 77, 4095, 32767])
    cs, sn = D.rope_cos_sin(pos, Dh, theta)
    xs = rng.standard_normal((len(pos), 2, Dh))
    y = D.rope(xs, cs, sn)
    half = Dh // 2
    pair = lambda z: z[..., :half] ** 2 + z[..., half:] ** 2
    assert np.allclose(pair(y), pair(xs), atol=1e-12)       # rotations keep pair norms
    # the same rotation written with complex numbers: (a + ib) * e^{i pos theta^{-2j/D}}
    z = (xs[..., :half] + 1j * xs[..., half:]) * np.exp(
        1j * pos[:, None, None] * theta ** (-2.0 * np.arange(half) / Dh))
    assert np.allclose(np.concatenate([z.real, z.imag], -1), y, atol=1e-10)
    # scores depend on the relative position only
    q, k = rng.standard_normal((1, 1, Dh)), rng.standard_normal((1, 1, Dh))
    rot = lambda v, p: D.rope(v, *D.rope_cos_sin(np.array([p]), Dh, theta))
    dot = lambda a, b: float((rot(q, a) * rot(k, b)).sum())
    assert abs(dot(9, 4) - dot(105, 100)) < 1e-10
    assert abs(dot(9, 4) - dot(9, 5)) > 1e-6


def test_rmsnorm_and_silu():
    rng = np.random.default_rng(4)
    x = rng.standard_normal((6, 32)) * 3
    y = D.rms_norm(x, np.ones(32), 1e-5)
    ms = np.mean(x * x, axis=1)
    assert np.allclose(np.mean(y * y, axis=1), ms / (ms + 1e-5), atol=1e-13)
    g = rng.standard_normal(32)
    ref = F.rms_norm(torch.from_numpy(x), (32,), torch.from_numpy(g), eps=1e-5).numpy()
    assert np.allclose(D.rms_norm(x, g, 1e-5), ref, atol=1e-13)
    assert np.allclose(D.silu(x), F.silu(torch.from_numpy(x)).numpy(), atol=1e-13)


def test_first_token_key_is_unrotated_projection():
    """Restart positions: every prompt's first key sits at position 0, where RoPE is the
    identity, so in layer 0 it is the plain projection of its normalised embedding,
    wherever the prompt sits in its packed row."""
    c = _case([4, 7, 3, 5], n_layers=1, **TINY)
    sh = D.Shape.of(c.shape)
    plan = ffd.pack(c.lengths, 12)
    out = D.prefill_packed_dense(plan, c.tokens, c.weights, sh)
    L0 = c.weights["layers"][0]
    E = c.weights["embed"].astype(np.float64)
    for i in range(len(c.lengths)):
        t = plan.prompt_kv_off[i]
        want = D.rms_norm(E[c.tokens[t]], L0["attn_norm"].astype(np.float64), sh.rms_eps) @ L0["wk"].T.astype(np.float64)
        assert np.allclose(out.k[0][t], want, atol=1e-12)


def test_round_bf16():
    x = np.array([1.0, 1.0 + 2.0 ** -8, 1.0 + 3 * 2.0 ** -8, -2.5, 1.0 + 2.0 ** -7, 3.0e38], dtype=np.float64)
    # 3e38 = 1.7632 * 2^127; 1.7632 * 128 = 225.7 rounds to 226
    want = np.array([1.0, 1.0, 1.0 + 2.0 ** -6, -2.5, 1.0 + 2.0 ** -7, 226 / 128 * 2.0 ** 127])
    got = D.round_bf16(x)
    assert np.array_equal(got, want)


# ----------------------------------------------------------------------------- long-prompt helpers
def test_causal_rows_equal_the_dense_causal_mask():
    n = 11
    dense = D.causal(n)
    lazy = D.CausalRows(n)
    assert np.array_equal(lazy[0:n], dense)
    assert np.array_equal(lazy[3:7], dense[3:7])
    idx = np.array([10, 0, 4, 4])
    assert np.array_equal(lazy[idx], dense[idx])


@pytest.mark.parametrize("n_layers", [1, 2])
@pytest.mark.parametrize("shape", [TINY, TINY_GQA], ids=["mha", "gqa"])
def test_last_layer_rows_match_hugging_face_and_the_full_pass(n_layers, shape):
    """Restricting the last layer to a few query rows (what the long-prompt GPU tests use)
    gives Hugging Face's hidden states at those rows and leaves every cache row unchanged."""
    c = _case([23], n_layers=n_layers, **shape)
    sh = D.Shape.of(c.shape)
    rows = np.array([22, 0, 7, 15, 16])
    part = D.prefill_prompt(c.tokens, c.weights, sh, last_rows=rows)
    full = D.prefill_prompt(c.tokens, c.weights, sh)
    h, ks, vs = hf_llama.run(hf_llama.build(c.shape, c.weights), c.tokens[None, :])
    assert part.hidden.shape == (len(rows), sh.d_model)
    assert D.errors(part.hidden, h[0][rows])[0] < 1e-5
    assert D.errors(part.hidden, full.hidden[rows])[0] < 1e-12
    for l in range(n_layers):
        assert D.errors(part.k[l], ks[l][0])[0] < 1e-5 and D.errors(part.v[l], vs[l][0])[0] < 1e-5
        assert np.array_equal(part.k[l], full.k[l]) and np.array_equal(part.v[l], full.v[l])
    # the bf16 rounding hook sees the same values at those rows
    part_r = D.prefill_prompt(c.tokens, c.weights, sh, rnd=D.round_bf16, last_rows=rows)
    full_r = D.prefill_prompt(c.tokens, c.weights, sh, rnd=D.round_bf16)
    assert D.errors(part_r.hidden, full_r.hidden[rows])[0] < 1e-12
