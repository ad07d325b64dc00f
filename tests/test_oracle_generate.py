"""Pins of the generation oracle (greedy decoding after the prefill; section 2.2 for
autoregressive sampling with a KV cache, section 4.8 for packing the caches during
generation).  The oracle recomputes the whole sequence for every token; Hugging Face's
generate decodes incrementally with its own KV cache, an independent implementation.
CPU only."""
import numpy as np
import pytest

from oracle import decoder as D
from oracle import generate as G
from paper_2404_09529_amd import workloads as W

from . import hf_llama

TINY = dict(d_model=64, n_heads=4, n_kv_heads=4, head_dim=16, ffn_dim=96, vocab=50)
TINY_GQA = dict(d_model=64, n_heads=4, n_kv_heads=2, head_dim=16, ffn_dim=96, vocab=50)


def _case(seed, lengths, n_layers=2, **shape):
    c = W.make_case(1, seed, n_layers=n_layers, lengths=lengths, random_gains=True, **shape)
    return c, W.draw_lm_head(c.wl, seed, c.shape), D.Shape.of(c.shape)


def _prompts(c):
    off = np.concatenate([[0], np.cumsum(c.lengths)])
    return [c.tokens[off[i]:off[i + 1]] for i in range(len(c.lengths))]


def _gap(logits):
    s = np.sort(logits)
    return s[-1] - s[-2]


@pytest.mark.parametrize("shape", [TINY, TINY_GQA], ids=["mha", "gqa"])
def test_matches_hugging_face_greedy_generate(shape):
    c, lm, sh = _case(0, [6, 1, 13], **shape)
    for p in _prompts(c):
        ours = G.generate(p, c.weights, sh, lm, 8)
        hf, hk, hv = hf_llama.greedy_generate(c.shape, c.weights, lm, p, 8)
        # every choice must be clear of a tie: HF forms RoPE angles in float32
        f = G.teacher_forced(p, ours[:-1], c.weights, sh, lm)
        first = D.prefill_prompt(p, c.weights, sh).hidden[-1] @ lm.T
        assert min([_gap(first)] + [_gap(r) for r in f.logits]) > 1e-4
        assert ours.tolist() == hf.tolist()
        # the cache rows HF appended while decoding are the teacher-forced rows
        for layer in range(sh.n_layers):
            assert np.max(np.abs(hk[layer] - f.k[layer][: len(ours) - 1])) < 1e-5
            assert np.max(np.abs(hv[layer] - f.v[layer][: len(ours) - 1])) < 1e-5


def test_first_generated_token_is_the_prefills_first_token():
    c, lm, sh = _case(1, [5, 9, 2, 17])
    ref = D.prefill_per_prompt(c.lengths, c.tokens, c.weights, sh)
    _, first = D.first_token(ref.hidden, c.lengths, lm)
    gen = G.generate_batch(c.lengths, c.tokens, c.weights, sh, lm, 1)
    assert gen[:, 0].tolist() == first.tolist()


def test_generation_is_argmax_of_the_teacher_forced_rows():
    c, lm, sh = _case(2, [11])
    p = _prompts(c)[0]
    gen = G.generate(p, c.weights, sh, lm, 6)
    f = G.teacher_forced(p, gen[:-1], c.weights, sh, lm)
    assert np.argmax(f.logits, axis=1).tolist() == gen[1:].tolist()


def test_teacher_forced_rows_are_prefix_invariant():
    """Causality: the rows of fed token t do not depend on the tokens fed after it, and the
    prompt's own rows are the prefill's."""
    c, lm, sh = _case(3, [7])
    p = _prompts(c)[0]
    fed = [3, 41, 0, 17, 17]
    full = G.teacher_forced(p, fed, c.weights, sh, lm)
    part = G.teacher_forced(p, fed[:2], c.weights, sh, lm)
    assert np.allclose(part.hidden, full.hidden[:2], rtol=0, atol=1e-12)
    for layer in range(sh.n_layers):
        assert np.allclose(part.k[layer], full.k[layer][:2], rtol=0, atol=1e-12)
    pre = D.prefill_prompt(p, c.weights, sh)
    seq = D.prefill_prompt(np.concatenate([p, fed]), c.weights, sh)
    for layer in range(sh.n_layers):
        assert np.allclose(seq.k[layer][:7], pre.k[layer], rtol=0, atol=1e-12)


def test_a_prompt_generates_the_same_in_any_batch():
    """Packing the caches must not couple prompts: generation is per prompt by definition,
    so a prompt's tokens do not depend on which other prompts share its batch."""
    c, lm, sh = _case(4, [4, 10, 1])
    alone = G.generate(_prompts(c)[1], c.weights, sh, lm, 5)
    batch = G.generate_batch(c.lengths, c.tokens, c.weights, sh, lm, 5)
    assert batch[1].tolist() == alone.tolist()
