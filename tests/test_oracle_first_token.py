"""Pins of the oracle's first-token step (section 2.3: time to first token = prefill plus the
generation of the first token): the LM head on each prompt's last token and the greedy
choice.  CPU only."""
import numpy as np
import pytest

from oracle import decoder as D
from paper_2404_09529_amd import workloads as W

from . import hf_llama

TINY = dict(d_model=64, n_heads=4, n_kv_heads=4, head_dim=16, ffn_dim=96, vocab=50)


def test_first_token_matches_hugging_face_causal_lm():
    # an independent implementation of the whole step: decoder, final norm and LM head
    c = W.make_case(1, 0, n_layers=2, lengths=[7, 1, 12, 4], random_gains=True, **TINY)
    lm_head = W.draw_lm_head(c.wl, 0, c.shape)
    sh = D.Shape.of(c.shape)
    ref = D.prefill_per_prompt(c.lengths, c.tokens, c.weights, sh)
    logits, tokens = D.first_token(ref.hidden, c.lengths, lm_head)
    off = np.concatenate([[0], np.cumsum(c.lengths)])
    for i in range(len(c.lengths)):
        hf = hf_llama.last_logits(c.shape, c.weights, lm_head, c.tokens[off[i]:off[i + 1]])
        assert np.max(np.abs(hf - logits[i])) < 1e-5   # HF forms RoPE angles in float32
        assert int(np.argmax(hf)) == int(tokens[i])


def test_last_token_rows_pick_each_prompts_last_row():
    # hidden row r = e_r, LM head = identity: prompt i's logits are the one-hot of its last row
    lengths = [3, 1, 4, 2]
    L = sum(lengths)
    logits, tokens = D.first_token(np.eye(L), lengths, np.eye(L))
    assert tokens.tolist() == [2, 3, 7, 9]
    assert np.array_equal(logits, np.eye(L)[[2, 3, 7, 9]])


def test_planted_maximum_and_lowest_id_on_ties():
    rng = np.random.default_rng(5)
    h = rng.standard_normal((6, 16))
    lengths = [2, 4]                 # last rows 1 and 5
    lm = 0.01 * rng.standard_normal((40, 16))
    lm[17] = 3.0 * h[1]              # logit 3 |h1|^2, far above the rest
    lm[29] = 3.0 * h[5]
    logits, tokens = D.first_token(h, lengths, lm)
    assert tokens.tolist() == [17, 29]
    assert logits[0, 17] == pytest.approx(3.0 * h[1] @ h[1])
    lm[4] = lm[17]                   # an equal maximum at a lower id wins
    assert D.first_token(h, lengths, lm)[1].tolist() == [4, 29]


def test_vocabulary_permutation_is_equivariant():
    rng = np.random.default_rng(6)
    h = rng.standard_normal((9, 12))
    lm = rng.standard_normal((30, 12))
    lengths = [4, 5]
    logits, tokens = D.first_token(h, lengths, lm)
    perm = rng.permutation(30)
    logits_p, tokens_p = D.first_token(h, lengths, lm[perm])
    assert np.array_equal(logits_p, logits[:, perm])
    assert perm[tokens_p].tolist() == tokens.tolist()


def test_rounding_hook_applies_to_the_hidden_row_only():
    rng = np.random.default_rng(7)
    h = rng.standard_normal((3, 8)) * (1 + 1e-3)
    lm = W.bf16_value(W.bf16_bits(rng.standard_normal((5, 8)).astype(np.float32))).reshape(5, 8)
    lg, _ = D.first_token(h, [3], lm, rnd=D.round_bf16)
    assert np.allclose(lg[0], D.round_bf16(h[2]) @ lm.T.astype(np.float64), rtol=0, atol=1e-12)
