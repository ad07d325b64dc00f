"""Oracle: greedy generation after the prefill, one prompt at a time.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

What is computed.  Autoregressive sampling runs one forward pass per new token
(section 2.2); the KV cache only saves recomputing the keys and values of
earlier tokens, it does not change the result.  So the plain definition of
generation, used here, recomputes everything: the token after a sequence s is
argmax over the vocabulary of hidden(s)[last] . W_lm (lowest id on ties,
numpy's argmax), with hidden(s) the decoder of ``oracle.decoder`` over s alone
(causal mask, positions 0..|s|-1).  Greedy generation of a prompt p appends
that token and repeats.  Packing the caches for generation (section 4.8) must
give each prompt exactly what it gets alone, so there is one mode: per prompt.

``teacher_forced`` is the same forward over the prompt followed by a given
list of fed tokens: row l + t of that single pass is what a decode step that
consumes fed token t at position l + t must produce (its key and value, which
the step appends to the cache, and the final hidden row whose logits choose
the next token), because causality makes row l + t independent of later rows.

Readings, where the paper is silent: generation is greedy; the
token consumed by the first decode step is the first token chosen from the
prefill (section 2.3); positions continue each prompt's own positions, l, l+1,
... (restart positions, section 3.2, carried into generation).

Parity pins: tests/test_oracle_generate.py (Hugging Face's greedy generate with
its own KV cache on tiny models, the prefill's first token, prefix invariance
of the caches, and self-consistency of the two functions).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import List, Sequence

import numpy as np

from . import decoder as D


@dataclass
class Forced:
    """Rows l .. l + n_fed - 1 of one pass over prompt + fed tokens."""
    hidden: np.ndarray            # [n_fed, d]   final hidden rows (after the final norm)
    logits: np.ndarray            # [n_fed, V]
    k: List[np.ndarray]           # per layer [n_fed, Hkv*D]: the cache rows the steps append
    v: List[np.ndarray]


def teacher_forced(prompt: Sequence[int], fed: Sequence[int], weights, shape: D.Shape, lm_head: np.ndarray,
                   rnd: D.Rounder = D._ident) -> Forced:
    """The prompt followed by ``fed`` in one causal pass; the rows of the fed tokens."""
    seq = np.concatenate([np.asarray(prompt, dtype=np.int64), np.asarray(fed, dtype=np.int64)])
    l = len(prompt)
    r = D.prefill_prompt(seq, weights, shape, rnd)
    h = r.hidden[l:]
    logits = rnd(h) @ np.asarray(lm_head, dtype=np.float64).T
    return Forced(hidden=h, logits=logits, k=[k[l:] for k in r.k], v=[v[l:] for v in r.v])


def generate(prompt: Sequence[int], weights, shape: D.Shape, lm_head: np.ndarray, n_tokens: int,
             rnd: D.Rounder = D._ident) -> np.ndarray:
    """The first ``n_tokens`` greedily generated tokens of one prompt, each chosen from a full
    recomputation over the prompt and the tokens chosen before it."""
    seq = [int(t) for t in prompt]
    lm = np.asarray(lm_head, dtype=np.float64)
    out = []
    for _ in range(n_tokens):
        h = D.prefill_prompt(np.asarray(seq, dtype=np.int64), weights, shape, rnd).hidden[-1]
        tok = int(np.argmax(rnd(h) @ lm.T))
        out.append(tok)
        seq.append(tok)
    return np.asarray(out, dtype=np.int64)


def generate_batch(lengths: Sequence[int], tokens: np.ndarray, weights, shape: D.Shape, lm_head: np.ndarray,
                   n_tokens: int, prompts: Sequence[int] = None) -> np.ndarray:
    """``generate`` for every prompt of a flat batch (original order): [k, n_tokens]; rows of
    prompts left out of ``prompts`` are -1."""
    lengths = np.asarray(lengths, dtype=np.int64)
    off = np.concatenate([[0], np.cumsum(lengths)])
    out = np.full((len(lengths), n_tokens), -1, dtype=np.int64)
    for i in (range(len(lengths)) if prompts is None else prompts):
        out[i] = generate(tokens[off[i]:off[i + 1]], weights, shape, lm_head, n_tokens)
    return out
