"""Oracle: Llama-style decoder prefill over prompts, packed rows or padded rows.

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

What is computed (section 2.1 for self-attention; the appendix model table
for the Llama / Mistral family the paper runs; section 3.2 for the masks and
positions; Algorithm 1 for the prefill-then-unpack structure):

  x = E[token]
  for every layer:
      xn      = RMSNorm(x) * g_attn            RMSNorm(x) = x / sqrt(mean(x^2) + eps)
      q, k, v = xn Wq^T, xn Wk^T, xn Wv^T       split into heads of size D
      q, k    = RoPE(q, k; position)            rotate-half pairs (i, i + D/2),
                                                angle = position * theta^(-2i/D)
      o       = softmax(q k^T / sqrt(D) + mask) v     per head; query head h reads
                                                      key/value head h // (H / Hkv)
      x       = x + o Wo^T
      hn      = RMSNorm(x) * g_mlp
      x       = x + (SiLU(hn Wg^T) * (hn Wu^T)) Wd^T
      cache   = (k after RoPE, v)               the layer's KV cache
  hidden = RMSNorm(x) * g_final

First token (section 2.3: the time to first token covers prefilling the KV
cache and generating the first token; section 4.3 adds the unpacking): for
every prompt, the logits of its last token, hidden[last] W_lm^T over the
vocabulary, and the greedy choice argmax, lowest id on ties (``first_token``).

Readings of the paper, where it is silent or ambiguous:
* the score scale is 1/sqrt(D), D the head size (the paper writes the
  single-head form with the model width);
* the mask is applied to the scores before the softmax, masked entries
  contributing exactly zero probability;
* a query with no allowed key (a pad slot under M') has output 0;
* the cached K is the post-RoPE K;
* RoPE angles are formed and evaluated in float64;
* the final hidden state is taken after the final RMSNorm;
* the first token is chosen greedily (the paper names no sampler).

Modes, which the paper asserts give the exact same caches (section 3.3):
* ``prefill_per_prompt`` -- every prompt alone, causal mask, positions
  0..l-1 (the plain definition of the result);
* ``prefill_packed_dense`` -- the packed rows of a plan under the literal
  independent mask M' and restart positions, then UNPACK;
* ``prefill_padded`` -- full batching: right-padded rows with a pad token and a
  key-padding mask, the pad outputs discarded.

Precision: float64 by default.  ``rnd`` (identity by default) is a hook
applied to the values a bfloat16 pipeline would store (normalised inputs of
the projections, q/k/v, rotated q/k, the attention probabilities fed to the
value product, attention outputs and the SwiGLU product, and the cache).  It
is used only to measure the rounding floor of an ideal bf16 pipeline; with
the identity hook the code is the plain definition above.

Parity pins: tests/test_oracle_decoder.py (Hugging Face's independent Llama
implementation on tiny shapes, textbook causal attention, closed forms and
invariants of every step, and agreement of the three modes).
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Callable, Dict, List, Optional, Sequence

import numpy as np

from . import ffd

Rounder = Callable[[np.ndarray], np.ndarray]


def _ident(x: np.ndarray) -> np.ndarray:
    return x


@dataclass
class Shape:
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    rms_eps: float
    rope_theta: float

    @classmethod
    def of(cls, s) -> "Shape":
        return cls(s.n_layers, s.d_model, s.n_heads, s.n_kv_heads, s.head_dim, s.ffn_dim,
                   float(s.rms_eps), float(s.rope_theta))


# ----------------------------------------------------------------------------- steps
def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def rope_cos_sin(positions: np.ndarray, head_dim: int, theta: float):
    """cos, sin of shape [n, D/2]; angle_i = position * theta^(-2i/D), all in float64."""
    i = np.arange(head_dim // 2, dtype=np.float64)
    inv_freq = theta ** (-2.0 * i / head_dim)
    ang = np.asarray(positions, dtype=np.float64)[:, None] * inv_freq[None, :]
    return np.cos(ang), np.sin(ang)


def rope(x: np.ndarray, cos: np.ndarray, sin: np.ndarray) -> np.ndarray:
    """Rotate pairs (x_i, x_{i+D/2}) by the angle of pair i.  x: [n, heads, D]."""
    half = x.shape[-1] // 2
    a, b = x[..., :half], x[..., half:]
    c, s = cos[:, None, :], sin[:, None, :]
    return np.concatenate([a * c - b * s, b * c + a * s], axis=-1)


def silu(x: np.ndarray) -> np.ndarray:
    return x / (1.0 + np.exp(-x))


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, allowed: np.ndarray,
              rnd: Rounder = _ident, q_chunk: int = 2048) -> np.ndarray:
    """softmax(q k^T / sqrt(D) + mask) v per head.

    q [nq, H, D]; k, v [n, Hkv, D]; allowed: [nq, n] boolean (query, key), or anything
    sliced like it.
    Rows are processed in chunks of ``q_chunk`` queries to bound memory; every
    row's arithmetic is the same whatever the chunking.
    """
    n, H, D = q.shape
    Hkv = k.shape[1]
    group = H // Hkv
    out = np.zeros_like(q)
    scale = 1.0 / np.sqrt(D)
    for h in range(H):
        g = h // group
        kh, vh = k[:, g, :], v[:, g, :]
        for a in range(0, n, q_chunk):
            b = min(n, a + q_chunk)
            s = (q[a:b, h, :] @ kh.T) * scale
            ok = allowed[a:b]
            s = np.where(ok, s, -np.inf)
            mx = np.max(s, axis=1, keepdims=True)
            has = np.isfinite(mx)
            e = np.where(ok, np.exp(s - np.where(has, mx, 0.0)), 0.0)
            den = np.sum(e, axis=1, keepdims=True)
            p = e / np.where(has, den, 1.0)
            o = rnd(p) @ vh
            out[a:b, h, :] = np.where(has, o, 0.0)
    return out


def causal(n: int) -> np.ndarray:
    return np.tril(np.ones((n, n), dtype=bool))


class CausalRows:
    """The causal mask of n tokens, produced a block of query rows at a time instead of as
    one [n, n] array: ``CausalRows(n)[rows]`` equals ``causal(n)[rows]`` for a slice or an
    index array.  Long prompts (tens of thousands of tokens) need it to stay in memory."""

    def __init__(self, n: int):
        self.n = n

    def __getitem__(self, rows) -> np.ndarray:
        q = np.arange(self.n)[rows]
        return np.arange(self.n)[None, :] <= q[:, None]


# ----------------------------------------------------------------------------- the stack
@dataclass
class Result:
    hidden: np.ndarray            # [n, d]
    k: List[np.ndarray]           # per layer [n, Hkv*D]
    v: List[np.ndarray]


def forward(x: np.ndarray, weights: Dict, shape: Shape, positions: np.ndarray,
            allowed, rnd: Rounder = _ident, dtype=np.float64,
            last_rows: Optional[np.ndarray] = None) -> Result:
    """The decoder over one sequence of embedded tokens x [n, d].

    ``allowed`` is the [n, n] boolean mask (query, key), or anything indexed like it
    (``CausalRows``).  ``last_rows`` (default: all) restricts what the LAST layer computes
    after its keys and values to those query rows: their attention output, MLP and final
    norm.  Every layer's keys and values, and every result at those rows, are the same as
    without the restriction, since no other row reads them; ``hidden`` then holds only those
    rows, in the order given."""
    s = shape
    H, Hkv, D = s.n_heads, s.n_kv_heads, s.head_dim
    n = x.shape[0]
    x = np.asarray(x, dtype=dtype)
    cos, sin = rope_cos_sin(positions, D, s.rope_theta)
    cos, sin = cos.astype(dtype), sin.astype(dtype)
    ks, vs = [], []
    eps = dtype(s.rms_eps)
    layers = weights["layers"][: s.n_layers]
    for li, L in enumerate(layers):
        W = {key: np.asarray(val, dtype=dtype) for key, val in L.items()}
        xn = rnd(rms_norm(x, W["attn_norm"], eps))
        k = rnd(xn @ W["wk"].T).reshape(n, Hkv, D)
        v = rnd(xn @ W["wv"].T).reshape(n, Hkv, D)
        k = rnd(rope(k, cos, sin))
        if last_rows is not None and li == len(layers) - 1:
            sel = np.asarray(last_rows, dtype=np.int64)
            xn, x, qcos, qsin, mask = xn[sel], x[sel], cos[sel], sin[sel], allowed[sel]
        else:
            qcos, qsin, mask = cos, sin, allowed
        nq = x.shape[0]
        q = rnd(xn @ W["wq"].T).reshape(nq, H, D)
        q = rnd(rope(q, qcos, qsin))
        o = rnd(attention(q, k, v, mask, rnd).reshape(nq, H * D))
        x = x + o @ W["wo"].T
        hn = rnd(rms_norm(x, W["mlp_norm"], eps))
        a = rnd(silu(hn @ W["wg"].T) * (hn @ W["wu"].T))
        x = x + a @ W["wd"].T
        ks.append(k.reshape(n, Hkv * D))
        vs.append(v.reshape(n, Hkv * D))
    hidden = rms_norm(x, np.asarray(weights["final_norm"], dtype=dtype), eps)
    return Result(hidden=hidden, k=ks, v=vs)


def embed(weights: Dict, tokens: np.ndarray, dtype=np.float64) -> np.ndarray:
    return np.asarray(weights["embed"], dtype=dtype)[np.asarray(tokens, dtype=np.int64)]


def _alloc(total: int, shape: Shape, dtype) -> Result:
    kv = shape.n_kv_heads * shape.head_dim
    return Result(hidden=np.zeros((total, shape.d_model), dtype=dtype),
                  k=[np.zeros((total, kv), dtype=dtype) for _ in range(shape.n_layers)],
                  v=[np.zeros((total, kv), dtype=dtype) for _ in range(shape.n_layers)])


def prefill_prompt(tokens: np.ndarray, weights: Dict, shape: Shape, rnd: Rounder = _ident,
                   dtype=np.float64, last_rows: Optional[np.ndarray] = None) -> Result:
    """One prompt alone: causal mask, positions 0..l-1.  ``last_rows`` as in ``forward``."""
    n = len(tokens)
    return forward(embed(weights, tokens, dtype), weights, shape, np.arange(n), CausalRows(n), rnd, dtype,
                   last_rows)


def prefill_per_prompt(lengths: Sequence[int], tokens: np.ndarray, weights: Dict, shape: Shape,
                       rnd: Rounder = _ident, dtype=np.float64,
                       prompts: Optional[Sequence[int]] = None) -> Result:
    """Each prompt prefilled on its own; results at the prompt's rows of the compact cache.

    ``prompts`` restricts the work to a subset (other rows stay zero).
    """
    lengths = np.asarray(lengths, dtype=np.int64)
    off = np.concatenate([[0], np.cumsum(lengths)])
    out = _alloc(int(off[-1]), shape, dtype)
    for i in (range(len(lengths)) if prompts is None else prompts):
        a, b = int(off[i]), int(off[i + 1])
        r = prefill_prompt(tokens[a:b], weights, shape, rnd, dtype)
        out.hidden[a:b] = r.hidden
        for l in range(shape.n_layers):
            out.k[l][a:b] = r.k[l]
            out.v[l][a:b] = r.v[l]
    return out


def prefill_packed_dense(plan: ffd.Plan, tokens: np.ndarray, weights: Dict, shape: Shape,
                         rnd: Rounder = _ident, dtype=np.float64) -> Result:
    """Algorithm 1 literally: packed rows, the dense independent mask M', restart positions,
    one forward per row, then UNPACK into per-prompt caches (original order)."""
    C = plan.capacity
    d = shape.d_model
    E = np.asarray(weights["embed"], dtype=dtype)
    out = _alloc(plan.total_len, shape, dtype)
    for row in range(plan.n_rows):
        sl = slice(row * C, (row + 1) * C)
        kv = plan.slot_kv[sl]
        x = np.zeros((C, d), dtype=dtype)
        real = kv >= 0
        x[real] = E[tokens[kv[real]]]
        r = forward(x, weights, shape, plan.slot_pos[sl], ffd.independent_mask(plan, row), rnd, dtype)
        out.hidden[kv[real]] = r.hidden[real]
        for l in range(shape.n_layers):
            out.k[l][kv[real]] = r.k[l][real]
            out.v[l][kv[real]] = r.v[l][real]
    return out


def prefill_padded(lengths: Sequence[int], tokens: np.ndarray, weights: Dict, shape: Shape,
                   pad_token: int = 0, rnd: Rounder = _ident, dtype=np.float64) -> Result:
    """Full batching: prompt i right-padded to m with ``pad_token``; a query may attend to
    keys at or before it that are not pads (the key-padding mask); pad outputs discarded."""
    lengths = np.asarray(lengths, dtype=np.int64)
    m = int(lengths.max())
    off = np.concatenate([[0], np.cumsum(lengths)])
    out = _alloc(int(off[-1]), shape, dtype)
    for i, l in enumerate(lengths):
        toks = np.full(m, pad_token, dtype=np.int64)
        toks[:l] = tokens[off[i]:off[i + 1]]
        keep = np.zeros(m, dtype=bool)
        keep[:l] = True
        allowed = causal(m) & keep[None, :]
        r = forward(embed(weights, toks, dtype), weights, shape, np.arange(m), allowed, rnd, dtype)
        a, b = int(off[i]), int(off[i + 1])
        out.hidden[a:b] = r.hidden[:l]
        for layer in range(shape.n_layers):
            out.k[layer][a:b] = r.k[layer][:l]
            out.v[layer][a:b] = r.v[layer][:l]
    return out


# ----------------------------------------------------------------------------- first token
def last_token_rows(lengths: Sequence[int]) -> np.ndarray:
    """Row of each prompt's last token in the unpacked hidden state (original order)."""
    return np.cumsum(np.asarray(lengths, dtype=np.int64)) - 1


def first_token(hidden: np.ndarray, lengths: Sequence[int], lm_head: np.ndarray,
                rnd: Rounder = _ident):
    """Greedy first token of every prompt (section 2.3).

    hidden [total_len, d] in original prompt order; lm_head [vocab, d].
    Returns (logits [k, vocab] float64, tokens [k] int64): logits of prompt i
    = rnd(hidden[last_i]) . lm_head[v] over v, token = the first v of maximal
    logit (numpy's argmax takes the first maximum).
    """
    h = rnd(np.asarray(hidden, dtype=np.float64)[last_token_rows(lengths)])
    logits = h @ np.asarray(lm_head, dtype=np.float64).T
    return logits, np.argmax(logits, axis=1)


# ----------------------------------------------------------------------------- bf16 floor
def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round to the nearest bfloat16 value (ties to even), returned in the input's dtype.

    float64 inputs are first rounded to float32; the double rounding this can
    cause is rare and immaterial for a rounding-floor estimate.
    """
    x = np.asarray(x)
    f = np.ascontiguousarray(x, dtype=np.float32)
    u = f.view(np.uint32).astype(np.uint64)
    u = ((u + 0x7FFF + ((u >> 16) & 1)) >> 16) << 16
    return u.astype(np.uint32).view(np.float32).astype(x.dtype).reshape(x.shape)


def errors(a: np.ndarray, b: np.ndarray):
    """(max |a-b|, mean |a-b|)."""
    d = np.abs(np.asarray(a, dtype=np.float64) - np.asarray(b, dtype=np.float64))
    return (float(d.max()) if d.size else 0.0, float(d.mean()) if d.size else 0.0)
