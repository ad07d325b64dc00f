"""Seeded synthetic workloads for packed prefill.

This module only draws numbers: prompt lengths, token ids and model weights.
It contains none of the method's arithmetic (no packing, no attention, no
normalisation), so that both the CPU oracle and the GPU path can be fed the
same inputs without sharing any code that computes a result.

The paper measures on text datasets whose prompt-length statistics are listed
in its appendix table of dataset lengths (min / mean / max per dataset) and on
Llama-family models whose shapes are listed in its appendix table of model
architectures.  Neither the datasets nor the trained checkpoints are available
here, so every workload is synthetic:

* prompt lengths are drawn from a per-workload distribution (uniform,
  lognormal, bimodal or Zipf) that stands in for a dataset's length mix;
* token ids are uniform over the vocabulary;
* weights are i.i.d. N(0, 0.02^2), rounded to bfloat16 (round to nearest even)
  for the bf16 workloads, so that both sides consume identical values.

Random streams: ``numpy.random.default_rng([workload_id, seed, stream])`` with
stream 0 = lengths, 1 = tokens, 2 = weights, 3 = norm gains (parity cases only;
the benchmark workloads use unit gains), 4 = the LM head (first-token step).
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import Callable, Dict, List, Optional

import numpy as np
from statistics import NormalDist

__all__ = [
    "ModelShape", "Workload", "Case", "WORKLOADS", "MODELS", "DATASETS", "workload", "make_case",
    "draw_lengths", "draw_tokens", "draw_weights", "bf16_bits", "bf16_value",
]


@dataclass(frozen=True)
class ModelShape:
    """Llama-style decoder shape (paper appendix, model-architecture table)."""
    n_layers: int
    d_model: int
    n_heads: int
    n_kv_heads: int
    head_dim: int
    ffn_dim: int
    vocab: int
    dtype: str            # "f32" or "bf16": storage/compute type of the GPU path
    rms_eps: float = 1e-5
    rope_theta: float = 10000.0

    def replace(self, **kw) -> "ModelShape":
        return dataclasses.replace(self, **kw)


@dataclass(frozen=True)
class Workload:
    wid: int
    name: str
    shape: ModelShape
    k: int                # prompts per batch
    capacity: int         # packed row length C
    lengths: Callable[[np.random.Generator, int], np.ndarray]
    description: str = ""


def _uniform(lo: int, hi: int):
    def f(rng: np.random.Generator, k: int) -> np.ndarray:
        return rng.integers(lo, hi + 1, k)
    return f


def _lognormal(median: float, sigma: float, lo: int, hi: int):
    def f(rng: np.random.Generator, k: int) -> np.ndarray:
        x = rng.lognormal(np.log(median), sigma, k)
        return np.clip(np.rint(x), lo, hi)
    return f


def _bimodal(short: tuple, long: tuple, frac_long: float):
    def f(rng: np.random.Generator, k: int) -> np.ndarray:
        n_long = int(round(frac_long * k))
        a = rng.integers(short[0], short[1] + 1, k - n_long)
        b = rng.integers(long[0], long[1] + 1, n_long)
        return rng.permutation(np.concatenate([a, b]))
    return f


def _zipf(a: float, scale: int, hi: int):
    def f(rng: np.random.Generator, k: int) -> np.ndarray:
        return np.minimum(scale * rng.zipf(a, k), hi)
    return f


_LLAMA2_7B = ModelShape(n_layers=4, d_model=4096, n_heads=32, n_kv_heads=32, head_dim=128,
                        ffn_dim=11008, vocab=32000, dtype="bf16", rope_theta=10000.0)

WORKLOADS: Dict[int, Workload] = {
    1: Workload(1, "tiny-fp32",
                ModelShape(n_layers=1, d_model=256, n_heads=4, n_kv_heads=4, head_dim=64,
                           ffn_dim=688, vocab=1000, dtype="f32"),
                k=8, capacity=128, lengths=_uniform(4, 64),
                description="tiny Llama-style decoder, 1 layer, fp32; 8 prompts U[4,64]; rows of 128"),
    2: Workload(2, "llama2-7b-lognormal", _LLAMA2_7B,
                k=64, capacity=4096, lengths=_lognormal(256, 1.0, 8, 4096),
                description="Llama-2-7B shape, 4 layers, bf16; 64 prompts lognormal(median 256, "
                            "sigma 1.0) clipped to [8,4096]; rows of 4096"),
    3: Workload(3, "llama2-7b-bimodal", _LLAMA2_7B,
                k=96, capacity=4096, lengths=_bimodal((16, 128), (1024, 4096), 0.2),
                description="Llama-2-7B shape, 4 layers, bf16; 96 prompts, 80% U[16,128] and "
                            "20% U[1024,4096]; rows of 4096"),
    4: Workload(4, "llama3-8b-gqa-lognormal",
                ModelShape(n_layers=4, d_model=4096, n_heads=32, n_kv_heads=8, head_dim=128,
                           ffn_dim=14336, vocab=128256, dtype="bf16", rope_theta=500000.0),
                k=128, capacity=8192, lengths=_lognormal(512, 1.2, 8, 8192),
                description="Llama-3-8B shape (GQA 32/8), 4 layers, bf16; 128 prompts "
                            "lognormal(median 512, sigma 1.2) clipped to [8,8192]; rows of 8192"),
    5: Workload(5, "llama-1.3b-long-zipf",
                ModelShape(n_layers=24, d_model=2048, n_heads=16, n_kv_heads=16, head_dim=128,
                           ffn_dim=5504, vocab=32000, dtype="bf16", rope_theta=10000.0),
                k=48, capacity=32768, lengths=_zipf(1.5, 32, 32768),
                description="1.3B shape, 24 layers, bf16; 48 prompts 32*Zipf(1.5) clipped to "
                            "32768; rows of 32768"),
}


# Prompt pools for the batch-size and regression sweeps (the paper's section on how the gain
# scales with the lengths in a batch, and its batch-size ablation): 5000 synthetic prompts with
# lengths uniform in [1, 512], taken in draw order in batches of k, each batch packed with the
# bin size equal to its own maximum length (capacity 0).  The model is chosen separately from
# MODELS; ``k`` here is the pool size, not a batch size.
WORKLOADS[6] = Workload(6, "uniform-1-512-pool", _LLAMA2_7B.replace(n_layers=24, d_model=2048, n_heads=16,
                                                                   n_kv_heads=16, ffn_dim=5504),
                        k=5000, capacity=0, lengths=_uniform(1, 512),
                        description="5000 prompts U[1,512] in draw order, batched k at a time, "
                                    "bin size = batch maximum")


def _lognormal_from_stats(lo: int, mean: float, hi: int, n: int):
    """Stand-in for a dataset known only by the min / mean / max of an n-prompt subsample:
    a lognormal whose mean is the stated mean and whose (1 - 1/n) quantile, where the largest
    of n draws sits, is the stated maximum; rounded and clipped to [min, max]."""
    z = NormalDist().inv_cdf(1.0 - 1.0 / n)
    c = float(np.log(hi / mean))            # = z sigma - sigma^2 / 2
    sigma = z - float(np.sqrt(z * z - 2.0 * c))
    mu = float(np.log(mean)) - sigma * sigma / 2.0

    def f(rng: np.random.Generator, k: int) -> np.ndarray:
        return np.clip(np.rint(rng.lognormal(mu, sigma, k)), lo, hi)
    return f


# Stand-ins for the paper's evaluation datasets (appendix table of dataset length statistics:
# 1000-prompt subsamples, min / mean / max prompt length).  The texts are not available, and
# only the lengths matter to the prefill cost.
DATASETS = {
    # name: (workload id, min, mean, max)
    "wiki256": (7, 1, 73, 256),
    "wiki512": (8, 6, 120, 512),
    "mmlu": (9, 4, 64, 1102),
    "hh-rlhf": (10, 22, 247, 1620),
    "alpaca": (11, 43, 126, 527),
    "samsum": (12, 21, 169, 942),
}
for _name, (_wid, _lo, _mean, _hi) in DATASETS.items():
    WORKLOADS[_wid] = Workload(_wid, f"{_name}-standin", WORKLOADS[6].shape, k=1000, capacity=0,
                               lengths=_lognormal_from_stats(_lo, _mean, _hi, 1000),
                               description=f"1000 prompts standing in for {_name} (min {_lo}, mean {_mean}, "
                                           f"max {_hi}): lognormal matched to the mean and to the max as the "
                                           f"0.999 quantile, clipped")

# Full-depth model shapes of the paper's appendix model table (bf16, random-init); Mistral 7B
# adds grouped-query attention (8 key/value heads) and a 14336-wide FFN.  Its sliding window
# (4096) is wider than every prompt of the sweeps, so plain causal attention is exact there.
MODELS: Dict[str, ModelShape] = {
    "llama-1.3b": _LLAMA2_7B.replace(n_layers=24, d_model=2048, n_heads=16, n_kv_heads=16, ffn_dim=5504),
    "llama2-7b": _LLAMA2_7B.replace(n_layers=32),
    "mistral-7b": _LLAMA2_7B.replace(n_layers=32, n_kv_heads=8, ffn_dim=14336),
}


def workload(wid: int) -> Workload:
    return WORKLOADS[wid]


# ----------------------------------------------------------------------------- bf16 storage
def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bfloat16 bit patterns (uint16), round to nearest even. Finite inputs only."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    out = np.empty(u.shape, dtype=np.uint16)
    flat_u, flat_o = u.reshape(-1), out.reshape(-1)
    step = 1 << 24
    for s in range(0, flat_u.size, step):
        c = flat_u[s:s + step]
        flat_o[s:s + step] = ((c + (np.uint32(0x7FFF) + ((c >> np.uint32(16)) & np.uint32(1))))
                              >> np.uint32(16)).astype(np.uint16)
    return out


def bf16_value(bits: np.ndarray) -> np.ndarray:
    """bfloat16 bit patterns (uint16) -> float32 values (exact)."""
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# ----------------------------------------------------------------------------- draws
def draw_lengths(wl: Workload, seed: int, k: Optional[int] = None) -> np.ndarray:
    rng = np.random.default_rng([wl.wid, seed, 0])
    return np.asarray(wl.lengths(rng, wl.k if k is None else k), dtype=np.int32)


def draw_tokens(wl: Workload, seed: int, total_len: int, vocab: Optional[int] = None) -> np.ndarray:
    rng = np.random.default_rng([wl.wid, seed, 1])
    return rng.integers(0, wl.shape.vocab if vocab is None else vocab, total_len).astype(np.int32)


def _normal(rng: np.random.Generator, shape, bf16: bool) -> np.ndarray:
    w = rng.standard_normal(shape, dtype=np.float32)
    w *= np.float32(0.02)
    if bf16:
        w = bf16_value(bf16_bits(w)).reshape(shape)
    return w


def draw_weights(wl: Workload, seed: int, shape: Optional[ModelShape] = None,
                 random_gains: bool = False) -> Dict[str, object]:
    """Model weights as float32 arrays (bf16-exact values for bf16 shapes).

    Layout follows the usual [out_features, in_features] convention:
    embed [V, d]; per layer wq [H*D, d], wk [Hkv*D, d], wv [Hkv*D, d], wo [d, H*D],
    wg [F, d], wu [F, d], wd [d, F]; attn_norm / mlp_norm / final_norm [d].
    Drawing order: embed, then per layer wq, wk, wv, wo, wg, wu, wd.
    """
    s = wl.shape if shape is None else shape
    bf = s.dtype == "bf16"
    rng = np.random.default_rng([wl.wid, seed, 2])
    d, H, Hkv, D, F = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim, s.ffn_dim
    out: Dict[str, object] = {"embed": _normal(rng, (s.vocab, d), bf)}
    layers: List[Dict[str, np.ndarray]] = []
    for _ in range(s.n_layers):
        L = {}
        L["wq"] = _normal(rng, (H * D, d), bf)
        L["wk"] = _normal(rng, (Hkv * D, d), bf)
        L["wv"] = _normal(rng, (Hkv * D, d), bf)
        L["wo"] = _normal(rng, (d, H * D), bf)
        L["wg"] = _normal(rng, (F, d), bf)
        L["wu"] = _normal(rng, (F, d), bf)
        L["wd"] = _normal(rng, (d, F), bf)
        layers.append(L)
    grng = np.random.default_rng([wl.wid, seed, 3])

    def gain():
        if not random_gains:
            return np.ones(d, dtype=np.float32)
        g = (1.0 + 0.1 * grng.standard_normal(d)).astype(np.float32)
        return bf16_value(bf16_bits(g)) if bf else g

    for L in layers:
        L["attn_norm"] = gain()
        L["mlp_norm"] = gain()
    out["layers"] = layers
    out["final_norm"] = gain()
    return out


def draw_lm_head(wl: Workload, seed: int, shape: Optional[ModelShape] = None) -> np.ndarray:
    """The LM head [vocab, d] (float32; bf16-exact values for bf16 shapes), own stream 4."""
    s = wl.shape if shape is None else shape
    rng = np.random.default_rng([wl.wid, seed, 4])
    return _normal(rng, (s.vocab, s.d_model), s.dtype == "bf16")


@dataclass
class Case:
    """One seeded batch: lengths, flat tokens (original prompt order) and weights."""
    wl: Workload
    shape: ModelShape
    seed: int
    capacity: int
    lengths: np.ndarray
    tokens: np.ndarray
    weights: Dict[str, object] = field(repr=False)

    @property
    def total_len(self) -> int:
        return int(self.lengths.sum())


def make_case(wid: int, seed: int = 0, *, n_layers: Optional[int] = None, k: Optional[int] = None,
              lengths: Optional[np.ndarray] = None, capacity: Optional[int] = None,
              random_gains: bool = False, with_weights: bool = True, **shape_overrides) -> Case:
    """A workload instance; the overrides shrink it for parity tests at the same layer shapes."""
    wl = WORKLOADS[wid]
    shape = wl.shape
    if n_layers is not None:
        shape = shape.replace(n_layers=n_layers)
    if shape_overrides:
        shape = shape.replace(**shape_overrides)
    if lengths is None:
        lengths = draw_lengths(wl, seed, k)
    lengths = np.asarray(lengths, dtype=np.int32)
    cap = wl.capacity if capacity is None else capacity
    tokens = draw_tokens(wl, seed, int(lengths.sum()), shape.vocab)
    weights = draw_weights(wl, seed, shape, random_gains) if with_weights else {}
    return Case(wl=wl, shape=shape, seed=seed, capacity=cap, lengths=lengths, tokens=tokens,
                weights=weights)
