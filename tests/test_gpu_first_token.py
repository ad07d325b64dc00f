"""First-token step on the GPU (section 2.3: time to first token = prefill + first token),
through its C-ABI entry point, against the oracle's ``first_token`` on the same inputs.

Bar, derived from the arithmetic: the GPU accumulates d products in float32, so each logit
may differ from the float64 value by at most d * 2^-24 * sum_j |h_j w_j| (the standard
bound for a float32 dot product; h is rounded to bf16 first in the bf16 model, on both
sides).  The argmax is an integer decided by those logits: where the oracle's best logit
leads the second by more than twice the bound the token must be the oracle's; otherwise it
must be a valid choice, a token whose exact logit is within twice the bound of the maximum.
"""
import numpy as np
import pytest
import torch

from oracle import decoder as D
from paper_2404_09529_amd import prepack as pp
from paper_2404_09529_amd import workloads as W

from .gpu_util import bf16_dev, f32_dev, rand_bf16, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _cfg(d, V, dtype=pp.PP_BF16):
    if dtype == pp.PP_BF16:
        return pp.PPConfig(n_layers=1, d_model=d, n_heads=d // 128, n_kv_heads=d // 128, head_dim=128,
                           ffn_dim=4 * d, vocab=V, dtype=dtype, rms_eps=1e-5, rope_theta=1e4)
    return pp.PPConfig(n_layers=1, d_model=d, n_heads=d // 64, n_kv_heads=d // 64, head_dim=64, ffn_dim=4 * d,
                       vocab=V, dtype=dtype, rms_eps=1e-5, rope_theta=1e4)


def _run(lengths, hidden, lm_head, dtype=pp.PP_BF16, want_logits=True):
    d = hidden.shape[1]
    V = lm_head.shape[0]
    cfg = _cfg(d, V, dtype)
    dplan = pp.DevicePlan(pp.pp_pack(lengths, 0))
    ws = torch.empty(pp.pp_first_token_workspace_size(cfg, dplan), dtype=torch.uint8, device="cuda")
    k = len(lengths)
    tokens = torch.full((k,), -7, dtype=torch.int32, device="cuda")
    logits = torch.empty((k, V), dtype=torch.float32, device="cuda") if want_logits else None
    w = bf16_dev(lm_head) if dtype == pp.PP_BF16 else f32_dev(lm_head)
    print(f"[first_token] k={k} V={V} d={d} dtype={dtype}", flush=True)
    pp.pp_first_token(cfg, dplan, f32_dev(hidden), w, ws, tokens, logits)
    torch.cuda.synchronize()
    return tokens.cpu().numpy(), (None if logits is None else logits.cpu().numpy().astype(np.float64))


def _check(lengths, hidden, lm_head, tokens, logits, bf16=True):
    rnd = D.round_bf16 if bf16 else (lambda x: x)
    ref, ref_tok = D.first_token(hidden, lengths, lm_head, rnd=rnd)
    h = rnd(np.asarray(hidden, dtype=np.float64)[D.last_token_rows(lengths)])
    bound = hidden.shape[1] * 2.0 ** -24 * (np.abs(h) @ np.abs(np.asarray(lm_head, dtype=np.float64)).T) + 1e-30
    if logits is not None:
        err = np.abs(logits - ref)
        assert np.all(err <= bound), f"logit error {err.max():.3g} > bound at {np.unravel_index(np.argmax(err - bound), err.shape)}"
    for i, t in enumerate(tokens):
        top = np.sort(ref[i])[::-1]
        slack = 2 * bound[i].max()
        if top[0] - top[1] > slack:
            assert t == ref_tok[i], f"prompt {i}: token {t}, oracle {ref_tok[i]}"
        else:
            assert 0 <= t < lm_head.shape[0] and ref[i, t] >= top[0] - slack, f"prompt {i}: token {t} not a maximum"


@pytest.mark.timeout(600)
@pytest.mark.parametrize("case", ["one-prompt", "one-prompt-d512", "ragged-vocab", "ragged-vocab-d512", "33-prompts-d1024",
                                  "two-prompt-chunks", "two-passes-of-128", "llama2-7b-vocab", "bimodal-96-prompts",
                                  "llama3-8b-vocab"])
def test_first_token_bf16(case):
    # up to 64 prompts are one pass of 64 (K in segments of 512 columns when d allows); more,
    # passes of 128 (the last one partial)
    if case in ("llama2-7b-vocab", "bimodal-96-prompts", "llama3-8b-vocab"):
        # full size: the prompts of the Llama-2-7B lognormal (64), bimodal (96) and Llama-3-8B (128)
        # workloads with their vocabularies, d 4096
        wl, V = {"llama2-7b-vocab": (2, 32000), "bimodal-96-prompts": (3, 32000), "llama3-8b-vocab": (4, 128256)}[case]
        lengths = W.draw_lengths(W.workload(wl), 0)
        d = 4096
    else:
        lengths = {"one-prompt": [37], "one-prompt-d512": [1], "ragged-vocab": [5, 1, 12, 3, 9],
                   "ragged-vocab-d512": [5, 1, 12, 3, 9],
                   "33-prompts-d1024": list(np.random.default_rng(5).integers(1, 50, 33)),
                   "two-prompt-chunks": list(np.random.default_rng(3).integers(1, 40, 70)),
                   "two-passes-of-128": list(np.random.default_rng(4).integers(1, 30, 150))}[case]
        V, d = {"one-prompt": (1000, 256), "one-prompt-d512": (129, 512), "ragged-vocab": (1000, 256),
                "ragged-vocab-d512": (1000, 512),
                "33-prompts-d1024": (777, 1024), "two-prompt-chunks": (3000, 512),
                "two-passes-of-128": (2000, 256)}[case]
    rng = np.random.default_rng([len(lengths), V, d])
    hidden = rng.standard_normal((int(np.sum(lengths)), d), dtype=np.float32)   # unit RMS, like a normed state
    lm_head = rand_bf16(rng, (V, d), 0.02)
    tokens, logits = _run(lengths, hidden, lm_head)
    _check(lengths, hidden, lm_head, tokens, logits)


def test_first_token_bf16_without_logits_matches_with():
    rng = np.random.default_rng(11)
    lengths = [4, 9, 2]
    hidden = rng.standard_normal((15, 256)).astype(np.float32)
    lm_head = rand_bf16(rng, (700, 256), 0.02)
    t1, _ = _run(lengths, hidden, lm_head, want_logits=False)
    t2, logits = _run(lengths, hidden, lm_head)
    assert np.array_equal(t1, t2)
    _check(lengths, hidden, lm_head, t1, logits)


@pytest.mark.parametrize("d", [256, 512])
def test_first_token_ties_go_to_the_lowest_id_and_nan_gives_minus_one(d):
    rng = np.random.default_rng(12)
    lengths = [3, 5, 2]                          # last rows 2, 7, 9
    V = 1000
    hidden = rng.standard_normal((10, d)).astype(np.float32)
    lm_head = rand_bf16(rng, (V, d), 0.02)
    hb = D.round_bf16(hidden[2].astype(np.float64))
    planted = D.round_bf16(0.05 * hb)            # logit ~ 0.05 |h|^2 ~ 13, far above the rest
    for v in (3, 900, 450):                      # equal maxima in three different workgroups
        lm_head[v] = planted
    hidden[9] = np.nan                           # every logit of prompt 2 is NaN
    tokens, _ = _run(lengths, hidden, lm_head)
    assert tokens[0] == 3
    assert tokens[2] == -1
    ref, ref_tok = D.first_token(hidden[:8], lengths[:2], lm_head, rnd=D.round_bf16)
    assert tokens[1] == ref_tok[1] or ref[1, tokens[1]] >= ref[1].max() - 1e-3


def test_first_token_f32():
    rng = np.random.default_rng(13)
    lengths = [6, 1, 11, 4]
    d, V = 64, 50
    hidden = rng.standard_normal((22, d)).astype(np.float32)
    lm_head = (0.02 * rng.standard_normal((V, d))).astype(np.float32)
    tokens, logits = _run(lengths, hidden, lm_head, dtype=pp.PP_F32)
    _check(lengths, hidden, lm_head, tokens, logits, bf16=False)
