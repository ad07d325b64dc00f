"""pp_first_token_noalloc, the first token for callers that cannot allocate device memory,
through the C ABI against pp_first_token (which takes a caller workspace) on the same inputs.
Both run the same kernels, so tokens and logits must be bit-identical; checked on two calls
in a row, the second with a smaller input (the static buffer keeps the first call's
contents), and on the float32 model.  Device memory free before and after the calls must be
the same: the entry point allocates nothing."""
import numpy as np
import pytest
import torch

from paper_2404_09529_amd import prepack as pp

from .gpu_util import bf16_dev, f32_dev, rand_bf16, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _cfg(d, V, dtype):
    D = 128 if dtype == pp.PP_BF16 else 64
    return pp.PPConfig(n_layers=1, d_model=d, n_heads=d // D, n_kv_heads=d // D, head_dim=D, ffn_dim=4 * d,
                       vocab=V, dtype=dtype, rms_eps=1e-5, rope_theta=1e4)


def _inputs(lengths, d, V, dtype, seed):
    rng = np.random.default_rng(seed)
    hidden = rng.standard_normal((int(sum(lengths)), d)).astype(np.float32)
    if dtype == pp.PP_BF16:
        lm = bf16_dev(rand_bf16(rng, (V, d), 0.02))
    else:
        lm = f32_dev((rng.standard_normal((V, d)) * 0.02).astype(np.float32))
    cfg = _cfg(d, V, dtype)
    dplan = pp.DevicePlan(pp.pp_pack(lengths, 0))
    return cfg, dplan, f32_dev(hidden), lm


def _reference(cfg, dplan, h, lm):
    k, V = dplan.plan.k, cfg.vocab
    ws = torch.empty(pp.pp_first_token_workspace_size(cfg, dplan), dtype=torch.uint8, device="cuda")
    tok = torch.full((k,), -7, dtype=torch.int32, device="cuda")
    lg = torch.empty((k, V), dtype=torch.float32, device="cuda")
    pp.pp_first_token(cfg, dplan, h, lm, ws, tok, lg)
    return tok, lg


CALLS = [
    # prompt lengths, d, vocab, dtype: the second call is smaller than the first
    ([1 + (37 * i) % 500 for i in range(64)], 4096, 32000, pp.PP_BF16),
    ([3, 150, 1, 40, 77], 4096, 1000, pp.PP_BF16),
    ([4, 60, 33, 12, 9, 50, 17, 28], 256, 1000, pp.PP_F32),
]


def test_noalloc_matches_first_token_on_consecutive_calls():
    cases = [_inputs(l, d, V, dt, seed) for seed, (l, d, V, dt) in enumerate(CALLS)]
    refs = [_reference(*c) for c in cases]
    outs = []
    for cfg, dplan, _, _ in cases:
        k = dplan.plan.k
        outs.append((torch.full((k,), -7, dtype=torch.int32, device="cuda"),
                     torch.full((k, cfg.vocab), float("nan"), dtype=torch.float32, device="cuda"),
                     torch.full((k,), -7, dtype=torch.int32, device="cuda")))
    torch.cuda.synchronize()
    free0, _ = torch.cuda.mem_get_info()
    for (cfg, dplan, h, lm), (tok, lg, tok_only) in zip(cases, outs):
        print(f"[noalloc] k={dplan.plan.k} V={cfg.vocab} d={cfg.d_model} dtype={cfg.dtype}", flush=True)
        pp.pp_first_token_noalloc(cfg, dplan, h, lm, tok, lg)
        pp.pp_first_token_noalloc(cfg, dplan, h, lm, tok_only)          # logits not wanted
        torch.cuda.synchronize()
    free1, _ = torch.cuda.mem_get_info()
    assert free1 == free0, f"device memory free changed by {free0 - free1} bytes"
    for (tok_ref, lg_ref), (tok, lg, tok_only) in zip(refs, outs):
        assert torch.equal(tok, tok_ref)
        assert torch.equal(tok_only, tok_ref)
        assert torch.equal(lg, lg_ref)
        assert int(tok.min()) >= 0


def test_noalloc_rejects_a_workspace_beyond_its_buffer():
    # float32, 2 prompts, vocab 2,000,000: 32 MB of per-row partial results > 16 MiB
    cfg, dplan, h, lm = _inputs([3, 5], 256, 1000, pp.PP_F32, 9)
    big = _cfg(256, 2_000_000, pp.PP_F32)
    tok = torch.empty(2, dtype=torch.int32, device="cuda")
    with pytest.raises(pp.PrepackError) as e:
        pp.pp_first_token_noalloc(big, dplan, h, lm, tok)
    assert e.value.code == pp.PP_ERR_BUFFER_TOO_SMALL
