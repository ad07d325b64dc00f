"""Parity for the batches the batch-size and regression sweeps time: prompts of the U[1,512]
pool in batches of 16 and 32, each packed with the bin size equal to the batch's maximum
length (the paper's choice, section 3.1) on the 1.3B and Mistral-7B (GQA 32/8) layer shapes.

* sampled prompts of a batch against the oracle, gated against the ideal-bf16 floor as the
  other bf16 parity tests are;
* packed and fully batched prefill of the same batch give bit-identical caches and hidden
  states on the real tokens (section 3.3), since the sweep's speedup compares exactly these.
"""
import numpy as np
import pytest

from oracle import decoder as D
from paper_2404_09529_amd import prepack as pp
from paper_2404_09529_amd import workloads as W

from .gpu_util import gate_vs_floor, gpu_prefill, oracle_weights, report, require_gpu

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    require_gpu()


def _errs(name, gpu, ref, n_layers, rows):
    h, k, v = gpu
    out = [report(f"{name} hidden", h[rows], ref.hidden[rows])]
    for l in range(n_layers):
        out.append(report(f"{name} K{l}", k[l][rows], ref.k[l][rows]))
        out.append(report(f"{name} V{l}", v[l][rows], ref.v[l][rows]))
    return out


def _case(model, bs, batch, n_layers):
    pool = W.draw_lengths(W.workload(6), 0)
    lengths = pool[batch * bs:(batch + 1) * bs]
    shape = W.MODELS[model]
    return W.make_case(6, 0, lengths=lengths, random_gains=True, n_layers=n_layers, d_model=shape.d_model,
                       n_heads=shape.n_heads, n_kv_heads=shape.n_kv_heads, ffn_dim=shape.ffn_dim)


@pytest.mark.parametrize("model,bs,batch,n_layers", [("llama-1.3b", 32, 0, 2), ("llama-1.3b", 16, 5, 2),
                                                      ("mistral-7b", 16, 1, 1)])
def test_sweep_batch_vs_oracle(model, bs, batch, n_layers):
    case = _case(model, bs, batch, n_layers)
    plan = pp.pp_pack(case.lengths, 0)
    print(f"[parity] sweep {model} bs{bs} batch {batch}: lengths {case.lengths.tolist()} -> {plan.n_rows} rows "
          f"x {plan.capacity}", flush=True)
    gpu = gpu_prefill(case, plan)
    order = np.argsort(case.lengths, kind="stable")
    picks = sorted({int(order[0]), int(order[len(order) // 2]), int(order[-1])})
    off = np.concatenate([[0], np.cumsum(case.lengths)])
    rows = np.concatenate([np.arange(off[i], off[i + 1]) for i in picks])
    shape = D.Shape.of(case.shape)
    w64 = oracle_weights(case.weights)
    ref = D.prefill_per_prompt(case.lengths, case.tokens, w64, shape, prompts=picks)
    flo = D.prefill_per_prompt(case.lengths, case.tokens, w64, shape, prompts=picks, rnd=D.round_bf16)
    name = f"sweep {model} bs{bs}"
    gate_vs_floor(name, _errs(name, gpu, ref, n_layers, rows),
                  _errs(name + " floor", (flo.hidden, flo.k, flo.v), ref, n_layers, rows))
    assert np.all(np.isfinite(gpu[0]))


@pytest.mark.parametrize("bs,batch", [(32, 3), (16, 11)])
def test_sweep_packed_equals_padded(bs, batch):
    case = _case("llama-1.3b", bs, batch, 1)
    a = gpu_prefill(case, pp.pp_pack(case.lengths, 0))
    b = gpu_prefill(case, pp.pp_pack_padded(case.lengths))
    assert np.array_equal(a[0], b[0])
    assert np.array_equal(a[1][0], b[1][0]) and np.array_equal(a[2][0], b[2][0])
