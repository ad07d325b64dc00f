"""Helpers for the GPU parity tests: device transfers, bf16 ulps, error summaries.

Expected values always come from ``oracle/`` run on the same seeded inputs; nothing
here computes a result of the method.
"""
import numpy as np
import torch

from oracle import decoder as D
from paper_2404_09529_amd import prepack as pp

DEV = "cuda"


def require_gpu():
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    pp.lib()  # raises LibraryMissing when the HIP library has not been built


def bf16_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV).to(torch.bfloat16)


def f32_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(DEV)


def i32_dev(a):
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.int32)).to(DEV)


def host64(t):
    torch.cuda.synchronize()
    return t.float().cpu().numpy().astype(np.float64)


def rand_bf16(rng, shape, scale=1.0):
    """Normal values already rounded to bf16 (float32 storage), so both sides see the same numbers."""
    return D.round_bf16(rng.standard_normal(shape).astype(np.float32) * np.float32(scale))


def oracle_weights(w):
    """The same weights as float64 arrays (exact: every value is a float32), so that the
    oracle's float64 products do not convert them again on every call; its results are
    unchanged."""
    if isinstance(w, dict):
        return {k: oracle_weights(v) for k, v in w.items()}
    if isinstance(w, (list, tuple)):
        return type(w)(oracle_weights(v) for v in w)
    if isinstance(w, np.ndarray) and w.dtype == np.float32:
        return w.astype(np.float64)
    return w


def bf16_ulp(x):
    """Spacing of bf16 numbers at |x| (8 significant bits)."""
    a = np.maximum(np.abs(np.asarray(x, dtype=np.float64)), np.finfo(np.float32).tiny)
    return np.exp2(np.floor(np.log2(a)) - 7)


def within_ulps(got, ref, n_ulps=1.0, atol=0.0):
    """|got - round_bf16(ref)| <= n_ulps * ulp(ref) + atol, elementwise; returns the worst ratio."""
    err = np.abs(got - D.round_bf16(ref))
    bound = n_ulps * bf16_ulp(ref) + atol
    return float(np.max(err / bound)) if err.size else 0.0


def report(name, got, ref):
    mx, mean = D.errors(got, ref)
    print(f"[parity] {name}: max |err| {mx:.3e}  mean |err| {mean:.3e}", flush=True)
    return mx, mean


def gpu_prefill(case, plan, stream=None):
    """Run pp_prefill through the C ABI; returns (hidden, [K_l], [V_l]) as float64 numpy."""
    model = pp.DeviceModel(case.shape, case.weights)
    dplan = pp.DevicePlan(plan)
    run = pp.Prefill(model, dplan)
    tokens = i32_dev(case.tokens)
    run(tokens, stream)
    torch.cuda.synchronize()
    h = host64(run.hidden)
    k = host64(run.k_cache)
    v = host64(run.v_cache)
    return h, [k[l] for l in range(case.shape.n_layers)], [v[l] for l in range(case.shape.n_layers)]


# bf16 end to end: the absolute bar (2e-2 max / 2e-3 mean |err|) is below what bf16 storage
# allows through several layers at these shapes, so every compared tensor (hidden states,
# each layer's K and V, logits) is gated against the error an ideal bf16 pipeline makes on
# the same inputs: the oracle with every stored value rounded to bf16 (rnd=round_bf16).
# Both the max and the mean |err| of the GPU may be at most this factor times the floor's.
FLOOR_FACTOR = 1.25


def gate_vs_floor(name, gpu_errs, floor_errs):
    """gpu_errs, floor_errs: matching lists of (max |err|, mean |err|) against the float64
    oracle, one entry per compared tensor."""
    assert len(gpu_errs) == len(floor_errs)
    worst = max(g[0] / max(f[0], 1e-300) for g, f in zip(gpu_errs, floor_errs)), \
        max(g[1] / max(f[1], 1e-300) for g, f in zip(gpu_errs, floor_errs))
    print(f"[parity] {name}: worst GPU / floor ratio max {worst[0]:.3f}, mean {worst[1]:.3f} "
          f"(gate {FLOOR_FACTOR})", flush=True)
    for i, ((gm, ga), (fm, fa)) in enumerate(zip(gpu_errs, floor_errs)):
        assert ga <= FLOOR_FACTOR * fa, f"{name} tensor {i}: mean {ga:.3e} > {FLOOR_FACTOR} x floor {fa:.3e}"
        assert gm <= FLOOR_FACTOR * fm, f"{name} tensor {i}: max {gm:.3e} > {FLOOR_FACTOR} x floor {fm:.3e}"


def check_bar(name, got, ref, bar_max=2e-2, bar_mean=2e-3, stored_bf16=True):
    """The absolute bar (max / mean |err|) wherever the output format allows it.

    For bf16-stored outputs the floor is the error of the correctly rounded exact result,
    round_bf16(ref) - ref.  Where that floor already exceeds the bar (outputs of large
    magnitude), the GPU must stay within 10% of the floor instead."""
    mx, mean = report(name, got, ref)
    if not stored_bf16:
        assert mx <= bar_max and mean <= bar_mean, name
        return mx, mean
    fmx, fmean = D.errors(D.round_bf16(ref), ref)
    lim_max = bar_max if fmx <= bar_max else 1.1 * fmx
    lim_mean = bar_mean if fmean <= bar_mean else 1.1 * fmean
    if (lim_max, lim_mean) != (bar_max, bar_mean):
        print(f"[parity] {name}: bf16 rounding floor {fmx:.3e} / {fmean:.3e} exceeds the bar; "
              f"gated at 1.1x the floor", flush=True)
    assert mx <= lim_max and mean <= lim_mean, (name, mx, mean, lim_max, lim_mean)
    return mx, mean
