#!/usr/bin/env python3
"""Packed-prefill benchmark on one MI355X.

A step is one pp_prefill call: the whole device path (TENSORIZE, every decoder layer under
the independent mask with restart positions, KV and hidden-state UNPACK) over one batch of
synthetic prompts, with weights, tokens and the device plan already resident in HBM.
pp_pack (host) and the plan upload are timed separately and never part of `value`.

Prints one JSON line:
  value            effective (non-pad) prefill tokens/s of the packed path
  tflops_effective algorithmic FLOP / time (pads and skipped work excluded)
  padded           the same kernels on the full-batching plan (the paper's baseline)
  roofline         the dominant kernel (the gate/up projection GEMM with SwiGLU epilogue),
                   timed live with HIP events on its stream, against the bf16 MFMA peak;
                   `traffic` is its HBM bytes per launch from the committed counter summary,
                   reported only while the kernel source still matches the one measured
  cpu_baseline     the CPU oracle timed on a bounded sample of the same workload

--traffic-pass runs only that kernel and a plain copy of known size, for the hardware
counter passes (rocprofv3 --pmc FETCH_SIZE, then WRITE_SIZE) that calibrate and measure it.
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_BF16_TFLOPS = 2500.0   # MI355X dense bf16 MFMA
PEAK_HBM_GBPS = 8000.0      # MI355X HBM3E
METRIC = "effective prefill tokens/s + TFLOP/s (% bf16 MFMA peak) vs padded prefill"
GEMM_SOURCE = os.path.join(ROOT, "paper_2404_09529_amd", "csrc", "k_gemm_bf16.hip")
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "gemm_swiglu_llama2-7b-lognormal_traffic.md")
COPY_BYTES = 1 << 30        # the calibration copy reads and writes 1 GiB


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def algorithmic_flops(shape, lengths):
    """Linear layers of every real token plus causal attention pairs; norms, RoPE, softmax = 0."""
    import numpy as np
    s = shape
    L = int(np.sum(lengths))
    lin = 2 * (s.d_model * (s.n_heads + 2 * s.n_kv_heads) * s.head_dim + s.n_heads * s.head_dim * s.d_model
               + 3 * s.d_model * s.ffn_dim)
    pairs = int(np.sum(np.asarray(lengths, dtype=np.int64) * (np.asarray(lengths, dtype=np.int64) + 1) // 2))
    return s.n_layers * (L * lin + 4 * s.n_heads * s.head_dim * pairs)


def time_steps(fn, steps, warmup):
    import torch
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    t0 = time.perf_counter()
    for a, b in ev:
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = sorted(a.elapsed_time(b) for a, b in ev)
    return {"ms_mean": sum(ms) / len(ms), "ms_median": ms[len(ms) // 2], "ms_p10": ms[len(ms) // 10],
            "ms_p90": ms[min(len(ms) - 1, (9 * len(ms)) // 10)], "wall_s": wall}


def source_sha256(path):
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def recorded_traffic():
    """HBM bytes per launch of the gate/up GEMM from the committed counter summary (a line
    `record: {json}`), or None when there is none or the kernel source has changed since."""
    try:
        with open(TRAFFIC_SUMMARY) as f:
            line = next(l for l in f if l.startswith("record: "))
        rec = json.loads(line[len("record: "):])
    except (OSError, StopIteration, ValueError):
        return None
    if rec.get("kernel_source_sha256") != source_sha256(GEMM_SOURCE):
        return None
    return rec


def calibration_copy():
    """A float32 copy of COPY_BYTES through a plain elementwise kernel (dst = src * 1.0), run
    three times: hardware byte counters read on it calibrate the same counters elsewhere."""
    import torch
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.mul(src, 1.0, out=dst)
    torch.cuda.synchronize()
    del src, dst


def traffic_pass(args):
    """The gate/up GEMM alone on the workload's packed plan (random bf16 operands: traffic does
    not depend on the values), then a float32 copy of COPY_BYTES through a plain elementwise
    kernel, whose counter readings calibrate the GEMM's."""
    import torch

    from paper_2404_09529_amd import prepack as pp
    from paper_2404_09529_amd import workloads as W

    wl = W.workload(args.workload)
    lengths = W.draw_lengths(wl, args.seed)
    plan = pp.pp_pack(lengths, wl.capacity)
    dplan = pp.DevicePlan(plan)
    shape = wl.shape
    T, d, F = plan.n_slots, shape.d_model, shape.ffn_dim
    gen = torch.Generator(device="cuda").manual_seed(1)
    A = torch.randn((T, d), generator=gen, device="cuda").to(torch.bfloat16)
    Wgu = (torch.randn((2 * F, d), generator=gen, device="cuda") * 0.02).to(torch.bfloat16)
    C = torch.empty((T, F), dtype=torch.bfloat16, device="cuda")
    for _ in range(args.kernel_launches):
        pp.pp_gemm(pp.PP_BF16, pp.PP_EPI_SWIGLU, A, d, Wgu, d, C, F, T, 2 * F, d, dplan)
    torch.cuda.synchronize()
    del A, Wgu, C
    calibration_copy()
    print(json.dumps({"traffic_pass": wl.name, "gemm_launches": args.kernel_launches, "T": T, "d": d, "F": F,
                      "total_len": int(lengths.sum()), "copy_read_bytes": COPY_BYTES,
                      "copy_write_bytes": COPY_BYTES, "kernel_source_sha256": source_sha256(GEMM_SOURCE)}),
          flush=True)


def cpu_baseline(case, budget_s):
    """The oracle (float64, per prompt, as it stands) on prompts of the workload taken in
    original order, skipping prompts longer than 512 tokens, until budget_s has elapsed."""
    import numpy as np
    from oracle import decoder as D
    try:
        from threadpoolctl import threadpool_info
        cores = max((i.get("num_threads", 1) for i in threadpool_info()), default=1)
    except Exception:
        cores = 1
    shape = D.Shape.of(case.shape)
    off = np.concatenate([[0], np.cumsum(case.lengths)])
    done, t0, used = 0, time.perf_counter(), []
    for i, l in enumerate(case.lengths):
        if l > 512:
            continue
        D.prefill_prompt(case.tokens[off[i]:off[i + 1]], case.weights, shape)
        done += int(l)
        used.append(i)
        if time.perf_counter() - t0 >= budget_s:
            break
    el = time.perf_counter() - t0
    return {"value": done / el, "unit": "tokens/s", "cores": int(cores), "kind": "oracle",
            "sample": f"{len(used)} prompts ({done} tokens) of the same batch in original order, prompts "
                      f"longer than 512 tokens skipped; float64 numpy oracle, all {shape.n_layers} layers; "
                      f"{el:.1f} s"}


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=2, help="workload id (2 = Llama-2-7B shape, lognormal)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-padded", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--cpu-budget-s", type=float, default=20.0)
    ap.add_argument("--kernel-launches", type=int, default=20)
    ap.add_argument("--traffic-pass", action="store_true",
                    help="run only the dominant kernel and the calibration copy (for counter passes)")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="end with the calibration copy (for byte-counter passes over the whole step)")
    args = ap.parse_args()
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU: the packed prefill is a single-GPU path (rows are independent, "
              "so it would shard by rows with no collective); run with --gpus 1", file=sys.stderr)
        sys.exit(2)

    import numpy as np
    import torch

    from paper_2404_09529_amd import prepack as pp
    from paper_2404_09529_amd import workloads as W

    assert torch.cuda.is_available(), "bench.py needs a GPU"
    pp.lib()
    torch.cuda.set_device(0)
    if args.traffic_pass:
        traffic_pass(args)
        return

    t = time.perf_counter()
    case = W.make_case(args.workload, args.seed)
    shape, lengths = case.shape, case.lengths
    log(f"workload {case.wl.name}: k={len(lengths)} L={case.total_len} m={lengths.max()} "
        f"(weights drawn in {time.perf_counter() - t:.1f} s)")

    # host planning, timed on its own
    n_pack = 50
    t = time.perf_counter()
    for _ in range(n_pack):
        plan = pp.pp_pack(lengths, case.capacity)
    pack_ms = (time.perf_counter() - t) * 1e3 / n_pack
    dplan = pp.DevicePlan(plan)          # first device allocations: allocator start-up, untimed
    torch.cuda.synchronize()
    n_up = 10
    t = time.perf_counter()
    for _ in range(n_up):
        dplan = pp.DevicePlan(plan)
    torch.cuda.synchronize()
    upload_ms = (time.perf_counter() - t) * 1e3 / n_up
    model = pp.DeviceModel(shape, case.weights)
    tokens = torch.from_numpy(case.tokens).cuda()
    step = pp.Prefill(model, dplan)
    log(f"packed plan: {plan.n_rows} rows x {plan.capacity}, fill {case.total_len / plan.n_slots:.3f}, "
        f"pack {pack_ms:.3f} ms, upload {upload_ms:.2f} ms")

    flops = algorithmic_flops(shape, lengths)
    packed = time_steps(lambda: step(tokens), args.steps, args.warmup)
    ms = packed["ms_mean"]
    value = case.total_len / (ms / 1e3)
    tflops = flops / (ms / 1e3) / 1e12
    log(f"packed: {ms:.3f} ms/step, {value:,.0f} tokens/s, {tflops:.1f} TFLOP/s effective")

    # dominant kernel: the gate/up GEMM with the SwiGLU epilogue, same launch as inside pp_prefill
    T, d, F = plan.n_slots, shape.d_model, shape.ffn_dim
    gen = torch.Generator(device="cuda").manual_seed(1)
    A = torch.randn((T, d), generator=gen, device="cuda").to(torch.bfloat16)
    Cb = torch.empty((T, F), dtype=torch.bfloat16, device="cuda")
    Wgu = model.layers[0]["w_gateup"]
    kstream = torch.cuda.current_stream()
    gemm = lambda: pp.pp_gemm(pp.PP_BF16, pp.PP_EPI_SWIGLU, A, d, Wgu, d, Cb, F, T, 2 * F, d, dplan, kstream)
    kt = time_steps(gemm, args.kernel_launches, 3)
    k_flops = 2.0 * case.total_len * (2 * F) * d
    achieved = k_flops / (kt["ms_mean"] / 1e3) / 1e12
    del A, Cb
    log(f"gate/up GEMM: {kt['ms_mean']:.3f} ms/launch, {achieved:.1f} TFLOP/s algorithmic")
    traffic = recorded_traffic()
    k_bytes = 2 * (case.total_len * d + 2 * F * d + case.total_len * F)   # A, W once; C written once

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": shape.dtype, "data": "synthetic",
        "config": {"workload": case.wl.name, "description": case.wl.description, "seed": args.seed,
                   "k": int(len(lengths)), "capacity": int(case.capacity), "total_len": case.total_len,
                   "max_len": int(lengths.max()), "n_rows": plan.n_rows, "fill": round(case.total_len / plan.n_slots, 4)},
        "tflops_effective": round(tflops, 2), "frac_bf16_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
        "algorithmic_flop": flops,
        "ms_median": round(packed["ms_median"], 4), "ms_p10": round(packed["ms_p10"], 4),
        "ms_p90": round(packed["ms_p90"], 4),
        "pack_ms": round(pack_ms, 4), "plan_upload_ms": round(upload_ms, 3),
        "roofline": {"kernel": "gemm_bf16_kernel<kSwiGLU> (gate/up projection)", "bound": "mfma",
                     "achieved": round(achieved, 1), "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                     "frac": round(achieved / PEAK_BF16_TFLOPS, 4),
                     "traffic": None if traffic is None else traffic["hbm_bytes_per_launch"],
                     "ms_per_launch": round(kt["ms_mean"], 4),
                     "algorithmic_flop_per_launch": k_flops, "algorithmic_bytes_per_launch": k_bytes,
                     "traffic_source": None if traffic is None else os.path.relpath(TRAFFIC_SUMMARY, ROOT)},
    }

    # time to first token (section 2.3): the prefill step plus the greedy first token of every
    # prompt (LM head on its last token, argmax); the LM head streams 2 V d bytes from HBM
    V = shape.vocab
    lm_head = torch.from_numpy(W.draw_lm_head(case.wl, args.seed, shape)).cuda().to(model.torch_dtype)
    cfg = pp.config_of(shape)
    ft_ws = torch.empty(pp.pp_first_token_workspace_size(cfg, dplan), dtype=torch.uint8, device="cuda")
    first = torch.empty(len(lengths), dtype=torch.int32, device="cuda")
    ftok = lambda: pp.pp_first_token(cfg, dplan, step.hidden, lm_head, ft_ws, first, None, kstream)
    ft = time_steps(ftok, args.kernel_launches, 3)
    both = time_steps(lambda: (step(tokens, kstream), ftok()), args.steps, args.warmup)
    lm_bytes = lm_head.numel() * lm_head.element_size()
    out["ttft"] = {"ms_median": round(both["ms_median"], 4), "ms_mean": round(both["ms_mean"], 4),
                   "first_token_ms": round(ft["ms_mean"], 4), "prefill_ms_median": round(packed["ms_median"], 4),
                   "first_token_roofline": {"bound": "hbm", "achieved": round(lm_bytes / (ft["ms_mean"] / 1e3) / 1e9, 1),
                                            "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                                            "frac": round(lm_bytes / (ft["ms_mean"] / 1e3) / 1e9 / PEAK_HBM_GBPS, 4),
                                            "algorithmic_bytes_per_launch": lm_bytes, "vocab": V}}
    log(f"first token: {ft['ms_mean'] * 1e3:.1f} us ({lm_bytes / (ft['ms_mean'] / 1e3) / 1e9:.0f} GB/s on the LM head); "
        f"TTFT {both['ms_median']:.3f} ms")
    del step, lm_head, ft_ws
    torch.cuda.empty_cache()

    if not args.no_padded:
        pplan = pp.pp_pack_padded(lengths)
        pstep = pp.Prefill(model, pp.DevicePlan(pplan))
        padded = time_steps(lambda: pstep(tokens), max(3, args.steps // 4), 1)
        pms = padded["ms_mean"]
        out["padded"] = {"ms_per_step": round(pms, 4), "tokens_per_s": round(case.total_len / (pms / 1e3), 1),
                         "tflops_effective": round(flops / (pms / 1e3) / 1e12, 2), "n_rows": pplan.n_rows,
                         "capacity": pplan.capacity}
        out["speedup_vs_padded"] = round(pms / ms, 3)
        log(f"padded: {pms:.3f} ms/step, speedup {pms / ms:.2f}x")
        del pstep
        torch.cuda.empty_cache()

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(case, args.cpu_budget_s)
        log(f"cpu oracle: {out['cpu_baseline']['value']:.1f} tokens/s on {out['cpu_baseline']['cores']} threads")

    if args.calibration_copy:
        calibration_copy()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
