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
  attention_pairs  causal (query, key) pairs per head and layer: algorithmic, and executed
                   by the attention kernel (tile inflation); the padded plan's executed count
                   sits under `padded`
  roofline         the dominant kernel (the gate/up projection GEMM with SwiGLU epilogue),
                   timed live with HIP events on its stream, against the bf16 MFMA peak;
                   `traffic` is its HBM bytes per launch from the committed counter summary,
                   reported only for the workload and seed it was measured on and while the
                   kernel source still matches the one measured (null otherwise)
  cpu_baseline     the CPU oracle (float32) timed on a stratified sample of the same batch that
                   includes its longest prompt, extrapolated to the whole batch by FLOP
  device_memory    workspace, outputs and peak device memory of packed and padded prefill
  pack_ms          the pp_pack C call (plan arrays allocated once)

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
PEAK_FP32_TFLOPS = 78.6     # fp32 FMA on the vector ALUs: 256 CUs x 4 SIMDs x 16 lanes x 2 FLOP x
                            # 2.4 GHz.  The published 157.3 counts packed FMAs (two per lane per
                            # clock), which this library is built without.
PEAK_HBM_GBPS = 8000.0      # MI355X HBM3E
METRIC = "effective prefill tokens/s + TFLOP/s (% bf16 MFMA peak) vs padded prefill"
GEMM_SOURCE = os.path.join(ROOT, "paper_2404_09529_amd", "csrc", "k_gemm_bf16.hip")
TRAFFIC_SUMMARY = os.path.join(ROOT, "profiles", "gemm_swiglu_llama2-7b-lognormal_traffic.md")
COPY_BYTES = 1 << 30        # the calibration copy reads and writes 1 GiB
CPU_SAMPLE_S = 12.0         # about this much timed oracle work for cpu_baseline (more layers while it fits)


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


def attention_pairs(plan, lengths, tiled=True, key_tile=64):
    """Causal (query, key) pairs per head and layer: what the method needs, sum of l(l+1)/2,
    and what the attention kernel computes.  The bf16 kernel (tiled) takes every query of a
    work item's query tile against key tiles of 64 up to the tile's last query (section 3.2:
    M' never leaves the prompt's diagonal block); the float32 kernel takes each real query's
    own keys only."""
    import numpy as np

    from paper_2404_09529_amd import prepack as pp
    L = np.asarray(lengths, dtype=np.int64)
    alg = int((L * (L + 1) // 2).sum())
    n = np.asarray(plan.seg_len, dtype=np.int64)[np.asarray(plan.qtile_seg, dtype=np.int64)]
    q0 = np.asarray(plan.qtile_q0, dtype=np.int64)
    qt = pp.PP_QTILE
    n_kv = np.minimum(q0 + qt, n)
    exe = int((qt * key_tile * ((n_kv + key_tile - 1) // key_tile)).sum()) if tiled else alg
    return {"algorithmic": alg, "executed": exe, "inflation": round(exe / max(alg, 1), 3)}


def prefill_memory(step, base_alloc):
    """Device memory of one pp_prefill setup (workspace, hidden states, K/V caches) and the
    peak allocated above what was resident before it (weights, tokens, plan), after one call."""
    import torch
    nb = lambda t: t.numel() * t.element_size()
    return {"workspace_bytes": nb(step.workspace), "outputs_bytes": nb(step.hidden) + nb(step.k_cache) + nb(step.v_cache),
            "extra_peak_bytes": int(torch.cuda.max_memory_allocated() - base_alloc),
            "peak_alloc_bytes": int(torch.cuda.max_memory_allocated())}


def model_bytes(model):
    import torch
    return int(sum(t.numel() * t.element_size() for t in vars(model).values() if isinstance(t, torch.Tensor)) +
               sum(t.numel() * t.element_size() for layer in model.layers for t in layer.values()
                   if isinstance(t, torch.Tensor)))


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


def time_cold(fn, steps, warmup, flush_bytes=1 << 30):
    """Like time_steps, but before every timed call a read of `flush_bytes` (more than the
    256 MB last-level cache) evicts what the previous call left there; the read is outside the
    timed region.  This is the state a call finds after a prefill, which streams gigabytes."""
    import torch
    buf = torch.zeros(flush_bytes // 4, dtype=torch.float32, device="cuda")
    for _ in range(warmup):
        fn()
    torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(steps)]
    for a, b in ev:
        buf.amax()
        a.record()
        fn()
        b.record()
    torch.cuda.synchronize()
    del buf
    ms = sorted(a.elapsed_time(b) for a, b in ev)
    return {"ms_mean": sum(ms) / len(ms), "ms_median": ms[len(ms) // 2], "ms_p10": ms[len(ms) // 10],
            "ms_p90": ms[min(len(ms) - 1, (9 * len(ms)) // 10)]}


def source_sha256(path):
    import hashlib
    with open(path, "rb") as f:
        return hashlib.sha256(f.read()).hexdigest()


def recorded_traffic(workload, seed):
    """HBM bytes per launch of the gate/up GEMM from the committed counter summary (a line
    `record: {json}`), or None when there is none, when it was taken on another workload or
    seed (the re-fetches depend on the plan's shape), or when the kernel source has changed
    since."""
    try:
        with open(TRAFFIC_SUMMARY) as f:
            line = next(l for l in f if l.startswith("record: "))
        rec = json.loads(line[len("record: "):])
    except (OSError, StopIteration, ValueError):
        return None
    if rec.get("workload") != workload or rec.get("seed") != seed:
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
    print(json.dumps({"traffic_pass": wl.name, "seed": args.seed, "gemm_launches": args.kernel_launches,
                      "T": T, "d": d, "F": F, "total_len": int(lengths.sum()), "copy_read_bytes": COPY_BYTES,
                      "copy_write_bytes": COPY_BYTES, "kernel_source_sha256": source_sha256(GEMM_SOURCE)}),
          flush=True)


def cpu_model():
    try:
        with open("/proc/cpuinfo") as f:
            for line in f:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def prompt_flops(shape, l):
    """Algorithmic FLOP of one prompt of l tokens through one decoder layer (as
    algorithmic_flops, per layer)."""
    s = shape
    lin = 2 * (s.d_model * (s.n_heads + 2 * s.n_kv_heads) * s.head_dim + s.n_heads * s.head_dim * s.d_model
               + 3 * s.d_model * s.ffn_dim)
    return l * lin + 4 * s.n_heads * s.head_dim * (l * (l + 1) // 2)


def cpu_baseline(case):
    """The oracle as it stands (per prompt, numpy), in float32, on the host's cores, over a
    stratified sample of the batch, extrapolated to the whole batch by algorithmic FLOP.

    The prompts are split by length into four quartiles; from each the prompt of median
    length is timed, and from the top quartile also the batch's longest prompt.  Each is
    timed through one decoder layer, then, while the timing stays near CPU_SAMPLE_S in all,
    through as many of the model's other layers as fit (the oracle's per-layer work is the
    same in every layer, so a quartile's per-layer time is the mean over the layers run, and
    n layers take n times that); a quartile's time is then scaled by its FLOP over its
    sampled prompts'.  The embedding and final norm are left out (no FLOP)."""
    import dataclasses

    import numpy as np
    from threadpoolctl import threadpool_limits

    from oracle import decoder as D
    affinity = len(os.sched_getaffinity(0))
    threads = int(os.environ.get("OMP_NUM_THREADS", affinity) or affinity)
    threads = max(1, min(threads, affinity))
    shape = D.Shape.of(case.shape)
    one = dataclasses.replace(shape, n_layers=1)
    lengths = np.asarray(case.lengths, dtype=np.int64)
    off = np.concatenate([[0], np.cumsum(lengths)])
    order = np.argsort(lengths, kind="stable")
    strata = [q for q in np.array_split(order, 4) if len(q)]
    longest = int(order[-1])
    picks = []
    for qi, q in enumerate(strata):
        picks.append([int(q[len(q) // 2])])
        if qi == len(strata) - 1 and longest not in picks[-1]:
            picks[-1].append(longest)

    def run(layers):                  # seconds per quartile for its picks through `layers`
        el = []
        for p in picks:
            t = time.perf_counter()
            for i in p:
                D.prefill_prompt(case.tokens[off[i]:off[i + 1]], case.weights, layers, dtype=np.float32)
            el.append(time.perf_counter() - t)
        return el

    t_all = time.perf_counter()
    with threadpool_limits(limits=threads):
        D.prefill_prompt(case.tokens[off[0]:off[0] + min(16, int(lengths[0]))], case.weights, one,
                         dtype=np.float32)                      # warm-up
        el = run(one)
        first = time.perf_counter() - t_all
        extra = int(min(shape.n_layers - 1, max(0.0, CPU_SAMPLE_S / max(first, 1e-9) - 1.0)))
        if extra:
            el = [a + b for a, b in zip(el, run(dataclasses.replace(shape, n_layers=extra)))]
    wall = time.perf_counter() - t_all
    total_s, timed = 0.0, []
    for q, p, e in zip(strata, picks, el):
        f_sample = sum(prompt_flops(shape, int(lengths[i])) for i in p)
        f_stratum = sum(prompt_flops(shape, int(lengths[i])) for i in q)
        total_s += e / (1 + extra) * f_stratum / f_sample * shape.n_layers
        timed += [(int(i), int(lengths[i])) for i in p]
    L = int(lengths.sum())
    return {"value": L / total_s, "unit": "tokens/s", "cores": threads, "kind": "oracle",
            "cpu_model": cpu_model(), "affinity_cpus": affinity, "dtype": "f32",
            "extrapolated_batch_s": round(total_s, 2),
            "sample": f"stratified: the median-length prompt of each length quartile plus the longest prompt, "
                      f"{len(timed)} prompts (ids, lengths) {timed}, each through {1 + extra} of the {shape.n_layers} "
                      f"layers; whole batch ({len(lengths)} prompts, {L} tokens, {shape.n_layers} layers) "
                      f"extrapolated by algorithmic FLOP per quartile; float32 numpy oracle on {threads} "
                      f"threads; {wall:.1f} s timed"}


def gemm_rows_executed(plan):
    """Rows of the packed batch the projection GEMMs compute: the plan's row tiles (every
    PP_MTILE-slot tile holding a slot of some span; tiles of row-tail padding alone are
    skipped)."""
    from paper_2404_09529_amd import prepack as pp
    T = plan.n_slots
    return int(sum(min(pp.PP_MTILE, T - int(m0)) for m0 in plan.mtile_m0))


# ----------------------------------------------------------------------------- sweeps
def batch_predictors(lengths, n_rows):
    """The two batch statistics the paper regresses the speedup on (section 4.7): the batch-size
    reduction r/k (packed rows over prompts) and the max absolute deviation m - L/k (the longest
    prompt minus the mean length)."""
    import numpy as np
    lengths = np.asarray(lengths, dtype=np.int64)
    k = len(lengths)
    return {"r_over_k": n_rows / k, "max_abs_dev": float(lengths.max() - lengths.sum() / k)}


def linear_fit(x, y):
    """Ordinary least squares y ~ a + b x: slope b, intercept a, Pearson correlation and R^2;
    None when x or y does not vary (a batch size of 1 has r/k = 1 for every batch)."""
    import numpy as np
    x, y = np.asarray(x, dtype=np.float64), np.asarray(y, dtype=np.float64)
    xm, ym = x.mean(), y.mean()
    sxx, syy, sxy = np.sum((x - xm) ** 2), np.sum((y - ym) ** 2), np.sum((x - xm) * (y - ym))
    if sxx == 0 or syy == 0:
        return None
    b = sxy / sxx
    r = sxy / np.sqrt(sxx * syy)
    return {"slope": float(b), "intercept": float(ym - b * xm), "pearson_r": float(r), "r2": float(r * r),
            "n": int(len(x))}


def device_weights(shape, seed):
    """Random-init weights drawn on the device with torch (N(0, 0.02^2), bf16; unit norm gains)
    for timing-only sweeps at full model depth, where drawing them on the host would take
    minutes.  Nothing compares these values with anything."""
    import torch
    g = torch.Generator(device="cuda").manual_seed(seed)
    s, dt = shape, torch.bfloat16

    def n(*sz):
        return (torch.randn(sz, generator=g, device="cuda") * 0.02).to(dt)

    ones = lambda: torch.ones(s.d_model, dtype=torch.float32, device="cuda")
    d, H, Hkv, D, F = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim, s.ffn_dim
    layers = [dict(wq=n(H * D, d), wk=n(Hkv * D, d), wv=n(Hkv * D, d), wo=n(d, H * D), wg=n(F, d), wu=n(F, d),
                   wd=n(d, F), attn_norm=ones(), mlp_norm=ones()) for _ in range(s.n_layers)]
    return {"embed": n(s.vocab, d), "final_norm": ones(), "layers": layers}


def time_plan(pp, model, plan, tokens, reps, warmup, lm_head=None):
    """Median of `reps` timed pp_prefill steps of one plan after `warmup` untimed ones; with an
    LM head also the time to first token, prefill and pp_first_token timed together."""
    import torch
    dplan = pp.DevicePlan(plan)
    step = pp.Prefill(model, dplan)
    out = {"ms": time_steps(lambda: step(tokens), reps, warmup)["ms_median"]}
    if lm_head is not None:
        cfg = model.config
        ws = torch.empty(max(pp.pp_first_token_workspace_size(cfg, dplan), 1), dtype=torch.uint8, device="cuda")
        first = torch.empty(max(plan.k, 1), dtype=torch.int32, device="cuda")
        out["ttft_ms"] = time_steps(lambda: (step(tokens), pp.pp_first_token(cfg, dplan, step.hidden, lm_head, ws,
                                                                             first)), reps, warmup)["ms_median"]
    return out


def measure_batch(pp, model, lengths, args, gen, lm_head=None):
    """One batch prefilled packed (FFD, bin size = the batch's maximum length) and fully
    batched (every prompt right-padded to that maximum): same kernels, same stream."""
    import torch
    shape = model.shape
    L = int(lengths.sum())
    tokens = torch.randint(0, shape.vocab, (L,), generator=gen, device="cuda", dtype=torch.int32)
    plan, pplan = pp.pp_pack(lengths, 0), pp.pp_pack_padded(lengths)
    rec = {"k": int(len(lengths)), "L": L, "m": int(lengths.max()), "r": plan.n_rows,
           **batch_predictors(lengths, plan.n_rows)}
    for name, pl in (("packed", plan), ("padded", pplan)):
        t = time_plan(pp, model, pl, tokens, args.reps, args.sweep_warmup, lm_head)
        rec[f"ms_{name}"] = t["ms"]
        if "ttft_ms" in t:
            rec[f"ttft_ms_{name}"] = t["ttft_ms"]
        rec[f"slots_{name}"] = pl.n_slots
    rec["speedup"] = rec["ms_padded"] / rec["ms_packed"]
    if lm_head is not None:
        rec["ttft_speedup"] = rec["ttft_ms_padded"] / rec["ttft_ms_packed"]
    rec["tflops_packed"] = algorithmic_flops(shape, lengths) / (rec["ms_packed"] / 1e3) / 1e12
    return rec


def sweep_pool(W, name, seed, n):
    """Prompt lengths of a sweep: the U[1,512] pool or a dataset stand-in, in draw order."""
    wid = 6 if name == "uniform" else W.DATASETS[name][0]
    return W.draw_lengths(W.workload(wid), seed)[:n]


def dataset_batches(pp, lengths, bs):
    """The four ways of batching a whole prompt set that the paper compares (section 4.6), as
    lists of (prompt ids, plan):
      full       batches of bs prompts in arrival (draw) order, right-padded to the batch maximum;
      batch      the same batches, each packed on its own (FFD, bin size = the batch maximum);
      ordered    prompts sorted by length, consecutive batches of bs, right-padded (length-ordered
                 batching: needs the whole set in advance);
      dataset    the whole set packed at once (FFD, bin size = the set's maximum), its rows taken
                 bs at a time (dataset prepacking: also needs the whole set).
    For `dataset`, FFD run again on the prompts of a group of rows of the whole-set packing (in
    their original order, same bin size) rebuilds exactly those rows, because every prompt still
    finds the same first row with room; the row count is checked."""
    import numpy as np
    lengths = np.asarray(lengths, dtype=np.int32)
    n = len(lengths)
    out = {"full": [], "batch": [], "ordered": [], "dataset": []}
    for b in range(0, n, bs):
        ids = np.arange(b, min(b + bs, n))
        out["full"].append((ids, pp.pp_pack_padded(lengths[ids])))
        out["batch"].append((ids, pp.pp_pack(lengths[ids], 0)))
    order = np.argsort(lengths, kind="stable")
    for b in range(0, n, bs):
        ids = order[b:b + bs]
        out["ordered"].append((ids, pp.pp_pack_padded(lengths[ids])))
    whole = pp.pp_pack(lengths, 0)
    C = whole.capacity
    for r0 in range(0, whole.n_rows, bs):
        r1 = min(r0 + bs, whole.n_rows)
        ids = np.sort(whole.seg_prompt[whole.row_seg_ptr[r0]:whole.row_seg_ptr[r1]])
        plan = pp.pp_pack(lengths[ids], C)
        if plan.n_rows != r1 - r0:
            raise RuntimeError(f"rows {r0}..{r1} of the whole-set packing rebuilt as {plan.n_rows} rows")
        out["dataset"].append((ids, plan))
    return out


def run_dataset_packing(pp, W, model, args, gen, out):
    """Per-prompt prefill time of the four batchings of each prompt set (section 4.6)."""
    import numpy as np
    import torch
    shape = model.shape
    for name in args.pools.split(","):
        lengths = sweep_pool(W, name, args.seed, args.prompts)
        tokens_all = torch.randint(0, shape.vocab, (int(lengths.sum()),), generator=gen, device="cuda",
                                   dtype=torch.int32)
        off = np.concatenate([[0], np.cumsum(lengths)])
        entry = {"pool": name, "prompts": int(len(lengths)), "min": int(lengths.min()),
                 "mean": float(lengths.mean()), "max": int(lengths.max()), "batch_size": args.batch}
        for method, batches in dataset_batches(pp, lengths, args.batch).items():
            total, slots, rows = 0.0, 0, 0
            for ids, plan in batches:
                tokens = torch.cat([tokens_all[off[i]:off[i + 1]] for i in ids.tolist()])
                total += time_plan(pp, model, plan, tokens, args.reps, args.sweep_warmup)["ms"]
                slots, rows = slots + plan.n_slots, rows + plan.n_rows
                torch.cuda.empty_cache()
            entry[method] = {"batches": len(batches), "ms_total": total, "ms_per_prompt": total / len(lengths),
                             "rows": rows, "slots": slots, "fill": float(lengths.sum()) / slots}
            log(f"  {name} {method}: {len(batches)} batches, {total:.1f} ms, {total / len(lengths):.4f} ms/prompt, "
                f"fill {entry[method]['fill']:.3f}")
        out["pools"].append(entry)


def decode_step_bytes(shape, lengths, n_new, padded):
    """Algorithmic HBM bytes of the n_new decode steps of one generate call: every step reads
    all decoder weights, the LM head and the keys and values of every prompt's cache so far
    (full batching: its padding too), and writes one key and value row per prompt."""
    import numpy as np
    s = shape
    e = 2 if s.dtype == "bf16" else 4
    d, H, Hkv, D, F, V = s.d_model, s.n_heads, s.n_kv_heads, s.head_dim, s.ffn_dim, s.vocab
    weights = s.n_layers * (d * (H + 2 * Hkv) * D + H * D * d + 3 * d * F) * e + V * d * e
    lengths = np.asarray(lengths, dtype=np.int64)
    ctx = len(lengths) * int(lengths.max()) if padded else int(lengths.sum())
    k = len(lengths)
    kv_row = 2 * s.n_layers * Hkv * D * e                    # one token's key and value, all layers
    total = 0
    for t in range(n_new):
        total += weights + (ctx + k * (t + 1)) * kv_row      # reads (the step's own row included) ...
        total += k * kv_row                                  # ... and the appended rows
    return total


def run_generate(args):
    """Greedy generation after the prefill with packed and with full-batching KV caches
    (section 4.8): --gen-lengths prompts (default: the paper's toy batch, nine prompts of one
    token and one of 1000), --gen-tokens decode steps after the first token, on --model.
    Times whole pp_generate calls (prefill and first token excluded), and reports the KV cache
    and peak device memory of each layout."""
    import numpy as np
    import torch

    from paper_2404_09529_amd import prepack as pp
    from paper_2404_09529_amd import workloads as W

    shape = W.MODELS[args.model]
    if args.layers:
        shape = shape.replace(n_layers=args.layers)
    lengths = np.asarray([int(x) for x in args.gen_lengths.split(",")], dtype=np.int32)
    n_new = args.gen_tokens
    model = pp.DeviceModel(shape, device_weights(shape, args.seed))
    g = torch.Generator(device="cuda").manual_seed(args.seed + 2)
    lm = (torch.randn((shape.vocab, shape.d_model), generator=g, device="cuda") * 0.02).to(model.torch_dtype)
    tokens = torch.randint(0, shape.vocab, (int(lengths.sum()),), generator=g, device="cuda", dtype=torch.int32)
    dplan = pp.DevicePlan(pp.pp_pack(lengths, 0))
    pre = pp.Prefill(model, dplan)
    pre(tokens)
    ws = torch.empty(max(pp.pp_first_token_workspace_size(model.config, dplan), 1), dtype=torch.uint8, device="cuda")
    first = torch.empty(len(lengths), dtype=torch.int32, device="cuda")
    pp.pp_first_token(model.config, dplan, pre.hidden, lm, ws, first)
    torch.cuda.synchronize()
    base_alloc = torch.cuda.memory_allocated()
    out = {"generate": args.model, "shape": shape.__dict__, "lengths": lengths.tolist(), "n_new": n_new,
           "reps": args.reps, "warmup": args.sweep_warmup}
    toks = {}
    for name, padded in (("packed", False), ("padded", True)):
        torch.cuda.synchronize()
        torch.cuda.reset_peak_memory_stats()
        gen = pp.Generation(model, pre, lengths, n_new, padded=padded)
        stream = torch.cuda.current_stream()
        t = time_steps(lambda: gen(first, lm, stream=stream), args.reps, args.sweep_warmup)
        torch.cuda.synchronize()
        toks[name] = gen.tokens.cpu().numpy()
        gen.capture(first, lm)                 # the same call recorded as one HIP graph
        tg = time_steps(gen.replay, args.reps, args.sweep_warmup)
        torch.cuda.synchronize()
        graph_same = bool(np.array_equal(gen.tokens.cpu().numpy(), toks[name]))
        nbytes = decode_step_bytes(shape, lengths, n_new, padded)
        ms = t["ms_median"]
        mg = tg["ms_median"]
        out[name] = {"ms": ms, "ms_per_token": ms / n_new, "ms_p10": t["ms_p10"], "ms_p90": t["ms_p90"],
                     "graph_ms": mg, "graph_ms_per_token": mg / n_new, "graph_tokens_identical": graph_same,
                     "graph_roofline_frac": round(nbytes / (mg / 1e3) / 1e9 / PEAK_HBM_GBPS, 4),
                     "kv_cache_bytes": gen.kv_cache_bytes(),
                     "peak_alloc_bytes": int(torch.cuda.max_memory_allocated()),
                     "extra_alloc_bytes": int(torch.cuda.max_memory_allocated() - base_alloc),
                     "algorithmic_bytes": nbytes,
                     "roofline": {"bound": "hbm", "achieved": round(nbytes / (ms / 1e3) / 1e9, 1),
                                  "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                                  "frac": round(nbytes / (ms / 1e3) / 1e9 / PEAK_HBM_GBPS, 4)}}
        log(f"{name}: {ms:.3f} ms for {n_new} tokens ({ms / n_new:.3f} ms/token; as one HIP graph "
            f"{mg:.3f} ms, {nbytes / (mg / 1e3) / 1e9:.0f} GB/s), KV cache "
            f"{gen.kv_cache_bytes() / 1e6:.1f} MB, peak {torch.cuda.max_memory_allocated() / 1e9:.2f} GB, "
            f"{nbytes / (ms / 1e3) / 1e9:.0f} GB/s algorithmic")
        del gen
        torch.cuda.empty_cache()
    out["tokens_identical"] = bool(np.array_equal(toks["packed"], toks["padded"]))
    out["time_saving"] = 1.0 - out["packed"]["ms"] / out["padded"]["ms"]
    out["graph_time_saving"] = 1.0 - out["packed"]["graph_ms"] / out["padded"]["graph_ms"]
    out["kv_memory_saving"] = 1.0 - out["packed"]["kv_cache_bytes"] / out["padded"]["kv_cache_bytes"]
    out["peak_memory_saving"] = 1.0 - out["packed"]["peak_alloc_bytes"] / out["padded"]["peak_alloc_bytes"]
    print(json.dumps(out), flush=True)


def run_attention_lengths(args):
    """pp_attention alone on batches of equal-length prompts filling 32,768 slots (rows of 4096),
    Llama-2-7B heads (32 x 128), random bf16 queries, keys and values: time per call against
    both rooflines of the kernel.  Algorithmic work per head: 4 D l(l+1)/2 FLOP per prompt;
    algorithmic bytes: every token's query, key, value and output once (4 x 2 D bytes per token
    and head).  Key/value re-reads by later query tiles are not algorithmic."""
    import numpy as np
    import torch

    from paper_2404_09529_amd import prepack as pp
    H, D, slots = 32, 128, 32768
    cfg = pp.PPConfig(n_layers=1, d_model=H * D, n_heads=H, n_kv_heads=H, head_dim=D, ffn_dim=11008, vocab=32000,
                      dtype=pp.PP_BF16, rms_eps=1e-5, rope_theta=1e4)
    out = {"sweep": "attention-lengths", "heads": H, "head_dim": D, "slots": slots, "rows": []}
    g = torch.Generator(device="cuda").manual_seed(args.seed)
    for n in [int(x) for x in args.lengths.split(",")]:
        lengths = np.full(slots // n, n, dtype=np.int32)
        plan = pp.pp_pack(lengths, 4096)
        dp = pp.DevicePlan(plan)
        q = torch.randn((plan.n_slots, H * D), generator=g, device="cuda").to(torch.bfloat16)
        kc = torch.randn((plan.total_len, H * D), generator=g, device="cuda").to(torch.bfloat16)
        vc = torch.randn((plan.total_len, H * D), generator=g, device="cuda").to(torch.bfloat16)
        o = torch.empty_like(q)
        t = time_steps(lambda: pp.pp_attention(cfg, dp, q, H * D, kc, vc, o), args.reps, args.sweep_warmup)
        ms = t["ms_median"]
        pairs = attention_pairs(plan, lengths)
        flop = 4 * H * D * pairs["algorithmic"]
        nbytes = 4 * 2 * D * H * plan.total_len
        rec = {"length": n, "prompts": int(len(lengths)), "us": round(ms * 1e3, 1),
               "tflops": round(flop / (ms / 1e3) / 1e12, 1), "frac_mfma": round(flop / (ms / 1e3) / 1e12 / PEAK_BF16_TFLOPS, 4),
               "gbps": round(nbytes / (ms / 1e3) / 1e9, 1), "frac_hbm": round(nbytes / (ms / 1e3) / 1e9 / PEAK_HBM_GBPS, 4),
               "bound_us": round(1e6 * max(flop / (PEAK_BF16_TFLOPS * 1e12), nbytes / (PEAK_HBM_GBPS * 1e9)), 1),
               "pairs_executed_over_algorithmic": pairs["inflation"]}
        out["rows"].append(rec)
        log(f"attention, prompts of {n}: {rec['us']} us, {rec['tflops']} TFLOP/s ({100 * rec['frac_mfma']:.1f}% of MFMA "
            f"peak), {rec['gbps']} GB/s algorithmic ({100 * rec['frac_hbm']:.1f}% of HBM)")
        del q, kc, vc, o
        torch.cuda.empty_cache()
    print(json.dumps(out), flush=True)


def run_sweep(args):
    """--sweep regression: batches of --batch prompts from the prompt pool, the speedup of
    packing over full batching per batch, and the linear fits of the speedup on r/k and on
    m - L/k.  --sweep batch: the mean speedup at each of --batch-sizes.  --sweep datasets: the
    prefill time and time to first token per batch of --batch prompts, packed and fully
    batched, over each pool of --pools.  --sweep dataset-packing: per-prompt prefill time of
    full batching, per-batch packing, length-ordered batching and whole-set packing."""
    import numpy as np
    import torch

    from paper_2404_09529_amd import prepack as pp
    from paper_2404_09529_amd import workloads as W

    shape = W.MODELS[args.model]
    if args.layers:
        shape = shape.replace(n_layers=args.layers)
    t = time.perf_counter()
    model = pp.DeviceModel(shape, device_weights(shape, args.seed))
    lm_head = None
    if args.sweep == "datasets":
        g = torch.Generator(device="cuda").manual_seed(args.seed + 2)
        lm_head = (torch.randn((shape.vocab, shape.d_model), generator=g, device="cuda") * 0.02).to(torch.bfloat16)
    torch.cuda.synchronize()
    log(f"sweep {args.sweep}: model {args.model} ({shape.n_layers} layers), weights drawn on the device in "
        f"{time.perf_counter() - t:.1f} s")
    gen = torch.Generator(device="cuda").manual_seed(args.seed + 1)
    out = {"sweep": args.sweep, "model": args.model, "shape": shape.__dict__, "seed": args.seed, "reps": args.reps,
           "warmup": args.sweep_warmup}
    if args.sweep == "dataset-packing":
        out["pools"] = []
        run_dataset_packing(pp, W, model, args, gen, out)
        print(json.dumps(out), flush=True)
        return
    pools = args.pools.split(",") if args.sweep == "datasets" else [args.pool]
    sizes = [int(b) for b in args.batch_sizes.split(",")] if args.sweep == "batch" else [args.batch]
    out["per_batch_size"] = []
    t0 = time.perf_counter()
    for name in pools:
        pool = sweep_pool(W, name, args.seed, args.prompts)
        for bs in sizes:
            n_b = len(pool) // bs
            if args.max_batches:
                n_b = min(n_b, args.max_batches)
            recs = []
            for b in range(n_b):
                recs.append(measure_batch(pp, model, pool[b * bs:(b + 1) * bs], args, gen, lm_head))
                if (b + 1) % 20 == 0 or b + 1 == n_b:
                    log(f"  {name} batch size {bs}: {b + 1}/{n_b} batches, last speedup {recs[-1]['speedup']:.2f}x "
                        f"({time.perf_counter() - t0:.0f} s)")
                torch.cuda.empty_cache()
            col = lambda key: np.array([r[key] for r in recs], dtype=np.float64)
            sp, mp, md = col("speedup"), col("ms_packed"), col("ms_padded")
            entry = {"pool": name, "prompts": int(len(pool)), "batch_size": bs, "batches": n_b,
                     "speedup_mean": float(sp.mean()), "speedup_std": float(sp.std()),
                     "ms_packed_mean": float(mp.mean()), "ms_packed_std": float(mp.std()),
                     "ms_padded_mean": float(md.mean()), "ms_padded_std": float(md.std()),
                     "total_time_ratio": float(md.sum() / mp.sum()),
                     "r_over_k_mean": float(col("r_over_k").mean()), "max_abs_dev_mean": float(col("max_abs_dev").mean()),
                     "tflops_packed_mean": float(col("tflops_packed").mean())}
            if lm_head is not None:
                tp, td = col("ttft_ms_packed"), col("ttft_ms_padded")
                entry.update({"ttft_ms_packed_mean": float(tp.mean()), "ttft_ms_packed_std": float(tp.std()),
                              "ttft_ms_padded_mean": float(td.mean()), "ttft_ms_padded_std": float(td.std()),
                              "ttft_speedup_mean": float(col("ttft_speedup").mean())})
            if n_b >= 3:
                for key, x in (("fit_r_over_k", "r_over_k"), ("fit_max_abs_dev", "max_abs_dev")):
                    fit = linear_fit(col(x), sp)
                    if fit is not None:
                        entry[key] = fit
            if args.sweep == "regression":
                entry["records"] = recs
            out["per_batch_size"].append(entry)
            log(f"{name} batch size {bs}: speedup {entry['speedup_mean']:.2f} +- {entry['speedup_std']:.2f}x over "
                f"{n_b} batches; packed {entry['ms_packed_mean']:.2f} ms, padded {entry['ms_padded_mean']:.2f} ms")
    print(json.dumps(out), flush=True)


def main():
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--workload", type=int, default=2, help="workload id (2 = Llama-2-7B shape, lognormal)")
    ap.add_argument("--seed", type=int, default=0)
    ap.add_argument("--no-padded", action="store_true")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--kernel-launches", type=int, default=20)
    ap.add_argument("--traffic-pass", action="store_true",
                    help="run only the dominant kernel and the calibration copy (for counter passes)")
    ap.add_argument("--calibration-copy", action="store_true",
                    help="end with the calibration copy (for byte-counter passes over the whole step)")
    ap.add_argument("--sweep", choices=["regression", "batch", "datasets", "dataset-packing", "attention-lengths"],
                    help="instead of the benchmark line: packing against full batching per batch of a prompt "
                         "pool, with linear fits of the speedup (regression), across batch sizes (batch), with "
                         "the time to first token over dataset stand-ins (datasets), or against length-ordered "
                         "batching and whole-set packing (dataset-packing); attention-lengths: the attention kernel "
                         "alone on prompts of each of --lengths against its MFMA and HBM rooflines")
    ap.add_argument("--pool", default="uniform", help="sweep regression/batch: uniform (U[1,512]) or a dataset "
                                                     "stand-in (wiki256, wiki512, mmlu, hh-rlhf, alpaca, samsum)")
    ap.add_argument("--pools", default="wiki256,wiki512,mmlu,hh-rlhf,alpaca,samsum",
                    help="sweep datasets/dataset-packing: prompt pools")
    ap.add_argument("--model", default="llama-1.3b", help="sweep model shape (llama-1.3b, llama2-7b, mistral-7b)")
    ap.add_argument("--layers", type=int, default=0, help="sweep: decoder layers (0 = the model's full depth)")
    ap.add_argument("--batch", type=int, default=32, help="sweep: prompts (dataset packing: rows) per batch")
    ap.add_argument("--batch-sizes", default="1,2,4,8,16,32,64", help="sweep batch: batch sizes")
    ap.add_argument("--lengths", default="16,32,64,128,256,512,1024,2048,4096",
                    help="sweep attention-lengths: prompt lengths (each batch fills 32,768 slots)")
    ap.add_argument("--prompts", type=int, default=5000, help="sweep: prompts taken from the pool")
    ap.add_argument("--max-batches", type=int, default=0, help="sweep: at most this many batches per size")
    ap.add_argument("--reps", type=int, default=3, help="sweep: timed steps per batch and layout (median)")
    ap.add_argument("--sweep-warmup", type=int, default=1, help="sweep: untimed steps per batch and layout")
    ap.add_argument("--generate", action="store_true",
                    help="instead of the benchmark line: greedy generation with packed vs full-batching KV caches")
    ap.add_argument("--gen-lengths", default=",".join(["1"] * 9 + ["1000"]),
                    help="generate: prompt lengths (default: nine of one token and one of 1000)")
    ap.add_argument("--gen-tokens", type=int, default=20, help="generate: decode steps after the first token")
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
    if args.sweep == "attention-lengths":
        run_attention_lengths(args)
        return
    if args.sweep:
        run_sweep(args)
        return
    if args.generate:
        run_generate(args)
        return

    t = time.perf_counter()
    case = W.make_case(args.workload, args.seed)
    shape, lengths = case.shape, case.lengths
    log(f"workload {case.wl.name}: k={len(lengths)} L={case.total_len} m={lengths.max()} "
        f"(weights drawn in {time.perf_counter() - t:.1f} s)")

    # host planning, timed on its own: the C call into plan arrays allocated once, and the
    # binding's pp_pack (which allocates the arrays and copies them out) for reference
    n_pack = 50
    bufs = pp.PlanBuffers(len(lengths), case.capacity)
    l32 = np.ascontiguousarray(lengths, dtype=np.int32)
    bufs.pack(l32, case.capacity)
    t = time.perf_counter()
    for _ in range(n_pack):
        bufs.pack(l32, case.capacity)
    pack_ms = (time.perf_counter() - t) * 1e3 / n_pack
    t = time.perf_counter()
    for _ in range(n_pack):
        plan = pp.pp_pack(lengths, case.capacity)
    pack_binding_ms = (time.perf_counter() - t) * 1e3 / n_pack
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
    torch.cuda.synchronize()
    base_alloc = torch.cuda.memory_allocated()
    torch.cuda.reset_peak_memory_stats()
    step = pp.Prefill(model, dplan)
    step(tokens)
    torch.cuda.synchronize()
    mem_packed = prefill_memory(step, base_alloc)
    log(f"packed plan: {plan.n_rows} rows x {plan.capacity}, fill {case.total_len / plan.n_slots:.3f}, "
        f"pack {pack_ms:.3f} ms, upload {upload_ms:.2f} ms")

    flops = algorithmic_flops(shape, lengths)
    packed = time_steps(lambda: step(tokens), args.steps, args.warmup)
    ms = packed["ms_mean"]
    value = case.total_len / (ms / 1e3)
    tflops = flops / (ms / 1e3) / 1e12
    log(f"packed: {ms:.3f} ms/step, {value:,.0f} tokens/s, {tflops:.1f} TFLOP/s effective")

    # dominant kernel: the gate/up GEMM (bf16: with the SwiGLU epilogue), same launch as inside
    # pp_prefill; the float32 model's is the FMA (vector ALU) GEMM storing gate and up
    T, d, F = plan.n_slots, shape.d_model, shape.ffn_dim
    bf = shape.dtype == "bf16"
    peak = PEAK_BF16_TFLOPS if bf else PEAK_FP32_TFLOPS
    gen = torch.Generator(device="cuda").manual_seed(1)
    kstream = torch.cuda.current_stream()
    Wgu = model.layers[0]["w_gateup"]
    if bf:
        A = torch.randn((T, d), generator=gen, device="cuda").to(torch.bfloat16)
        Cb = torch.empty((T, F), dtype=torch.bfloat16, device="cuda")
        gemm = lambda: pp.pp_gemm(pp.PP_BF16, pp.PP_EPI_SWIGLU, A, d, Wgu, d, Cb, F, T, 2 * F, d, dplan, kstream)
        k_name, k_bytes = "gemm_bf16_kernel<kSwiGLU> (gate/up projection)", 2 * (case.total_len * d + 2 * F * d
                                                                              + case.total_len * F)
    else:
        A = torch.randn((T, d), generator=gen, device="cuda")
        Cb = torch.empty((T, 2 * F), dtype=torch.float32, device="cuda")
        gemm = lambda: pp.pp_gemm(pp.PP_F32, pp.PP_EPI_STORE, A, d, Wgu, d, Cb, 2 * F, T, 2 * F, d, None, kstream)
        k_name, k_bytes = "gemm_f32_kernel (gate/up projection)", 4 * (case.total_len * d + 2 * F * d
                                                                        + case.total_len * 2 * F)
    kt = time_steps(gemm, args.kernel_launches, 3)
    k_flops = 2.0 * case.total_len * (2 * F) * d
    achieved = k_flops / (kt["ms_mean"] / 1e3) / 1e12
    del A, Cb
    log(f"gate/up GEMM: {kt['ms_mean']:.3f} ms/launch, {achieved:.1f} TFLOP/s algorithmic")
    traffic = recorded_traffic(case.wl.name, args.seed) if bf else None   # A, W once; C written once (k_bytes)

    out = {
        "metric": METRIC, "value": round(value, 1), "unit": "tokens/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": shape.dtype, "data": "synthetic",
        "config": {"workload": case.wl.name, "description": case.wl.description, "seed": args.seed,
                   "k": int(len(lengths)), "capacity": int(case.capacity), "total_len": case.total_len,
                   "max_len": int(lengths.max()), "n_rows": plan.n_rows, "fill": round(case.total_len / plan.n_slots, 4)},
        "tflops_effective": round(tflops, 2), "frac_bf16_peak": round(tflops / PEAK_BF16_TFLOPS, 4),
        "frac_peak": round(tflops / peak, 4), "peak_tflops": peak,
        "algorithmic_flop": flops,
        "ms_median": round(packed["ms_median"], 4), "ms_p10": round(packed["ms_p10"], 4),
        "ms_p90": round(packed["ms_p90"], 4),
        "pack_ms": round(pack_ms, 4), "pack_binding_ms": round(pack_binding_ms, 4),
        "plan_upload_ms": round(upload_ms, 3),
        "gemm_rows_executed_over_L": round(gemm_rows_executed(plan) / case.total_len, 4),
        "device_memory": {"packed": mem_packed, "weights_bytes": model_bytes(model)},
        "attention_pairs": attention_pairs(plan, lengths, tiled=bf),
        "roofline": {"kernel": k_name, "bound": "mfma" if bf else "alu",
                     "achieved": round(achieved, 1), "peak": peak, "unit": "TFLOP/s",
                     "frac": round(achieved / peak, 4),
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
    # the LM head read from HBM, as after a prefill (the roofline figure), and warm: repeated
    # calls, where part of it may still sit in the last-level cache
    ft = time_cold(ftok, args.kernel_launches, 3)
    ft_warm = time_steps(ftok, args.kernel_launches, 3)
    both = time_steps(lambda: (step(tokens, kstream), ftok()), args.steps, args.warmup)
    lm_bytes = lm_head.numel() * lm_head.element_size()
    out["ttft"] = {"ms_median": round(both["ms_median"], 4), "ms_mean": round(both["ms_mean"], 4),
                   "first_token_ms": round(ft["ms_mean"], 4), "first_token_ms_warm": round(ft_warm["ms_mean"], 4),
                   "prefill_ms_median": round(packed["ms_median"], 4),
                   "first_token_roofline": {"bound": "hbm", "achieved": round(lm_bytes / (ft["ms_mean"] / 1e3) / 1e9, 1),
                                            "peak": PEAK_HBM_GBPS, "unit": "GB/s",
                                            "frac": round(lm_bytes / (ft["ms_mean"] / 1e3) / 1e9 / PEAK_HBM_GBPS, 4),
                                            "algorithmic_bytes_per_launch": lm_bytes, "vocab": V,
                                            "cache": "last-level cache cleared before each call"}}
    log(f"first token: {ft['ms_mean'] * 1e3:.1f} us ({lm_bytes / (ft['ms_mean'] / 1e3) / 1e9:.0f} GB/s on the LM head; "
        f"warm {ft_warm['ms_mean'] * 1e3:.1f} us); "
        f"TTFT {both['ms_median']:.3f} ms")
    del step, lm_head, ft_ws
    torch.cuda.empty_cache()

    if not args.no_padded:
        pplan = pp.pp_pack_padded(lengths)
        pdplan = pp.DevicePlan(pplan)
        torch.cuda.synchronize()
        base_alloc = torch.cuda.memory_allocated()
        torch.cuda.reset_peak_memory_stats()
        pstep = pp.Prefill(model, pdplan)
        pstep(tokens)
        torch.cuda.synchronize()
        out["device_memory"]["padded"] = prefill_memory(pstep, base_alloc)
        out["device_memory"]["padded_over_packed"] = round(
            out["device_memory"]["padded"]["extra_peak_bytes"] / out["device_memory"]["packed"]["extra_peak_bytes"], 3)
        padded = time_steps(lambda: pstep(tokens), max(3, args.steps // 4), 1)
        pms = padded["ms_mean"]
        out["padded"] = {"ms_per_step": round(pms, 4), "tokens_per_s": round(case.total_len / (pms / 1e3), 1),
                         "tflops_effective": round(flops / (pms / 1e3) / 1e12, 2), "n_rows": pplan.n_rows,
                         "capacity": pplan.capacity,
                         "attention_pairs_executed": attention_pairs(pplan, lengths, tiled=bf)["executed"]}
        out["speedup_vs_padded"] = round(pms / ms, 3)
        log(f"padded: {pms:.3f} ms/step, speedup {pms / ms:.2f}x")
        del pstep
        torch.cuda.empty_cache()

    if not args.no_cpu_baseline:
        out["cpu_baseline"] = cpu_baseline(case)
        log(f"cpu oracle: {out['cpu_baseline']['value']:.1f} tokens/s on {out['cpu_baseline']['cores']} threads "
            f"({out['cpu_baseline']['cpu_model']})")

    if args.calibration_copy:
        calibration_copy()
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
