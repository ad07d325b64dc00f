"""Host-side statistics of the batch-size and regression sweeps (section 4.7 of the paper):
the two predictors of the speedup, batch-size reduction r/k and max absolute deviation
m - L/k, and the least-squares line fitted to them.  CPU only, no GPU work."""
import os

import numpy as np
import pytest
from scipy import stats

import bench
from oracle import ffd
from paper_2404_09529_amd import prepack as pp
from paper_2404_09529_amd import workloads as W


def test_predictors_hand_worked():
    # lengths 3, 5, 8 in two rows: r/k = 2/3; mean 16/3, so m - L/k = 8 - 16/3 = 8/3
    p = bench.batch_predictors([3, 5, 8], 2)
    assert p["r_over_k"] == pytest.approx(2 / 3, abs=0)
    assert p["max_abs_dev"] == pytest.approx(8 / 3, rel=1e-15)


def test_predictors_degenerate_batches():
    # equal lengths: no deviation; one prompt: one row, no deviation
    assert bench.batch_predictors([7] * 5, 5) == {"r_over_k": 1.0, "max_abs_dev": 0.0}
    assert bench.batch_predictors([300], 1) == {"r_over_k": 1.0, "max_abs_dev": 0.0}


def test_pool_is_uniform_1_512():
    pool = W.draw_lengths(W.workload(6), 0)
    assert len(pool) == 5000 and pool.min() >= 1 and pool.max() <= 512
    # mean of U{1..512} is 256.5, sd 147.8: the pool mean sits within 4 standard errors
    assert abs(pool.mean() - 256.5) < 4 * 147.8 / np.sqrt(5000)


@pytest.mark.skipif(not os.path.exists(pp.LIB_PATH), reason="libprepack.so is not built")
@pytest.mark.parametrize("bs", [16, 32])
def test_sweep_rows_match_oracle_ffd(bs):
    """r of every sweep batch (bin size = the batch maximum) is the oracle FFD's, bit for bit."""
    pool = W.draw_lengths(W.workload(6), 0)
    for b in range(0, 40 * bs, bs):
        lengths = pool[b:b + bs]
        r = pp.pp_pack(lengths, 0).n_rows
        assert r == len(ffd.ffd(lengths.tolist(), int(lengths.max())))
        assert ffd.lower_bound(lengths.tolist(), int(lengths.max())) <= r <= len(lengths)


def test_linear_fit_exact_line():
    x = np.array([0.1, 0.4, 0.5, 0.9])
    f = bench.linear_fit(x, 3.0 - 2.5 * x)
    assert f["slope"] == pytest.approx(-2.5, rel=1e-12)
    assert f["intercept"] == pytest.approx(3.0, rel=1e-12)
    assert f["pearson_r"] == pytest.approx(-1.0, rel=1e-12)
    assert f["r2"] == pytest.approx(1.0, rel=1e-12)


def test_linear_fit_matches_scipy_linregress():
    rng = np.random.default_rng(7)
    x = rng.uniform(0.3, 0.9, 157)
    y = 4.0 - 3.0 * x + rng.normal(0, 0.2, 157)
    f = bench.linear_fit(x, y)
    ref = stats.linregress(x, y)
    assert f["slope"] == pytest.approx(ref.slope, rel=1e-10)
    assert f["intercept"] == pytest.approx(ref.intercept, rel=1e-10)
    assert f["pearson_r"] == pytest.approx(ref.rvalue, rel=1e-10)
    assert f["n"] == 157


def test_linear_fit_residuals_orthogonal():
    """Normal equations: residuals sum to zero and are orthogonal to x."""
    rng = np.random.default_rng(3)
    x = rng.uniform(0, 300, 60)
    y = 1.0 + 0.01 * x + rng.normal(0, 0.3, 60)
    f = bench.linear_fit(x, y)
    res = y - (f["intercept"] + f["slope"] * x)
    assert abs(res.sum()) < 1e-9
    assert abs(np.dot(res, x)) < 1e-6
    assert f["r2"] == pytest.approx(1 - np.sum(res ** 2) / np.sum((y - y.mean()) ** 2), rel=1e-10)


# ----------------------------------------------------------------------------- dataset stand-ins and batchings
@pytest.mark.parametrize("name", list(W.DATASETS))
def test_dataset_standins_match_stated_statistics(name):
    """min / max inside the stated range, the mean within 10% of the stated one."""
    wid, lo, mean, hi = W.DATASETS[name]
    lengths = W.draw_lengths(W.workload(wid), 0)
    assert len(lengths) == 1000 and lengths.min() >= lo and lengths.max() <= hi
    assert abs(lengths.mean() - mean) <= 0.1 * mean


@pytest.mark.skipif(not os.path.exists(pp.LIB_PATH), reason="libprepack.so is not built")
@pytest.mark.parametrize("name,bs", [("uniform", 16), ("mmlu", 16), ("hh-rlhf", 32), ("wiki256", 8)])
def test_dataset_batchings_cover_every_prompt_once(name, bs):
    lengths = bench.sweep_pool(W, name, 0, 1000)
    out = bench.dataset_batches(pp, lengths, bs)
    for method, batches in out.items():
        ids = np.concatenate([i for i, _ in batches])
        assert np.array_equal(np.sort(ids), np.arange(len(lengths))), method
        for i, plan in batches:
            assert plan.total_len == int(lengths[i].sum())
    # full batching and its length-ordered form pad to the batch maximum; length ordering
    # never needs more slots
    slots = {m: sum(p.n_slots for _, p in b) for m, b in out.items()}
    assert slots["ordered"] <= slots["full"]
    assert slots["batch"] <= slots["full"]


@pytest.mark.skipif(not os.path.exists(pp.LIB_PATH), reason="libprepack.so is not built")
@pytest.mark.parametrize("name,bs", [("mmlu", 16), ("samsum", 4), ("uniform", 32)])
def test_dataset_packing_rebuilds_the_oracle_rows(name, bs):
    """Whole-set FFD from the oracle; each group of bs of its rows, packed again on its own,
    holds the same prompts row for row."""
    lengths = bench.sweep_pool(W, name, 0, 1000)
    bins = ffd.ffd(lengths.tolist(), int(lengths.max()))
    groups = bench.dataset_batches(pp, lengths, bs)["dataset"]
    assert len(groups) == (len(bins) + bs - 1) // bs
    for g, (ids, plan) in enumerate(groups):
        want = [sorted(b) for b in bins[g * bs:(g + 1) * bs]]
        got = []
        for r in range(plan.n_rows):
            segs = plan.seg_prompt[plan.row_seg_ptr[r]:plan.row_seg_ptr[r + 1]]
            got.append(sorted(int(ids[s]) for s in segs))
        assert sorted(got) == sorted(want)


def test_linear_fit_of_a_constant_predictor_is_none():
    # batch size 1: every batch has r/k = 1
    assert bench.linear_fit([1.0, 1.0, 1.0], [0.99, 1.0, 1.01]) is None
    assert bench.linear_fit([0.5, 0.6, 0.7], [1.0, 1.0, 1.0]) is None


def test_attention_pairs_brute_force():
    # causal pairs per head and layer, counted one by one on a tiny plan: the method needs
    # l(l+1)/2 per prompt; the tiled kernel computes each work item's whole query tile
    # against key tiles of 64 up to the item's last key
    lengths = [1, 130, 64, 300]
    plan = pp.pp_pack(lengths, 512)
    got = bench.attention_pairs(plan, lengths)
    want_alg = sum(1 for n in lengths for q in range(n) for key in range(q + 1))
    want_exe = 0
    for s, q0 in zip(plan.qtile_seg.tolist(), plan.qtile_q0.tolist()):
        n = int(plan.seg_len[s])
        last_key = min(q0 + pp.PP_QTILE, n) - 1
        want_exe += sum(1 for q in range(pp.PP_QTILE) for key in range(64 * (last_key // 64 + 1)))
    assert got["algorithmic"] == want_alg
    assert got["executed"] == want_exe
    assert got["inflation"] >= 1.0
    # the float32 kernel takes each real query's own keys only
    assert bench.attention_pairs(plan, lengths, tiled=False)["executed"] == want_alg
