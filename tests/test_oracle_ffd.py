"""Pins for the packing oracle (oracle/ffd.py): brute force, bounds, special cases,
invariants and hand-worked examples.  CPU only."""
import itertools
import json
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st

from oracle import ffd


def _golden(golden_dir):
    with open(os.path.join(golden_dir, "ffd_examples.json")) as f:
        return json.load(f)["examples"]


def _bins_from_plan(p):
    return [list(map(int, p.seg_prompt[p.row_seg_ptr[r]:p.row_seg_ptr[r + 1]]))
            for r in range(p.n_rows)]


def test_hand_worked_examples(golden_dir):
    for ex in _golden(golden_dir):
        p = ffd.pack(ex["lengths"], ex["capacity"])
        assert ffd.ffd(ex["lengths"], p.capacity) == ex["bins"], ex["name"]
        assert _bins_from_plan(p) == ex["bins"]
        assert p.seg_start.tolist() == ex["seg_start"]
        assert p.prompt_kv_off.tolist() == ex["prompt_kv_off"]
        assert p.slot_kv.tolist() == ex["slot_kv"]
        assert p.slot_pos.tolist() == ex["slot_pos"]
        for key in ("mask_row0", "mask_row2"):
            if key in ex:
                row = int(key[-1])
                want = np.array([[c == "1" for c in line] for line in ex[key]])
                assert np.array_equal(ffd.independent_mask(p, row), want)


@pytest.mark.parametrize("seed", range(40))
def test_brute_force_optimum_and_ffd_bound(seed):
    rng = np.random.default_rng(seed)
    k = int(rng.integers(1, 9))
    C = int(rng.integers(4, 20))
    lengths = rng.integers(1, C + 1, k).tolist()
    opt = ffd.optimal_bins(lengths, C)
    r = len(ffd.ffd(lengths, C))
    assert ffd.lower_bound(lengths, C) <= opt <= r <= ffd.dosa_bound(opt) + 1e-9
    assert r <= k
    if k <= 6:
        assert ffd.optimal_bins_by_partition(lengths, C) == opt


def test_ffd_is_not_optimal_here():
    # rows of 10, lengths 4,4,3,3,3,3: FFD puts both 4s together (room 2), then three 3s
    # (room 1) and opens a third row; the optimum is {4,3,3} twice.  11/9*2 + 6/9 >= 3.
    lengths = [4, 4, 3, 3, 3, 3]
    assert ffd.ffd(lengths, 10) == [[0, 1], [2, 3, 4], [5]]
    assert ffd.optimal_bins(lengths, 10) == 2
    assert ffd.optimal_bins_by_partition(lengths, 10) == 2
    assert 3 <= ffd.dosa_bound(2)


def test_special_cases():
    # all prompts longer than half a row: no two share a row, r = k
    assert len(ffd.ffd([6, 7, 8, 9], 10)) == 4
    # everything fits one row
    p = ffd.pack([3, 2, 4], 10)
    assert p.n_rows == 1
    # bin size = m and all equal lengths: one prompt per row
    assert ffd.pack([5, 5, 5]).n_rows == 3
    # empty batch
    p = ffd.pack([], 16)
    assert p.n_rows == 0 and p.total_len == 0
    # invalid inputs
    with pytest.raises(ValueError):
        ffd.pack([3, 0, 2], 8)
    with pytest.raises(ValueError):
        ffd.pack([3, 9, 2], 8)


def _check_plan_invariants(lengths, p):
    lengths = np.asarray(lengths)
    k = len(lengths)
    C = p.capacity
    # each prompt in exactly one segment; rows hold at most C tokens
    assert sorted(p.seg_prompt.tolist()) == list(range(k))
    assert np.array_equal(p.seg_len, lengths[p.seg_prompt])
    for r in range(p.n_rows):
        segs = range(p.row_seg_ptr[r], p.row_seg_ptr[r + 1])
        col = 0
        for s in segs:   # contiguous from column 0, no overlap
            assert p.seg_start[s] == r * C + col
            col += int(p.seg_len[s])
        assert 0 < col <= C
        # pads only at the row tail
        tail = p.slot_kv[r * C + col:(r + 1) * C]
        assert np.all(tail == -1)
    # slot_kv is a bijection from real slots onto [0, L)
    real = p.slot_kv[p.slot_kv >= 0]
    assert np.array_equal(np.sort(real), np.arange(lengths.sum()))
    # closed forms of positions and cache rows
    for s in range(k):
        a, n, i = int(p.seg_start[s]), int(p.seg_len[s]), int(p.seg_prompt[s])
        assert np.array_equal(p.slot_pos[a:a + n], np.arange(n))
        assert np.array_equal(p.slot_kv[a:a + n], p.prompt_kv_off[i] + np.arange(n))
        assert np.all(p.slot_seg[a:a + n] == s)


@settings(max_examples=200, deadline=None)
@given(st.lists(st.integers(1, 40), min_size=1, max_size=30), st.integers(0, 60))
def test_plan_invariants(lengths, extra):
    C = max(lengths) + extra
    p = ffd.pack(lengths, C)
    _check_plan_invariants(lengths, p)
    assert ffd.lower_bound(lengths, C) <= p.n_rows <= len(lengths)
    assert np.array_equal(ffd.split_lengths(p), np.asarray(lengths))


@settings(max_examples=100, deadline=None)
@given(st.lists(st.integers(1, 40), min_size=1, max_size=20))
def test_padded_plan(lengths):
    p = ffd.pack_padded(lengths)
    m = max(lengths)
    assert p.n_rows == len(lengths) and p.capacity == m
    for i, l in enumerate(lengths):
        row = slice(i * m, (i + 1) * m)
        assert np.array_equal(p.slot_pos[row], np.arange(m))
        assert np.all(p.slot_seg[row] == i)
        assert np.array_equal(p.slot_kv[row][:l], p.prompt_kv_off[i] + np.arange(l))
        assert np.all(p.slot_kv[row][l:] == -1)
    assert np.all(p.seg_len == m)


def test_mask_is_block_diagonal_lower_triangular():
    p = ffd.pack([3, 4, 2, 5, 1], 8)
    for r in range(p.n_rows):
        M = ffd.independent_mask(p, r)
        base = r * p.capacity
        seg = p.slot_seg[base:base + p.capacity]
        for i, j in itertools.product(range(p.capacity), repeat=2):
            want = seg[i] >= 0 and seg[i] == seg[j] and j <= i
            assert M[i, j] == want
