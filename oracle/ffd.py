"""Oracle: bin packing and the packed / padded plans (integer work).

TEST INFRASTRUCTURE ONLY (see ``oracle/__init__.py``).

What the paper fixes, and how it is read here:

* BINPACK (Algorithm 1; section 3.1): the prompt lengths are packed into the
  fewest bins of a fixed size, by the first-fit-decreasing heuristic.  The
  paper uses a third-party Python implementation that is not available; this
  is the textbook FFD: take the prompts in order of decreasing length (ties by
  original index), put each into the lowest-numbered bin that still has room,
  and open a new bin when none has.  Inside a bin the prompts sit back to back
  from position 0 in the order they were placed; the rest of the bin is
  padding (section 3.1: bins that are not full are padded to the bin size).
* Bin size: the paper takes the maximum prompt length m (section 3.1).  A
  ``capacity`` argument generalises it; ``capacity == 0`` means m.
* RESTART-PE (section 3.2): the position of a token is its offset inside its
  own prompt, restarting at 0 at every prompt start.
* INDEPENDENT-MASK (section 3.2): for every prompt occupying positions
  [a, b) of a bin, M'[a:b, a:b] is lower triangular; every other entry is 0.
* UNPACK (Algorithm 1): per-prompt caches in the original prompt order; the
  cache of prompt i occupies rows [off_i, off_i + l_i) of a compact cache,
  off = exclusive prefix sum of the lengths in original order.
* Full batching baseline (section 4.2): every prompt is padded at its end to
  the batch maximum m; one row per prompt; each row is one causal span of
  length m whose pad tokens never influence the real ones.

Parity pins (tests/test_oracle_ffd.py): brute-force optimum on tiny inputs and
the tight FFD bound, special cases, invariants, and hand-worked examples in
``tests/golden/``.  Parity with the third-party library's exact bin
assignment is unpinned (it is not available), which is why the packing
choices above are pinned only against their own definition and invariants.
"""
from __future__ import annotations

import itertools
from dataclasses import dataclass
from typing import List, Optional, Sequence

import numpy as np


def ffd(lengths: Sequence[int], capacity: int) -> List[List[int]]:
    """First-fit decreasing.  Returns bins as lists of prompt indices in placement order."""
    order = sorted(range(len(lengths)), key=lambda i: (-int(lengths[i]), i))
    bins: List[List[int]] = []
    room: List[int] = []
    for i in order:
        li = int(lengths[i])
        for b in range(len(bins)):
            if room[b] >= li:
                bins[b].append(i)
                room[b] -= li
                break
        else:
            bins.append([i])
            room.append(capacity - li)
    return bins


def optimal_bins(lengths: Sequence[int], capacity: int) -> int:
    """Fewest bins of size ``capacity`` holding all lengths, by exhaustive search (tiny k only)."""
    k = len(lengths)
    assert k <= 10, "brute force is for tiny inputs"
    best = k
    items = sorted((int(x) for x in lengths), reverse=True)

    def place(j: int, loads: List[int]) -> None:
        nonlocal best
        if len(loads) >= best:
            return
        if j == k:
            best = len(loads)
            return
        seen = set()
        for b in range(len(loads)):
            if loads[b] + items[j] <= capacity and loads[b] not in seen:
                seen.add(loads[b])
                loads[b] += items[j]
                place(j + 1, loads)
                loads[b] -= items[j]
        loads.append(items[j])
        place(j + 1, loads)
        loads.pop()

    place(0, [])
    return best


def optimal_bins_by_partition(lengths: Sequence[int], capacity: int) -> int:
    """Second brute force: try every assignment of items to bins (k <= 7)."""
    k = len(lengths)
    assert k <= 7
    for r in range(1, k + 1):
        for assign in itertools.product(range(r), repeat=k):
            loads = [0] * r
            for i, b in enumerate(assign):
                loads[b] += int(lengths[i])
            if max(loads) <= capacity and len(set(assign)) == r:
                return r
    return k


@dataclass
class Plan:
    """Everything the prefill needs about where each token sits.

    Segments (attention spans) are listed row by row; inside a row in
    placement order.  Slot t of the packed batch is row t // capacity,
    column t % capacity.
    """
    k: int
    capacity: int
    n_rows: int
    max_len: int
    total_len: int
    row_seg_ptr: np.ndarray    # [n_rows + 1]
    seg_prompt: np.ndarray     # [k]
    seg_start: np.ndarray      # [k] global slot of the span's first token
    seg_len: np.ndarray        # [k] span length (packed: the prompt length; padded: m)
    prompt_kv_off: np.ndarray  # [k + 1]
    slot_seg: np.ndarray       # [n_rows * capacity], -1 outside every span
    slot_pos: np.ndarray       # [n_rows * capacity], 0 outside every span
    slot_kv: np.ndarray        # [n_rows * capacity], -1 at pads

    @property
    def n_slots(self) -> int:
        return self.n_rows * self.capacity


def _prefix(lengths: np.ndarray) -> np.ndarray:
    off = np.zeros(len(lengths) + 1, dtype=np.int64)
    for i, l in enumerate(lengths):
        off[i + 1] = off[i] + int(l)
    return off


def _check_lengths(lengths: np.ndarray) -> None:
    if np.any(lengths <= 0):
        raise ValueError("every prompt needs at least one token")


def pack(lengths: Sequence[int], capacity: int = 0) -> Plan:
    """Algorithm 1 up to the model call: BINPACK, TENSORIZE layout, RESTART-PE, UNPACK map."""
    lengths = np.asarray(lengths, dtype=np.int64)
    k = len(lengths)
    if k:
        _check_lengths(lengths)
    m = int(lengths.max()) if k else 0
    C = m if capacity == 0 else int(capacity)
    if k and m > C:
        raise ValueError(f"prompt of length {m} does not fit a row of {C}")
    bins = ffd(lengths, C) if k else []
    off = _prefix(lengths)
    r = len(bins)
    row_seg_ptr = np.zeros(r + 1, dtype=np.int32)
    seg_prompt, seg_start, seg_len = [], [], []
    for b, items in enumerate(bins):
        col = 0
        for i in items:
            seg_prompt.append(i)
            seg_start.append(b * C + col)
            seg_len.append(int(lengths[i]))
            col += int(lengths[i])
        row_seg_ptr[b + 1] = row_seg_ptr[b] + len(items)
    T = r * C
    slot_seg = np.full(T, -1, dtype=np.int32)
    slot_pos = np.zeros(T, dtype=np.int32)
    slot_kv = np.full(T, -1, dtype=np.int32)
    for s in range(len(seg_prompt)):
        p, a, n = seg_prompt[s], seg_start[s], seg_len[s]
        for j in range(n):
            slot_seg[a + j] = s
            slot_pos[a + j] = j                 # restart positions
            slot_kv[a + j] = off[p] + j         # UNPACK target row
    return Plan(k=k, capacity=C, n_rows=r, max_len=m, total_len=int(off[-1]),
                row_seg_ptr=row_seg_ptr, seg_prompt=np.array(seg_prompt, dtype=np.int32),
                seg_start=np.array(seg_start, dtype=np.int32),
                seg_len=np.array(seg_len, dtype=np.int32), prompt_kv_off=off.astype(np.int32),
                slot_seg=slot_seg, slot_pos=slot_pos, slot_kv=slot_kv)


def pack_padded(lengths: Sequence[int]) -> Plan:
    """Full batching (section 4.2): prompt i alone in row i, right-padded to m.

    Row i is one causal span of length m starting at slot i*m; positions run
    0..m-1 over the whole row; only the first l_i slots carry a real token.
    """
    lengths = np.asarray(lengths, dtype=np.int64)
    k = len(lengths)
    if k:
        _check_lengths(lengths)
    m = int(lengths.max()) if k else 0
    off = _prefix(lengths)
    T = k * m
    slot_seg = np.zeros(T, dtype=np.int32)
    slot_pos = np.zeros(T, dtype=np.int32)
    slot_kv = np.full(T, -1, dtype=np.int32)
    for i in range(k):
        for j in range(m):
            slot_seg[i * m + j] = i
            slot_pos[i * m + j] = j
            if j < lengths[i]:
                slot_kv[i * m + j] = off[i] + j
    seg_len = np.full(k, m, dtype=np.int32)
    return Plan(k=k, capacity=m, n_rows=k, max_len=m, total_len=int(off[-1]),
                row_seg_ptr=np.arange(k + 1, dtype=np.int32),
                seg_prompt=np.arange(k, dtype=np.int32),
                seg_start=(np.arange(k, dtype=np.int64) * m).astype(np.int32),
                seg_len=seg_len, prompt_kv_off=off.astype(np.int32),
                slot_seg=slot_seg, slot_pos=slot_pos, slot_kv=slot_kv)


def independent_mask(plan: Plan, row: int) -> np.ndarray:
    """The literal M' of one row (section 3.2): boolean [C, C], True where attention is allowed."""
    C = plan.capacity
    M = np.zeros((C, C), dtype=bool)
    base = row * C
    for s in range(plan.row_seg_ptr[row], plan.row_seg_ptr[row + 1]):
        a = int(plan.seg_start[s]) - base
        b = a + int(plan.seg_len[s])
        M[a:b, a:b] = np.tril(np.ones((b - a, b - a), dtype=bool))
    return M


def row_fill(plan: Plan) -> np.ndarray:
    """Real tokens per row."""
    fill = np.zeros(plan.n_rows, dtype=np.int64)
    for t in range(plan.n_slots):
        if plan.slot_kv[t] >= 0:
            fill[t // plan.capacity] += 1
    return fill


def dosa_bound(opt: int) -> float:
    """Tight worst-case bound of FFD: FFD <= 11/9 OPT + 6/9 (Dosa 2007)."""
    return 11.0 * opt / 9.0 + 6.0 / 9.0


def lower_bound(lengths: Sequence[int], capacity: int) -> int:
    total = int(np.sum(lengths))
    return -(-total // capacity) if total else 0


def split_lengths(plan: Plan) -> Optional[np.ndarray]:
    """Prompt lengths recovered from the plan (for round-trip checks)."""
    return np.diff(plan.prompt_kv_off.astype(np.int64))
