"""Pins of the top-k reranking oracle (oracle/topk.py) on the CPU: numpy's lexsort, a counting
brute force, special values and invariants."""
from __future__ import annotations

import numpy as np
import pytest

from oracle.topk import topk


def _lexsort_topk(s, off, k):
    """Reference by a different route: numpy's lexsort per group (NaN flag, then -score, then
    index as the keys, last key primary)."""
    n_groups = len(off) - 1
    idx = np.full((n_groups, k), -1, np.int32)
    for g in range(n_groups):
        a, b = off[g], off[g + 1]
        seg = s[a:b].astype(np.float64)
        nan = np.isnan(seg)
        neg = np.where(nan, 0.0, -seg)
        order = np.lexsort((np.arange(a, b), neg, nan))
        top = np.arange(a, b)[order][:k]
        idx[g, :len(top)] = top
    return idx


def _count_rank_topk(s, off, k):
    """Brute force: the rank of document i in its group is the number of members that precede it
    (higher score; or equal score and lower index; NaN after numbers)."""
    n_groups = len(off) - 1
    idx = np.full((n_groups, k), -1, np.int32)
    for g in range(n_groups):
        a, b = off[g], off[g + 1]
        for i in range(a, b):
            rank = 0
            for j in range(a, b):
                si, sj = s[i], s[j]
                if np.isnan(sj):
                    before = np.isnan(si) and j < i
                elif np.isnan(si):
                    before = True
                else:
                    before = sj > si or (sj == si and j < i)
                rank += before
            if rank < k:
                idx[g, rank] = i
    return idx


def _random_case(seed, n_groups, max_size, pool=None):
    rng = np.random.default_rng(seed)
    sizes = rng.integers(0, max_size + 1, n_groups)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    n = int(off[-1])
    s = rng.standard_normal(n).astype(np.float32) if pool is None else \
        rng.choice(np.asarray(pool, np.float32), n)
    return s, off


@pytest.mark.parametrize("seed", range(8))
def test_matches_lexsort_and_brute_force(seed):
    pool = None if seed % 2 == 0 else [0.0, -0.0, 1.0, -1.0, 2.5, np.inf, -np.inf, np.nan, 1e-45]
    s, off = _random_case(seed, n_groups=25, max_size=40, pool=pool)
    for k in (1, 3, 20, 64):
        idx, vals = topk(s, off, k)
        assert np.array_equal(idx, _lexsort_topk(s, off, k))
        assert np.array_equal(idx, _count_rank_topk(s, off, k))
        got = np.where(idx >= 0, s[np.maximum(idx, 0)], np.nan)
        assert np.array_equal(got, vals, equal_nan=True)


def test_hand_worked_group():
    # scores of docs 0..6; expected order: 3.0 (doc 5), then the 2.0 tie (docs 1, 4 by index),
    # then +-0.0 tie (docs 0, 6; -0.0 equals +0.0), then -inf (doc 2), then NaN (doc 3)
    s = np.array([0.0, 2.0, -np.inf, np.nan, 2.0, 3.0, -0.0], np.float32)
    off = np.array([0, 7], np.int64)
    idx, vals = topk(s, off, 7)
    assert idx.tolist() == [[5, 1, 4, 0, 6, 2, 3]]
    idx3, vals3 = topk(s, off, 3)
    assert idx3.tolist() == [[5, 1, 4]] and vals3.tolist() == [[3.0, 2.0, 2.0]]


def test_padding_and_empty_groups():
    s = np.array([1.0, 5.0, 3.0], np.float32)
    off = np.array([0, 0, 2, 3, 3], np.int64)  # empty, {0,1}, {2}, empty
    idx, vals = topk(s, off, 3)
    assert idx.tolist() == [[-1, -1, -1], [1, 0, -1], [2, -1, -1], [-1, -1, -1]]
    assert np.isnan(vals[0]).all() and vals[1, :2].tolist() == [5.0, 1.0] and np.isnan(vals[1, 2])


def test_invariants():
    s, off = _random_case(11, n_groups=12, max_size=60)
    k = 10
    idx, vals = topk(s, off, k)
    # a permutation of the documents inside each group leaves the selected scores unchanged
    rng = np.random.default_rng(3)
    perm = np.arange(len(s))
    for g in range(len(off) - 1):
        a, b = off[g], off[g + 1]
        perm[a:b] = a + rng.permutation(b - a)
    _, vals_p = topk(s[perm], off, k)
    assert np.array_equal(vals, vals_p, equal_nan=True)
    # scaling by 2 (exact) keeps the order; negating reverses it (for distinct scores)
    assert np.array_equal(topk(s * np.float32(2), off, k)[0], idx)
    full, _ = topk(s, off, 64)
    rev, _ = topk(-s, off, 64)
    for g in range(len(off) - 1):
        n = off[g + 1] - off[g]
        assert full[g, :n].tolist() == rev[g, :n][::-1].tolist()
    # k >= group size: every member exactly once
    for g in range(len(off) - 1):
        n = off[g + 1] - off[g]
        assert sorted(full[g, :n].tolist()) == list(range(off[g], off[g + 1]))


def test_rejects_k_below_one():
    with pytest.raises(ValueError):
        topk(np.zeros(3, np.float32), np.array([0, 3]), 0)


@pytest.mark.parametrize("mutant", ["ties_by_higher_index", "nan_first", "signed_zero_ordered",
                                    "ascending"])
def test_pins_reject_plausible_mistakes(monkeypatch, mutant):
    """A plausible mistake in the oracle's order must be caught by the lexsort pin."""
    import math
    import oracle.topk as ot

    def key(score, index):
        if mutant == "nan_first" and math.isnan(score):
            return (-1, 0.0, index)
        if math.isnan(score):
            return (1, 0.0, index)
        if mutant == "ties_by_higher_index":
            return (0, -score, -index)
        if mutant == "signed_zero_ordered":
            return (0, -score, -math.copysign(1.0, score), index)
        if mutant == "ascending":
            return (0, score, index)
        return (0, -score, index)

    monkeypatch.setattr(ot, "sort_key", key)
    s, off = _random_case(5, n_groups=30, max_size=30,
                          pool=[0.0, -0.0, 1.0, 2.0, np.nan, -np.inf, 7.0])
    idx, _ = ot.topk(s, off, 8)
    assert not np.array_equal(idx, _lexsort_topk(s, off, 8)), mutant
