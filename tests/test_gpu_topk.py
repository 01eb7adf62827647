"""GPU per-query top-k reranking through the C ABI, against oracle/topk.py on the same float32
scores (the order is decided on identical values, so indices must match exactly)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from oracle.topk import topk as oracle_topk
import workloads as W
from _gpu import assert_scores_close, dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def T():
    import paper_1212_2287_amd as T
    T.load_library()
    return T


def _gpu_topk(T, s, off, k):
    import torch
    idx, vals = T.tree_ens_topk(dev(np.asarray(s, np.float32)), dev(np.asarray(off, np.int64)), k)
    torch.cuda.synchronize()
    return idx.cpu().numpy(), vals.cpu().numpy()


def _check(T, s, off, k, what):
    idx, vals = _gpu_topk(T, s, off, k)
    ref_idx, ref_vals = oracle_topk(s, off, k)
    assert np.array_equal(idx, ref_idx), f"{what}: indices differ at " \
        f"{np.argwhere(idx != ref_idx)[:3].tolist()}"
    assert np.array_equal(vals, ref_vals, equal_nan=True), what


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("k", [1, 20, 64, 1024])
def test_random_groups_and_special_values(T, seed, k):
    rng = np.random.default_rng(seed)
    sizes = np.concatenate([[0, 1, k - 1 if k > 1 else 0, k, k + 1, 200, 5000],
                            rng.integers(0, 300, 40)])
    rng.shuffle(sizes)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    n = int(off[-1])
    if seed % 2:
        pool = np.array([0.0, -0.0, 1.0, -1.0, 2.5, np.inf, -np.inf, np.nan, 1e-45, -1e-45],
                        np.float32)
        s = rng.choice(pool, n)
    else:
        s = rng.standard_normal(n).astype(np.float32)
    _check(T, s, off, k, f"seed {seed} k {k}")


def test_all_equal_and_many_ties(T):
    # every score equal: the first k by index; and a group made of a few distinct values
    s = np.concatenate([np.full(3000, 1.5, np.float32),
                        np.repeat(np.array([3.0, -0.0, 0.0, np.nan], np.float32), 700)])
    off = np.array([0, 3000, len(s)], np.int64)
    for k in (1, 7, 700, 1024):
        _check(T, s, off, k, f"ties k {k}")


def test_ill_formed_offsets_are_clamped(T):
    s = np.random.default_rng(1).standard_normal(100).astype(np.float32)
    # each offset is clamped into [0, 100] on its own; a group ending before it starts is empty:
    # [0, 30), [30, 30), [20, 100), [100, 100)
    off = np.array([-5, 30, 20, 150, 80], np.int64)
    groups = [(0, 30), (30, 30), (20, 100), (100, 100)]
    idx, vals = _gpu_topk(T, s, off, 8)
    for g, (a, b) in enumerate(groups):
        ref_idx, ref_vals = oracle_topk(s, np.array([a, b], np.int64), 8)
        assert np.array_equal(idx[g], ref_idx[0]), g
        assert np.array_equal(vals[g], ref_vals[0], equal_nan=True), g


def test_argument_errors(T):
    import torch
    s = dev(np.zeros(10, np.float32))
    off = dev(np.array([0, 10], np.int64))
    for bad_k in (0, 1025):
        with pytest.raises(T.TreeEnsError) as ei:
            T.tree_ens_topk(s, off, bad_k)
        assert ei.value.code == T.TREE_ENS_E_ARG
    empty = dev(np.zeros(1, np.int64))  # zero groups: no launch
    idx, vals = T.tree_ens_topk(s, empty, 5)
    torch.cuda.synchronize()
    assert idx.shape == (0, 5)


def test_predict_topk_on_ranking_workload(T):
    """Scoring and reranking of the ranking-shaped workload's query groups (20-200 candidates per
    query, the best 20 kept), in one call."""
    import torch
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg)
    sizes = W.make_query_groups(cfg)
    off = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)
    with T.TreeEnsemble.from_ensemble(ens) as m:
        scores, idx, vals = m.predict_topk(dev(X), dev(off), 20)
        torch.cuda.synchronize()
        scores, idx, vals = scores.cpu().numpy(), idx.cpu().numpy(), vals.cpu().numpy()
    ref, _, _ = oracle.score(ens, X, want_leaves=False)
    assert_scores_close(scores, ref, "rank_1kx32 scores")
    ref_idx, ref_vals = oracle_topk(scores, off, 20)
    assert np.array_equal(idx, ref_idx)
    assert np.array_equal(vals, ref_vals, equal_nan=True)
