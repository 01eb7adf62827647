"""Seeded random models across every LDS plan the packer chooses (64, 32, 16 and 8 documents per
block, two-workgroup and one-workgroup plans, narrow and wide records, float and threshold-coded
documents, 1, 2 or 4 trees per lane, complete-depth tiles), with IEEE corner values in the
thresholds and documents, both tie rules, vector-valued leaves and bags: scores, leaf ids and the
feature trace against the oracle. (This sweep found the whole-chunk slot and the accumulation
issues that tests/test_gpu_limits.py and tests/test_gpu_accuracy.py now pin.)"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import workloads as W
from _gpu import assert_leaves_equal, assert_scores_close, dev

pytestmark = pytest.mark.gpu

_POOL = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf, np.nan, 1e-45, 3.4e38, -1.5],
                 np.float32)


@pytest.fixture(scope="module")
def T():
    import paper_1212_2287_amd as T
    T.load_library()
    return T


def _case(seed):
    rng = np.random.default_rng(1000 + seed)
    F = int(rng.choice([1, 5, 40, 136, 137, 300, 700, 1100, 1500, 2500, 3000]))
    n_trees = int(rng.integers(1, 400))
    max_leaves = int(rng.choice([1, 2, 8, 32, 64, 200]))
    pooled = bool(rng.random() < 0.3)
    rule = int(rng.integers(0, 2))
    ens = W.random_ensemble(5000 + seed, n_trees=n_trees, n_features=F, min_leaves=1,
                            max_leaves=max_leaves, thr_values=_POOL[:8] if pooled else None)
    n_docs = int(rng.choice([1, 7, 63, 64, 65, 500, 3000, 20000]))
    X = W.random_docs(5000 + seed, n_docs, F, values=_POOL if pooled else None,
                      zero_frac=float(rng.random() * 0.6))
    n_out = int(rng.choice([1, 1, 1, 3, 6]))
    vals = None if n_out == 1 else W.make_leaf_vectors(ens, n_out, "dense", seed=seed)
    n_bags = int(rng.integers(1, 3))
    return ens, X, rule, vals, n_bags


@pytest.mark.parametrize("seed", range(60))
def test_random_plan(T, seed):
    import torch
    ens, X, rule, vals, n_bags = _case(seed)
    what = f"seed {seed}: {ens.n_trees} trees, {X.shape[1]} features, {X.shape[0]} docs, rule {rule}"
    flags = T.TREE_ENS_RIGHT_IF_GT if rule else T.TREE_ENS_RIGHT_IF_GE
    with T.TreeEnsemble.from_ensemble(ens, flags, leaf_values=vals, n_bags=n_bags) as m:
        x = dev(X)
        s = m.predict(x)
        ids = m.predict_leaves(x)
        cnt, masks = m.feature_usage(x)
        torch.cuda.synchronize()
        s, ids = s.cpu().numpy().astype(np.float64), ids.cpu().numpy()
        cnt, masks = cnt.cpu().numpy(), masks.cpu().numpy().view(np.uint32)
    if vals is None:
        ref, ref_ids, _ = oracle.score(ens, X, rule=rule)
        ref = ref / n_bags
    else:
        _, ref_ids, _ = oracle.score(ens, X, rule=rule)
        ref = oracle.score_multi(ens, vals, X, n_bags=n_bags, rule=rule)
    assert_scores_close(s.ravel(), ref.ravel(), what)
    assert_leaves_equal(ids, ref_ids, what)
    ref_cnt, ref_masks = oracle.feature_usage(ens, X, rule=rule)
    assert np.array_equal(cnt, ref_cnt) and np.array_equal(masks, ref_masks), what + ": trace"
