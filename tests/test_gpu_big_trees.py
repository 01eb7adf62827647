"""Trees too large for one LDS tile (up to the 65,535-node limit: 32,768 leaves), walked from
device memory by the scoring kernel: 8,192- and 32,768-leaf trees at 136 and 700 features,
alone and next to tiled trees, float and threshold-coded documents, both tie rules, small
(split) and large (whole-block) batches; leaf ids bit-exact and scores within the tolerance
against the oracle, plus the feature trace and vector-valued leaves."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import workloads as W
from _gpu import assert_leaves_equal, assert_scores_close, dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def T():
    import paper_1212_2287_amd as T
    T.load_library()
    return T


def _stack(parts, n_feat, seed):
    trees = [e.tree(t) for e in parts for t in range(e.n_trees)]
    order = np.random.default_rng(seed).permutation(len(trees))
    trees = [trees[i] for i in order]
    offs = np.cumsum([0] + [len(t[0]) for t in trees]).astype(np.int64)
    cat = [np.concatenate([np.asarray(t[k], dt) for t in trees]) for k, dt in
           enumerate((np.int32, np.float32, np.int32, np.int32, np.float32))]
    return W.Ensemble(offs, *cat, n_feat)


def _model(n_feat, big_leaves, n_small, small_leaves=40, seed=0, thr_values=None):
    parts = []
    if n_small:
        parts.append(W.random_ensemble(seed + 500, n_trees=n_small, n_features=n_feat, min_leaves=1,
                                       max_leaves=small_leaves, thr_values=thr_values))
    for i, L in enumerate(big_leaves):
        parts.append(W.random_ensemble(seed + 600 + i, n_trees=1, n_features=n_feat, min_leaves=L,
                                       max_leaves=L, thr_values=thr_values))
    return _stack(parts, n_feat, seed)


def _check(T, ens, X, what, flags=0, expect_tiles=None):
    import torch
    with T.TreeEnsemble.from_ensemble(ens, flags) as m:
        if expect_tiles is not None:
            assert (m.info()["n_tiles"] > 0) == expect_tiles, (what, m.info())
        x = dev(X)
        s = m.predict(x)
        ids = m.predict_leaves(x)
        torch.cuda.synchronize()
        s, ids = s.cpu().numpy(), ids.cpu().numpy()
    ref, ref_ids, _ = oracle.score(ens, X, rule=flags)
    assert_scores_close(s, ref, what)
    assert_leaves_equal(ids, ref_ids, what)


@pytest.mark.parametrize("n_feat", [136, 700])
@pytest.mark.parametrize("big_leaves", [8192, 32768])
def test_one_big_tree(T, n_feat, big_leaves):
    print(f"[big] {big_leaves} leaves alone, {n_feat} features", flush=True)
    ens = _model(n_feat, [big_leaves], 0, seed=big_leaves + n_feat)
    X = W.random_docs(n_feat + big_leaves, 5000, n_feat, zero_frac=0.2)
    _check(T, ens, X, f"{big_leaves} leaves, {n_feat} features", expect_tiles=False)


@pytest.mark.parametrize("n_feat,n_docs", [(136, 3000), (136, 70000), (700, 2000), (700, 40000)])
def test_big_trees_next_to_tiled_trees(T, n_feat, n_docs):
    print(f"[big] mixed model, {n_feat} features, {n_docs} docs", flush=True)
    ens = _model(n_feat, [8192, 32768, 3000], 200, seed=n_feat)
    X = W.random_docs(n_feat, n_docs, n_feat, zero_frac=0.3)
    for flags in (0, 1):
        _check(T, ens, X, f"mixed, {n_feat} features, {n_docs} docs, rule {flags}", flags,
               expect_tiles=True)


def test_big_trees_with_threshold_codes_and_ties(T):
    """A model whose tiled trees make the 700-feature plan code its documents (16-bit codes in
    LDS), plus big trees; thresholds from a small pool, so documents tie with them often."""
    import torch
    pool = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf], np.float32)
    ens = _model(700, [8192, 20000], 300, small_leaves=400, seed=3, thr_values=pool)
    X = W.random_docs(3, 3000, 700, values=np.append(pool, np.nan).astype(np.float32), zero_frac=0.2)
    for flags in (0, 1):
        _check(T, ens, X, f"coded, rule {flags}", flags, expect_tiles=True)
    with T.TreeEnsemble.from_ensemble(ens) as m:
        cnt, masks = m.feature_usage(dev(X))
        torch.cuda.synchronize()
        cnt, masks = cnt.cpu().numpy(), masks.cpu().numpy().view(np.uint32)
    ref_cnt, ref_masks = oracle.feature_usage(ens, X)
    assert np.array_equal(cnt, ref_cnt) and np.array_equal(masks, ref_masks)


def test_big_trees_feature_trace_and_vector_leaves(T):
    import torch
    ens = _model(136, [8192, 4000], 100, seed=9)
    X = W.random_docs(9, 4000, 136, zero_frac=0.1)
    with T.TreeEnsemble.from_ensemble(ens) as m:
        cnt, masks = m.feature_usage(dev(X))
        torch.cuda.synchronize()
        cnt, masks = cnt.cpu().numpy(), masks.cpu().numpy().view(np.uint32)
    ref_cnt, ref_masks = oracle.feature_usage(ens, X)
    assert np.array_equal(cnt, ref_cnt) and np.array_equal(masks, ref_masks)
    vals = W.make_leaf_vectors(ens, 6, "dense", seed=4)
    with T.TreeEnsemble.from_ensemble(ens, leaf_values=vals, n_bags=2) as m:
        s = m.predict(dev(X))
        torch.cuda.synchronize()
        s = s.cpu().numpy()
    ref = oracle.score_multi(ens, vals, X, n_bags=2)
    assert_scores_close(s, ref, "vector leaves with big trees")
