"""Scores that cancel near zero: the tolerance |g - r| <= 1e-6 + 1e-5 |r| is then nearly
absolute, so the GPU's accumulation must stay far below 1e-6 although the leaf values are of
order 1. Each tree is paired with a copy whose leaf values are negated and nudged by ~1e-3, so a
document's score is a sum of nudges while the sum of |leaf value| is in the thousands (a float
sum of groups of four leaf values, the earlier accumulation, misses the tolerance here)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import workloads as W
from _gpu import assert_scores_close, dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def T():
    import paper_1212_2287_amd as T
    T.load_library()
    return T


def _cancelling_ensemble(n_pairs, n_features, seed):
    base = W.random_ensemble(seed, n_trees=n_pairs, n_features=n_features, min_leaves=2, max_leaves=24)
    rng = np.random.default_rng(seed)
    nudge = (rng.normal(0.0, 1e-3, base.value.shape[0])).astype(np.float32)
    mirror_value = np.where(base.feature < 0, -base.value + nudge, 0.0).astype(np.float32)
    n = base.feature.shape[0]
    offs = np.concatenate([base.tree_offsets, base.tree_offsets[1:] + n]).astype(np.int64)
    cat = lambda a, b: np.concatenate([a, b])
    ens = W.Ensemble(offs, cat(base.feature, base.feature), cat(base.threshold, base.threshold),
                     cat(base.left, base.left), cat(base.right, base.right), cat(base.value, mirror_value),
                     n_features)
    return ens


@pytest.mark.parametrize("n_pairs", [500, 1500])
def test_scores_cancelling_near_zero(T, n_pairs):
    import torch
    F = 24
    ens = _cancelling_ensemble(n_pairs, F, 77 + n_pairs)
    X = W.random_docs(78, 3000, F, zero_frac=0.1)
    ref, _, _ = oracle.score(ens, X, want_leaves=False)
    leaf_abs = np.abs(ens.value[ens.feature < 0]).mean() * ens.n_trees
    assert np.median(np.abs(ref)) < 0.1 and leaf_abs > 500  # cancelling scores, large leaf mass
    with T.TreeEnsemble.from_ensemble(ens) as m:
        s = m.predict(dev(X))
        torch.cuda.synchronize()
    assert_scores_close(s.cpu().numpy(), ref, f"{n_pairs} cancelling pairs")


def test_vector_outputs_cancelling_near_zero(T):
    import torch
    F = 24
    ens = _cancelling_ensemble(800, F, 91)
    vals = np.stack([ens.value, 0.5 * ens.value, -ens.value, 2.0 * ens.value, ens.value], axis=1)
    X = W.random_docs(92, 2000, F, zero_frac=0.1)
    ref = oracle.score_multi(ens, vals, X)
    with T.TreeEnsemble.from_ensemble(ens, leaf_values=vals) as m:
        s = m.predict(dev(X))
        torch.cuda.synchronize()
    assert_scores_close(s.cpu().numpy().astype(np.float64).ravel(), ref.ravel(), "vector, cancelling")
