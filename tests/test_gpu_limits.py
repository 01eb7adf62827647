"""Maximum sizes on the GPU: every document-block width the LDS plans choose (64, 32, 16 and 8
documents per block, float and threshold-coded rows) up to the largest feature id accepted,
and the largest single tree one LDS tile holds, against the oracle (scores within tolerance,
leaf ids bit-exact)."""
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


def _check(T, ens, X, what, expect_dl=None, expect_coded=None):
    import torch
    with T.TreeEnsemble.from_ensemble(ens) as m:
        info = m.info()
        if expect_dl is not None:
            assert info["docs_per_block"] == expect_dl, (what, info)
        x = dev(X)
        s = m.predict(x)
        ids = m.predict_leaves(x)
        torch.cuda.synchronize()
        s, ids = s.cpu().numpy(), ids.cpu().numpy()
    ref, ref_ids, _ = oracle.score(ens, X)
    assert_scores_close(s, ref, what)
    assert_leaves_equal(ids, ref_ids, what)


def _wide(seed, n_cols, n_trees, max_leaves):
    ens = W.random_ensemble(seed, n_trees=n_trees, n_features=n_cols, min_leaves=2, max_leaves=max_leaves)
    # make sure the last column is read
    internal = np.nonzero(ens.feature >= 0)[0]
    ens.feature[internal[0]] = n_cols - 1
    return ens


# (columns the model reads, documents per block the plan must pick)
@pytest.mark.parametrize("n_cols,dl", [(383, 64), (384, 32), (767, 32), (768, 16), (1535, 16),
                                       (1536, 8), (3071, 8)])
def test_block_widths_up_to_the_largest_feature_id(T, n_cols, dl):
    ens = _wide(n_cols, n_cols, n_trees=40, max_leaves=12)
    X = W.random_docs(n_cols, 700, n_cols, zero_frac=0.3)
    _check(T, ens, X, f"{n_cols} columns", expect_dl=dl)


@pytest.mark.parametrize("n_cols,dl", [(800, 32), (1600, 16), (3071, 16)])
def test_coded_rows_for_wide_features_and_large_trees(T, n_cols, dl):
    # trees too large for the float blocks switch the plan to 16-bit codes (twice the
    # documents per block)
    ens = _wide(7 + n_cols, n_cols, n_trees=30, max_leaves=400)
    X = W.random_docs(n_cols, 500, n_cols, zero_frac=0.3)
    _check(T, ens, X, f"{n_cols} columns, coded", expect_dl=dl)


def test_largest_tree_one_tile_holds(T):
    # 2,923 leaves (5,845 nodes) is the largest tree accepted at 136 features; one more leaf
    # is refused at create
    ens = W.random_ensemble(1, n_trees=1, n_features=136, min_leaves=2923, max_leaves=2923)
    X = W.make_docs(W.WORKLOADS["rank_1kx32"], n_docs=3000)
    _check(T, ens, X, "largest tree")
    big = W.random_ensemble(1, n_trees=1, n_features=136, min_leaves=2924, max_leaves=2924)
    with pytest.raises(T.TreeEnsError) as ei:
        T.TreeEnsemble.from_ensemble(big)
    assert ei.value.code == T.TREE_ENS_E_MODEL
