"""Maximum sizes on the GPU: every document-block width the LDS plans choose (64, 32, 16 and 8
documents per block, float and threshold-coded rows) up to the largest feature id accepted,
the largest single tree one LDS tile holds and the smallest one it does not, against the oracle (scores within tolerance,
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
    # 2,923 leaves (5,845 nodes) is the largest tree one tile holds at 136 features (it is
    # tiled); one more leaf makes it a big tree, walked from device memory
    ens = W.random_ensemble(1, n_trees=1, n_features=136, min_leaves=2923, max_leaves=2923)
    X = W.make_docs(W.WORKLOADS["rank_1kx32"], n_docs=3000)
    with T.TreeEnsemble.from_ensemble(ens) as m:
        assert m.info()["n_tiles"] == 1
    _check(T, ens, X, "largest tiled tree")
    big = W.random_ensemble(1, n_trees=1, n_features=136, min_leaves=2924, max_leaves=2924)
    with T.TreeEnsemble.from_ensemble(big) as m:
        assert m.info()["n_tiles"] == 0
    _check(T, big, X, "smallest big tree")


# (features, leaves per tree at most, documents per block): float plans with 4, 2 and 1 trees
# per lane and two threshold-coded plans (the emulator test pins each plan's shape)
@pytest.mark.parametrize("n_features,max_leaves,dl", [(380, 100, 64), (760, 100, 32), (3000, 40, 8),
                                                      (1530, 200, 32), (3000, 200, 16)])
def test_slots_of_whole_chunks(T, n_features, max_leaves, dl):
    """Near the top of each block-width band the document tile and the trace's bitmasks leave
    less than 64 KiB for the tile slot of one-workgroup plans, which the packer sizes to whole
    1,024-record chunks (the unit a window is copied in); large trees fill the last chunk (the
    emulator test pins each plan). A batch of more blocks than the GPU holds at once runs whole
    blocks at tiling 0: scores, leaf ids and the feature trace (whose bitmasks follow the slot,
    as the zero record of idle tree slots does) against the oracle, under the strict rule."""
    import torch
    pool = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf], np.float32)
    ens = W.random_ensemble(5066, n_trees=160, n_features=n_features, min_leaves=1,
                            max_leaves=max_leaves, thr_values=pool)
    n_docs = 300 * dl  # 300 blocks: more than the 256 resident workgroups
    X = W.random_docs(5066, n_docs, n_features, values=np.append(pool, np.nan).astype(np.float32),
                      zero_frac=0.2)
    with T.TreeEnsemble.from_ensemble(ens, T.TREE_ENS_RIGHT_IF_GT) as m:
        assert m.info()["docs_per_block"] == dl
        x = dev(X)
        s = m.predict(x)
        ids = m.predict_leaves(x)
        cnt, masks = m.feature_usage(x)
        torch.cuda.synchronize()
        s, ids = s.cpu().numpy(), ids.cpu().numpy()
        cnt, masks = cnt.cpu().numpy(), masks.cpu().numpy().view(np.uint32)
    ref, ref_ids, _ = oracle.score(ens, X, rule=1)
    assert_scores_close(s, ref, f"{n_features} features")
    assert_leaves_equal(ids, ref_ids, f"{n_features} features")
    ref_cnt, ref_masks = oracle.feature_usage(ens, X, rule=1)
    assert np.array_equal(masks, ref_masks) and np.array_equal(cnt, ref_cnt), f"{n_features} features: trace"
