"""The model-specialised kernel (TREE_ENS_CODEGEN, compiled with hiprtc at create time) on the
GPU through the C ABI, against the oracle: |g - r| <= 1e-6 + 1e-5 |r| per document (the
hand-worked ensemble exactly)."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import workloads as W
from _golden import load_hand_ensemble
from _gpu import assert_leaves_equal, assert_scores_close, dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def T():
    import paper_1212_2287_amd as T
    T.load_library()
    return T


def _gpu(T, ens, X, flags=0, n_bags=1):
    import torch
    flags |= T.TREE_ENS_CODEGEN
    if n_bags == 1:
        h = T.tree_ens_create(ens.tree_offsets, ens.feature, ens.threshold, ens.left, ens.right, ens.value, flags)
    else:
        h = T.tree_ens_create_multi(ens.tree_offsets, ens.feature, ens.threshold, ens.left, ens.right,
                                    ens.value, 1, n_bags, flags)
    with T.TreeEnsemble(h) as m:
        s = m.predict(dev(X))
        torch.cuda.synchronize()
        return s.cpu().numpy()


@pytest.mark.parametrize("rule,name", [(0, "ge"), (1, "gt")])
def test_hand_ensemble_exact(T, rule, name):
    ens, X, expects = load_hand_ensemble()
    got = _gpu(T, ens, X, T.TREE_ENS_RIGHT_IF_GT if rule else T.TREE_ENS_RIGHT_IF_GE)
    assert got.tolist() == [e[1] for e in expects[name]]


@pytest.mark.parametrize("wl,n_trees,n_docs", [("tiny_10x8", None, None), ("rank_1kx32", 150, 20000), ("wide_1kx64_f700", 40, 5000),
                                                   ("shallow_20kx8_1M", 300, 100000)])
def test_workload_prefixes(T, wl, n_trees, n_docs):
    cfg = W.WORKLOADS[wl]
    ens = W.make_ensemble(cfg, n_trees=n_trees)
    X = W.make_docs(cfg, n_docs=n_docs)
    ref, _, _ = oracle.score(ens, X, want_leaves=False)
    assert_scores_close(_gpu(T, ens, X), ref, f"{wl} prefix")


_POOL = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf, np.nan, 1e-45], dtype=np.float32)


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("n_docs", [1, 255, 257, 3000])
def test_random_ensembles_corner_values(T, seed, n_docs):
    rule = seed % 2
    ens = W.random_ensemble(seed, n_trees=50, n_features=20, min_leaves=1, max_leaves=40,
                            thr_values=_POOL[:8] if seed < 2 else None)
    X = W.random_docs(seed, n_docs, 20, values=_POOL if seed < 2 else None, zero_frac=0.2)
    flags = T.TREE_ENS_RIGHT_IF_GT if rule else T.TREE_ENS_RIGHT_IF_GE
    ref, _, _ = oracle.score(ens, X, rule=rule, want_leaves=False)
    assert_scores_close(_gpu(T, ens, X, flags), ref, f"seed {seed}")
    assert_scores_close(_gpu(T, ens, X, flags, n_bags=3), ref / 3, f"seed {seed}, 3 bags")


def test_other_entry_points_keep_the_generic_kernels(T):
    import torch
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg, n_trees=60)
    X = W.make_docs(cfg, n_docs=900)
    h = T.tree_ens_create(ens.tree_offsets, ens.feature, ens.threshold, ens.left, ens.right, ens.value,
                          T.TREE_ENS_CODEGEN)
    with T.TreeEnsemble(h) as m:
        x = dev(X)
        ids = m.predict_leaves(x)
        c, _ = m.feature_usage(x)
        torch.cuda.synchronize()
        assert_leaves_equal(ids.cpu().numpy(), oracle.score(ens, X)[1], "codegen model leaves")
        assert np.array_equal(c.cpu().numpy(), oracle.feature_usage(ens, X)[0])
