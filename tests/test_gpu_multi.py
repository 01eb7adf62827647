"""GPU vector-valued leaves and bagged ensembles (tree_ens_create_multi) through the C ABI
against the oracle's oracle_score_multi: every output within |g - r| <= 1e-6 + 1e-5 |r| of the
fp64 oracle, leaf ids bit-exact."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import workloads as W
from _golden import load_hand_ensemble
from _gpu import assert_leaves_equal, assert_scores_close, dev

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def T():
    import paper_1212_2287_amd as T
    T.load_library()
    return T


def _gpu(T, ens, vals, X, n_bags=1, flags=0):
    import torch
    with T.TreeEnsemble.from_ensemble(ens, flags, leaf_values=vals, n_bags=n_bags) as m:
        s = m.predict(dev(X))
        torch.cuda.synchronize()
        return s.cpu().numpy()


def _close(got, ref, what):
    got = np.asarray(got, np.float64).reshape(ref.shape)
    assert_scores_close(got.ravel(), ref.ravel(), what)


@pytest.mark.parametrize("rule,name", [(0, "ge"), (1, "gt")])
@pytest.mark.parametrize("n_bags", [1, 2, 3])
def test_golden_hand_ensemble(T, rule, name, n_bags):
    ens, X, expects = load_hand_ensemble()
    s = np.array([e[1] for e in expects[name]])
    leaf = ens.feature < 0
    vals = np.zeros((ens.n_nodes, 3), np.float32)
    vals[leaf, 0] = ens.value[leaf]
    vals[leaf, 1] = 2 * ens.value[leaf] + 1
    vals[leaf, 2] = -ens.value[leaf]
    flags = T.TREE_ENS_RIGHT_IF_GT if rule else T.TREE_ENS_RIGHT_IF_GE
    got = _gpu(T, ens, vals, X, n_bags, flags)
    _close(got, np.stack([s, 2 * s + 3, -s], axis=1) / n_bags, f"golden {name} bags {n_bags}")


@pytest.mark.parametrize("wl,n_out,kind", [("tiny_10x8", 3, "probs"), ("rank_1kx32", 5, "dense"), ("rank_1kx32", 4, "class"),
                                               ("wide_1kx64_f700", 6, "dense")])
def test_workloads_full(T, wl, n_out, kind):
    cfg = W.WORKLOADS[wl]
    _say(f"[multi] {wl}: {n_out} outputs ({kind}), {cfg.n_docs} docs")
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg)
    vals = W.make_leaf_vectors(ens, n_out, kind, seed=cfg.seed_key)
    got = _gpu(T, ens, vals, X)
    assert got.shape == (cfg.n_docs, n_out)
    _close(got, oracle.score_multi(ens, vals, X), f"{wl} {kind}")


@pytest.mark.parametrize("wl,n_out", [("shallow_20kx8_1M", 6), ("large_5kx256_f700_1M", 2)])
def test_workload_1M_sampled(T, wl, n_out):
    import torch
    cfg = W.WORKLOADS[wl]
    _say(f"[multi] {wl} at full size, {n_out} outputs: generating")
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg)
    vals = W.make_leaf_vectors(ens, n_out, "dense", sigma=0.01, seed=cfg.seed_key)
    sample = np.sort(np.random.default_rng(20 + cfg.seed_key).choice(cfg.n_docs, size=2048, replace=False))
    _say(f"[multi] {wl}: scoring {cfg.n_docs} docs on the GPU")
    with T.TreeEnsemble.from_ensemble(ens, leaf_values=vals) as m:
        s = m.predict(dev(X))
        torch.cuda.synchronize()
        s = s.cpu().numpy()
    _say(f"[multi] {wl}: oracle on {sample.size} sampled docs")
    _close(s[sample], oracle.score_multi(ens, vals, X[sample]), f"{wl} sample")


@pytest.mark.parametrize("n_docs", [1, 63, 65, 4097, 67331])
def test_ragged_batches_and_splits(T, n_docs):
    # small batches split blocks over workgroups: four partial sums per document and launch,
    # reduced into the right columns (5 outputs: two launches, the second one partial)
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg, n_trees=300)
    X = W.make_docs(cfg, n_docs=n_docs)
    vals = W.make_leaf_vectors(ens, 5, "dense", seed=7)
    _close(_gpu(T, ens, vals, X, n_bags=3), oracle.score_multi(ens, vals, X, n_bags=3),
           f"{n_docs} docs")


@pytest.mark.parametrize("n_docs", [65, 5000])
def test_coded_documents(T, n_docs):
    cfg = W.WORKLOADS["large_5kx256_f700_1M"]
    ens = W.make_ensemble(cfg, n_trees=80)
    X = W.make_docs(cfg, n_docs=n_docs)
    vals = W.make_leaf_vectors(ens, 9, "probs", seed=2)
    with T.TreeEnsemble.from_ensemble(ens, leaf_values=vals) as m:
        assert m.info()["docs_per_block"] == 64
    _close(_gpu(T, ens, vals, X), oracle.score_multi(ens, vals, X), "coded")


def test_bagging_scalar(T):
    import torch
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg, n_trees=400)
    X = W.make_docs(cfg, n_docs=3000)
    for b in (3, 7):
        got = _gpu(T, ens, None, X, n_bags=b)
        assert got.shape == (3000,)
        _close(got, oracle.score(ens, X, want_leaves=False)[0] / b, f"{b} bags")
    # four bags: an exact power-of-two scaling of the unbagged GPU scores
    with T.TreeEnsemble.from_ensemble(ens) as m1, T.TreeEnsemble.from_ensemble(ens, n_bags=4) as m4:
        x = dev(X)
        s1, s4 = m1.predict(x), m4.predict(x)
        torch.cuda.synchronize()
        assert np.array_equal(s4.cpu().numpy(), s1.cpu().numpy() * np.float32(0.25))


def test_leaves_and_usage_of_a_vector_model(T):
    import torch
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg, n_trees=100)
    X = W.make_docs(cfg, n_docs=700)
    vals = W.make_leaf_vectors(ens, 3, "dense", seed=1)
    with T.TreeEnsemble.from_ensemble(ens, leaf_values=vals) as m:
        ids = m.predict_leaves(dev(X))
        c, _ = m.feature_usage(dev(X))
        torch.cuda.synchronize()
        assert_leaves_equal(ids.cpu().numpy(), oracle.score(ens, X)[1], "vector model leaves")
        assert np.array_equal(c.cpu().numpy(), oracle.feature_usage(ens, X)[0])


def test_empty_model_and_errors(T):
    import torch
    F = 8
    X = W.random_docs(1, 50, F)
    empty = W.Ensemble(np.zeros(1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.float32),
                       np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32), F)
    with T.TreeEnsemble.from_ensemble(empty, leaf_values=np.zeros((0, 3), np.float32)) as m:
        s = m.predict(dev(X))
        torch.cuda.synchronize()
        assert s.shape == (50, 3) and not s.cpu().numpy().any()
    ens, Xh, _ = load_hand_ensemble()
    vals = np.ones((ens.n_nodes, 2), np.float32)
    for n_out, n_bags in ((0, 1), (257, 1), (2, 0)):
        with pytest.raises(T.TreeEnsError) as ei:
            T.tree_ens_create_multi(ens.tree_offsets, ens.feature, ens.threshold, ens.left, ens.right,
                                    np.ones(ens.n_nodes * max(n_out, 1), np.float32), n_out, n_bags)
        assert ei.value.code == T.TREE_ENS_E_ARG
    with T.TreeEnsemble.from_ensemble(ens, leaf_values=vals) as m:
        assert (m.n_outputs, m.n_bags) == (2, 1)
        with pytest.raises(T.TreeEnsError) as ei:
            m.predict_topk(dev(Xh), dev(np.array([0, 7], np.int64)), 3)
        assert ei.value.code == T.TREE_ENS_E_ARG
