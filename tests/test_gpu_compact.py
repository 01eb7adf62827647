"""Compact packets on the GPU: coded 64-document plans whose trees have at most 511 nodes (the
700-feature workload's shape) walk 4-byte records, two trees per lane, reading each children
pair whole, with leaf payloads in device memory. Leaf ids bit-exact and scores within the
tolerance against the oracle, for batch sizes that take every launch shape (a single document,
split tails, whole-block heads), both tie rules, models mixed with small and single-leaf trees
(idle slots in the last group), vector-valued leaves, repeat calls bitwise equal, and a seeded
sweep of 24 random models of that shape with IEEE corner values and bags. The CPU
emulator (tests/test_pack_emu.py) pins that these models get compact packets and walks them
with the kernel's addressing."""
from __future__ import annotations

import numpy as np
import pytest

import _compact_cases as CC
import oracle
import workloads as W
from _gpu import assert_leaves_equal, assert_scores_close, dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def T():
    import paper_1212_2287_amd as T
    T.load_library()
    return T


def _run(T, ens, X, flags=0):
    import torch
    with T.TreeEnsemble.from_ensemble(ens, flags) as m:
        x = dev(X)
        s = m.predict(x)
        ids = m.predict_leaves(x)
        s2 = m.predict(x)
        torch.cuda.synchronize()
        return s.cpu().numpy(), ids.cpu().numpy(), s2.cpu().numpy()


def _check(T, ens, X, what, flags=0):
    print(what, flush=True)
    s, ids, s2 = _run(T, ens, X, flags)
    ref, ref_ids, _ = oracle.score(ens, X, rule=flags)
    assert_scores_close(s, ref, what)
    assert_leaves_equal(ids, ref_ids, what)
    assert np.array_equal(s.view(np.uint32), s2.view(np.uint32)), f"{what}: repeat call differs"


@pytest.mark.parametrize("n_docs", [1, 65, 3000, 40000])
def test_large_workload_prefix(T, n_docs):
    cfg = W.WORKLOADS["large_5kx256_f700_1M"]
    ens = W.make_ensemble(cfg, n_trees=300)
    X = W.make_docs(cfg, n_docs=n_docs)
    for flags in (0, 1):
        _check(T, ens, X, f"large prefix, {n_docs} docs, rule {flags}", flags)


def _mixed(seed):
    rng = np.random.default_rng(900 + seed)
    pool = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf], np.float32)
    big = W.random_ensemble(900 + seed, n_trees=int(rng.integers(20, 120)), n_features=700, min_leaves=150,
                            max_leaves=256, thr_values=pool if seed % 2 == 0 else None)
    small = W.random_ensemble(950 + seed, n_trees=int(rng.integers(1, 9)), n_features=700, min_leaves=1,
                              max_leaves=int(rng.choice([1, 2, 9])))
    trees = [big.tree(t) for t in range(big.n_trees)] + [small.tree(t) for t in range(small.n_trees)]
    trees = [trees[i] for i in rng.permutation(len(trees))]
    offs = np.cumsum([0] + [len(t[0]) for t in trees]).astype(np.int64)
    cat = [np.concatenate([np.asarray(t[k], dt) for t in trees]) for k, dt in
           enumerate((np.int32, np.float32, np.int32, np.int32, np.float32))]
    ens = W.Ensemble(offs, *cat, 700)
    n_docs = int(rng.choice([7, 130, 5000]))
    X = W.random_docs(900 + seed, n_docs=n_docs, n_features=700, zero_frac=0.3,
                      values=np.append(pool, np.nan).astype(np.float32) if seed % 2 == 0 else None)
    internal = np.nonzero(ens.feature >= 0)[0]
    for _ in range(300):
        n = internal[rng.integers(0, internal.size)]
        X[rng.integers(0, n_docs), ens.feature[n]] = ens.threshold[n]
    return ens, X


@pytest.mark.parametrize("seed", range(4))
def test_random_coded_models_with_small_trees(T, seed):
    ens, X = _mixed(seed)
    for flags in (0, 1):
        _check(T, ens, X, f"mixed model {seed}, {X.shape[0]} docs, rule {flags}", flags)


@pytest.mark.parametrize("n_docs", [90, 9000])
def test_vector_valued_leaves(T, n_docs):
    import torch
    cfg = W.WORKLOADS["large_5kx256_f700_1M"]
    ens = W.make_ensemble(cfg, n_trees=120)
    X = W.make_docs(cfg, n_docs=n_docs)
    vals = W.make_leaf_vectors(ens, 6, "dense", seed=cfg.seed_key)
    print(f"vector leaves, {n_docs} docs", flush=True)
    with T.TreeEnsemble.from_ensemble(ens, 0, leaf_values=vals) as m:
        got = m.predict(dev(X))
        torch.cuda.synchronize()
        got = got.cpu().numpy()
    ref = oracle.score_multi(ens, vals, X)
    assert_scores_close(got.ravel(), ref.ravel(), "vector-valued leaves")


def test_packets_of_several_groups(T):
    """Small trees share a window (several groups per packet: bodies one after another, one
    root pair per group in the header) next to large ones that keep the plan coded."""
    big = W.random_ensemble(41, n_trees=150, n_features=700, min_leaves=200, max_leaves=256)
    small = W.random_ensemble(42, n_trees=130, n_features=700, min_leaves=16, max_leaves=32)
    trees = [big.tree(t) for t in range(big.n_trees)] + [small.tree(t) for t in range(small.n_trees)]
    offs = np.cumsum([0] + [len(t[0]) for t in trees]).astype(np.int64)
    cat = [np.concatenate([np.asarray(t[k], dt) for t in trees]) for k, dt in
           enumerate((np.int32, np.float32, np.int32, np.int32, np.float32))]
    ens = W.Ensemble(offs, *cat, 700)
    for n_docs in (100, 7000):
        X = W.random_docs(43, n_docs, 700)
        for flags in (0, 1):
            _check(T, ens, X, f"several groups, {n_docs} docs, rule {flags}", flags)


def test_kernel_timing_events(T):
    """The measurement aid times each scoring launch of later eager predicts: one launch per
    predict (the coding pass and the split reduction are not counted), positive durations,
    nothing after it is switched off, and a new start clears the record."""
    import torch
    cfg = W.WORKLOADS["large_5kx256_f700_1M"]
    ens = W.make_ensemble(cfg, n_trees=60)
    X = dev(W.make_docs(cfg, n_docs=3000))
    with T.TreeEnsemble.from_ensemble(ens) as m:
        m.kernel_timing(True)
        for _ in range(3):
            m.predict(X)
        torch.cuda.synchronize()
        ms, n = m.kernel_time()
        assert n == 3 and ms > 0.0, (ms, n)
        m.kernel_timing(False)
        m.predict(X)
        torch.cuda.synchronize()
        assert m.kernel_time()[1] == 3
        m.kernel_timing(True)
        assert m.kernel_time() == (0.0, 0)
        m.kernel_timing(False)


def test_widest_coded_tile(T):
    """767 features: the widest coded 64-document tile (98,304 bytes) next to the 32 windows,
    the whole LDS."""
    ens = W.random_ensemble(1577, n_trees=90, n_features=767, min_leaves=200, max_leaves=256)
    internal = np.nonzero(ens.feature >= 0)[0]
    ens.feature[internal[0]] = 766
    X = W.random_docs(62, 3000, 767, zero_frac=0.2)
    for flags in (0, 1):
        _check(T, ens, X, f"767 features, rule {flags}", flags)


@pytest.mark.parametrize("n_features,min_leaves,max_leaves", [(700, 257, 400)])
def test_coded_models_that_keep_8_byte_packets(T, n_features, min_leaves, max_leaves):
    """Coded 64-document models the compact packets do not take (trees over 511 nodes) walk the
    8-byte records with threshold codes staged unshifted; the emulator test pins which models
    take which."""
    ens = W.random_ensemble(60 + n_features, n_trees=90, n_features=n_features, min_leaves=min_leaves,
                            max_leaves=max_leaves)
    X = W.random_docs(61, 3000, n_features, zero_frac=0.2)
    with T.TreeEnsemble.from_ensemble(ens) as m:
        assert m.info()["docs_per_block"] == 64
    for flags in (0, 1):
        _check(T, ens, X, f"8-byte coded packets, {n_features} features, rule {flags}", flags)


@pytest.mark.parametrize("seed", range(CC.N_CASES))
def test_random_compact_models(T, seed):
    """Seeded random models of the compact packets' shape (tests/_compact_cases.py: 420-767
    features, large trees mixed with small and single-leaf ones, IEEE corner values, exact ties,
    one to 9,000 documents, either rule, vector-valued leaves, bags): scores and leaf ids
    against the oracle. The emulator test pins that 22 of the 24 take the compact packets."""
    import torch
    ens, X, rule, vals, n_bags = CC.case(seed)
    what = f"compact case {seed}: {ens.n_trees} trees, {X.shape[1]} features, {X.shape[0]} docs, rule {rule}"
    print(what, flush=True)
    with T.TreeEnsemble.from_ensemble(ens, rule, leaf_values=vals, n_bags=n_bags) as m:
        x = dev(X)
        s = m.predict(x)
        ids = m.predict_leaves(x)
        torch.cuda.synchronize()
        s, ids = s.cpu().numpy().astype(np.float64), ids.cpu().numpy()
    _, ref_ids, _ = oracle.score(ens, X, rule=rule)
    if vals is None:
        ref = oracle.score(ens, X, rule=rule)[0] / n_bags
    else:
        ref = oracle.score_multi(ens, vals, X, n_bags=n_bags, rule=rule)
    assert_scores_close(s.ravel(), ref.ravel(), what)
    assert_leaves_equal(ids, ref_ids, what)
