"""GPU feature-access trace (tree_ens_feature_usage, Section 6 / Table 4) through the C ABI
against the oracle's trace: per-document feature bitmasks and counts must match exactly."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import workloads as W
from _golden import load_hand_ensemble
from _gpu import dev

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def T():
    import paper_1212_2287_amd as T
    T.load_library()
    return T


def _gpu_usage(T, ens, X, flags=0, want_masks=True):
    import torch
    with T.TreeEnsemble.from_ensemble(ens, flags) as m:
        c, mk = m.feature_usage(dev(X), want_masks=want_masks)
        torch.cuda.synchronize()
        return c.cpu().numpy(), None if mk is None else mk.cpu().numpy().view(np.uint32)


def _assert_usage_equal(got, ref, what):
    gc, gm = got
    rc, rm = ref
    assert gc.shape == rc.shape, what
    if gm is not None:
        assert gm.shape == rm.shape, (what, gm.shape, rm.shape)
        if not np.array_equal(gm, rm):
            d, w = np.argwhere(gm != rm)[0]
            raise AssertionError(f"{what}: {int((gm != rm).any(axis=1).sum())} documents differ; "
                                 f"first doc {d} word {w}: gpu {gm[d, w]:#010x} oracle {rm[d, w]:#010x}")
    if not np.array_equal(gc, rc):
        d = int(np.argwhere(gc != rc)[0][0])
        raise AssertionError(f"{what}: counts differ at doc {d}: gpu {gc[d]} oracle {rc[d]}")


@pytest.mark.parametrize("rule,name", [(0, "ge"), (1, "gt")])
def test_golden_hand_ensemble(T, rule, name):
    ens, X, expects = load_hand_ensemble()
    flags = T.TREE_ENS_RIGHT_IF_GT if rule else T.TREE_ENS_RIGHT_IF_GE
    counts, masks = _gpu_usage(T, ens, X, flags)
    for d, feats in expects["usage_" + name]:
        want = sum(1 << f for f in feats)
        assert int(masks[d, 0]) == want, (d, masks[d, 0], feats)
        assert counts[d] == len(feats)


@pytest.mark.parametrize("wl", ["tiny_10x8", "rank_1kx32", "wide_1kx64_f700"])
def test_workload_full(T, wl):
    cfg = W.WORKLOADS[wl]
    _say(f"[usage] {wl}: {cfg.n_trees} trees, {cfg.n_docs} docs")
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg)
    got = _gpu_usage(T, ens, X)
    _assert_usage_equal(got, oracle.feature_usage(ens, X), f"{wl}")


@pytest.mark.parametrize("wl", ["shallow_20kx8_1M", "large_5kx256_f700_1M"])
def test_workload_1M_sampled(T, wl):
    import torch
    cfg = W.WORKLOADS[wl]
    _say(f"[usage] {wl} at full size: generating")
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg)
    sample = np.sort(np.random.default_rng(10 + cfg.seed_key).choice(cfg.n_docs, size=4096, replace=False))
    _say(f"[usage] {wl}: tracing {cfg.n_docs} docs on the GPU")
    with T.TreeEnsemble.from_ensemble(ens) as m:
        c, mk = m.feature_usage(dev(X))
        torch.cuda.synchronize()
        c, mk = c.cpu().numpy(), mk.cpu().numpy().view(np.uint32)
    _say(f"[usage] {wl}: oracle on {sample.size} sampled docs")
    ref = oracle.feature_usage(ens, X[sample])
    _assert_usage_equal((c[sample], mk[sample]), ref, f"{wl} sample")
    # properties over every document: the count is the mask's popcount and at least the number
    # of distinct root features
    pop = np.unpackbits(mk.view(np.uint8), axis=1).sum(axis=1)
    assert np.array_equal(pop, c)
    roots = {int(ens.feature[int(o)]) for o in ens.tree_offsets[:-1] if ens.feature[int(o)] >= 0}
    assert (c >= len(roots)).all()


@pytest.mark.parametrize("n_docs", [1, 63, 64, 65, 4097])
@pytest.mark.parametrize("wl", ["rank_1kx32", "wide_1kx64_f700"])
def test_ragged_batches(T, wl, n_docs):
    # wide_1kx64_f700 (700 features) runs the one-workgroup float kernels
    cfg = W.WORKLOADS[wl]
    ens = W.make_ensemble(cfg, n_trees=150)
    X = W.make_docs(cfg, n_docs=n_docs)
    _assert_usage_equal(_gpu_usage(T, ens, X), oracle.feature_usage(ens, X),
                        f"{wl}, {n_docs} docs")


_POOL = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf, np.nan], dtype=np.float32)


@pytest.mark.parametrize("seed", range(6))
def test_random_ensembles_rules_and_special_values(T, seed):
    rule = seed % 2
    F = (40, 70, 136, 33, 5, 300)[seed]
    ens = W.random_ensemble(seed, n_trees=60, n_features=F, min_leaves=1, max_leaves=40,
                            thr_values=_POOL[:8] if seed % 3 == 0 else None)
    X = W.random_docs(seed, 333, F, values=_POOL if seed % 3 == 0 else None, zero_frac=0.2)
    X[7, :] = np.nan
    flags = T.TREE_ENS_RIGHT_IF_GT if rule else T.TREE_ENS_RIGHT_IF_GE
    _assert_usage_equal(_gpu_usage(T, ens, X, flags), oracle.feature_usage(ens, X, rule=rule),
                        f"seed {seed} rule {rule}")


def test_extra_document_columns_and_counts_only(T):
    # documents wider than the model reads: the mask rows follow the document width and the
    # words past the model's features are zero; counts alone when no mask is wanted
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg, n_trees=80)
    X = W.make_docs(cfg, n_docs=500)
    wide = np.concatenate([X, np.full((500, 100), 0.5, np.float32)], axis=1)
    wide_ens = W.Ensemble(ens.tree_offsets, ens.feature, ens.threshold, ens.left, ens.right, ens.value,
                          wide.shape[1])
    got = _gpu_usage(T, ens, wide)
    _assert_usage_equal(got, oracle.feature_usage(wide_ens, wide), "wide documents")
    assert not got[1][:, (136 + 31) // 32:].any()
    c, m = _gpu_usage(T, ens, X, want_masks=False)
    assert m is None and np.array_equal(c, oracle.feature_usage(ens, X)[0])


def test_leaf_only_and_empty_models(T):
    import torch
    F = 20
    X = W.random_docs(3, 100, F)
    leaves = W.Ensemble(np.arange(4, dtype=np.int64), np.full(3, -1, np.int32), np.zeros(3, np.float32),
                        np.full(3, -1, np.int32), np.full(3, -1, np.int32), np.ones(3, np.float32), F)
    c, m = _gpu_usage(T, leaves, X)
    assert not c.any() and not m.any()
    empty = W.Ensemble(np.zeros(1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.float32),
                       np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32), F)
    with T.TreeEnsemble.from_ensemble(empty) as mdl:
        cnt = torch.full((100,), 7, dtype=torch.int32, device="cuda")
        msk = torch.full((100, 1), 7, dtype=torch.int32, device="cuda")
        T.tree_ens_feature_usage(mdl.handle, dev(X), cnt, msk)
        torch.cuda.synchronize()
        assert not cnt.cpu().numpy().any() and not msk.cpu().numpy().any()
        c0, m0 = mdl.feature_usage(dev(X[:0]))
        assert c0.shape == (0,)


def test_argument_errors(T):
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg, n_trees=20)
    X = W.make_docs(cfg, n_docs=10)
    with T.TreeEnsemble.from_ensemble(ens) as m:
        with pytest.raises(T.TreeEnsError) as ei:
            m.feature_usage(dev(X[:, :10].copy()))
        assert ei.value.code == T.TREE_ENS_E_SHAPE
