"""Property tests (hypothesis) of the HIP path through the C ABI: random small ensembles and
documents against the oracle (scores and leaves, vector-valued leaves with bags, the feature
trace), and invariants of the mathematics checked on the GPU alone —
doubling leaf values doubles every score exactly, permuting documents permutes the scores bit
for bit, renumbering nodes maps the leaf ids and keeps the scores bit for bit, reordering trees
keeps the scores within the tolerance."""
from __future__ import annotations

import numpy as np
import pytest
from hypothesis import HealthCheck, given, settings, strategies as st

import oracle
import workloads as W
from _gpu import assert_leaves_equal, assert_scores_close, dev

pytestmark = pytest.mark.gpu

_POOL = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf, np.nan, 1e-45, 3.4e38],
                 dtype=np.float32)

SETTINGS = settings(max_examples=25, deadline=None, database=None, derandomize=True,
                    suppress_health_check=[HealthCheck.too_slow, HealthCheck.function_scoped_fixture])


@pytest.fixture(scope="module")
def T():
    import paper_1212_2287_amd as T
    T.load_library()
    return T


cases = st.fixed_dictionaries({
    "seed": st.integers(0, 10_000),
    "n_trees": st.integers(1, 40),
    "n_features": st.integers(1, 60),
    "max_leaves": st.integers(1, 48),
    "n_docs": st.integers(1, 300),
    "pooled": st.booleans(),
    "rule": st.integers(0, 1),
})


def _make(c):
    pool = _POOL[:8] if c["pooled"] else None
    ens = W.random_ensemble(c["seed"], n_trees=c["n_trees"], n_features=c["n_features"],
                            min_leaves=1, max_leaves=c["max_leaves"], thr_values=pool)
    X = W.random_docs(c["seed"], c["n_docs"], c["n_features"], values=_POOL if c["pooled"] else None,
                      zero_frac=0.1)
    return ens, X


def _run(T, ens, X, rule, leaves=True):
    import torch
    flags = T.TREE_ENS_RIGHT_IF_GT if rule else T.TREE_ENS_RIGHT_IF_GE
    with T.TreeEnsemble.from_ensemble(ens, flags) as m:
        x = dev(X)
        s = m.predict(x)
        ids = m.predict_leaves(x) if leaves else None
        torch.cuda.synchronize()
        return s.cpu().numpy(), None if ids is None else ids.cpu().numpy()


@SETTINGS
@given(c=cases)
def test_random_ensembles_match_the_oracle(T, c):
    ens, X = _make(c)
    s, ids = _run(T, ens, X, c["rule"])
    ref, ref_ids, _ = oracle.score(ens, X, rule=c["rule"])
    assert_scores_close(s, ref, str(c))
    assert_leaves_equal(ids, ref_ids, str(c))


@SETTINGS
@given(c=cases)
def test_invariants_on_the_gpu(T, c):
    ens, X = _make(c)
    rule = c["rule"]
    s, ids = _run(T, ens, X, rule)
    # doubling every leaf value doubles every score exactly (fp64 accumulation
    # and the final rounding all commute with an exact power-of-two scaling)
    ens2 = W.Ensemble(ens.tree_offsets, ens.feature, ens.threshold, ens.left, ens.right,
                      (ens.value * 2).astype(np.float32), ens.n_features)
    s2, _ = _run(T, ens2, X, rule, leaves=False)
    assert np.array_equal(s2, 2 * s)
    # permuting the documents permutes the scores bit for bit (a document's trees are summed
    # in the same order whichever lane holds it)
    perm = np.random.default_rng(c["seed"]).permutation(X.shape[0])
    sp, ip = _run(T, ens, X[perm], rule)
    assert np.array_equal(sp, s[perm]) and np.array_equal(ip, ids[perm])
    # renumbering the nodes maps the leaf ids and keeps the scores bit for bit
    ens4, maps = W.relabel_nodes(ens, c["seed"])
    s4, i4 = _run(T, ens4, X, rule)
    assert np.array_equal(s4, s)
    for t in range(ens.n_trees):
        assert np.array_equal(i4[:, t], maps[t][ids[:, t]])
    # reversing the tree order keeps the scores within the tolerance, the leaves exactly
    order = list(range(ens.n_trees))[::-1]
    feats, thrs, lefts, rights, vals, offs = [], [], [], [], [], [0]
    for t in order:
        f, th, l, r, v = ens.tree(t)
        feats.append(f); thrs.append(th); lefts.append(l); rights.append(r); vals.append(v)
        offs.append(offs[-1] + f.shape[0])
    rev = W.Ensemble(np.asarray(offs, np.int64), np.concatenate(feats), np.concatenate(thrs),
                     np.concatenate(lefts), np.concatenate(rights), np.concatenate(vals), ens.n_features)
    sr, ir = _run(T, rev, X, rule)
    assert_scores_close(sr, s.astype(np.float64), "reversed trees")
    assert np.array_equal(ir[:, ::-1], ids)


@SETTINGS
@given(c=cases, n_out=st.integers(2, 9), n_bags=st.integers(1, 4))
def test_vector_leaves_and_bags_match_the_oracle(T, c, n_out, n_bags):
    import torch
    ens, X = _make(c)
    vals = W.make_leaf_vectors(ens, n_out, ("dense", "class", "probs")[c["seed"] % 3], seed=c["seed"])
    flags = T.TREE_ENS_RIGHT_IF_GT if c["rule"] else T.TREE_ENS_RIGHT_IF_GE
    with T.TreeEnsemble.from_ensemble(ens, flags, leaf_values=vals, n_bags=n_bags) as m:
        s = m.predict(dev(X))
        torch.cuda.synchronize()
        s = s.cpu().numpy().astype(np.float64)
    ref = oracle.score_multi(ens, vals, X, n_bags=n_bags, rule=c["rule"])
    assert_scores_close(s.ravel(), ref.ravel(), str(c))


@SETTINGS
@given(c=cases)
def test_feature_trace_matches_the_oracle(T, c):
    import torch
    ens, X = _make(c)
    flags = T.TREE_ENS_RIGHT_IF_GT if c["rule"] else T.TREE_ENS_RIGHT_IF_GE
    with T.TreeEnsemble.from_ensemble(ens, flags) as m:
        cnt, masks = m.feature_usage(dev(X))
        torch.cuda.synchronize()
        cnt, masks = cnt.cpu().numpy(), masks.cpu().numpy().view(np.uint32)
    ref_c, ref_m = oracle.feature_usage(ens, X, rule=c["rule"])
    assert np.array_equal(cnt, ref_c) and np.array_equal(masks, ref_m), str(c)
