"""Pins for the oracle's feature-access trace (oracle_feature_usage: the distinct features a
document's walks compare, over the whole ensemble -- Section 6 and its Table 4). Each check ties
it to something other than itself: hand-worked sets, the path-conjunction brute force, closed
forms for stumps and oblivious trees, and invariants. CPU only."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from oracle import brute
import workloads as W
from _golden import load_hand_ensemble

RULES = (oracle.RULE_GE, oracle.RULE_GT)


def _mask_of(sets, n_features):
    """uint32 [n_docs][(F + 31) // 32] bitmask of per-document feature sets."""
    words = (n_features + 31) // 32
    m = np.zeros((len(sets), words), np.uint32)
    for d, s in enumerate(sets):
        for f in s:
            m[d, f // 32] |= np.uint32(1) << np.uint32(f % 32)
    return m


def _sets_of(masks, n_features):
    return [sorted(f for f in range(n_features) if (int(masks[d, f // 32]) >> (f % 32)) & 1)
            for d in range(masks.shape[0])]


def _check(ens, X, rule, sets):
    counts, masks = oracle.feature_usage(ens, X, rule=rule)
    got = _sets_of(masks, ens.n_features)
    for d, s in enumerate(sets):
        assert got[d] == sorted(s), (d, got[d], sorted(s))
    assert np.array_equal(masks, _mask_of(sets, ens.n_features))
    assert counts.tolist() == [len(set(s)) for s in sets]


@pytest.mark.parametrize("rule,name", [(0, "ge"), (1, "gt")])
def test_golden_hand_ensemble(rule, name):
    ens, X, expects = load_hand_ensemble()
    sets = [fs for _, fs in sorted(expects["usage_" + name])]
    assert len(sets) == X.shape[0]
    _check(ens, X, rule, sets)


_POOL = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf], dtype=np.float32)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("rule", RULES)
def test_brute_force_path_features(seed, rule):
    # the brute force finds each document's leaf by testing every leaf's whole path conjunction
    # (no walk); the features on that path, over all trees, are the expected set. More than 32
    # features so that the set spans several mask words.
    F = 37 if seed % 2 else 70
    ens = W.random_ensemble(seed, n_trees=9, n_features=F, min_leaves=1, max_leaves=20,
                            thr_values=_POOL[:6] if seed % 2 else None)
    X = W.random_docs(seed, 50, F, values=_POOL if seed % 2 else None, zero_frac=0.2)
    X[3, :] = np.nan
    X[5, ::2] = np.nan
    ids = brute.leaves(ens, X, rule)
    path_feats = []
    for t in range(ens.n_trees):
        fe, th, le, ri, _ = ens.tree(t)
        path_feats.append({leaf: {f for f, _, _ in path} for leaf, path in brute.leaf_paths(fe, th, le, ri)})
    sets = [set().union(*(path_feats[t][int(ids[d, t])] for t in range(ens.n_trees)))
            for d in range(X.shape[0])]
    _check(ens, X, rule, sets)


def test_stumps_and_single_leaves_closed_form():
    # a stump compares its one feature for every document, whatever the value (NaN included);
    # a single-leaf tree compares nothing
    rng = np.random.default_rng(2)
    F = 45
    f = rng.integers(0, F, size=12)
    feats, thrs, lefts, rights, vals, offs = [], [], [], [], [], [0]
    for k in range(12):
        feats += [f[k], -1, -1]
        thrs += [rng.random(), 0, 0]
        lefts += [1, -1, -1]
        rights += [2, -1, -1]
        vals += [0, 1, 2]
        offs.append(offs[-1] + 3)
        feats += [-1]; thrs += [0]; lefts += [-1]; rights += [-1]; vals += [0.5]
        offs.append(offs[-1] + 1)
    ens = W.Ensemble(np.asarray(offs, np.int64), np.asarray(feats, np.int32), np.asarray(thrs, np.float32),
                     np.asarray(lefts, np.int32), np.asarray(rights, np.int32), np.asarray(vals, np.float32), F)
    X = W.random_docs(4, 30, F, zero_frac=0.1)
    X[0] = np.nan
    X[1] = np.inf
    for rule in RULES:
        _check(ens, X, rule, [set(f.tolist())] * 30)
    leaves_only = W.Ensemble(np.arange(5, dtype=np.int64), np.full(4, -1, np.int32), np.zeros(4, np.float32),
                             np.full(4, -1, np.int32), np.full(4, -1, np.int32), np.ones(4, np.float32), F)
    counts, masks = oracle.feature_usage(leaves_only, X)
    assert not counts.any() and not masks.any()


@pytest.mark.parametrize("depth", [1, 3, 6])
def test_oblivious_trees_closed_form(depth):
    # every node on level k of tree t compares f_{t,k}: every walk of a complete tree compares
    # exactly {f_{t,k} : k < depth}, whatever the document
    rng = np.random.default_rng(10 + depth)
    F, n_trees = 40, 7
    feats, thrs, lefts, rights, offs, want = [], [], [], [], [0], set()
    for t in range(n_trees):
        fe, le, ri = W.grow_complete_structure(np.random.default_rng(200 + t), depth, F)
        level = np.zeros(fe.shape[0], np.int64)
        for n in range(fe.shape[0]):  # creation order: parents precede children
            if fe[n] >= 0:
                level[le[n]] = level[ri[n]] = level[n] + 1
        fk = rng.integers(0, F, size=depth)
        internal = fe >= 0
        fe = fe.copy()
        fe[internal] = fk[level[internal]]
        want |= set(fk.tolist())
        feats.append(fe); lefts.append(le); rights.append(ri)
        thrs.append(rng.random(fe.shape[0]).astype(np.float32))
        offs.append(offs[-1] + fe.shape[0])
    n = offs[-1]
    ens = W.Ensemble(np.asarray(offs, np.int64), np.concatenate(feats), np.concatenate(thrs),
                     np.concatenate(lefts), np.concatenate(rights), np.zeros(n, np.float32), F)
    X = W.random_docs(depth, 60, F)
    X[7] = np.nan
    _check(ens, X, oracle.RULE_GE, [want] * 60)


def _slice(ens, a, b):
    lo, hi = int(ens.tree_offsets[a]), int(ens.tree_offsets[b])
    return W.Ensemble(ens.tree_offsets[a:b + 1] - lo, ens.feature[lo:hi], ens.threshold[lo:hi],
                      ens.left[lo:hi], ens.right[lo:hi], ens.value[lo:hi], ens.n_features)


def test_invariants():
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg, n_trees=80)
    X = W.make_docs(cfg, n_docs=300)
    F = ens.n_features
    counts, masks = oracle.feature_usage(ens, X)
    # the count is the mask's population; no bit past the last feature is set
    pop = np.array([sum(bin(int(w)).count("1") for w in row) for row in masks])
    assert np.array_equal(counts, pop)
    tail = F % 32
    if tail:
        assert not (masks[:, -1] >> np.uint32(tail)).any()
    # union over a split of the trees; and at least one feature per tree with an internal root
    ca, ma = oracle.feature_usage(_slice(ens, 0, 30), X)
    cb, mb = oracle.feature_usage(_slice(ens, 30, ens.n_trees), X)
    assert np.array_equal(ma | mb, masks)
    assert (counts >= np.maximum(ca, cb)).all()
    assert (counts >= 1).all() and (counts <= F).all()
    # the root features of all trees are always examined
    roots = {int(ens.feature[int(o)]) for o in ens.tree_offsets[:-1] if ens.feature[int(o)] >= 0}
    for s in _sets_of(masks, F):
        assert roots <= set(s)
    # the set size is at most the number of comparisons the walks made
    for d in range(0, 300, 37):
        _, _, visits = oracle.score(ens, X[d:d + 1])
        assert counts[d] <= visits
    # permuting documents permutes the rows
    perm = np.random.default_rng(1).permutation(X.shape[0])
    c2, m2 = oracle.feature_usage(ens, X[perm])
    assert np.array_equal(c2, counts[perm]) and np.array_equal(m2, masks[perm])
    # renaming feature ids (and moving the document columns with them) renames the set
    fperm = np.random.default_rng(2).permutation(F)  # old id -> new id
    fe = np.where(ens.feature >= 0, fperm[np.maximum(ens.feature, 0)], -1).astype(np.int32)
    ens_p = W.Ensemble(ens.tree_offsets, fe, ens.threshold, ens.left, ens.right, ens.value, F)
    Xp = np.empty_like(X)
    Xp[:, fperm] = X
    _, m3 = oracle.feature_usage(ens_p, Xp)
    assert _sets_of(m3, F) == [sorted(int(fperm[f]) for f in s) for s in _sets_of(masks, F)]
    # renumbering nodes changes nothing
    ens4, _ = W.relabel_nodes(ens, 5)
    assert np.array_equal(oracle.feature_usage(ens4, X)[1], masks)


def test_thread_count_does_not_change_results():
    cfg = W.WORKLOADS["wide_1kx64_f700"]
    ens = W.make_ensemble(cfg, n_trees=40)
    X = W.make_docs(cfg, n_docs=500)
    a = oracle.feature_usage(ens, X, threads=1)
    b = oracle.feature_usage(ens, X, threads=4)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1])


def test_malformed_model_is_reported():
    ens, X, _ = load_hand_ensemble()
    bad = W.Ensemble(ens.tree_offsets, ens.feature, ens.threshold, ens.left.copy(), ens.right, ens.value,
                     ens.n_features)
    bad.left[0] = 99
    with pytest.raises(oracle.OracleError):
        oracle.feature_usage(bad, X)
    badf = W.Ensemble(ens.tree_offsets, ens.feature.copy(), ens.threshold, ens.left, ens.right, ens.value,
                      ens.n_features)
    badf.feature[0] = ens.n_features  # feature id past the document's columns
    with pytest.raises(oracle.OracleError):
        oracle.feature_usage(badf, X)
