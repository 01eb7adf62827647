"""Pins for the oracle's vector-valued leaves and bagged ensembles (oracle_score_multi;
Section 3: a leaf may hold a class, a real or another model; Section 5.3: several bagged
boosted ensembles averaged). Each check ties it to something other than itself: the hand-worked
golden sums, the scalar oracle per component, closed forms for one-tree-per-class models and
bagged copies, separately scored bags, and the path-conjunction brute force. CPU only."""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle
from oracle import brute
import workloads as W
from _golden import load_hand_ensemble

RULES = (oracle.RULE_GE, oracle.RULE_GT)


@pytest.mark.parametrize("rule,name", [(0, "ge"), (1, "gt")])
def test_golden_hand_ensemble(rule, name):
    # leaf rows (v, 2v + 1, -v): over the three trees the sums are (s, 2s + 3, -s), exact
    ens, X, expects = load_hand_ensemble()
    s = np.array([e[1] for e in expects[name]])
    leaf = ens.feature < 0
    vals = np.zeros((ens.n_nodes, 3), np.float32)
    vals[leaf, 0] = ens.value[leaf]
    vals[leaf, 1] = 2 * ens.value[leaf] + 1
    vals[leaf, 2] = -ens.value[leaf]
    out = oracle.score_multi(ens, vals, X, rule=rule)
    assert np.array_equal(out, np.stack([s, 2 * s + 3, -s], axis=1))
    # two bags: halves, exact (a power of two)
    assert np.array_equal(oracle.score_multi(ens, vals, X, n_bags=2, rule=rule), out / 2)


@pytest.mark.parametrize("kind", ["dense", "class", "probs"])
@pytest.mark.parametrize("rule", RULES)
def test_each_component_is_the_scalar_score(kind, rule):
    # component c equals the scalar oracle's score of the ensemble whose leaf values are
    # column c (the same fp64 sum in the same tree order): pins the row stride and the column
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg, n_trees=70)
    X = W.make_docs(cfg, n_docs=300)
    vals = W.make_leaf_vectors(ens, 5, kind, seed=3)
    out = oracle.score_multi(ens, vals, X, rule=rule)
    for c in range(5):
        e = W.Ensemble(ens.tree_offsets, ens.feature, ens.threshold, ens.left, ens.right,
                       np.ascontiguousarray(vals[:, c]), ens.n_features)
        assert np.array_equal(out[:, c], oracle.score(e, X, rule=rule, want_leaves=False)[0]), c


def test_one_tree_per_class_closed_form():
    # multi-class boosting layout: tree t feeds class t % C only, so class c's output is the
    # scalar score of the sub-ensemble of trees c, c + C, c + 2C, ... (adding exact zeros
    # elsewhere changes nothing)
    cfg = W.WORKLOADS["rank_1kx32"]
    C = 4
    ens = W.make_ensemble(cfg, n_trees=41)
    X = W.make_docs(cfg, n_docs=250)
    out = oracle.score_multi(ens, W.make_leaf_vectors(ens, C, "class"), X)
    for c in range(C):
        trees = list(range(c, ens.n_trees, C))
        sub = _select(ens, trees)
        assert np.array_equal(out[:, c], oracle.score(sub, X, want_leaves=False)[0]), c


def test_probability_leaves_sum_to_tree_count():
    # every leaf row of a forest classifier sums to 1: the outputs of a document sum to the
    # number of trees (up to float32 rounding of the rows)
    cfg = W.WORKLOADS["tiny_10x8"]
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg)
    vals = W.make_leaf_vectors(ens, 3, "probs", seed=1)
    out = oracle.score_multi(ens, vals, X)
    assert np.allclose(out.sum(axis=1), ens.n_trees, rtol=0, atol=1e-5)
    assert (out >= 0).all()


def _select(ens, trees):
    feats, thrs, lefts, rights, vals, offs = [], [], [], [], [], [0]
    for t in trees:
        f, th, l, r, v = ens.tree(t)
        feats.append(f); thrs.append(th); lefts.append(l); rights.append(r); vals.append(v)
        offs.append(offs[-1] + f.shape[0])
    return W.Ensemble(np.asarray(offs, np.int64), np.concatenate(feats), np.concatenate(thrs),
                      np.concatenate(lefts), np.concatenate(rights), np.concatenate(vals), ens.n_features)


def _concat_all(parts):
    offs = [np.zeros(1, np.int64)]
    base = 0
    for p in parts:
        offs.append(p.tree_offsets[1:] + base)
        base += int(p.tree_offsets[-1])
    return W.Ensemble(np.concatenate(offs), np.concatenate([p.feature for p in parts]),
                      np.concatenate([p.threshold for p in parts]), np.concatenate([p.left for p in parts]),
                      np.concatenate([p.right for p in parts]), np.concatenate([p.value for p in parts]),
                      parts[0].n_features)


@pytest.mark.parametrize("n_bags", [2, 3, 5])
def test_bags_average_separately_scored_bags(n_bags):
    # bags of different sizes, scored one by one and averaged, against the concatenation
    bags = [W.random_ensemble(10 + b, n_trees=7 + 3 * b, n_features=9, max_leaves=20) for b in range(n_bags)]
    X = W.random_docs(4, 120, 9)
    ens = _concat_all(bags)
    vals = np.ascontiguousarray(ens.value[:, None])
    out = oracle.score_multi(ens, vals, X, n_bags=n_bags)[:, 0]
    per_bag = np.stack([oracle.score(b, X, want_leaves=False)[0] for b in bags])
    assert np.allclose(out, per_bag.mean(axis=0), rtol=1e-14, atol=1e-15)
    assert not np.allclose(out, per_bag.sum(axis=0), rtol=1e-6)


@pytest.mark.parametrize("n_bags", [2, 4])
def test_identical_bags_equal_one_bag(n_bags):
    # B copies of one ensemble averaged: exactly the single ensemble's score (B a power of two:
    # the B-fold sum and the division are exact)
    ens = W.random_ensemble(3, n_trees=30, n_features=12, max_leaves=16)
    X = W.random_docs(3, 200, 12)
    vals = W.make_leaf_vectors(ens, 2, "dense", seed=0)
    one = oracle.score_multi(ens, vals, X)
    cat = _concat_all([ens] * n_bags)
    assert np.array_equal(oracle.score_multi(cat, np.concatenate([vals] * n_bags), X, n_bags=n_bags), one)


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("rule", RULES)
def test_brute_force_fsum(seed, rule):
    pool = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf], dtype=np.float32)
    ens = W.random_ensemble(seed, n_trees=11, n_features=6, max_leaves=14,
                            thr_values=pool[:6] if seed % 2 else None)
    X = W.random_docs(seed, 60, 6, values=pool if seed % 2 else None, zero_frac=0.2)
    X[2] = np.nan
    C, B = 3, 1 + seed % 3
    vals = W.make_leaf_vectors(ens, C, "dense", sigma=1.0, seed=seed)
    out = oracle.score_multi(ens, vals, X, n_bags=B, rule=rule)
    ids = brute.leaves(ens, X, rule)
    for d in range(X.shape[0]):
        rows = [vals[int(ens.tree_offsets[t]) + int(ids[d, t])] for t in range(ens.n_trees)]
        for c in range(C):
            terms = [float(r[c]) for r in rows]
            exact = math.fsum(terms) / B
            bound = (len(terms) - 1) * 2.0 ** -53 * sum(abs(v) for v in terms) / B + 1e-300
            assert abs(out[d, c] - exact) <= bound + 2.0 ** -53 * abs(exact), (d, c)


def test_argument_errors():
    ens, X, _ = load_hand_ensemble()
    with pytest.raises(ValueError):
        oracle.score_multi(ens, np.zeros((ens.n_nodes - 1, 2), np.float32), X)
    with pytest.raises(oracle.OracleError):
        oracle.score_multi(ens, np.zeros((ens.n_nodes, 2), np.float32), X, n_bags=0)
