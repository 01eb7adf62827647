"""Pins for the oracle: each check ties the oracle to something other than itself -- hand-worked
values, closed forms, a path-conjunction brute force, the paper's own known-answer generator,
an error bound, and invariants of the mathematics. CPU only."""
from __future__ import annotations

import math

import numpy as np
import pytest

import oracle
from oracle import brute
import workloads as W
from _golden import load_hand_ensemble

RULES = (oracle.RULE_GE, oracle.RULE_GT)


def _fsum_bound(ens, X, ids):
    """Recursive-summation error bound (n-1) * u * sum|v| per document (u = 2^-53), for the
    oracle's double-precision tree-order sum against the correctly rounded sum."""
    vals = np.abs(np.array([[float(ens.value[int(ens.tree_offsets[t]) + int(ids[d, t])])
                             for t in range(ens.n_trees)] for d in range(ids.shape[0])]))
    return max(ens.n_trees - 1, 0) * 2.0 ** -53 * vals.sum(axis=1) + 1e-300


# ------------------------------------------------------------------------------------------
# hand-worked fixture (tests/golden/hand_ensemble.txt)
# ------------------------------------------------------------------------------------------
@pytest.mark.parametrize("rule,name", [(0, "ge"), (1, "gt")])
def test_golden_hand_ensemble(rule, name):
    ens, X, expects = load_hand_ensemble()
    exp_scores = np.array([e[1] for e in expects[name]])
    exp_visits = sum(e[2] for e in expects[name])
    exp_ids = np.array([e[3] for e in expects[name]], dtype=np.int32)
    for walk in (0, 1):
        s, ids, visits = oracle.score(ens, X, rule=rule, walk=walk)
        assert np.array_equal(s, exp_scores), (walk, s, exp_scores)
        assert np.array_equal(ids, exp_ids)
        assert visits == exp_visits
    s, ids = oracle.score_padded(ens, X, rule=rule)
    assert np.array_equal(s, exp_scores) and np.array_equal(ids, exp_ids)
    assert np.array_equal(brute.leaves(ens, X, rule), exp_ids)
    assert np.array_equal(brute.scores(ens, X, rule), exp_scores)


# ------------------------------------------------------------------------------------------
# brute force (path conjunction, exactly one leaf) and fsum
# ------------------------------------------------------------------------------------------
_POOL = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf], dtype=np.float32)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("rule", RULES)
def test_brute_force_matches(seed, rule):
    # thresholds and feature values from one small pool: ties x == theta are frequent
    ens = W.random_ensemble(seed, n_trees=7, n_features=5, min_leaves=1, max_leaves=12,
                            thr_values=_POOL[:6] if seed % 2 else None)
    X = W.random_docs(seed, 40, 5, values=_POOL if seed % 2 else None, zero_frac=0.2)
    X[3, 1] = np.nan
    X[5, :] = np.nan
    ids_b = brute.leaves(ens, X, rule)
    s_b = brute.scores(ens, X, rule, ids_b)
    for walk in (0, 1):
        s, ids, _ = oracle.score(ens, X, rule=rule, walk=walk)
        assert np.array_equal(ids, ids_b)
        assert np.all(np.abs(s - s_b) <= _fsum_bound(ens, X, ids_b))
    s, ids = oracle.score_padded(ens, X, rule=rule)
    assert np.array_equal(ids, ids_b)


def test_fp64_sum_within_recursive_summation_bound():
    # many trees, many terms: the oracle's sum must be within (n-1) u sum|v| of fsum
    ens = W.random_ensemble(77, n_trees=400, n_features=8, min_leaves=2, max_leaves=6, leaf_sigma=1e3)
    X = W.random_docs(77, 25, 8)
    s, ids, _ = oracle.score(ens, X)
    ref = brute.scores(ens, X, 0, ids)
    err = np.abs(s - ref)
    assert np.all(err <= _fsum_bound(ens, X, ids))
    # and the same sum in float32 would not be: the pin can tell fp32 from fp64 accumulation
    vals = np.array([[ens.value[int(ens.tree_offsets[t]) + ids[d, t]] for t in range(ens.n_trees)]
                     for d in range(ids.shape[0])], dtype=np.float32)
    s32 = np.zeros(ids.shape[0], dtype=np.float32)
    for t in range(ens.n_trees):
        s32 = (s32 + vals[:, t]).astype(np.float32)
    assert np.any(np.abs(s32.astype(np.float64) - ref) > _fsum_bound(ens, X, ids))


# ------------------------------------------------------------------------------------------
# closed forms
# ------------------------------------------------------------------------------------------
def _stump_ensemble(rng, n_trees, n_features):
    feats, thrs, lefts, rights, vals, offs = [], [], [], [], [], [0]
    a = rng.integers(-512, 512, size=n_trees) / 256.0  # dyadic: every sum is exact
    b = rng.integers(-512, 512, size=n_trees) / 256.0
    f = rng.integers(0, n_features, size=n_trees)
    th = rng.random(n_trees, dtype=np.float32)
    for k in range(n_trees):
        feats += [f[k], -1, -1]
        thrs += [th[k], 0, 0]
        lefts += [1, -1, -1]
        rights += [2, -1, -1]
        vals += [0, a[k], b[k]]
        offs.append(offs[-1] + 3)
    ens = W.Ensemble(np.asarray(offs, np.int64), np.asarray(feats, np.int32), np.asarray(thrs, np.float32),
                     np.asarray(lefts, np.int32), np.asarray(rights, np.int32), np.asarray(vals, np.float32),
                     n_features)
    return ens, f, th, a, b


@pytest.mark.parametrize("rule", RULES)
def test_stump_closed_form(rule):
    rng = np.random.default_rng(5)
    ens, f, th, a, b = _stump_ensemble(rng, 300, 11)
    X = W.random_docs(5, 200, 11)
    for k in range(0, 300, 7):  # exact ties x == theta
        X[k % 200, f[k]] = th[k]
    cmp = X[:, f] >= th if rule == 0 else X[:, f] > th
    expected = np.where(cmp, b, a).sum(axis=1)  # exact: dyadic values, |sum| < 2^10
    s, ids, visits = oracle.score(ens, X, rule=rule)
    assert np.array_equal(s, expected)
    assert np.array_equal(ids, np.where(cmp, 2, 1))
    assert visits == 200 * 300


def _levels_and_inorder_leaves(feature, left, right):
    """Level of every node (root 0) and the leaves in left-to-right order -- read off the
    structure alone, without any feature values."""
    level = np.zeros(len(feature), dtype=np.int64)
    order = []

    def visit(n, d):
        level[n] = d
        if feature[n] < 0:
            order.append(n)
            return
        visit(int(left[n]), d + 1)
        visit(int(right[n]), d + 1)

    visit(0, 0)
    return level, order


@pytest.mark.parametrize("depth", [1, 2, 3, 5, 7])
@pytest.mark.parametrize("rule", RULES)
def test_complete_oblivious_tree_closed_form(depth, rule):
    # every node on level k tests the same (f_k, theta_k): bit b_k = [x[f_k] >= theta_k] no
    # longer depends on the path, and the leaf reached is the one at left-to-right position
    # sum_k b_k 2^(d-1-k) (the implicit layout i -> 2i+1+b of the Pred form, Section 3).
    rng = np.random.default_rng(depth)
    n_trees, F = 6, 9
    ens = W.make_ensemble(W.scaled(W.WORKLOADS["shallow_20kx8_1M"], n_trees=n_trees))
    ens = W.Ensemble(ens.tree_offsets, ens.feature.copy(), ens.threshold.copy(), ens.left, ens.right,
                     ens.value, F)
    if depth != 3:
        feats, lefts, rights, offs = [], [], [], [0]
        for t in range(n_trees):
            fe, le, ri = W.grow_complete_structure(np.random.default_rng(100 + t), depth, F)
            feats.append(fe); lefts.append(le); rights.append(ri)
            offs.append(offs[-1] + fe.shape[0])
        n = offs[-1]
        ens = W.Ensemble(np.asarray(offs, np.int64), np.concatenate(feats), np.zeros(n, np.float32),
                         np.concatenate(lefts), np.concatenate(rights),
                         rng.integers(-64, 64, size=n).astype(np.float32) / 8, F)
    fk = rng.integers(0, F, size=(n_trees, depth))
    tk = rng.random((n_trees, depth), dtype=np.float32)
    pos_order = []
    for t in range(n_trees):
        a = int(ens.tree_offsets[t])
        fe, _, le, ri, _ = ens.tree(t)
        level, order = _levels_and_inorder_leaves(fe, le, ri)
        internal = np.nonzero(fe >= 0)[0]
        ens.feature[a + internal] = fk[t, level[internal]]
        ens.threshold[a + internal] = tk[t, level[internal]]
        pos_order.append(order)
    X = W.random_docs(depth, 300, F)
    for t in range(n_trees):
        X[t, fk[t, 0]] = tk[t, 0]  # exact ties at the root
    exp_ids = np.empty((300, n_trees), dtype=np.int32)
    for t in range(n_trees):
        bits = (X[:, fk[t]] >= tk[t]) if rule == 0 else (X[:, fk[t]] > tk[t])
        pos = (bits.astype(np.int64) << np.arange(depth - 1, -1, -1)).sum(axis=1)
        exp_ids[:, t] = np.asarray(pos_order[t])[pos]
    s, ids, visits = oracle.score(ens, X, rule=rule)
    assert np.array_equal(ids, exp_ids)
    assert visits == 300 * n_trees * depth
    exp_s = np.array([sum(float(ens.value[int(ens.tree_offsets[t]) + exp_ids[d, t]]) for t in range(n_trees))
                      for d in range(300)])
    assert np.array_equal(s, exp_s)  # eighths, exact
    s2, ids2 = oracle.score_padded(ens, X, rule=rule)
    assert np.array_equal(ids2, exp_ids)


@pytest.mark.parametrize("seed", range(4))
def test_all_thresholds_infinite(seed):
    ens = W.random_ensemble(seed, n_trees=20, n_features=6, min_leaves=1, max_leaves=30)
    X = W.random_docs(seed, 50, 6) * 2e30 - 1e30  # large finite values
    leftmost, rightmost = [], []
    for t in range(ens.n_trees):
        fe, _, le, ri, _ = ens.tree(t)
        n = 0
        while fe[n] >= 0:
            n = int(le[n])
        leftmost.append(n)
        n = 0
        while fe[n] >= 0:
            n = int(ri[n])
        rightmost.append(n)
    internal = ens.feature >= 0
    pos = W.Ensemble(ens.tree_offsets, ens.feature, np.where(internal, np.float32(np.inf), 0).astype(np.float32),
                     ens.left, ens.right, ens.value, ens.n_features)
    neg = W.Ensemble(ens.tree_offsets, ens.feature, np.where(internal, np.float32(-np.inf), 0).astype(np.float32),
                     ens.left, ens.right, ens.value, ens.n_features)
    for rule in RULES:
        _, ids, _ = oracle.score(pos, X, rule=rule)
        assert np.all(ids == np.asarray(leftmost)[None, :])
    _, ids, _ = oracle.score(neg, X, rule=0)
    assert np.all(ids == np.asarray(rightmost)[None, :])
    Xn = X.copy()
    Xn[:, :] = -np.inf  # -inf >= -inf: right under the paper's rule, left under the strict one
    _, ids, _ = oracle.score(neg, Xn, rule=0)
    assert np.all(ids == np.asarray(rightmost)[None, :])
    _, ids, _ = oracle.score(neg, Xn, rule=1)
    assert np.all(ids == np.asarray(leftmost)[None, :])


# ------------------------------------------------------------------------------------------
# the paper's leaf-equiprobable generator as a known-answer test (Section 4.1)
# ------------------------------------------------------------------------------------------
def _known_answer_docs(ens, t, rule, rng):
    """For every leaf of tree t, a document built from the leaf's root path: each ancestor
    contributes a value below its threshold when the path goes left and at/above it when it
    goes right (Section 4.1). When a feature repeats on the path, the constraints are
    intersected; a leaf whose interval is empty is unreachable and skipped."""
    fe, th, le, ri, _ = ens.tree(t)
    docs, want = [], []
    for leaf, path in brute.leaf_paths(fe, th, le, ri):
        lo = {}
        hi = {}
        for f, theta, went_right in path:
            theta = float(theta)
            if went_right:  # x >= theta (ge) or x > theta (gt)
                lo[f] = max(lo.get(f, -math.inf), theta)
            else:
                hi[f] = min(hi.get(f, math.inf), theta)
        x = rng.random(ens.n_features, dtype=np.float32) * 4 - 2
        ok = True
        for f in set(lo) | set(hi):
            a, b = lo.get(f, -math.inf), hi.get(f, math.inf)
            if rule == 0:  # need a <= x < b
                v = np.float32(a) if a > -math.inf else np.nextafter(np.float32(b), np.float32(-np.inf))
                ok &= bool(v >= np.float32(a)) and bool(v < np.float32(b))
            else:  # need a < x <= b
                v = np.float32(b) if b < math.inf else np.nextafter(np.float32(a), np.float32(np.inf))
                ok &= bool(v > np.float32(a)) and bool(v <= np.float32(b))
            x[f] = v
        if ok:
            docs.append(x)
            want.append(leaf)
    return np.asarray(docs, dtype=np.float32).reshape(-1, ens.n_features), want


@pytest.mark.parametrize("seed", range(5))
@pytest.mark.parametrize("rule", RULES)
def test_leaf_equiprobable_known_answers(seed, rule):
    rng = np.random.default_rng(seed)
    ens = W.random_ensemble(seed, n_trees=8, n_features=4, min_leaves=2, max_leaves=40)
    for t in range(ens.n_trees):
        X, want = _known_answer_docs(ens, t, rule, rng)
        assert len(want) >= 1
        single = ens.take_trees(t + 1)
        _, ids, _ = oracle.score(single, X, rule=rule)
        assert np.array_equal(ids[:, t], np.asarray(want, dtype=np.int32))


# ------------------------------------------------------------------------------------------
# the three walks agree on the configurations' own shapes
# ------------------------------------------------------------------------------------------
@pytest.mark.parametrize("wl", ["tiny_10x8", "rank_1kx32", "wide_1kx64_f700", "shallow_20kx8_1M", "large_5kx256_f700_1M"])
@pytest.mark.parametrize("rule", RULES)
def test_walks_agree_on_workloads(wl, rule):
    cfg = W.WORKLOADS[wl]
    ens = W.make_ensemble(cfg, n_trees=min(cfg.n_trees, 40))
    X = W.make_docs(cfg, n_docs=300)
    s0, i0, v0 = oracle.score(ens, X, rule=rule, walk=0)
    s1, i1, v1 = oracle.score(ens, X, rule=rule, walk=1)
    assert np.array_equal(i0, i1) and np.array_equal(s0, s1) and v0 == v1
    s2, i2 = oracle.score_padded(ens, X, rule=rule, max_depth=24)
    assert np.array_equal(i0, i2) and np.array_equal(s0, s2)


# ------------------------------------------------------------------------------------------
# invariants
# ------------------------------------------------------------------------------------------
def _slice(ens, a, b):
    """Trees [a, b) of an ensemble as an ensemble of their own."""
    lo, hi = int(ens.tree_offsets[a]), int(ens.tree_offsets[b])
    return W.Ensemble(ens.tree_offsets[a:b + 1] - lo, ens.feature[lo:hi], ens.threshold[lo:hi],
                      ens.left[lo:hi], ens.right[lo:hi], ens.value[lo:hi], ens.n_features)


def _cat(a, b):
    return W.Ensemble(np.concatenate([a.tree_offsets, b.tree_offsets[1:] + a.tree_offsets[-1]]),
                      np.concatenate([a.feature, b.feature]), np.concatenate([a.threshold, b.threshold]),
                      np.concatenate([a.left, b.left]), np.concatenate([a.right, b.right]),
                      np.concatenate([a.value, b.value]), a.n_features)


def test_invariants():
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg, n_trees=60)
    X = W.make_docs(cfg, n_docs=400)
    s, ids, _ = oracle.score(ens, X)
    # additivity over a split of the trees
    a, b = _slice(ens, 0, 25), _slice(ens, 25, ens.n_trees)
    sa, ia, _ = oracle.score(a, X)
    sb, ib, _ = oracle.score(b, X)
    assert np.array_equal(np.concatenate([ia, ib], axis=1), ids)
    assert np.allclose(sa + sb, s, rtol=1e-13, atol=1e-13)
    assert np.array_equal(oracle.score(_cat(a, b), X)[0], s)
    # scaling leaf values by 2 scales the scores exactly
    ens2 = W.Ensemble(ens.tree_offsets, ens.feature, ens.threshold, ens.left, ens.right,
                      (ens.value * 2).astype(np.float32), ens.n_features)
    assert np.array_equal(oracle.score(ens2, X)[0], 2 * s)
    # scaling features and thresholds by 2 (exact in binary) keeps every leaf
    ens3 = W.Ensemble(ens.tree_offsets, ens.feature, (ens.threshold * 2).astype(np.float32), ens.left,
                      ens.right, ens.value, ens.n_features)
    assert np.array_equal(oracle.score(ens3, (X * 2).astype(np.float32))[1], ids)
    # permuting documents permutes scores
    perm = np.random.default_rng(1).permutation(X.shape[0])
    sp, ip, _ = oracle.score(ens, X[perm])
    assert np.array_equal(sp, s[perm]) and np.array_equal(ip, ids[perm])
    # renumbering nodes maps the leaf ids and keeps the scores
    ens4, maps = W.relabel_nodes(ens, 3)
    s4, i4, _ = oracle.score(ens4, X)
    assert np.array_equal(s4, s)
    for t in range(ens.n_trees):
        assert np.array_equal(i4[:, t], maps[t][ids[:, t]])
    # reversing the tree order keeps the scores up to rounding
    rev = _slice(ens, 0, 1)
    for t in range(1, ens.n_trees):
        rev = _cat(_slice(ens, t, t + 1), rev)
    sr, ir, _ = oracle.score(rev, X)
    assert np.array_equal(ir[:, ::-1], ids)
    assert np.allclose(sr, s, rtol=1e-12, atol=1e-13)


def test_strict_rule_equals_nudged_threshold():
    # right iff x > theta  <=>  right iff x >= next float32 above theta (no float32 lies
    # strictly between them); theta = +inf has no successor: x > +inf is never true, which is
    # what a NaN threshold gives under >=.
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg, n_trees=50)
    X = W.make_docs(cfg, n_docs=500)
    internal = ens.feature >= 0
    thr = ens.threshold.copy()
    thr[internal.nonzero()[0][:5]] = np.float32(np.inf)
    ens = W.Ensemble(ens.tree_offsets, ens.feature, thr, ens.left, ens.right, ens.value, ens.n_features)
    nudged = np.nextafter(thr, np.float32(np.inf)).astype(np.float32)
    nudged[np.isposinf(thr)] = np.float32(np.nan)
    ens_n = W.Ensemble(ens.tree_offsets, ens.feature, np.where(internal, nudged, thr).astype(np.float32),
                       ens.left, ens.right, ens.value, ens.n_features)
    _, ids_gt, _ = oracle.score(ens, X, rule=1)
    _, ids_ge, _ = oracle.score(ens_n, X, rule=0)
    assert np.array_equal(ids_gt, ids_ge)
    # and ties really occur here (thresholds are drawn from feature values)
    _, ids_ge0, _ = oracle.score(ens, X, rule=0)
    assert not np.array_equal(ids_ge0, ids_gt)


def test_thread_count_does_not_change_results():
    cfg = W.WORKLOADS["wide_1kx64_f700"]
    ens = W.make_ensemble(cfg, n_trees=30)
    X = W.make_docs(cfg, n_docs=700)
    a = oracle.score(ens, X, threads=1)
    b = oracle.score(ens, X, threads=4)
    assert np.array_equal(a[0], b[0]) and np.array_equal(a[1], b[1]) and a[2] == b[2]


def test_malformed_model_is_reported():
    ens, X, _ = load_hand_ensemble()
    bad = W.Ensemble(ens.tree_offsets, ens.feature, ens.threshold, ens.left.copy(), ens.right, ens.value,
                     ens.n_features)
    bad.left[0] = 99  # out of range child
    with pytest.raises(oracle.OracleError):
        oracle.score(bad, X)
    cyc = W.Ensemble(ens.tree_offsets, ens.feature, ens.threshold, ens.left.copy(), ens.right, ens.value,
                     ens.n_features)
    a = int(ens.tree_offsets[1])
    cyc.left[a + 3] = 0  # node 3 of tree 1 points back to the root
    with pytest.raises(oracle.OracleError):
        oracle.score(cyc, np.full((1, 3), 0.5, dtype=np.float32))  # root -> 3 -> (left) root ...
