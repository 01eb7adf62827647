"""The seeded generators produce the configured shapes and distributions, deterministically."""
from __future__ import annotations

import numpy as np
import pytest

import workloads as W


def _depths(fe, le, ri):
    d = np.zeros(len(fe), dtype=np.int64)
    stack = [0]
    while stack:
        n = stack.pop()
        if fe[n] >= 0:
            d[le[n]] = d[ri[n]] = d[n] + 1
            stack += [int(le[n]), int(ri[n])]
    return d


@pytest.mark.parametrize("wl", sorted(W.WORKLOADS))
def test_workload_shapes_and_seeds(wl):
    cfg = W.WORKLOADS[wl]
    T = min(cfg.n_trees, 200)
    ens = W.make_ensemble(cfg, n_trees=T)
    assert ens.n_trees == T
    assert ens.tree_offsets[0] == 0 and np.all(np.diff(ens.tree_offsets) == 2 * cfg.n_leaves - 1)
    not_bfs = 0
    for t in range(T):
        fe, th, le, ri, va = ens.tree(t)
        internal = fe >= 0
        assert (fe < 0).sum() == cfg.n_leaves
        assert np.all(fe[internal] < cfg.n_features)
        assert np.all(le[~internal] == -1) and np.all(ri[~internal] == -1)
        assert np.all(ri[internal] == le[internal] + 1)  # a split appends left then right
        d = _depths(fe, le, ri)
        if cfg.max_depth is not None:
            assert d[~internal].max() <= cfg.max_depth
        if cfg.complete:
            assert np.all(d[~internal] == cfg.max_depth)
        bfs = np.argsort(d, kind="stable")
        not_bfs += int(not np.array_equal(bfs, np.arange(len(fe))))
        if cfg.thresholds == "uniform":
            assert np.all((th[internal] >= 0) & (th[internal] < 1))
        if cfg.thresholds == "sample_nonzero":
            assert np.all(th[internal] != 0)
    assert not_bfs > T // 2  # creation order is usually not breadth-first
    X = W.make_docs(cfg, n_docs=3000)
    assert X.shape == (3000, cfg.n_features) and X.dtype == np.float32 and X.flags.c_contiguous
    assert abs(float((X == 0).mean()) - cfg.zero_frac) < 0.01
    assert np.all(np.isfinite(X)) and np.all(X >= 0)
    if cfg.nonzero == "uniform":
        assert X.max() < 1


def test_determinism_and_prefixes():
    cfg = W.WORKLOADS["rank_1kx32"]
    a = W.make_ensemble(cfg, n_trees=30)
    b = W.make_ensemble(cfg, n_trees=10)
    c = a.take_trees(10)
    for name in ("tree_offsets", "feature", "threshold", "left", "right", "value"):
        assert np.array_equal(getattr(b, name), getattr(c, name))
    X1 = W.make_docs(cfg, n_docs=9000)
    X2 = W.make_docs(cfg, n_docs=2500, start=4000)
    assert np.array_equal(X1[4000:6500], X2)
    assert not np.array_equal(W.make_docs(W.WORKLOADS["shallow_20kx8_1M"], n_docs=10), W.make_docs(W.WORKLOADS["tiny_10x8"], n_docs=10))


def test_thresholds_come_from_the_sample():
    cfg = W.WORKLOADS["large_5kx256_f700_1M"]
    S = W.make_threshold_sample(cfg)
    ens = W.make_ensemble(cfg, n_trees=5)
    internal = ens.feature >= 0
    for n in np.nonzero(internal)[0][:300]:
        assert ens.threshold[n] in S[:, ens.feature[n]]
    assert (ens.threshold[internal] == 0).mean() > 0.3  # half the sample is zeros


def test_query_groups():
    g = W.make_query_groups(W.WORKLOADS["rank_1kx32"])
    assert g.sum() == W.WORKLOADS["rank_1kx32"].n_docs
    assert g[:-1].min() >= 20 and g.max() <= 200


def test_relabel_keeps_structure():
    ens = W.random_ensemble(3, 5, 4, min_leaves=1, max_leaves=9)
    rel, maps = W.relabel_nodes(ens, 1)
    for t in range(ens.n_trees):
        fe, th, le, ri, va = ens.tree(t)
        f2, t2, l2, r2, v2 = rel.tree(t)
        m = maps[t]
        assert np.array_equal(f2[m], fe) and np.array_equal(v2[m], va)
        internal = fe >= 0
        assert np.array_equal(l2[m][internal], m[le[internal]])
