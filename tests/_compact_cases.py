"""Seeded random models of the shape the compact packets take: 420 to 767 features, so that
64 float rows leave too little LDS for the trees and the documents are staged as threshold
codes; 5-150 trees of 100-256 leaves (at most 511 nodes) mixed with up to 40 smaller ones
(single leaves among them) in random order; IEEE corner values in thresholds and documents for
about a third of the cases; batches from one document to several thousand. Shared by the GPU
sweep (tests/test_gpu_compact.py) and the host emulator's check that these models do take the
compact packets (tests/test_pack_emu.py). Inputs only: no scoring arithmetic here."""
from __future__ import annotations

import numpy as np

import workloads as W

N_CASES = 24

_POOL = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf, np.nan, 1e-45, 3.4e38, -1.5],
                 np.float32)


def case(seed: int):
    """(ensemble, documents, tie rule, leaf vectors or None, bags) of case `seed`."""
    rng = np.random.default_rng(7000 + seed)
    F = int(rng.choice([420, 500, 600, 700, 767]))
    pooled = bool(rng.random() < 0.3)
    thr = _POOL[:8] if pooled else None
    big = W.random_ensemble(7100 + seed, n_trees=int(rng.integers(5, 150)), n_features=F,
                            min_leaves=int(rng.choice([100, 150, 200])), max_leaves=256, thr_values=thr)
    trees = [big.tree(t) for t in range(big.n_trees)]
    n_small = int(rng.integers(0, 40))
    if n_small:
        small = W.random_ensemble(7200 + seed, n_trees=n_small, n_features=F, min_leaves=1,
                                  max_leaves=int(rng.choice([1, 4, 40, 120])), thr_values=thr)
        trees += [small.tree(t) for t in range(small.n_trees)]
    trees = [trees[i] for i in rng.permutation(len(trees))]
    offs = np.cumsum([0] + [len(t[0]) for t in trees]).astype(np.int64)
    cat = [np.concatenate([np.asarray(t[k], dt) for t in trees]) for k, dt in
           enumerate((np.int32, np.float32, np.int32, np.int32, np.float32))]
    ens = W.Ensemble(offs, *cat, F)
    n_docs = int(rng.choice([1, 63, 64, 65, 200, 3000, 9000]))
    X = W.random_docs(7300 + seed, n_docs, F, values=_POOL if pooled else None,
                      zero_frac=float(rng.random() * 0.6))
    # documents that sit exactly on thresholds (ties under either rule)
    internal = np.nonzero(ens.feature >= 0)[0]
    for _ in range(min(200, 4 * n_docs)):
        n = internal[rng.integers(0, internal.size)]
        X[rng.integers(0, n_docs), ens.feature[n]] = ens.threshold[n]
    rule = int(rng.integers(0, 2))
    n_out = int(rng.choice([1, 1, 1, 3, 6]))
    vals = None if n_out == 1 else W.make_leaf_vectors(ens, n_out, "dense", seed=seed)
    n_bags = int(rng.integers(1, 3))
    return ens, X, rule, vals, n_bags
