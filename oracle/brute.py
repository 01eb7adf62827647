"""Path-conjunction brute force for tiny ensembles -- TEST INFRASTRUCTURE ONLY.

A tree partitions feature space into one region per leaf: a document lies in leaf l's region
exactly when every predicate on the root-to-l path holds -- ``x[f] < theta`` for each step into
a left child and ``x[f] >= theta`` for each step into a right child (Section 3 of the paper;
with ``rule=1`` a right step needs ``x[f] > theta`` and a left step ``not (x[f] > theta)``).
This module does not walk the tree for a document: it enumerates every leaf's path once and
tests each document against every leaf's full conjunction. Exactly one leaf must match per
(document, tree); anything else raises. Scores are ``math.fsum`` of the matched leaves' values
(correctly rounded), so they pin the oracle's double-precision tree-order sum.
"""
from __future__ import annotations

import math

import numpy as np


def leaf_paths(feature, threshold, left, right):
    """For one tree, ``[(leaf_id, [(f, theta, went_right), ...]), ...]`` for every leaf,
    found by expanding the tree from the root (each node expanded once)."""
    out = []
    stack = [(0, [])]
    seen = 0
    n_nodes = len(feature)
    while stack:
        node, path = stack.pop()
        seen += 1
        if seen > n_nodes:
            raise ValueError("tree has a cycle or a shared node")
        if feature[node] < 0:
            out.append((node, path))
            continue
        f, th = int(feature[node]), np.float32(threshold[node])
        stack.append((int(left[node]), path + [(f, th, False)]))
        stack.append((int(right[node]), path + [(f, th, True)]))
    return out


def _pred_holds(xf: np.float32, th: np.float32, went_right: bool, rule: int) -> bool:
    right_side = bool(xf >= th) if rule == 0 else bool(xf > th)
    return right_side if went_right else not right_side


def leaves(ens, X: np.ndarray, rule: int = 0) -> np.ndarray:
    """Leaf id reached by every (document, tree): int32 ``[n_docs][n_trees]``."""
    X = np.asarray(X, dtype=np.float32)
    n_docs = X.shape[0]
    out = np.empty((n_docs, ens.n_trees), dtype=np.int32)
    for t in range(ens.n_trees):
        f, th, l, r, _ = ens.tree(t)
        paths = leaf_paths(f, th, l, r)
        for d in range(n_docs):
            x = X[d]
            hits = [leaf for leaf, path in paths
                    if all(_pred_holds(x[pf], pth, pr, rule) for pf, pth, pr in path)]
            if len(hits) != 1:
                raise AssertionError(f"doc {d} tree {t}: {len(hits)} leaves match (expected exactly 1)")
            out[d, t] = hits[0]
    return out


def scores(ens, X: np.ndarray, rule: int = 0, leaf_ids: np.ndarray | None = None) -> np.ndarray:
    """Correctly rounded ``math.fsum`` of the reached leaves' values, float64 ``[n_docs]``."""
    ids = leaves(ens, X, rule) if leaf_ids is None else leaf_ids
    out = np.empty(ids.shape[0], dtype=np.float64)
    for d in range(ids.shape[0]):
        terms = [float(ens.value[int(ens.tree_offsets[t]) + int(ids[d, t])]) for t in range(ens.n_trees)]
        out[d] = math.fsum(terms)
    return out
