"""Seeded synthetic inputs for tree-ensemble scoring.

This module builds regression-tree ensembles and dense feature matrices shaped like the
workloads of the paper (synthetic trees, Section 4.1; learning-to-rank shaped ensembles,
Section 4.2 and Table 1) at five fixed configurations, plus a generic random-ensemble builder
for property tests. It is shared by the oracle tests, the GPU parity tests, ``smoke()`` and
``bench.py``.

It holds none of the scoring arithmetic: nothing here walks a tree, compares a feature with a
threshold or sums leaf values. It only draws structures, feature ids, thresholds, leaf values
and feature matrices from seeded streams.

Flat ensemble format (the format the C ABI takes):

* ``tree_offsets`` int64 ``[T+1]``: tree ``t`` owns flat nodes ``[off[t], off[t+1])``;
* ``feature`` int32: feature id of an internal node, ``-1`` for a leaf;
* ``threshold`` float32: threshold of an internal node (0 for leaves, ignored);
* ``left`` / ``right`` int32: tree-local child ids of an internal node, ``-1`` for a leaf;
* ``value`` float32: regression value of a leaf (0 for internal nodes, ignored).

Nodes are stored in *creation order*: the root is node 0 and splitting a leaf appends its left
then its right child. For random trees this order is not breadth-first, so any consumer that
needs a breadth-first layout has to build it.

Seeding: every stream is a numpy PCG64 generator seeded by
``SeedSequence(12122287, spawn_key=(cfg, stream, index...))``. Trees and document chunks have
streams of their own, so the first ``n`` trees (or documents) of a configuration are the same
whatever total count is requested. That lets tests run a prefix of a 1M-document configuration
and compare it with the bench's full-size run.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Optional

import numpy as np

ROOT_SEED = 12122287  # the arXiv number of the paper, as a fixed root entropy

# stream ids inside one configuration
_S_STRUCT, _S_THRESH, _S_LEAF, _S_X, _S_SAMPLE, _S_QUERY = range(6)

X_CHUNK_ROWS = 4096  # documents per independently seeded chunk of X
SAMPLE_ROWS = 10_000  # rows of the seeded sample that thresholds are drawn from


def _rng(*key: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence(ROOT_SEED, spawn_key=tuple(key))))


@dataclass
class Ensemble:
    """A tree ensemble in the flat creation-order format described in the module docstring."""

    tree_offsets: np.ndarray  # int64 [T+1]
    feature: np.ndarray  # int32 [N]
    threshold: np.ndarray  # float32 [N]
    left: np.ndarray  # int32 [N]
    right: np.ndarray  # int32 [N]
    value: np.ndarray  # float32 [N]
    n_features: int  # number of feature columns the documents carry

    @property
    def n_trees(self) -> int:
        return int(self.tree_offsets.shape[0] - 1)

    @property
    def n_nodes(self) -> int:
        return int(self.feature.shape[0])

    def tree(self, t: int):
        """Arrays of tree ``t`` (tree-local views): feature, threshold, left, right, value."""
        a, b = int(self.tree_offsets[t]), int(self.tree_offsets[t + 1])
        return (self.feature[a:b], self.threshold[a:b], self.left[a:b], self.right[a:b], self.value[a:b])

    def take_trees(self, n: int) -> "Ensemble":
        """The first ``n`` trees as an ensemble of their own."""
        end = int(self.tree_offsets[n])
        return Ensemble(self.tree_offsets[: n + 1].copy(), self.feature[:end].copy(),
                        self.threshold[:end].copy(), self.left[:end].copy(), self.right[:end].copy(),
                        self.value[:end].copy(), self.n_features)


@dataclass(frozen=True)
class Config:
    """One synthetic workload: ensemble shape, threshold rule, leaf and feature distributions."""

    seed_key: int  # first spawn key of the workload's random streams
    name: str
    n_trees: int
    n_leaves: int
    max_depth: Optional[int]  # cap on leaf depth (edges) for random trees; None = no cap
    complete: bool  # complete (perfectly balanced) trees of depth log2(n_leaves)
    n_features: int
    n_docs: int
    zero_frac: float  # fraction of feature values that are exactly +0.0
    nonzero: str  # "uniform" -> U[0,1), "lognormal" -> exp(N(0,1))
    thresholds: str  # "uniform" | "sample" | "sample_nonzero"
    leaf_sigma: float  # leaf values ~ N(0, leaf_sigma) (standard deviation)
    query_groups: bool = False  # docs come in query groups of U{20..200}
    notes: str = ""


_ALL = (
    Config(1, "tiny_10x8", 10, 8, None, False, 136, 1_000, 0.0, "uniform", "uniform", 1.0,
           notes="10 trees x 8 leaves, 7 uniform leaf splits (unbalanced), U[0,1) features"),
    Config(2, "rank_1kx32", 1_000, 32, 16, False, 136, 100_000, 0.30, "lognormal", "sample", 0.1,
           query_groups=True,
           notes="MSLR-shaped: 136 features, 1k trees x 32 leaves, depth <= 16"),
    Config(3, "wide_1kx64_f700", 1_000, 64, 20, False, 700, 50_000, 0.60, "uniform", "sample_nonzero", 0.1,
           notes="wide features: 700 features, 1k trees x 64 leaves, depth <= 20"),
    Config(4, "shallow_20kx8_1M", 20_000, 8, 3, True, 136, 1_000_000, 0.0, "uniform", "uniform", 0.01,
           notes="20k complete depth-3 trees, 1M docs"),
    Config(5, "large_5kx256_f700_1M", 5_000, 256, 24, False, 700, 1_000_000, 0.50, "lognormal", "sample", 0.01,
           notes="5k trees x 256 leaves, depth <= 24, 700 features, 1M docs (model exceeds LDS)"),
)
# the five workloads by name
WORKLOADS = {c.name: c for c in _ALL}


# ----------------------------------------------------------------------------------------------
# feature values
# ----------------------------------------------------------------------------------------------
def _feature_block(rng_mask: np.random.Generator, rng_val: np.random.Generator, rows: int, cols: int,
                   zero_frac: float, nonzero: str) -> np.ndarray:
    """``rows x cols`` float32 block: exact +0.0 with probability ``zero_frac``, else the
    nonzero distribution. Values are drawn for every cell (zeros then overwrite), so the block
    is a fixed function of the two streams."""
    if nonzero == "uniform":
        vals = rng_val.random((rows, cols), dtype=np.float32)
    elif nonzero == "lognormal":
        vals = np.exp(rng_val.standard_normal((rows, cols))).astype(np.float32)
    else:
        raise ValueError(f"unknown nonzero distribution {nonzero!r}")
    if zero_frac > 0.0:
        zero = rng_mask.random((rows, cols)) < zero_frac
        vals[zero] = np.float32(0.0)
    return vals


def make_docs(cfg: Config, n_docs: Optional[int] = None, start: int = 0) -> np.ndarray:
    """Documents ``[start, start+n_docs)`` of configuration ``cfg`` as a row-major float32
    ``[n_docs][n_features]`` array. Every chunk of ``X_CHUNK_ROWS`` rows is drawn whole from
    streams of its own, so any row range is reproducible on its own."""
    n = cfg.n_docs - start if n_docs is None else int(n_docs)
    F = cfg.n_features
    out = np.empty((n, F), dtype=np.float32)
    end = start + n
    if n <= 0:
        return out
    for k in range(start // X_CHUNK_ROWS, (end - 1) // X_CHUNK_ROWS + 1):
        c0 = k * X_CHUNK_ROWS
        blk = _feature_block(_rng(cfg.seed_key, _S_X, k, 0), _rng(cfg.seed_key, _S_X, k, 1), X_CHUNK_ROWS, F,
                             cfg.zero_frac, cfg.nonzero)
        lo, hi = max(start, c0), min(end, c0 + X_CHUNK_ROWS)
        out[lo - start:hi - start] = blk[lo - c0:hi - c0]
    return out


def make_threshold_sample(cfg: Config) -> np.ndarray:
    """The seeded ``SAMPLE_ROWS x n_features`` sample (same distribution as the documents,
    independent stream) that data-driven thresholds are drawn from."""
    return _feature_block(_rng(cfg.seed_key, _S_SAMPLE, 0), _rng(cfg.seed_key, _S_SAMPLE, 1), SAMPLE_ROWS,
                          cfg.n_features, cfg.zero_frac, cfg.nonzero)


def make_query_groups(cfg: Config, n_docs: Optional[int] = None) -> np.ndarray:
    """Query-group sizes U{20..200} covering ``n_docs`` documents (the last group truncated)."""
    n = cfg.n_docs if n_docs is None else int(n_docs)
    rng = _rng(cfg.seed_key, _S_QUERY)
    sizes = []
    total = 0
    while total < n:
        s = int(rng.integers(20, 201))
        s = min(s, n - total)
        sizes.append(s)
        total += s
    return np.asarray(sizes, dtype=np.int64)


# ----------------------------------------------------------------------------------------------
# tree structures (creation order: root 0, a split appends left then right)
# ----------------------------------------------------------------------------------------------
def grow_random_structure(rng: np.random.Generator, n_leaves: int, max_depth: Optional[int],
                          n_features: int):
    """Random unbalanced binary tree with exactly ``n_leaves`` leaves: ``n_leaves-1`` times,
    split a leaf chosen uniformly among the leaves whose depth is below ``max_depth`` and give
    the new internal node a feature id uniform on ``[0, n_features)``.

    Returns (feature, left, right) int32 arrays in creation order."""
    n_split = n_leaves - 1
    u = rng.random(n_split)
    fids = rng.integers(0, n_features, size=n_split)
    n_nodes = 2 * n_leaves - 1
    feature = np.full(n_nodes, -1, dtype=np.int32)
    left = np.full(n_nodes, -1, dtype=np.int32)
    right = np.full(n_nodes, -1, dtype=np.int32)
    depth = [0] * n_nodes
    elig = [0]  # leaves that may still be split, in a deterministic order
    nxt = 1
    cap = max_depth if max_depth is not None else n_nodes
    for s in range(n_split):
        if not elig:
            raise ValueError(f"cannot place {n_leaves} leaves under max depth {max_depth}")
        i = int(u[s] * len(elig))
        node = elig[i]
        elig[i] = elig[-1]
        elig.pop()
        feature[node] = fids[s]
        left[node] = nxt
        right[node] = nxt + 1
        d = depth[node] + 1
        depth[nxt] = depth[nxt + 1] = d
        if d < cap:
            elig.append(nxt)
            elig.append(nxt + 1)
        nxt += 2
    return feature, left, right


def grow_complete_structure(rng: np.random.Generator, depth: int, n_features: int):
    """Complete tree of the given depth (``2**depth`` leaves), nodes created depth-first
    (split a node, then fully grow its left subtree, then its right one), so the creation order
    differs from breadth-first order for ``depth >= 2``. Feature ids uniform on
    ``[0, n_features)``, drawn in creation order of the internal nodes."""
    n_int = (1 << depth) - 1
    fids = rng.integers(0, n_features, size=n_int)
    n_nodes = 2 * n_int + 1
    feature = np.full(n_nodes, -1, dtype=np.int32)
    left = np.full(n_nodes, -1, dtype=np.int32)
    right = np.full(n_nodes, -1, dtype=np.int32)
    state = {"next": 1, "k": 0}

    def grow(node: int, d: int) -> None:
        if d == depth:
            return
        feature[node] = fids[state["k"]]
        state["k"] += 1
        l, r = state["next"], state["next"] + 1
        state["next"] += 2
        left[node], right[node] = l, r
        grow(l, d + 1)
        grow(r, d + 1)

    grow(0, 0)
    return feature, left, right


def _draw_thresholds(cfg: Config, rng: np.random.Generator, feature: np.ndarray,
                     sample: Optional[np.ndarray], nz_cols: Optional[list]) -> np.ndarray:
    thr = np.zeros(feature.shape[0], dtype=np.float32)
    internal = np.nonzero(feature >= 0)[0]
    if cfg.thresholds == "uniform":
        thr[internal] = rng.random(internal.shape[0], dtype=np.float32)
    elif cfg.thresholds == "sample":
        rows = rng.integers(0, sample.shape[0], size=internal.shape[0])
        thr[internal] = sample[rows, feature[internal]]
    elif cfg.thresholds == "sample_nonzero":
        u = rng.random(internal.shape[0])
        for j, n in enumerate(internal):
            col = nz_cols[feature[n]]
            thr[n] = col[int(u[j] * col.shape[0])]
    else:
        raise ValueError(f"unknown threshold rule {cfg.thresholds!r}")
    return thr


def make_ensemble(cfg: Config, n_trees: Optional[int] = None) -> Ensemble:
    """The first ``n_trees`` trees (default: all) of configuration ``cfg``."""
    T = cfg.n_trees if n_trees is None else int(n_trees)
    sample = nz_cols = None
    if cfg.thresholds in ("sample", "sample_nonzero"):
        sample = make_threshold_sample(cfg)
        if cfg.thresholds == "sample_nonzero":
            nz_cols = [sample[:, f][sample[:, f] != 0] for f in range(cfg.n_features)]
            if any(c.shape[0] == 0 for c in nz_cols):
                raise ValueError("a sample column has no nonzero entry")
    feats, thrs, lefts, rights, vals = [], [], [], [], []
    offsets = np.zeros(T + 1, dtype=np.int64)
    for t in range(T):
        rs = _rng(cfg.seed_key, _S_STRUCT, t)
        if cfg.complete:
            depth = int(cfg.n_leaves).bit_length() - 1
            if (1 << depth) != cfg.n_leaves:
                raise ValueError("complete trees need a power-of-two leaf count")
            f, l, r = grow_complete_structure(rs, depth, cfg.n_features)
        else:
            f, l, r = grow_random_structure(rs, cfg.n_leaves, cfg.max_depth, cfg.n_features)
        thr = _draw_thresholds(cfg, _rng(cfg.seed_key, _S_THRESH, t), f, sample, nz_cols)
        val = np.zeros(f.shape[0], dtype=np.float32)
        leaves = np.nonzero(f < 0)[0]
        val[leaves] = (_rng(cfg.seed_key, _S_LEAF, t).normal(0.0, cfg.leaf_sigma, leaves.shape[0])
                       .astype(np.float32))
        feats.append(f)
        thrs.append(thr)
        lefts.append(l)
        rights.append(r)
        vals.append(val)
        offsets[t + 1] = offsets[t] + f.shape[0]
    return Ensemble(offsets, np.concatenate(feats), np.concatenate(thrs), np.concatenate(lefts),
                    np.concatenate(rights), np.concatenate(vals), cfg.n_features)


def make_leaf_vectors(ens: Ensemble, n_outputs: int, kind: str = "dense", sigma: float = 0.1,
                      seed: int = 0) -> np.ndarray:
    """float32 [n_nodes, n_outputs] leaf rows for a vector-valued version of ``ens`` (internal
    nodes' rows are zero):
      * "dense": every component N(0, sigma) (multi-output regression);
      * "class": tree t adds to class t % n_outputs only, with the tree's own leaf value (the
        one-tree-per-class-per-round layout of multi-class boosting);
      * "probs": a probability vector per leaf, the normalised magnitudes of N(0, 1) draws
        (a forest classifier's class distributions)."""
    rng = _rng(9000, seed, n_outputs)
    leaf = ens.feature < 0
    out = np.zeros((ens.n_nodes, n_outputs), dtype=np.float32)
    if kind == "dense":
        out[leaf] = rng.normal(0.0, sigma, (int(leaf.sum()), n_outputs)).astype(np.float32)
    elif kind == "class":
        tree_of = np.repeat(np.arange(ens.n_trees), np.diff(ens.tree_offsets))
        rows = np.nonzero(leaf)[0]
        out[rows, tree_of[rows] % n_outputs] = ens.value[rows]
    elif kind == "probs":
        m = np.abs(rng.normal(0.0, 1.0, (int(leaf.sum()), n_outputs)))
        out[leaf] = (m / m.sum(axis=1, keepdims=True)).astype(np.float32)
    else:
        raise ValueError(f"unknown leaf vector kind {kind!r}")
    return out


def scaled(cfg: Config, n_docs: Optional[int] = None, n_trees: Optional[int] = None) -> Config:
    """Same configuration with fewer documents and/or trees (a prefix of the full one)."""
    from dataclasses import replace
    return replace(cfg, n_docs=cfg.n_docs if n_docs is None else int(n_docs),
                   n_trees=cfg.n_trees if n_trees is None else int(n_trees))


# ----------------------------------------------------------------------------------------------
# generic random ensembles for property tests
# ----------------------------------------------------------------------------------------------
def random_ensemble(seed: int, n_trees: int, n_features: int, min_leaves: int = 1, max_leaves: int = 16,
                    max_depth: Optional[int] = None, thr_values: Optional[np.ndarray] = None,
                    leaf_sigma: float = 1.0) -> Ensemble:
    """Small random ensemble: each tree gets a leaf count uniform on
    ``[min_leaves, max_leaves]`` (1 = a single-leaf tree), random unbalanced structure,
    thresholds U[0,1) or drawn from ``thr_values`` (to create ties with documents built from
    the same values), leaf values N(0, leaf_sigma)."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(ROOT_SEED, spawn_key=(1000, seed))))
    feats, thrs, lefts, rights, vals = [], [], [], [], []
    offsets = np.zeros(n_trees + 1, dtype=np.int64)
    for t in range(n_trees):
        L = int(rng.integers(min_leaves, max_leaves + 1))
        if max_depth is not None:
            L = min(L, 1 << max_depth)
        f, l, r = grow_random_structure(rng, L, max_depth, n_features)
        thr = np.zeros(f.shape[0], dtype=np.float32)
        internal = np.nonzero(f >= 0)[0]
        if thr_values is None:
            thr[internal] = rng.random(internal.shape[0], dtype=np.float32)
        else:
            thr[internal] = np.asarray(thr_values, dtype=np.float32)[
                rng.integers(0, len(thr_values), size=internal.shape[0])]
        val = np.zeros(f.shape[0], dtype=np.float32)
        lv = np.nonzero(f < 0)[0]
        val[lv] = rng.normal(0.0, leaf_sigma, lv.shape[0]).astype(np.float32)
        feats.append(f)
        thrs.append(thr)
        lefts.append(l)
        rights.append(r)
        vals.append(val)
        offsets[t + 1] = offsets[t] + f.shape[0]
    return Ensemble(offsets, np.concatenate(feats), np.concatenate(thrs), np.concatenate(lefts),
                    np.concatenate(rights), np.concatenate(vals), n_features)


def random_docs(seed: int, n_docs: int, n_features: int, values: Optional[np.ndarray] = None,
                zero_frac: float = 0.0) -> np.ndarray:
    """``n_docs x n_features`` float32 documents, U[0,1) or drawn from ``values``, with an
    optional fraction of exact zeros."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(ROOT_SEED, spawn_key=(2000, seed))))
    if values is None:
        X = rng.random((n_docs, n_features), dtype=np.float32)
    else:
        X = np.asarray(values, dtype=np.float32)[rng.integers(0, len(values), size=(n_docs, n_features))]
    if zero_frac > 0:
        X[rng.random((n_docs, n_features)) < zero_frac] = np.float32(0.0)
    return np.ascontiguousarray(X)


def relabel_nodes(ens: Ensemble, seed: int) -> tuple[Ensemble, list]:
    """Same ensemble with each tree's non-root nodes renumbered by a random permutation (the
    root stays node 0). Returns the new ensemble and, per tree, the map old id -> new id."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(ROOT_SEED, spawn_key=(3000, seed))))
    feats, thrs, lefts, rights, vals, maps = [], [], [], [], [], []
    for t in range(ens.n_trees):
        f, th, l, r, v = ens.tree(t)
        n = f.shape[0]
        perm = np.concatenate([[0], 1 + rng.permutation(n - 1)]).astype(np.int64)  # old -> new
        nf = np.empty_like(f)
        nth = np.empty_like(th)
        nl = np.empty_like(l)
        nr = np.empty_like(r)
        nv = np.empty_like(v)
        nf[perm] = f
        nth[perm] = th
        nv[perm] = v
        nl[perm] = np.where(l >= 0, perm[np.maximum(l, 0)], -1)
        nr[perm] = np.where(r >= 0, perm[np.maximum(r, 0)], -1)
        feats.append(nf)
        thrs.append(nth)
        lefts.append(nl)
        rights.append(nr)
        vals.append(nv)
        maps.append(perm)
    return (Ensemble(ens.tree_offsets.copy(), np.concatenate(feats), np.concatenate(thrs),
                     np.concatenate(lefts), np.concatenate(rights), np.concatenate(vals), ens.n_features),
            maps)
