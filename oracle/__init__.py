"""Oracle for tree-ensemble scoring -- TEST INFRASTRUCTURE ONLY.

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may import
this package. The GPU library never loads it and shares no code with it.

* ``liboracle.so`` (built from ``oracle.c`` with plain ``gcc -O2 -fopenmp``): the definition of
  the score written out -- a branching walk, a predicated walk and the literal padded
  breadth-first predicated walk (Section 3 of the paper), leaf values summed in double precision
  in tree order (Section 5.3); and the feature-access trace, the distinct features each
  document's walks compare (Section 6, Table 4); vector-valued leaves and bagged ensembles
  (Sections 3 and 5.3).
* ``brute.py``: a path-conjunction brute force for tiny inputs (a document reaches leaf l iff
  every predicate on the root-to-l path holds), summed with ``math.fsum``.

Every function here is pinned by the CPU tests in ``tests/test_oracle_*.py`` against hand-worked
values, closed forms, invariants and the brute force.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from typing import Optional

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "oracle.c")
LIB = os.path.join(HERE, "liboracle.so")

RULE_GE = 0  # right iff x >= theta (the paper's convention)
RULE_GT = 1  # right iff x > theta

_lib = None


def build(out: str = LIB, src: str = SRC, extra: tuple = ()) -> str:
    """Compile the oracle with plain ``gcc -O2 -fopenmp`` (no vectorisation tricks)."""
    cmd = ["gcc", "-O2", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-Wall", "-Werror",
           *extra, src, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def _bind(lib: ctypes.CDLL) -> ctypes.CDLL:
    P = ctypes.c_void_p
    i32, i64 = ctypes.c_int32, ctypes.c_int64
    lib.oracle_score.restype = ctypes.c_int
    lib.oracle_score.argtypes = [i32, P, P, P, P, P, P, P, i64, i32, i32, i32, i32, P, P, P]
    lib.oracle_score_padded.restype = ctypes.c_int
    lib.oracle_score_padded.argtypes = [i32, P, P, P, P, P, P, P, i64, i32, i32, i32, P, P]
    lib.oracle_score_multi.restype = ctypes.c_int
    lib.oracle_score_multi.argtypes = [i32, P, P, P, P, P, P, i32, i32, P, i64, i32, i32, i32, P]
    lib.oracle_feature_usage.restype = ctypes.c_int
    lib.oracle_feature_usage.argtypes = [i32, P, P, P, P, P, P, i64, i32, i32, i32, P, P]
    lib.oracle_max_threads.restype = ctypes.c_int
    lib.oracle_max_threads.argtypes = []
    return lib


def load(path: Optional[str] = None) -> ctypes.CDLL:
    """Load the built oracle (building it first only if no library exists)."""
    global _lib
    if path is not None:
        return _bind(ctypes.CDLL(path))
    if _lib is None:
        override = os.environ.get("ORACLE_LIB")  # mutation tests load a deliberately broken build
        if override:
            _lib = _bind(ctypes.CDLL(override))
        else:
            if not os.path.exists(LIB):
                build()
            _lib = _bind(ctypes.CDLL(LIB))
    return _lib


def _p(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data


def _model_arrays(ens):
    return (np.ascontiguousarray(ens.tree_offsets, dtype=np.int64),
            np.ascontiguousarray(ens.feature, dtype=np.int32),
            np.ascontiguousarray(ens.threshold, dtype=np.float32),
            np.ascontiguousarray(ens.left, dtype=np.int32),
            np.ascontiguousarray(ens.right, dtype=np.int32),
            np.ascontiguousarray(ens.value, dtype=np.float32))


class OracleError(RuntimeError):
    pass


def score(ens, X: np.ndarray, rule: int = RULE_GE, walk: int = 0, threads: int = 0,
          want_leaves: bool = True, lib: Optional[ctypes.CDLL] = None):
    """Score documents ``X`` (float32 ``[n_docs][n_features]``) with ensemble ``ens``.

    ``walk`` 0 = branching walk, 1 = predicated walk over explicit children.
    Returns ``(scores float64 [n_docs], leaf_ids int32 [n_docs][n_trees] or None, visits)``
    where ``visits`` counts the internal nodes visited over all (document, tree) pairs."""
    lib = lib or load()
    off, fe, th, le, ri, va = _model_arrays(ens)
    X = np.ascontiguousarray(X, dtype=np.float32)
    n_docs, n_feat = X.shape
    scores = np.empty(n_docs, dtype=np.float64)
    leaves = np.empty((n_docs, ens.n_trees), dtype=np.int32) if want_leaves else None
    visits = np.zeros(1, dtype=np.int64)
    rc = lib.oracle_score(ens.n_trees, _p(off), _p(fe), _p(th), _p(le), _p(ri), _p(va), _p(X),
                          n_docs, n_feat, rule, walk, threads, _p(scores), _p(leaves), _p(visits))
    if rc != 0:
        raise OracleError(f"oracle_score failed with code {rc}")
    return scores, leaves, int(visits[0])


def score_padded(ens, X: np.ndarray, rule: int = RULE_GE, max_depth: int = 20,
                 lib: Optional[ctypes.CDLL] = None):
    """Scores and leaf ids through the literal padded breadth-first Pred walk."""
    lib = lib or load()
    off, fe, th, le, ri, va = _model_arrays(ens)
    X = np.ascontiguousarray(X, dtype=np.float32)
    n_docs, n_feat = X.shape
    scores = np.empty(n_docs, dtype=np.float64)
    leaves = np.empty((n_docs, ens.n_trees), dtype=np.int32)
    rc = lib.oracle_score_padded(ens.n_trees, _p(off), _p(fe), _p(th), _p(le), _p(ri), _p(va), _p(X),
                                 n_docs, n_feat, rule, max_depth, _p(scores), _p(leaves))
    if rc != 0:
        raise OracleError(f"oracle_score_padded failed with code {rc}")
    return scores, leaves


def score_multi(ens, leaf_values: np.ndarray, X: np.ndarray, n_bags: int = 1, rule: int = RULE_GE,
                threads: int = 0, lib: Optional[ctypes.CDLL] = None) -> np.ndarray:
    """Vector-valued leaves, bagged ensembles: float64 [n_docs, n_outputs] = (sum over trees of
    the reached leaves' rows of ``leaf_values`` [n_nodes, n_outputs]) / n_bags."""
    lib = lib or load()
    off, fe, th, le, ri, _ = _model_arrays(ens)
    vals = np.ascontiguousarray(leaf_values, dtype=np.float32)
    if vals.ndim != 2 or vals.shape[0] != ens.n_nodes:
        raise ValueError("leaf_values must be [n_nodes, n_outputs]")
    X = np.ascontiguousarray(X, dtype=np.float32)
    n_docs, n_feat = X.shape
    out = np.empty((n_docs, vals.shape[1]), dtype=np.float64)
    rc = lib.oracle_score_multi(ens.n_trees, _p(off), _p(fe), _p(th), _p(le), _p(ri), _p(vals),
                                vals.shape[1], n_bags, _p(X), n_docs, n_feat, rule, threads, _p(out))
    if rc != 0:
        raise OracleError(f"oracle_score_multi failed with code {rc}")
    return out


def feature_usage(ens, X: np.ndarray, rule: int = RULE_GE, threads: int = 0,
                  lib: Optional[ctypes.CDLL] = None):
    """Features examined per document over all trees (Section 6, Table 4): (counts int32
    [n_docs], masks uint32 [n_docs][(n_features + 31) // 32], bit f % 32 of word f // 32)."""
    lib = lib or load()
    off, fe, th, le, ri, _ = _model_arrays(ens)
    X = np.ascontiguousarray(X, dtype=np.float32)
    n_docs, n_feat = X.shape
    counts = np.empty(n_docs, dtype=np.int32)
    masks = np.empty((n_docs, (n_feat + 31) // 32), dtype=np.uint32)
    rc = lib.oracle_feature_usage(ens.n_trees, _p(off), _p(fe), _p(th), _p(le), _p(ri), _p(X), n_docs,
                                  n_feat, rule, threads, _p(counts), _p(masks))
    if rc != 0:
        raise OracleError(f"oracle_feature_usage failed with code {rc}")
    return counts, masks


def max_threads(lib: Optional[ctypes.CDLL] = None) -> int:
    return int((lib or load()).oracle_max_threads())
