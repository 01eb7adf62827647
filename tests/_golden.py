"""Parser for the hand-worked fixtures under tests/golden/ (format described in each file)."""
from __future__ import annotations

import os

import numpy as np

from workloads import Ensemble

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _f(tok: str) -> float:
    return float.fromhex(tok) if tok.lower().startswith(("0x", "-0x")) else float(tok)


def load_hand_ensemble(name: str = "hand_ensemble.txt"):
    """Returns (ensemble, X float32, expects) where expects[rule] = list of
    (doc, score, visits, [leaf ids]) and expects["usage_" + rule] = list of (doc, [feature ids])."""
    trees: list[dict] = []
    docs: dict[int, list[float]] = {}
    expects: dict[str, list] = {"ge": [], "gt": [], "usage_ge": [], "usage_gt": []}
    n_features = None
    with open(os.path.join(GOLDEN, name)) as fh:
        for line in fh:
            line = line.split("#", 1)[0].strip()
            if not line:
                continue
            tok = line.split()
            if tok[0] == "features":
                n_features = int(tok[1])
            elif tok[0] == "tree":
                assert int(tok[1]) == len(trees)
                trees.append({})
            elif tok[0] == "node":
                trees[-1][int(tok[1])] = (int(tok[2]), _f(tok[3]), int(tok[4]), int(tok[5]), _f(tok[6]))
            elif tok[0] == "doc":
                docs[int(tok[1])] = [_f(t) for t in tok[2:]]
            elif tok[0] == "expect":
                expects[tok[1]].append((int(tok[2]), _f(tok[3]), int(tok[4]), [int(t) for t in tok[5:]]))
            elif tok[0] == "usage":
                expects["usage_" + tok[1]].append((int(tok[2]), [int(t) for t in tok[3:]]))
            else:
                raise ValueError(f"bad golden line: {line}")
    feats, thrs, lefts, rights, vals, offs = [], [], [], [], [], [0]
    for tr in trees:
        n = len(tr)
        assert sorted(tr) == list(range(n))
        for i in range(n):
            f, th, l, r, v = tr[i]
            feats.append(f); thrs.append(th); lefts.append(l); rights.append(r); vals.append(v)
        offs.append(offs[-1] + n)
    ens = Ensemble(np.asarray(offs, np.int64), np.asarray(feats, np.int32), np.asarray(thrs, np.float32),
                   np.asarray(lefts, np.int32), np.asarray(rights, np.int32), np.asarray(vals, np.float32),
                   n_features)
    X = np.asarray([docs[d] for d in sorted(docs)], dtype=np.float32)
    assert X.shape[1] == n_features
    return ens, X, expects
