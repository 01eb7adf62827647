"""Host code under AddressSanitizer and UndefinedBehaviorSanitizer: the packer, the code
generator, the tile-image emulator and the oracle, built with g++/gcc -fsanitize=address,undefined
into one driver (``tests/sanitize_driver.cpp``) and run on seeded models — the hand-worked
ensemble, prefixes of the five workloads (float and coded plans, complete-depth tiles), random
ensembles with IEEE corner values, vector-valued leaves, empty and single-leaf models, and
malformed models that the packer must reject. The emulator's leaf ids must equal the oracle's;
any sanitizer report fails the run."""
from __future__ import annotations

import os
import subprocess

import numpy as np
import pytest

import workloads as W
from _golden import load_hand_ensemble

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1212_2287_amd", "csrc")
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1"]


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    d = tmp_path_factory.mktemp("san")
    obj = str(d / "oracle.o")
    exe = str(d / "sanitize_driver")
    subprocess.run(["gcc", "-std=c11", *SAN, "-c", os.path.join(ROOT, "oracle", "oracle.c"), "-o", obj],
                   check=True)
    subprocess.run(["g++", "-std=c++17", *SAN, "-I", CSRC, os.path.join(ROOT, "tests", "sanitize_driver.cpp"),
                    os.path.join(ROOT, "tests", "pack_emu.cpp"), os.path.join(CSRC, "pack.cpp"),
                    os.path.join(CSRC, "codegen.cpp"), obj, "-lm", "-o", exe], check=True)
    return exe, d


def _write(path, ens, X, values=None, valid=True):
    vals = ens.value if values is None else values
    n_out = 1 if values is None else values.shape[1]
    X = np.ascontiguousarray(X, np.float32)
    with open(path, "wb") as f:
        f.write(np.array([ens.n_trees, X.shape[1]], np.int32).tobytes())
        f.write(np.array([ens.feature.shape[0], X.shape[0]], np.int64).tobytes())
        f.write(np.array([n_out, int(valid)], np.int32).tobytes())
        f.write(np.ascontiguousarray(ens.tree_offsets, np.int64).tobytes())
        f.write(np.ascontiguousarray(ens.feature, np.int32).tobytes())
        f.write(np.ascontiguousarray(ens.threshold, np.float32).tobytes())
        f.write(np.ascontiguousarray(ens.left, np.int32).tobytes())
        f.write(np.ascontiguousarray(ens.right, np.int32).tobytes())
        f.write(np.ascontiguousarray(vals, np.float32).tobytes())
        f.write(X.tobytes())
    return str(path)


def _run(exe, files):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe, *files], capture_output=True, text=True, env=env, timeout=900)
    assert r.returncode == 0, (r.stdout[-2000:], r.stderr[-4000:])
    assert r.stdout.count("ok ") == len(files)


_POOL = np.array([0.0, -0.0, 0.25, 0.5, 1.0, np.inf, -np.inf, np.nan, 1e-45, -3.4e38], np.float32)


def test_valid_models(driver):
    exe, d = driver
    files = []
    ens, X, _ = load_hand_ensemble()
    files.append(_write(d / "hand.bin", ens, X))
    for wl, n_trees, n_docs in (("tiny_10x8", None, 130), ("rank_1kx32", 150, 70), ("wide_1kx64_f700", 60, 40),
                                ("shallow_20kx8_1M", 400, 70), ("large_5kx256_f700_1M", 30, 66)):
        cfg = W.WORKLOADS[wl]
        files.append(_write(d / f"{wl}.bin", W.make_ensemble(cfg, n_trees=n_trees),
                            W.make_docs(cfg, n_docs=n_docs)))
    for seed in range(6):
        F = (1, 7, 33, 136, 260, 5)[seed]
        ens = W.random_ensemble(seed, n_trees=40, n_features=F, min_leaves=1, max_leaves=30,
                                thr_values=_POOL[:7] if seed % 2 else None)
        X = W.random_docs(seed, 97, F, values=_POOL if seed % 2 else None, zero_frac=0.2)
        files.append(_write(d / f"rand{seed}.bin", ens, X))
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg, n_trees=50)
    files.append(_write(d / "vec.bin", ens, W.make_docs(cfg, n_docs=65),
                        values=W.make_leaf_vectors(ens, 3, "dense", seed=1)))
    F = 9
    empty = W.Ensemble(np.zeros(1, np.int64), np.zeros(0, np.int32), np.zeros(0, np.float32),
                       np.zeros(0, np.int32), np.zeros(0, np.int32), np.zeros(0, np.float32), F)
    files.append(_write(d / "empty.bin", empty, W.random_docs(1, 10, F)))
    leaves = W.Ensemble(np.arange(4, dtype=np.int64), np.full(3, -1, np.int32), np.zeros(3, np.float32),
                        np.full(3, -1, np.int32), np.full(3, -1, np.int32), np.ones(3, np.float32), F)
    files.append(_write(d / "leaves.bin", leaves, W.random_docs(2, 10, F)))
    _run(exe, files)


def test_malformed_models(driver):
    """Each malformation must come back as a model error from the packer, with no memory error
    in the packer, the emulator or the oracle on the way."""
    exe, d = driver
    ens, X, _ = load_hand_ensemble()
    t1 = int(ens.tree_offsets[1])  # tree 1's root, an internal node
    cases = {}

    def variant(name, **changes):
        arrs = {k: getattr(ens, k).copy() for k in ("feature", "threshold", "left", "right")}
        for k, (i, v) in changes.items():
            arrs[k][i] = v
        cases[name] = W.Ensemble(ens.tree_offsets, arrs["feature"], arrs["threshold"], arrs["left"],
                                 arrs["right"], ens.value, ens.n_features)

    variant("child_out_of_range", left=(t1, 99))
    variant("child_names_root", left=(t1, 0))
    variant("same_children", left=(t1, int(ens.right[t1])))
    variant("nan_threshold", threshold=(t1, np.nan))
    variant("feature_below_minus_one", feature=(t1, -7))
    # tree 1: root 0 -> (5, 3), node 3 -> (6, 1), node 1 -> (4, 2); node 1's right child becomes
    # its own parent 3: a cycle, node 3 with two parents, node 2 unreachable
    assert int(ens.right[t1 + 3]) == 1 and int(ens.right[t1 + 1]) == 2
    variant("cycle", right=(t1 + 1, 3))
    files = [_write(d / f"bad_{name}.bin", e, X, valid=False) for name, e in cases.items()]
    _run(exe, files)
