"""The packer's tile images, walked on the host exactly as the scoring kernel addresses them
(``tests/pack_emu.cpp``): every LDS access stays in its region, every tree is walked once per
document block, leaves absorb further steps, and the leaf each document reaches matches the
oracle's, at every tiling the launch may pick. This pins the layout before any GPU run."""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle
import workloads as W
import _compact_cases as _CC
from _golden import load_hand_ensemble

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_1212_2287_amd", "csrc")
LEVELS = 5


@pytest.fixture(scope="module")
def emu(tmp_path_factory):
    out = str(tmp_path_factory.mktemp("emu") / "libpackemu.so")
    subprocess.run(["g++", "-O2", "-std=c++17", "-shared", "-fPIC", "-I", CSRC,
                    os.path.join(ROOT, "tests", "pack_emu.cpp"), os.path.join(CSRC, "pack.cpp"),
                    "-o", out], check=True)
    lib = ctypes.CDLL(out)
    P = ctypes.c_void_p
    lib.emu_walk.restype = ctypes.c_int
    lib.emu_walk.argtypes = [ctypes.c_int32, P, P, P, P, P, P, ctypes.c_int32, ctypes.c_uint32, P,
                             ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, P, P, P]
    lib.emu_walk_compact.restype = ctypes.c_int
    lib.emu_walk_compact.argtypes = [ctypes.c_int32, P, P, P, P, P, P, ctypes.c_int32, ctypes.c_uint32, P,
                                     ctypes.c_int64, ctypes.c_int32, P, P, P]
    lib.emu_code_check.restype = ctypes.c_int
    lib.emu_code_check.argtypes = [ctypes.c_int32, P, P, P, P, P, P, ctypes.c_uint32, P]
    lib.emu_message.restype = ctypes.c_char_p
    lib.emu_tree_order.restype = ctypes.c_int
    lib.emu_tree_order.argtypes = [ctypes.c_int32, P, P, P, P, P, P, ctypes.c_uint32, P, P, ctypes.c_int32]
    return lib


def _walk(lib, ens, X, level, flags=0, leaf_values=None):
    vals = ens.value if leaf_values is None else leaf_values
    n_out = 1 if leaf_values is None else leaf_values.shape[1]
    arrs = [np.ascontiguousarray(ens.tree_offsets, np.int64), np.ascontiguousarray(ens.feature, np.int32),
            np.ascontiguousarray(ens.threshold, np.float32), np.ascontiguousarray(ens.left, np.int32),
            np.ascontiguousarray(ens.right, np.int32), np.ascontiguousarray(vals, np.float32)]
    X = np.ascontiguousarray(X, np.float32)
    leaves = np.empty((X.shape[0], ens.n_trees), np.int32)
    scores = np.empty((X.shape[0], n_out), np.float64)
    plan = np.zeros(10, np.int32)
    rc = lib.emu_walk(ens.n_trees, *[a.ctypes.data for a in arrs], n_out, flags, X.ctypes.data,
                      X.shape[0], X.shape[1], level, leaves.ctypes.data, scores.ctypes.data, plan.ctypes.data)
    assert rc == 0, lib.emu_message().decode()
    return leaves, (scores[:, 0] if leaf_values is None else scores), plan


def _walk_compact(lib, ens, X, flags=0, leaf_values=None):
    """Leaf ids, scores and trees per lane of the compact packets, or None when the model has
    none."""
    vals = ens.value if leaf_values is None else leaf_values
    n_out = 1 if leaf_values is None else leaf_values.shape[1]
    arrs = [np.ascontiguousarray(ens.tree_offsets, np.int64), np.ascontiguousarray(ens.feature, np.int32),
            np.ascontiguousarray(ens.threshold, np.float32), np.ascontiguousarray(ens.left, np.int32),
            np.ascontiguousarray(ens.right, np.int32), np.ascontiguousarray(vals, np.float32)]
    X = np.ascontiguousarray(X, np.float32)
    leaves = np.empty((X.shape[0], ens.n_trees), np.int32)
    scores = np.empty((X.shape[0], n_out), np.float64)
    k = np.zeros(2, np.int32)
    rc = lib.emu_walk_compact(ens.n_trees, *[a.ctypes.data for a in arrs], n_out, flags, X.ctypes.data,
                              X.shape[0], X.shape[1], leaves.ctypes.data, scores.ctypes.data, k.ctypes.data)
    if rc == 2:
        return None
    assert rc == 0, lib.emu_message().decode()
    return leaves, (scores[:, 0] if leaf_values is None else scores), int(k[0]), int(k[1])


def _check(lib, ens, X, flags=0, levels=range(LEVELS)):
    ref_scores, ref_leaves, _ = oracle.score(ens, X, rule=flags)
    plans = []
    for lv in levels:
        leaves, scores, plan = _walk(lib, ens, X, lv, flags)
        np.testing.assert_array_equal(leaves, ref_leaves, err_msg=f"tiling {lv}")
        np.testing.assert_allclose(scores, ref_scores, rtol=1e-12, atol=1e-12, err_msg=f"tiling {lv}")
        plans.append(plan)
    # the compact packets, where the model has them, reach the same leaves
    compact = _walk_compact(lib, ens, X, flags)
    if compact is not None:
        leaves, scores = compact[:2]
        np.testing.assert_array_equal(leaves, ref_leaves, err_msg="compact packets")
        np.testing.assert_allclose(scores, ref_scores, rtol=1e-12, atol=1e-12, err_msg="compact packets")
    return plans[0]


@pytest.mark.parametrize("seed", range(8))
def test_random_wide_models(emu, seed):
    """Wide documents: one-workgroup plans of 64-, 32- and 16-document blocks, float and
    threshold-coded, with walker packets (one or two walkers per wave) or shared tiles."""
    rng = np.random.default_rng(100 + seed)
    n_feat = int(rng.choice([200, 300, 700, 1100]))
    ens = W.random_ensemble(100 + seed, n_trees=int(rng.integers(1, 200)), n_features=n_feat,
                            min_leaves=1, max_leaves=int(rng.choice([8, 64, 200, 300])))
    X = W.random_docs(100 + seed, n_docs=int(rng.integers(1, 80)), n_features=n_feat)
    _check(emu, ens, X, flags=seed % 2, levels=(0,))


def test_hand_ensemble_both_rules(emu):
    ens, X, _ = load_hand_ensemble()
    for flags in (0, 1):
        _check(emu, ens, X, flags)


@pytest.mark.parametrize("seed", range(6))
def test_random_ensembles(emu, seed):
    rng = np.random.default_rng(seed)
    n_feat = int(rng.integers(1, 300))
    ens = W.random_ensemble(seed, n_trees=int(rng.integers(1, 400)), n_features=n_feat,
                            min_leaves=1, max_leaves=int(rng.integers(2, 200)))
    X = W.random_docs(seed, n_docs=int(rng.integers(1, 150)), n_features=n_feat)
    _check(emu, ens, X, flags=seed % 2)


@pytest.mark.parametrize("wl,n_trees,n_docs,expect", [
    ("tiny_10x8", None, 200, dict(dl=64, coded=0)),
    ("rank_1kx32", None, 130, dict(dl=64, coded=0)),
    ("wide_1kx64_f700", 300, 70, dict(dl=32, coded=0)),
    ("shallow_20kx8_1M", 3000, 70, dict(dl=64, coded=0)),
    ("large_5kx256_f700_1M", 200, 70, dict(dl=64, coded=1, narrow=0)),
])
def test_workload_shapes(emu, wl, n_trees, n_docs, expect):
    """Prefixes of the benchmark workloads: both record formats, float and coded documents,
    complete-depth tiles (shallow_20kx8_1M), several interleave factors."""
    cfg = W.WORKLOADS[wl]
    ens = W.make_ensemble(cfg, n_trees=n_trees)
    X = W.make_docs(cfg, n_docs=n_docs)
    plan = _check(emu, ens, X, levels=(0, 4))
    assert plan[0] == expect["dl"] and plan[3] == expect["coded"], plan
    if "narrow" in expect:
        assert plan[2] == expect["narrow"], plan


@pytest.mark.parametrize("wl,n_trees,n_out,kind", [
    ("tiny_10x8", None, 3, "probs"),
    ("rank_1kx32", 120, 5, "class"),
    ("shallow_20kx8_1M", 800, 2, "dense"),  # complete-depth tiles
    ("large_5kx256_f700_1M", 60, 7, "dense"),  # coded documents
])
def test_vector_valued_leaves(emu, wl, n_trees, n_out, kind):
    """Leaf records name their row of the leaf-vector table (row 0 = the zero record's); the
    rows summed over the walks equal the oracle's vector-valued scores."""
    cfg = W.WORKLOADS[wl]
    ens = W.make_ensemble(cfg, n_trees=n_trees)
    X = W.make_docs(cfg, n_docs=90)
    vals = W.make_leaf_vectors(ens, n_out, kind, seed=cfg.seed_key)
    ref = oracle.score_multi(ens, vals, X)
    _, ref_leaves, _ = oracle.score(ens, X)
    for lv in (0, 4):
        leaves, scores, _ = _walk(emu, ens, X, lv, leaf_values=vals)
        np.testing.assert_array_equal(leaves, ref_leaves, err_msg=f"tiling {lv}")
        np.testing.assert_allclose(scores, ref, rtol=1e-12, atol=1e-12, err_msg=f"tiling {lv}")
    compact = _walk_compact(emu, ens, X, leaf_values=vals)
    assert (compact is not None) == (wl == "large_5kx256_f700_1M")
    if compact is not None:
        np.testing.assert_array_equal(compact[0], ref_leaves, err_msg="compact packets")
        np.testing.assert_allclose(compact[1], ref, rtol=1e-12, atol=1e-12, err_msg="compact packets")


def test_coded_documents_with_corner_values(emu):
    """Coded plan: NaN, +-inf, +-0 and values equal to thresholds; the emulator checks every
    staged code of the coding kernel's branch-free descent against a plain count."""
    cfg = W.WORKLOADS["large_5kx256_f700_1M"]
    ens = W.make_ensemble(cfg, n_trees=40)
    X = W.make_docs(cfg, n_docs=80)
    rng = np.random.default_rng(0)
    internal = np.nonzero(ens.feature >= 0)[0]
    for k in range(400):  # exact ties with thresholds of the features the nodes read
        n = internal[rng.integers(0, internal.size)]
        X[rng.integers(0, 80), ens.feature[n]] = ens.threshold[n]
    X[1] = np.nan
    X[2] = np.inf
    X[3] = -np.inf
    X[4] = -0.0
    X[5, ::3] = np.float32(3.4e38)
    plan = _check(emu, ens, X, levels=(0,))
    assert plan[3] == 1, plan


def _order(lib, ens, flags=0):
    arrs = [np.ascontiguousarray(ens.tree_offsets, np.int64), np.ascontiguousarray(ens.feature, np.int32),
            np.ascontiguousarray(ens.threshold, np.float32), np.ascontiguousarray(ens.left, np.int32),
            np.ascontiguousarray(ens.right, np.int32), np.ascontiguousarray(ens.value, np.float32)]
    order = np.empty(ens.n_trees, np.int32)
    tiles = np.empty(4096, np.int32)
    n = lib.emu_tree_order(ens.n_trees, *[a.ctypes.data for a in arrs], flags, order.ctypes.data,
                           tiles.ctypes.data, tiles.size)
    assert n >= 0, lib.emu_message().decode()
    assert np.array_equal(np.sort(order), np.arange(ens.n_trees))
    return order, tiles[:min(n, tiles.size)]


def _stack(trees, n_features):
    offs = np.cumsum([0] + [len(t[0]) for t in trees]).astype(np.int64)
    cat = [np.concatenate([np.asarray(t[k], dt) for t in trees]) for k, dt in
           enumerate((np.int32, np.float32, np.int32, np.int32, np.float32))]
    return W.Ensemble(offs, *cat, n_features)


def test_tree_order_known_answer(emu):
    """Trees are ordered by the expected longest of 64 paths, each split's chance of going right
    estimated by the share of the model's thresholds on its feature below its own. A complete
    tree's key is its depth; a deep chain whose root threshold is the lowest of its feature
    sends every document right to a leaf at depth 1 (key 1); complete trees come first among
    equal keys. Ordering by depth, deepest first, would put the chain first."""
    complete2 = ([0, 0, 0, -1, -1, -1, -1], [0.5, 0.25, 0.75, 0, 0, 0, 0], [1, 3, 5, -1, -1, -1, -1],
                 [2, 4, 6, -1, -1, -1, -1], [0, 0, 0, 1, 2, 3, 4])
    # root (lowest threshold) -> right leaf 2; left: a chain 1 -> 3 -> 5 of depth 4
    chain = ([0, 0, -1, 0, -1, 0, -1, -1, -1], [-1.0, 0.1, 0, 0.2, 0, 0.3, 0, 0, 0],
             [1, 3, -1, 5, -1, 7, -1, -1, -1], [2, 4, -1, 6, -1, 8, -1, -1, -1], [0] * 9)
    stump = ([0, -1, -1], [0.6, 0, 0], [1, -1, -1], [2, -1, -1], [0, 5, 6])
    ens = _stack([chain, stump, complete2], 1)
    for flags in (0, 1):
        order, _ = _order(emu, ens, flags)
        assert order.tolist() == [2, 1, 0], (flags, order)


@pytest.mark.parametrize("seed", range(8))
def test_tree_order_ignores_node_numbering(emu, seed):
    """The order depends on the trees, not on how their nodes are numbered (special thresholds,
    +inf under the strict rule included)."""
    pool = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf], dtype=np.float32)
    ens = W.random_ensemble(seed, n_trees=60, n_features=1 + seed, min_leaves=1, max_leaves=24,
                            thr_values=pool if seed % 2 == 0 else None)
    ren, _ = W.relabel_nodes(ens, seed)
    for flags in (0, 1):
        assert np.array_equal(_order(emu, ens, flags)[0], _order(emu, ren, flags)[0]), flags


def test_tree_order_keeps_complete_trees_together(emu):
    """Complete trees of one depth stay contiguous in a mixed model, and a model of complete trees
    is cut into complete-depth tiles only."""
    rand = W.make_ensemble(W.WORKLOADS["rank_1kx32"], n_trees=300)
    comp = W.make_ensemble(W.WORKLOADS["shallow_20kx8_1M"], n_trees=500)
    trees = []
    for i in range(800):
        e, t = (comp, i // 2) if i % 8 < 5 and i // 2 < 500 else (rand, i % 300)
        trees.append(e.tree(t))
    ens = _stack(trees, 136)
    order, tiles = _order(emu, ens)
    is_complete = np.array([len(trees[t][0]) == 15 for t in order])
    pos = np.nonzero(is_complete)[0]
    assert pos.size > 0 and pos[-1] - pos[0] + 1 == pos.size
    _, tiles = _order(emu, comp)
    assert tiles.size > 1 and (tiles == 3).all()


def _deep_tree(n_internal, depth):
    """A tree of n_internal splits whose longest path has `depth` edges: a chain of `depth`
    splits down the right children, then the remaining splits on leaves near the root."""
    fe, th, le, ri = [-1], [0.0], [-1], [-1]
    level = [0]

    def split(n):
        le[n], ri[n], fe[n], th[n] = len(fe), len(fe) + 1, 0, 0.5
        for _ in range(2):
            fe.append(-1), th.append(0.0), le.append(-1), ri.append(-1), level.append(level[n] + 1)

    node = 0
    for _ in range(depth):
        split(node)
        node = ri[node]
    for _ in range(n_internal - depth):
        split(next(i for i in range(len(fe)) if fe[i] < 0 and level[i] < depth - 1))
    return fe, th, le, ri, [1.0 if f < 0 else 0.0 for f in fe]


def test_deep_tree_of_complete_size_is_not_complete(emu):
    """255 nodes is the size of a complete tree of depth 7; a tree of 255 nodes and depth 71 is
    not complete (the check must not shift by the depth: 2 << 71 wraps to 2 << 7 on x86), so its
    tile keeps the leaf-tested walk, and its leaves still match the oracle."""
    tree = _deep_tree(127, 71)
    assert len(tree[0]) == 255
    ens = _stack([tree, tree], 1)
    _, tiles = _order(emu, ens)
    assert tiles.size >= 1 and (tiles == -1).all(), tiles
    X = np.array([[0.75], [0.25], [0.5], [np.nan]], np.float32)
    _check(emu, ens, X, levels=(0,))


def test_tree_order_shortens_the_lockstep_walk(emu):
    """On the ranking-shaped model, groups of 4 trees taken in the packed order need fewer
    lockstep steps (per 64-document wave, the longest path of any tree in the group) than in the
    input order: the estimate tracks the real path lengths."""
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg, n_docs=64 * 16)
    _, leaves, _ = oracle.score(ens, X)
    depth = np.zeros(ens.feature.shape[0], np.int64)
    for t in range(ens.n_trees):
        a = int(ens.tree_offsets[t])
        for q in range(int(ens.tree_offsets[t + 1]) - a):  # creation order: parents first
            if ens.feature[a + q] >= 0:
                depth[a + ens.left[a + q]] = depth[a + ens.right[a + q]] = depth[a + q] + 1
    paths = depth[ens.tree_offsets[:-1][None, :] + leaves]
    wave_max = paths.reshape(-1, 64, ens.n_trees).max(axis=1)

    def steps(order):
        return wave_max[:, order].reshape(wave_max.shape[0], -1, 4).max(axis=2).sum()

    order, _ = _order(emu, ens)
    assert steps(order) < 0.9 * steps(np.arange(ens.n_trees))


# feature counts near the top of a block-width band of one-workgroup plans, where the document
# tile and the trace's bitmasks leave less than 64 KiB for the tile slot: (features, leaves per
# tree at most, documents per block, trees per lane, coded documents)
BAND_TOP_PLANS = [(380, 100, 64, 4, 0), (760, 100, 32, 2, 0), (3000, 40, 8, 1, 0),
                  (1530, 200, 32, 1, 1), (3000, 200, 16, 1, 1)]


@pytest.mark.parametrize("n_features,max_leaves,dl,k,coded", BAND_TOP_PLANS)
def test_slots_of_whole_chunks(emu, n_features, max_leaves, dl, k, coded):
    """The kernel writes a tile window as whole 1,024-record chunks, so the slot of these plans
    must be a whole number of chunks (a slot of 64,768 bytes once let the last chunk overwrite
    the zero record and the trace's bitmasks). Large trees fill the last chunk."""
    pool = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf], np.float32)
    ens = W.random_ensemble(5066, n_trees=160, n_features=n_features, min_leaves=1,
                            max_leaves=max_leaves, thr_values=pool)
    X = W.random_docs(5066, 70, n_features)
    plan = _check(emu, ens, X, flags=1, levels=(0, 1))
    assert (plan[0], plan[1], plan[3]) == (dl, k, coded), plan
    tile_bytes, slot_recs = int(plan[6]), int(plan[7])
    assert plan[5] == 160 * 1024 and tile_bytes % 8192 == 0 and tile_bytes < 64 * 1024, plan
    assert tile_bytes - 8192 < slot_recs * 8 <= tile_bytes, plan  # the last chunk is in use


def test_walker_packets_or_shared_tiles(emu):
    """Plans of 64- and 32-document blocks stream per-wave packets when every group of K trees
    fits a walker's part of a sub-slot (the ranking and shallow workloads in two-workgroup
    plans; the large 700-feature workload's 511-node trees and the wide workload's two
    half-wave walkers per wave in one-workgroup plans, whose sub-slots take all of the LDS past
    the document tile), and keep the shared tiles otherwise (a group larger than a part). The
    walk over the packets (every LDS access in the walker's own part or on the packets' zero
    record, every tree once per block, leaf ids equal to the oracle's) is what _check runs in
    both cases."""
    for wl, packets in (("rank_1kx32", True), ("shallow_20kx8_1M", True), ("large_5kx256_f700_1M", True),
                        ("wide_1kx64_f700", True)):
        cfg = W.WORKLOADS[wl]
        ens = W.make_ensemble(cfg, n_trees=min(cfg.n_trees, 800 if wl != "large_5kx256_f700_1M" else 120))
        plan = _check(emu, ens, W.make_docs(cfg, n_docs=70), levels=(0,))
        assert (plan[8] > 0) == packets, (wl, plan)
        if packets and plan[5] == 80 * 1024:
            assert plan[8] % 64 == 0 and 16 * plan[8] * 8 <= plan[6], plan
        elif packets:
            # a 701-column tile of 64 codes or 32 floats (89,728 B); 16 sub-slots of 576 records
            assert plan[5] == 160 * 1024 and plan[0] * (2 if plan[3] else 4) == 128 and plan[8] == 576, plan
    # one-workgroup plan of 64-document blocks whose trees outgrow a 576-record sub-slot
    wide = W.random_ensemble(5, n_trees=24, n_features=300, min_leaves=300, max_leaves=320)
    plan = _check(emu, wide, W.random_docs(5, 70, 300), levels=(0,))
    assert plan[5] == 160 * 1024 and plan[0] == 64 and plan[8] == 0, plan
    # two-workgroup plan whose single trees outgrow a sub-slot
    big = W.random_ensemble(3, n_trees=30, n_features=136, min_leaves=150, max_leaves=220)
    plan = _check(emu, big, W.random_docs(3, 70, 136), levels=(0,))
    assert plan[5] == 80 * 1024 and plan[0] == 64 and plan[8] == 0, plan


def _big_model(seed, n_feat, n_small, small_leaves, big_leaves):
    """n_small trees of up to small_leaves leaves followed by trees of the given leaf counts
    (too large for one LDS tile), in one ensemble."""
    parts = []
    if n_small:
        parts.append(W.random_ensemble(seed, n_trees=n_small, n_features=n_feat, min_leaves=1,
                                       max_leaves=small_leaves))
    for i, L in enumerate(big_leaves):
        parts.append(W.random_ensemble(seed * 10 + i, n_trees=1, n_features=n_feat, min_leaves=L, max_leaves=L))
    trees = [e.tree(t) for e in parts for t in range(e.n_trees)]
    rng = np.random.default_rng(seed)
    order = rng.permutation(len(trees))  # big trees anywhere in the input order
    return _stack([trees[i] for i in order], n_feat)


@pytest.mark.parametrize("n_feat,n_small,big_leaves,coded", [
    (136, 40, [3000, 8192], 0),      # two-workgroup plan: a 45 KiB slot holds 2,923 leaves at most
    (136, 0, [8192, 32768], 0),      # only big trees: no tile at all
    (700, 30, [4500, 8192], 0),      # one-workgroup plan of 32 float documents
    (700, 300, [300, 8192], 1),      # threshold-coded documents
])
def test_big_trees_walked_from_device_memory(emu, n_feat, n_small, big_leaves, coded):
    """Trees larger than one LDS tile (up to 65,535 nodes) are packed after the tiled ones in
    the big-tree format and walked from the packed array: every child link stays inside its
    tree, leaves absorb a further step, and the leaf ids equal the oracle's, under both rules."""
    ens = _big_model(7 + n_small, n_feat, n_small, 400 if coded else 40, big_leaves)
    X = W.random_docs(9, 70, n_feat, zero_frac=0.2)
    for flags in (0, 1):
        plan = _check(emu, ens, X, flags=flags, levels=(0, 4))
        # a tree is big when its records, the tile header and K root copies exceed the slot
        cap = int(plan[6]) // 8 - 2 - int(plan[1])
        sizes = np.diff(ens.tree_offsets)
        assert plan[9] == int((sizes <= cap).sum()) and (sizes > cap).sum() >= 1, (plan, cap)
        assert plan[3] == coded, plan


def test_big_trees_with_vector_leaves(emu):
    ens = _big_model(3, 136, 20, 30, [8192])
    X = W.random_docs(4, 65, 136)
    vals = W.make_leaf_vectors(ens, 5, "dense", seed=2)
    ref = oracle.score_multi(ens, vals, X)
    _, ref_leaves, _ = oracle.score(ens, X)
    leaves, scores, plan = _walk(emu, ens, X, 0, leaf_values=vals)
    assert plan[9] == 20
    np.testing.assert_array_equal(leaves, ref_leaves)
    np.testing.assert_allclose(scores, ref, rtol=1e-12, atol=1e-12)


def test_tree_size_limit(emu):
    """65,535 nodes (32,768 leaves) is the largest tree accepted; one more leaf is refused."""
    ok = W.random_ensemble(11, n_trees=1, n_features=5, min_leaves=32768, max_leaves=32768)
    X = W.random_docs(11, 10, 5)
    plan = _check(emu, ok, X, levels=(0,))
    assert plan[9] == 0
    too_big = W.random_ensemble(12, n_trees=1, n_features=5, min_leaves=32769, max_leaves=32769)
    arrs = [np.ascontiguousarray(too_big.tree_offsets, np.int64), np.ascontiguousarray(too_big.feature, np.int32),
            np.ascontiguousarray(too_big.threshold, np.float32), np.ascontiguousarray(too_big.left, np.int32),
            np.ascontiguousarray(too_big.right, np.int32), np.ascontiguousarray(too_big.value, np.float32)]
    leaves = np.empty((10, 1), np.int32)
    scores = np.empty((10, 1), np.float64)
    plan = np.zeros(10, np.int32)
    rc = emu.emu_walk(1, *[a.ctypes.data for a in arrs], 1, 0, X.ctypes.data, 10, 5, 0,
                      leaves.ctypes.data, scores.ctypes.data, plan.ctypes.data)
    assert rc == -2 and b"65535" in emu.emu_message()


def _compact_k(lib, ens, X, flags=0, groups=False):
    got = _walk_compact(lib, ens, X, flags)
    return None if got is None else (got[2:] if groups else got[2])


@pytest.mark.parametrize("seed", range(_CC.N_CASES))
def test_compact_sweep_cases(emu, seed):
    """The GPU sweep's random models (tests/_compact_cases.py): all but two take the compact
    packets (cases 0 and 7 keep the 8-byte records), some with several groups in a packet; the
    compact walk of their first 200 documents reaches the oracle's leaves under the case's rule."""
    ens, X, rule, _, _ = _CC.case(seed)
    X = X[:200]
    got = _walk_compact(emu, ens, X, rule)
    if seed in (0, 7):
        assert got is None
        return
    assert got is not None and got[2] == 2
    ref_scores, ref_leaves, _ = oracle.score(ens, X, rule=rule)
    np.testing.assert_array_equal(got[0], ref_leaves)
    np.testing.assert_allclose(got[1], ref_scores, rtol=1e-12, atol=1e-12)
    if seed in (4, 21):
        assert got[3] == 3, "three groups in one packet"


def test_compact_packets_of_the_large_workload(emu):
    """The 700-feature coded workload's 511-node trees take the compact packets with two trees
    per lane (a 2,040-byte tree fills a 2 KiB window but its zero pair); its leaves and scores
    through them equal the oracle's (checked inside _check), under both rules."""
    cfg = W.WORKLOADS["large_5kx256_f700_1M"]
    ens = W.make_ensemble(cfg, n_trees=150)
    X = W.make_docs(cfg, n_docs=130)
    for flags in (0, 1):
        _check(emu, ens, X, flags=flags, levels=(0,))
        assert _compact_k(emu, ens, X, flags) == 2


@pytest.mark.parametrize("seed", range(6))
def test_compact_packets_random_coded_models(emu, seed):
    """Random coded models (700 features and trees of a few hundred nodes: float documents would
    not fit 64 per block) mixed with small and single-leaf trees, so that groups, windows and
    idle slots of a last partial group vary; +-inf and special thresholds under both rules, and
    documents with NaN, +-inf and exact ties, all reach the oracle's leaves."""
    rng = np.random.default_rng(900 + seed)
    pool = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf], np.float32)
    big = W.random_ensemble(900 + seed, n_trees=int(rng.integers(3, 70)), n_features=700, min_leaves=150,
                            max_leaves=256, thr_values=pool if seed % 3 == 0 else None)
    small = W.random_ensemble(950 + seed, n_trees=int(rng.integers(1, 8)), n_features=700, min_leaves=1,
                              max_leaves=int(rng.choice([1, 2, 9])))
    trees = [big.tree(t) for t in range(big.n_trees)] + [small.tree(t) for t in range(small.n_trees)]
    ens = _stack([trees[i] for i in rng.permutation(len(trees))], 700)
    X = W.random_docs(900 + seed, n_docs=int(rng.integers(1, 140)), n_features=700, zero_frac=0.3)
    X[:3, :50] = np.array([np.nan, np.inf, -np.inf], np.float32)[:X.shape[0], None][:3]
    internal = np.nonzero(ens.feature >= 0)[0]
    for _ in range(200):
        n = internal[rng.integers(0, internal.size)]
        X[rng.integers(0, X.shape[0]), ens.feature[n]] = ens.threshold[n]
    for flags in (0, 1):
        plan = _check(emu, ens, X, flags=flags, levels=(0,))
        assert plan[3] == 1, plan
        assert _compact_k(emu, ens, X, flags) == 2


def test_compact_packets_of_several_groups(emu):
    """Trees small enough to share a window (here 130 trees of 16-32 leaves next to 150 of
    200-256, which keep the plan coded) are packed several groups to a packet: the windows hold
    one body after another and the header one root pair per group."""
    big = W.random_ensemble(41, n_trees=150, n_features=700, min_leaves=200, max_leaves=256)
    small = W.random_ensemble(42, n_trees=130, n_features=700, min_leaves=16, max_leaves=32)
    ens = _stack([big.tree(t) for t in range(big.n_trees)] + [small.tree(t) for t in range(small.n_trees)], 700)
    X = W.random_docs(43, 100, 700)
    for flags in (0, 1):
        _check(emu, ens, X, flags=flags, levels=(0,))
        k, groups = _compact_k(emu, ens, X, flags, groups=True)
        assert k == 2 and groups > 1, (k, groups)


@pytest.mark.parametrize("n_features", [750, 767])
def test_compact_packets_for_the_widest_coded_tiles(emu, n_features):
    """The windows fit next to every coded 64-document tile (up to 768 columns, 96 KiB: 98,304 +
    16 x 4,096 bytes is the whole LDS; the packet header stays in registers)."""
    wide = W.random_ensemble(810 + n_features, n_trees=90, n_features=n_features, min_leaves=200,
                             max_leaves=256)
    internal = np.nonzero(wide.feature >= 0)[0]
    wide.feature[internal[0]] = n_features - 1  # the last column is read
    Xw = W.random_docs(61, 70, n_features)
    plan = _check(emu, wide, Xw, levels=(0,))
    assert plan[0] == 64 and plan[3] == 1, plan  # coded, 64 documents
    assert _compact_k(emu, wide, Xw) == 2


def test_compact_packets_not_built_where_they_do_not_apply(emu):
    """Float documents, trees over 511 nodes, and coded models with more distinct thresholds
    per feature than the 11-bit field holds keep the 8-byte packets only."""
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg, n_trees=50)
    assert _compact_k(emu, ens, W.make_docs(cfg, n_docs=10)) is None
    big = W.random_ensemble(4, n_trees=20, n_features=700, min_leaves=257, max_leaves=300)
    X = W.random_docs(4, 10, 700)
    _check(emu, big, X, levels=(0,))
    assert _compact_k(emu, big, X) is None
    # 2,100 distinct thresholds on feature 0 (codes beyond 2,046)
    many = W.random_ensemble(5, n_trees=20, n_features=700, min_leaves=200, max_leaves=256)
    internal = np.nonzero(many.feature >= 0)[0]
    many.feature[internal[:2100]] = 0
    many.threshold[internal[:2100]] = np.arange(2100, dtype=np.float32) / 2100.0
    Xm = W.random_docs(5, 10, 700)
    _check(emu, many, Xm, levels=(0,))
    assert _compact_k(emu, many, Xm) is None


def test_coding_search_tables_long_lists(emu):
    """The coding kernel's breadth-first search tables hold a feature's list padded with NaN to
    2^s - 1 entries: lists of 5,000 and 16,383 distinct thresholds (the longest that fits one
    coding workgroup's 16,384 slots) code exactly (the emulator checks every staged code of the
    descent against a plain count), and the model's leaves match the oracle's."""
    cfg = W.WORKLOADS["large_5kx256_f700_1M"]
    ens = W.make_ensemble(cfg, n_trees=100)
    internal = np.nonzero(ens.feature >= 0)[0]
    rng = np.random.default_rng(7)
    pick = rng.permutation(internal)
    ens.feature[np.isin(ens.feature, (3, 10))] = 20  # features 3 and 10: only the lists below
    ens.feature[pick[:16383]] = 10
    ens.threshold[pick[:16383]] = (np.arange(16383, dtype=np.float32) + 0.5) / 16383
    ens.feature[pick[16383:21383]] = 3
    ens.threshold[pick[16383:21383]] = rng.random(5000, dtype=np.float32)
    assert np.unique(ens.threshold[pick[:16383]]).size == 16383
    X = W.make_docs(cfg, n_docs=150)
    X[:, 10] = rng.random(150, dtype=np.float32)
    X[:20, 10] = ens.threshold[pick[:20]]  # exact ties
    X[20, [3, 10]] = np.nan
    X[21, [3, 10]] = np.inf
    plan = _check(emu, ens, X, levels=(0,))
    assert plan[3] == 1, plan
    for flags in (0, 1):
        assert _code_check(emu, ens, flags) > 2 * (16383 + 5000)


def _code_check(lib, ens, flags=0):
    arrs = [np.ascontiguousarray(ens.tree_offsets, np.int64), np.ascontiguousarray(ens.feature, np.int32),
            np.ascontiguousarray(ens.threshold, np.float32), np.ascontiguousarray(ens.left, np.int32),
            np.ascontiguousarray(ens.right, np.int32), np.ascontiguousarray(ens.value, np.float32)]
    n = np.zeros(1, np.int64)
    rc = lib.emu_code_check(ens.n_trees, *[a.ctypes.data for a in arrs], flags, n.ctypes.data)
    assert rc == 0, lib.emu_message().decode()
    return int(n[0])


@pytest.mark.parametrize("seed", range(4))
def test_coding_search_tables_at_every_threshold(emu, seed):
    """Coded models with +-inf and special thresholds, both rules: the search gives the plain
    count at every threshold, just below it, at +-inf, +-0 and NaN."""
    pool = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf], np.float32)
    ens = W.random_ensemble(300 + seed, n_trees=40, n_features=700, min_leaves=200, max_leaves=256,
                            thr_values=pool if seed % 2 else None)
    for flags in (0, 1):
        assert _code_check(emu, ens, flags) > 0
