"""The C ABI on a host without a GPU: the library loads, exports every function the header
declares, and reports model and argument errors before any HIP call."""
from __future__ import annotations

import ctypes

import numpy as np
import pytest

import paper_1212_2287_amd as T
import workloads as W
from _golden import load_hand_ensemble


@pytest.fixture(scope="module")
def lib():
    return T.load_library()


def test_exports_every_declared_function(lib):
    names = T.header_functions()
    assert set(names) >= {"tree_ens_create", "tree_ens_predict", "tree_ens_predict_leaves",
                          "tree_ens_info", "tree_ens_destroy", "tree_ens_last_error"}
    for n in names:
        assert hasattr(lib, n), f"{n} declared in include/tree_ens.h but not exported"


def _create(ens, **kw):
    arrs = dict(tree_offsets=ens.tree_offsets, feature=ens.feature, threshold=ens.threshold,
                left=ens.left, right=ens.right, value=ens.value)
    arrs.update(kw)
    flags = arrs.pop("flags", 0)
    return T.tree_ens_create(arrs["tree_offsets"], arrs["feature"], arrs["threshold"], arrs["left"],
                             arrs["right"], arrs["value"], flags)


def _expect(code, ens, match=None, **kw):
    with pytest.raises(T.TreeEnsError) as ei:
        _create(ens, **kw)
    assert ei.value.code == code, str(ei.value)
    if match:
        assert match in ei.value.message, ei.value.message


def test_model_errors_are_reported_without_a_device():
    ens, _, _ = load_hand_ensemble()
    a = int(ens.tree_offsets[1])  # tree 1 starts here
    l, r, f, th = ens.left.copy(), ens.right.copy(), ens.feature.copy(), ens.threshold.copy()
    l2 = l.copy(); l2[a + 0] = 0
    _expect(T.TREE_ENS_E_MODEL, ens, "naming the root", left=l2)
    l3 = l.copy(); l3[a + 0] = 7
    _expect(T.TREE_ENS_E_MODEL, ens, "out of range", left=l3)
    l4 = l.copy(); l4[a + 3] = 4  # node 3's left becomes node 4, which node 1 also owns
    _expect(T.TREE_ENS_E_MODEL, ens, "two parents", left=l4)
    r5 = r.copy(); r5[a + 0] = 5  # left == right
    _expect(T.TREE_ENS_E_MODEL, ens, "same left and right", right=r5)
    th6 = th.copy(); th6[a + 0] = np.nan
    _expect(T.TREE_ENS_E_MODEL, ens, "NaN threshold", threshold=th6)
    f7 = f.copy(); f7[a + 0] = -2
    _expect(T.TREE_ENS_E_MODEL, ens, "feature id", feature=f7)
    # a cycle that is not connected to the root: nodes 1 and 2 of a 3-node tree point at each
    # other, each with exactly one parent, and the root is a leaf
    cyc = W.Ensemble(np.array([0, 3], np.int64), np.array([-1, 0, 0], np.int32), np.zeros(3, np.float32),
                     np.array([-1, 2, 1], np.int32), np.array([-1, 2, 1], np.int32), np.zeros(3, np.float32), 1)
    with pytest.raises(T.TreeEnsError) as ei:
        _create(cyc)
    assert ei.value.code == T.TREE_ENS_E_MODEL
    off = ens.tree_offsets.copy(); off[2] = off[1]  # an empty tree
    _expect(T.TREE_ENS_E_MODEL, ens, "has no node", tree_offsets=off)
    off0 = ens.tree_offsets.copy(); off0[0] = 1
    _expect(T.TREE_ENS_E_MODEL, ens, "tree_offsets[0]", tree_offsets=off0)
    _expect(T.TREE_ENS_E_ARG, ens, "flag", flags=4)
    # features beyond the LDS document tile
    fbig = f.copy(); fbig[0] = 5000
    _expect(T.TREE_ENS_E_MODEL, ens, "document-tile limit", feature=fbig)


def test_oversized_tree_is_rejected():
    # 65,535 nodes (32,768 leaves) is the largest tree accepted; a tree of 32,769 leaves is
    # refused during validation, before any device call
    n_leaves = 32769
    fe, le, ri = W.grow_random_structure(np.random.default_rng(0), n_leaves, None, 136)
    n = fe.shape[0]
    ens = W.Ensemble(np.array([0, n], np.int64), fe, np.zeros(n, np.float32), le, ri, np.zeros(n, np.float32), 136)
    with pytest.raises(T.TreeEnsError) as ei:
        _create(ens)
    assert ei.value.code == T.TREE_ENS_E_MODEL and "65535 nodes" in ei.value.message


def test_valid_model_reaches_the_device_step():
    # on a host without a GPU a valid model passes validation and fails at the upload
    import torch
    ens = W.make_ensemble(W.WORKLOADS["tiny_10x8"])
    if torch.cuda.is_available():
        pytest.skip("a GPU is present")
    with pytest.raises(T.TreeEnsError) as ei:
        _create(ens)
    assert ei.value.code == T.TREE_ENS_E_DEVICE


def test_null_arguments(lib):
    assert lib.tree_ens_create(None, 0, None, None, None, None, None, None, 0) == T.TREE_ENS_E_ARG
    assert "NULL" in T.tree_ens_last_error()
    assert lib.tree_ens_predict(None, None, None, 10, 4, None) == T.TREE_ENS_E_ARG
    assert lib.tree_ens_predict_leaves(None, None, None, 10, 4, None) == T.TREE_ENS_E_ARG
    assert lib.tree_ens_info(None, None, None, None, None, None, None) == T.TREE_ENS_E_ARG
    assert lib.tree_ens_kernel_timing(None, 1) == T.TREE_ENS_E_ARG
    assert lib.tree_ens_kernel_time(None, None, None) == T.TREE_ENS_E_ARG
    lib.tree_ens_destroy(None)  # accepted
    h = ctypes.c_void_p()
    assert lib.tree_ens_create(ctypes.byref(h), -1, None, None, None, None, None, None, 0) == T.TREE_ENS_E_ARG
    assert h.value is None


def test_c_client_reports_errors_without_a_device(tmp_path):
    """A plain C program linked against the library (no Python, no torch) sees the same model
    and argument errors through include/tree_ens.h."""
    import subprocess
    from paper_1212_2287_amd import _build
    exe = _build.build_c_client(out=str(tmp_path / "c_client"))
    r = subprocess.run([exe, "errors"], capture_output=True, text=True, timeout=60)
    assert r.returncode == 0, r.stdout + r.stderr
