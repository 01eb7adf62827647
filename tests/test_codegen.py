"""The model-specialised kernel source (TREE_ENS_CODEGEN) on the CPU: the generated program,
compiled as plain C++ with tests/codegen_shim.h and run once per document, must reproduce the
oracle (hand-worked ensemble exactly, random ensembles with ties and IEEE corner values under
both rules); the same source compiles for gfx950 with hiprtc; limits and errors are reported
before any device call."""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np
import pytest

import oracle
import paper_1212_2287_amd as T
import workloads as W
from _golden import load_hand_ensemble

HERE = os.path.dirname(os.path.abspath(__file__))

_DRIVER = r"""
#include "codegen_shim.h"
#include "generated.hip"
extern "C" void run(const float *X, long long n_docs, int n_features, float *scores, double scale) {
    for (long long d = 0; d < n_docs; d++) {
        blockIdx.x = unsigned(d / 256);
        threadIdx.x = unsigned(d % 256);
        tree_ens_cg(X, n_docs, n_features, scores, scale);
    }
}
"""


def _source(ens, flags=0):
    return T.tree_ens_codegen_source(ens.tree_offsets, ens.feature, ens.threshold, ens.left, ens.right,
                                     ens.value, flags)


def _run_on_cpu(tmp_path, src, X, scale=1.0):
    (tmp_path / "generated.hip").write_text(src)
    (tmp_path / "driver.cpp").write_text(_DRIVER)
    lib = tmp_path / "libcg.so"
    subprocess.run(["g++", "-O1", "-std=c++17", "-shared", "-fPIC", "-I", HERE, "-I", str(tmp_path),
                    "-ffp-contract=off", "-fno-fast-math", str(tmp_path / "driver.cpp"), "-o", str(lib)],
                   check=True)
    dll = ctypes.CDLL(str(lib))
    X = np.ascontiguousarray(X, np.float32)
    out = np.empty(X.shape[0], np.float32)
    dll.run(ctypes.c_void_p(X.ctypes.data), ctypes.c_longlong(X.shape[0]), ctypes.c_int(X.shape[1]),
            ctypes.c_void_p(out.ctypes.data), ctypes.c_double(scale))
    return out


@pytest.mark.parametrize("rule,name", [(0, "ge"), (1, "gt")])
def test_generated_program_on_the_hand_ensemble(tmp_path, rule, name):
    ens, X, expects = load_hand_ensemble()
    got = _run_on_cpu(tmp_path, _source(ens, rule), X)
    assert got.tolist() == [e[1] for e in expects[name]]


_POOL = np.array([0.0, -0.0, 0.25, 0.5, 0.75, 1.0, np.inf, -np.inf, np.nan, 1e-45], dtype=np.float32)


@pytest.mark.parametrize("seed", range(4))
def test_generated_program_matches_the_oracle(tmp_path, seed):
    rule = seed % 2
    ens = W.random_ensemble(seed, n_trees=70, n_features=12, min_leaves=1, max_leaves=30,
                            thr_values=_POOL[:8] if seed < 2 else None)
    X = W.random_docs(seed, 300, 12, values=_POOL if seed < 2 else None, zero_frac=0.2)
    got = _run_on_cpu(tmp_path, _source(ens, rule), X, scale=1.0 / 3)
    ref, _, _ = oracle.score(ens, X, rule=rule, want_leaves=False)
    ref = ref / 3
    assert np.all(np.abs(got - ref) <= 1e-6 + 1e-5 * np.abs(ref))


def test_generated_source_compiles_for_gfx950():
    # hiprtc needs no device
    ens = W.make_ensemble(W.WORKLOADS["tiny_10x8"])
    src = _source(ens).encode()
    rtc = ctypes.CDLL("libhiprtc.so")
    prog = ctypes.c_void_p()
    assert rtc.hiprtcCreateProgram(ctypes.byref(prog), src, b"cg.hip", 0, None, None) == 0
    opts = [b"--offload-arch=gfx950", b"-O3", b"-fno-gpu-flush-denormals-to-zero",
            b"-Xclang", b"-target-feature", b"-Xclang", b"-packed-fp32-ops"]
    arr = (ctypes.c_char_p * len(opts))(*opts)
    rc = rtc.hiprtcCompileProgram(prog, len(opts), arr)
    size = ctypes.c_size_t()
    rtc.hiprtcGetCodeSize(prog, ctypes.byref(size))
    rtc.hiprtcDestroyProgram(ctypes.byref(prog))
    assert rc == 0 and size.value > 0


def test_source_shape_and_limits():
    ens, _, _ = load_hand_ensemble()
    src = _source(ens)
    assert 'extern "C" __global__' in src and "tree_ens_cg" in src and "x[1] >= 0x0p+0f" in src
    assert "x[1] > 0x0p+0f" in _source(ens, T.TREE_ENS_RIGHT_IF_GT)
    big = W.make_ensemble(W.WORKLOADS["shallow_20kx8_1M"], n_trees=5000)  # 75,000 nodes
    with pytest.raises(T.TreeEnsError) as ei:
        _source(big)
    assert ei.value.code == T.TREE_ENS_E_MODEL and "65536" in ei.value.message
    # model errors first, and create refuses code generation for vector-valued leaves
    bad_left = ens.left.copy()
    bad_left[3] = 0
    with pytest.raises(T.TreeEnsError) as ei:
        T.tree_ens_codegen_source(ens.tree_offsets, ens.feature, ens.threshold, bad_left, ens.right, ens.value)
    assert ei.value.code == T.TREE_ENS_E_MODEL
    with pytest.raises(T.TreeEnsError) as ei:
        T.tree_ens_create_multi(ens.tree_offsets, ens.feature, ens.threshold, ens.left, ens.right,
                                np.ones(ens.n_nodes * 2, np.float32), 2, 1, T.TREE_ENS_CODEGEN)
    assert ei.value.code == T.TREE_ENS_E_ARG
