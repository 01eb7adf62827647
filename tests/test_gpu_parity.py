"""GPU parity on the five workload configurations: the HIP path through the C ABI against the
oracle, scores within |g - r| <= 1e-6 + 1e-5 |r| of the fp64 oracle sum and leaf ids bit-exact.
Configurations with 1M documents run at full size in the launch configuration the bench times
and are compared on a seeded sample of documents that the oracle scores one by one."""
from __future__ import annotations

import sys

import numpy as np
import pytest

import oracle
import workloads as W
from _gpu import assert_leaves_equal, assert_scores_close, dev

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def T():
    import paper_1212_2287_amd as T
    T.load_library()
    return T


def _run(T, ens, X, leaves_rows=None, flags=0):
    import torch
    with T.TreeEnsemble.from_ensemble(ens, flags) as m:
        Xd = dev(X)
        s = m.predict(Xd)
        ids = None
        if leaves_rows is not None:
            ids = m.predict_leaves(Xd[:leaves_rows].contiguous())
        torch.cuda.synchronize()
        return s.cpu().numpy(), None if ids is None else ids.cpu().numpy()


@pytest.mark.parametrize("cfg_id", [1, 2, 3])
def test_config_full(T, cfg_id):
    cfg = W.CONFIGS[cfg_id]
    _say(f"[parity] config {cfg_id} ({cfg.name}): {cfg.n_trees} trees, {cfg.n_docs} docs")
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg)
    rows = min(cfg.n_docs, 8192)
    s, ids = _run(T, ens, X, leaves_rows=rows)
    ref, _, _ = oracle.score(ens, X, want_leaves=False)
    assert_scores_close(s, ref, f"config {cfg_id}")
    _, ref_ids, _ = oracle.score(ens, X[:rows])
    assert_leaves_equal(ids, ref_ids, f"config {cfg_id}")


def test_config2_latency_batch(T):
    # the 100-document batch: too few documents to fill the GPU, so the trees are split over
    # workgroups and partial sums are reduced by a second kernel
    cfg = W.CONFIGS[2]
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg, n_docs=100)
    s, ids = _run(T, ens, X, leaves_rows=100)
    ref, ref_ids, _ = oracle.score(ens, X)
    assert_scores_close(s, ref, "config 2, 100 docs")
    assert_leaves_equal(ids, ref_ids, "config 2, 100 docs")


@pytest.mark.parametrize("cfg_id", [4, 5])
def test_config_1M_sampled(T, cfg_id):
    import torch
    cfg = W.CONFIGS[cfg_id]
    _say(f"[parity] config {cfg_id} ({cfg.name}) at full size: generating")
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg)
    rng = np.random.default_rng(cfg_id)
    sample = np.sort(rng.choice(cfg.n_docs, size=4096, replace=False))
    _say(f"[parity] config {cfg_id}: scoring {cfg.n_docs} docs on the GPU")
    with T.TreeEnsemble.from_ensemble(ens) as m:
        Xd = dev(X)
        s = m.predict(Xd)
        lo = cfg.n_docs - 2048  # leaf ids for a slice that ends at the last (ragged) block
        ids = m.predict_leaves(Xd[lo:].contiguous())
        torch.cuda.synchronize()
        s = s.cpu().numpy()
        ids = ids.cpu().numpy()
        del Xd
    _say(f"[parity] config {cfg_id}: oracle on the sample")
    ref, _, _ = oracle.score(ens, X[sample], want_leaves=False)
    assert_scores_close(s[sample], ref, f"config {cfg_id} sample")
    _, ref_ids, _ = oracle.score(ens, X[lo:])
    assert_leaves_equal(ids, ref_ids, f"config {cfg_id} last 2048 docs")
    assert np.all(np.isfinite(s))
