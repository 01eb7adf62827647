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


@pytest.mark.parametrize("wl", ["tiny_10x8", "rank_1kx32", "wide_1kx64_f700"])
def test_workload_full(T, wl):
    cfg = W.WORKLOADS[wl]
    _say(f"[parity] {wl}: {cfg.n_trees} trees, {cfg.n_docs} docs")
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg)
    # every score and every leaf id (up to 100,000 x 1,000 of them)
    s, ids = _run(T, ens, X, leaves_rows=cfg.n_docs)
    ref, ref_ids, _ = oracle.score(ens, X)
    assert_scores_close(s, ref, f"{wl}")
    assert_leaves_equal(ids, ref_ids, f"{wl}")


@pytest.mark.parametrize("wl", ["rank_1kx32", "wide_1kx64_f700"])
def test_workload_full_strict_rule(T, wl):
    # right iff x > theta: the packer stores the next float above each threshold (and +inf as
    # "never right"); every score and the leaf ids of the first 8,192 documents
    cfg = W.WORKLOADS[wl]
    _say(f"[parity] {wl}, strict rule: {cfg.n_trees} trees, {cfg.n_docs} docs")
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg)
    rows = min(cfg.n_docs, 8192)
    s, ids = _run(T, ens, X, leaves_rows=rows, flags=T.TREE_ENS_RIGHT_IF_GT)
    ref, _, _ = oracle.score(ens, X, rule=1, want_leaves=False)
    assert_scores_close(s, ref, f"{wl} strict")
    _, ref_ids, _ = oracle.score(ens, X[:rows], rule=1)
    assert_leaves_equal(ids, ref_ids, f"{wl} strict")
    if wl == "rank_1kx32":
        # thresholds sampled from feature values (zeros included) tie with document values, so
        # the two rules send documents to different leaves (wide_1kx64_f700 has no such ties)
        _, ge_ids, _ = oracle.score(ens, X[:rows], rule=0)
        assert not np.array_equal(ge_ids, ref_ids)


def test_rank_1kx32_latency_batch(T):
    # the 100-document batch: too few documents to fill the GPU, so the trees are split over
    # workgroups and partial sums are reduced by a second kernel
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg, n_docs=100)
    s, ids = _run(T, ens, X, leaves_rows=100)
    ref, ref_ids, _ = oracle.score(ens, X)
    assert_scores_close(s, ref, "rank_1kx32, 100 docs")
    assert_leaves_equal(ids, ref_ids, "rank_1kx32, 100 docs")


LEAF_CHUNK = 131_072  # documents per leaf-id launch: whole rounds of workgroups, no splits


@pytest.mark.parametrize("wl", ["shallow_20kx8_1M", "large_5kx256_f700_1M"])
def test_workload_1M_sampled(T, wl):
    import torch
    cfg = W.WORKLOADS[wl]
    _say(f"[parity] {wl} at full size: generating")
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg)
    rng = np.random.default_rng(cfg.seed_key)
    sample = np.sort(rng.choice(cfg.n_docs, size=4096, replace=False))
    _say(f"[parity] {wl}: scoring {cfg.n_docs} docs on the GPU")
    with T.TreeEnsemble.from_ensemble(ens) as m:
        Xd = dev(X)
        s = m.predict(Xd)
        torch.cuda.synchronize()
        s = s.cpu().numpy()
        # leaf ids of the seeded sample: every document's leaves are computed by launches of
        # LEAF_CHUNK documents (the path in which each workgroup walks every tree of its block)
        # and the sample's rows are kept
        ids = np.empty((sample.size, cfg.n_trees), np.int32)
        for a in range(0, cfg.n_docs, LEAF_CHUNK):
            b = min(cfg.n_docs, a + LEAF_CHUNK)
            sel = np.nonzero((sample >= a) & (sample < b))[0]
            if sel.size == 0:
                continue
            _say(f"[parity] {wl}: leaf ids of docs {a}..{b}")
            chunk = m.predict_leaves(Xd[a:b].contiguous())
            rows = torch.from_numpy(sample[sel] - a).to(chunk.device)
            ids[sel] = chunk.index_select(0, rows).cpu().numpy()
            del chunk
        # the last 4,096 documents in one launch: a small batch, its blocks split over the tiles
        lo = cfg.n_docs - 4096
        tail_ids = m.predict_leaves(Xd[lo:].contiguous())
        torch.cuda.synchronize()
        tail_ids = tail_ids.cpu().numpy()
        del Xd
    _say(f"[parity] {wl}: oracle on the sample")
    ref, ref_ids, _ = oracle.score(ens, X[sample])
    assert_scores_close(s[sample], ref, f"{wl} sample")
    assert_leaves_equal(ids, ref_ids, f"{wl} sample leaf ids")
    _, ref_tail, _ = oracle.score(ens, X[lo:])
    assert_leaves_equal(tail_ids, ref_tail, f"{wl} last 4096 docs")
    assert np.all(np.isfinite(s))
