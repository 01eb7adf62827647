"""The allocation-free entry point (tree_ens_predict_noalloc), through the C ABI, against
tree_ens_predict on the same handle: two calls in a row, the second with a smaller batch, on
float and threshold-coded models and vector-valued leaves; scores equal bit for bit where the
launch shape is the same and within the oracle tolerance always. A batch whose codes exceed
the static scratch is refused."""
from __future__ import annotations

import numpy as np
import pytest

import oracle
import workloads as W
from _gpu import assert_scores_close, dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def T():
    import paper_1212_2287_amd as T
    T.load_library()
    return T


CASES = [
    # workload, trees (None = all), first and second batch sizes
    ("rank_1kx32", None, 5000, 100),
    ("tiny_10x8", None, 1000, 3),
    ("wide_1kx64_f700", 200, 3000, 700),
    ("large_5kx256_f700_1M", 40, 4000, 257),  # threshold-coded documents
    ("shallow_20kx8_1M", 2000, 40000, 6400),
]


@pytest.mark.parametrize("wl,n_trees,n1,n2", CASES)
def test_noalloc_matches_predict(T, wl, n_trees, n1, n2):
    import torch
    cfg = W.WORKLOADS[wl]
    print(f"[noalloc] {wl}: {n1} then {n2} docs", flush=True)
    ens = W.make_ensemble(cfg, n_trees=n_trees)
    X = W.make_docs(cfg, n_docs=n1)
    with T.TreeEnsemble.from_ensemble(ens) as m:
        for n in (n1, n2):
            x = dev(X[:n])
            ref = m.predict(x)
            out = torch.full((n,), float("nan"), dtype=torch.float32, device="cuda")
            m.predict_noalloc(x, out)
            torch.cuda.synchronize()
            got, want = out.cpu().numpy(), ref.cpu().numpy()
            assert np.array_equal(got, want), f"{wl}, {n} docs: noalloc differs from predict"
            oref, _, _ = oracle.score(ens, X[:n], want_leaves=False)
            assert_scores_close(got, oref, f"{wl}, {n} docs")


def test_noalloc_vector_leaves(T):
    import torch
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg, n_trees=300)
    vals = W.make_leaf_vectors(ens, 6, "dense", seed=3)
    X = W.make_docs(cfg, n_docs=2000)
    with T.TreeEnsemble.from_ensemble(ens, leaf_values=vals, n_bags=3) as m:
        for n in (2000, 90):
            x = dev(X[:n])
            ref = m.predict(x)
            out = torch.empty((n, 6), dtype=torch.float32, device="cuda")
            m.predict_noalloc(x, out)
            torch.cuda.synchronize()
            assert torch.equal(out, ref), n


def test_noalloc_refuses_codes_beyond_the_static_scratch(T):
    import torch
    cfg = W.WORKLOADS["large_5kx256_f700_1M"]
    ens = W.make_ensemble(cfg, n_trees=10)
    n = 16 * 1024 * 1024 // (700 * 2) + 64  # codes of n x 700 features exceed 16 MiB
    X = W.make_docs(cfg, n_docs=n)
    with T.TreeEnsemble.from_ensemble(ens) as m:
        assert m.info()["docs_per_block"] == 64
        x = dev(X)
        out = torch.empty(n, dtype=torch.float32, device="cuda")
        with pytest.raises(T.TreeEnsError) as ei:
            m.predict_noalloc(x, out)
        assert ei.value.code == T.TREE_ENS_E_ARG and "allocation-free" in ei.value.message
        # the refusal launches nothing and leaves the handle usable
        small = dev(X[:500])
        o2 = torch.empty(500, dtype=torch.float32, device="cuda")
        m.predict_noalloc(small, o2)
        assert torch.equal(o2, m.predict(small))
