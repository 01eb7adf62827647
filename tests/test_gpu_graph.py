"""HIP graph capture of the predict path: a small batch (split over the tiles, partials in the
handle's scratch, a second reduction kernel) and a large one captured with torch's graph API
and replayed several times with eager work of the same handle in between; every replay must
equal the eager result bit for bit (the launches are deterministic)."""
from __future__ import annotations

import numpy as np
import pytest

import workloads as W
from _gpu import dev

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def T():
    import paper_1212_2287_amd as T
    T.load_library()
    return T


@pytest.mark.parametrize("n_docs", [100, 20000])
def test_captured_predict_replays_match_eager(T, n_docs):
    import torch
    cfg = W.WORKLOADS["rank_1kx32"]
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg, n_docs=n_docs)
    other_X = W.make_docs(cfg, n_docs=3000, start=n_docs)
    with T.TreeEnsemble.from_ensemble(ens) as m:
        x, ox = dev(X), dev(other_X)
        eager = m.predict(x).clone()
        eager_other = m.predict(ox).clone()
        torch.cuda.synchronize()
        out = torch.empty(n_docs, dtype=torch.float32, device="cuda")
        side = torch.cuda.Stream()
        side.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(side):
            for _ in range(3):
                m.predict(x, out)
        torch.cuda.current_stream().wait_stream(side)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=side):
            m.predict(x, out)
        torch.cuda.synchronize()
        for i in range(4):
            out.fill_(-1.0)
            o = m.predict(ox)  # eager call of another batch size on the same handle
            g.replay()
            torch.cuda.synchronize()
            assert torch.equal(out, eager), f"replay {i}"
            assert torch.equal(o, eager_other), f"eager call between replays {i}"


@pytest.mark.parametrize("wl,n_trees,n_docs", [("rank_1kx32", None, 100),
                                               ("large_5kx256_f700_1M", 60, 300)])
def test_captured_replays_race_free_next_to_eager_calls(T, wl, n_trees, n_docs):
    """A captured small batch (split partial sums; threshold codes on the coded 700-feature
    model) replayed on one stream while eager predicts of the same handle run on another, with
    no host synchronisation between them: the captured call owns its scratch, so every replay
    and every eager result equals its eager reference bit for bit."""
    import torch
    cfg = W.WORKLOADS[wl]
    ens = W.make_ensemble(cfg, n_trees=n_trees)
    X = W.make_docs(cfg, n_docs=n_docs)
    other_X = W.make_docs(cfg, n_docs=n_docs + 37, start=n_docs)
    with T.TreeEnsemble.from_ensemble(ens) as m:
        x, ox = dev(X), dev(other_X)
        ref = m.predict(x).clone()
        ref_other = m.predict(ox).clone()
        torch.cuda.synchronize()
        cap, eager = torch.cuda.Stream(), torch.cuda.Stream()
        out = torch.empty(n_docs, dtype=torch.float32, device="cuda")
        cap.wait_stream(torch.cuda.current_stream())
        with torch.cuda.stream(cap):
            for _ in range(3):
                m.predict(x, out)
        torch.cuda.current_stream().wait_stream(cap)
        torch.cuda.synchronize()
        g = torch.cuda.CUDAGraph()
        with torch.cuda.graph(g, stream=cap):
            m.predict(x, out)
        torch.cuda.synchronize()
        reps = 16
        outs = torch.empty((reps, n_docs), dtype=torch.float32, device="cuda")
        others = torch.empty((reps, n_docs + 37), dtype=torch.float32, device="cuda")
        eager.wait_stream(torch.cuda.current_stream())
        cap.wait_stream(torch.cuda.current_stream())
        for i in range(reps):
            with torch.cuda.stream(eager):
                m.predict(ox, others[i])
                m.predict(ox, others[i])
            with torch.cuda.stream(cap):
                g.replay()
                outs[i].copy_(out)
        torch.cuda.synchronize()
        for i in range(reps):
            assert torch.equal(outs[i], ref), f"replay {i}"
            assert torch.equal(others[i], ref_other), f"eager call {i}"
