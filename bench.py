#!/usr/bin/env python3
"""Throughput of tree-ensemble scoring on one MI355X.

A step is one call of tree_ens_predict over the whole workload: stage every document's
features, walk every (document, tree) pair to its leaf, sum the leaf values, store one score
per document. The headline workload is the learning-to-rank shaped ensemble (1,000 trees x 32
leaves, depth <= 16, 136 features) over 100,000 documents, inputs resident in HBM.

Prints ONE JSON line on stdout (progress goes to stderr):
  value        doc*tree evaluations per second (whole job, one GPU)
  ns_per_doc   wall time per document
  latency_100doc_us   one 100-document batch: host wall clock of predict + stream sync
  rerank       per-query top-20 of the headline workload's query groups (Section 6's reranking)
  kernel_ms    device time per step (HIP events between steps: every kernel of the call)
  score_kernel_ms  the scoring kernel's mean launch duration (HIP events the library records
               right before and after each scoring launch, tree_ens_kernel_timing)
  roofline     the scoring kernel against the LDS byte roofline (node bytes: 8 per comparison
               and 4 per leaf, over 256 B/clk/CU), per score_kernel_ms
  roofline_hbm the same kernel against HBM (feature + score bytes)
  roofline_lds_issue  the node bytes against the LDS instruction ceiling of the walk
  cpu_baseline the oracle on the host cores, same workload
  workloads_extra the other workloads (1M-document ones included), same measurements
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import statistics
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "doc·tree evals/sec; ns/doc at 1k×32-leaf trees; µs per 100-doc batch"
HEADLINE = "rank_1kx32"

# MI355X figures: 256 CUs at 2.4 GHz; LDS read width 256 B/clk/CU (a ds_read_b128 probe
# reached 240); HBM3E 8 TB/s.
N_CU = 256
CLOCK_HZ = 2.4e9
LDS_BYTES_PER_CLK_CU = 256
LDS_PEAK_GBS = N_CU * CLOCK_HZ * LDS_BYTES_PER_CLK_CU / 1e9  # 157,286 GB/s
HBM_PEAK_GBS = 8000.0
# The LDS pipe's instruction ceiling for the walk: SQ_LDS_IDX_ACTIVE / SQ_INSTS_LDS of the
# scoring kernel on the ranking workload is 2.2 busy cycles per wave-level LDS instruction, and
# a comparison takes two (feature, node record), so at most 64 x 8 node bytes move per 4.4
# cycles per CU whatever the byte width allows.
LDS_CLK_PER_INSTR = 2.2
LDS_ISSUE_NODE_GBS = N_CU * CLOCK_HZ * 64 * 8 / (2 * LDS_CLK_PER_INSTR) / 1e9  # 71,494 GB/s
KERNEL_SRC = os.path.join(ROOT, "paper_1212_2287_amd", "csrc", "tree_ens.hip")
TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic.json")


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def kernel_hash() -> str:
    """Hash of the kernel and packer sources with comments and whitespace removed: stored
    counter results stay valid across comment edits and lapse on any code change."""
    import re
    h = hashlib.sha256()
    for p in (KERNEL_SRC, os.path.join(ROOT, "paper_1212_2287_amd", "csrc", "pack.cpp"),
              os.path.join(ROOT, "paper_1212_2287_amd", "csrc", "pack.hpp")):
        with open(p) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
        text = re.sub(r"//[^\n]*", "", text)
        h.update("".join(text.split()).encode())
    return h.hexdigest()[:16]


def node_depths(ens):
    """Depth (edges from the root) of every flat node, read off the tree structure."""
    import numpy as np
    depth = np.zeros(ens.n_nodes, dtype=np.int32)
    for t in range(ens.n_trees):
        a = int(ens.tree_offsets[t])
        fe, _, le, ri, _ = ens.tree(t)
        stack = [0]
        while stack:
            n = stack.pop()
            if fe[n] >= 0:
                depth[a + le[n]] = depth[a + ri[n]] = depth[a + n] + 1
                stack += [int(le[n]), int(ri[n])]
    return depth


def count_visits(model, ens, Xd, max_docs=None):
    """Internal nodes visited over all (document, tree) pairs, from the leaves the GPU reaches
    (leaf depth = comparisons made). With max_docs, counted on a prefix and scaled."""
    import torch
    n = Xd.shape[0] if max_docs is None else min(max_docs, Xd.shape[0])
    depth = torch.from_numpy(node_depths(ens)).to(Xd.device).to(torch.int64)
    offs = torch.from_numpy(ens.tree_offsets[:-1]).to(Xd.device)
    total = 0
    chunk = max(1, 50_000_000 // ens.n_trees)
    for a in range(0, n, chunk):
        ids = model.predict_leaves(Xd[a:min(n, a + chunk)].contiguous())
        total += int(depth[offs[None, :] + ids.to(torch.int64)].sum().item())
        del ids
    return total * (Xd.shape[0] / n), n < Xd.shape[0]


def step_stats(samples_s):
    """Median, mean and the 95% confidence interval of the mean (Student's t) of per-step
    times, in ms (the paper reports means of repeated trials with 95% intervals)."""
    n = len(samples_s)
    ms = [v * 1e3 for v in samples_s]
    mean = statistics.fmean(ms)
    half = 0.0
    if n > 1:
        try:
            from scipy.stats import t as student_t
            q = float(student_t.ppf(0.975, n - 1))
        except ImportError:  # normal quantile as a fallback
            q = 1.96
        half = q * statistics.stdev(ms) / n ** 0.5
    return {"n": n, "median_ms": statistics.median(ms), "mean_ms": mean, "ci95_ms": half,
            "min_ms": min(ms), "max_ms": max(ms)}


def time_steps(model, Xd, out, steps, warmup):
    """Host wall time per step over the timed region, mean device time per step from HIP events
    on the launch stream, the per-step event times (an event between consecutive steps), and the
    scoring kernel's own mean launch duration (HIP events the library records on the same stream
    right before and after each scoring launch: the dominant kernel alone, without the coding
    pass, the split reduction or launch gaps) with its launch count per step. The launch events
    come from a second pass of the same steps: recording them between the kernels of a call
    adds gaps to the stream, so the timed steps run without them."""
    import torch
    for _ in range(warmup):
        model.predict(Xd, out)
    torch.cuda.synchronize()
    evs = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    t0 = time.perf_counter()
    evs[0].record()
    for i in range(steps):
        model.predict(Xd, out)
        evs[i + 1].record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    model.kernel_timing(True)
    for _ in range(steps):
        model.predict(Xd, out)
    torch.cuda.synchronize()
    model.kernel_timing(False)
    launch_ms, launches = model.kernel_time()
    per = [evs[i].elapsed_time(evs[i + 1]) / 1e3 for i in range(steps)]
    return (wall / steps, evs[0].elapsed_time(evs[steps]) / 1e3 / steps, per,
            launch_ms / 1e3 / max(launches, 1), launches / steps)


def roofline(kernel_s, lds_bytes, hbm_bytes, traffic):
    return ({"bound": "lds", "achieved": round(lds_bytes / kernel_s / 1e9, 1), "peak": LDS_PEAK_GBS,
             "unit": "GB/s", "frac": round(lds_bytes / kernel_s / 1e9 / LDS_PEAK_GBS, 4),
             "traffic": traffic},
            {"bound": "hbm", "achieved": round(hbm_bytes / kernel_s / 1e9, 1), "peak": HBM_PEAK_GBS,
             "unit": "GB/s", "frac": round(hbm_bytes / kernel_s / 1e9 / HBM_PEAK_GBS, 4)},
            {"bound": "lds_issue", "achieved": round(lds_bytes / kernel_s / 1e9, 1),
             "peak": round(LDS_ISSUE_NODE_GBS, 1), "unit": "GB/s",
             "frac": round(lds_bytes / kernel_s / 1e9 / LDS_ISSUE_NODE_GBS, 4)})


def load_traffic(workload: str):
    """HBM bytes per launch measured with rocprofv3 FETCH_SIZE / WRITE_SIZE (scaled by a copy
    kernel of known size), if taken on the current kernel source; else None."""
    try:
        with open(TRAFFIC_FILE) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        return None
    ent = rec.get("workloads", {}).get(workload)
    if not ent or rec.get("kernel_hash") != kernel_hash():
        return None
    return ent.get("hbm_bytes_per_launch")


def measure_workload(T, W, wl, steps, warmup, n_docs=None, visits_sample=None):
    import torch
    cfg = W.WORKLOADS[wl]
    if n_docs is not None:
        cfg = W.scaled(cfg, n_docs=n_docs)
    t0 = time.perf_counter()
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg)
    log(f"{wl}: generated {cfg.n_trees} trees, {cfg.n_docs} docs in "
        f"{time.perf_counter() - t0:.1f}s")
    model = T.TreeEnsemble.from_ensemble(ens)
    Xd = torch.from_numpy(X).to("cuda")
    out = torch.empty(cfg.n_docs, dtype=torch.float32, device="cuda")
    del X
    wall_s, kern_s, per_step, launch_s, launches = time_steps(model, Xd, out, steps, warmup)
    doc_trees = cfg.n_docs * cfg.n_trees
    visits, sampled = count_visits(model, ens, Xd, visits_sample)
    lds_bytes = visits * 8 + doc_trees * 4
    hbm_bytes = cfg.n_docs * cfg.n_features * 4 + cfg.n_docs * 4 + model.info()["packed_bytes"]
    # the roofline of the dominant kernel: one scoring launch per step walks the whole batch
    rl, rl_hbm, rl_issue = roofline(launch_s, lds_bytes, hbm_bytes, load_traffic(cfg.name))
    rec = {"workload": cfg.name, "n_trees": cfg.n_trees, "n_leaves": cfg.n_leaves,
           "n_features": cfg.n_features, "n_docs": cfg.n_docs,
           "value": doc_trees / wall_s, "ms_per_step": wall_s * 1e3, "kernel_ms": kern_s * 1e3,
           "score_kernel_ms": launch_s * 1e3, "score_launches_per_step": launches,
           "ns_per_doc": wall_s * 1e9 / cfg.n_docs, "step_stats": step_stats(per_step),
           "visits": int(visits), "visits_sampled": sampled,
           "roofline": rl, "roofline_hbm": rl_hbm, "roofline_lds_issue": rl_issue,
           "model": model.info()}
    log(f"{wl}: {rec['ms_per_step']:.3f} ms/step, {rec['value']:.3e} doc*tree/s, "
        f"LDS frac {rl['frac']:.3f} (issue ceiling {rl_issue['frac']:.3f})")
    return rec, model, ens, Xd, out


def latency_100(model, Xd, reps=1000):
    import torch
    x = Xd[:100].contiguous()
    out = torch.empty(100, dtype=torch.float32, device="cuda")
    stream = torch.cuda.current_stream()
    for _ in range(20):
        model.predict(x, out)
    torch.cuda.synchronize()
    walls = []
    for _ in range(reps):
        t0 = time.perf_counter()
        model.predict(x, out)
        stream.synchronize()
        walls.append(time.perf_counter() - t0)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(reps):
        model.predict(x, out)
    ev1.record()
    torch.cuda.synchronize()
    walls.sort()
    return {"median_us": statistics.median(walls) * 1e6, "p99_us": walls[int(0.99 * (len(walls) - 1))] * 1e6,
            "device_us_per_call": ev0.elapsed_time(ev1) * 1e3 / reps, "reps": reps}


def rerank(T, W, model, Xd, cfg, k=20, reps=50):
    """Section 6's reranking step on the headline workload: every query's candidates (20-200
    documents) scored and cut to the best k, in one call (tree_ens_predict_topk), and the top-k
    kernel alone over already computed scores (tree_ens_topk)."""
    import numpy as np
    import torch
    sizes = W.make_query_groups(cfg)
    off = torch.from_numpy(np.concatenate([[0], np.cumsum(sizes)]).astype(np.int64)).to("cuda")
    scores, idx, vals = model.predict_topk(Xd, off, k)
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    for _ in range(3):
        T.tree_ens_topk(scores, off, k, idx, vals)
    torch.cuda.synchronize()
    ev0.record()
    for _ in range(reps):
        T.tree_ens_topk(scores, off, k, idx, vals)
    ev1.record()
    torch.cuda.synchronize()
    topk_us = ev0.elapsed_time(ev1) * 1e3 / reps
    ev0.record()
    for _ in range(reps):
        model.predict_topk(Xd, off, k)
    ev1.record()
    torch.cuda.synchronize()
    fused_ms = ev0.elapsed_time(ev1) / reps
    return {"queries": int(len(sizes)), "k": k, "docs": int(cfg.n_docs),
            "topk_us": topk_us, "predict_topk_ms": fused_ms,
            "queries_per_s": len(sizes) / (fused_ms * 1e-3)}


def feature_usage(model, Xd, cfg, visits, reps=5):
    """Section 6 / Table 4's measure on a workload: the share of the features each document's
    walks compare over the whole ensemble (tree_ens_feature_usage, bitmasks included), and the
    time of one trace of the batch. LDS roofline of the trace: per comparison a node record
    (8 B), a feature (4 B) and an atomic OR into the document's bitmask (4 B)."""
    import numpy as np
    import torch
    counts, masks = model.feature_usage(Xd)
    torch.cuda.synchronize()
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    ev0.record()
    for _ in range(reps):
        model.feature_usage(Xd)
    ev1.record()
    torch.cuda.synchronize()
    ms = ev0.elapsed_time(ev1) / reps
    c = counts.cpu().numpy().astype(np.float64)
    n = int(Xd.shape[0])
    lds = visits * 16
    return {"docs": n, "n_features": cfg.n_features, "avg_features": float(c.mean()),
            "avg_pct": float(100.0 * c.mean() / cfg.n_features), "min": int(c.min()), "max": int(c.max()),
            "ms": ms, "doc_tree_per_s": n * cfg.n_trees / (ms * 1e-3), "reps": reps,
            "roofline": {"bound": "lds", "achieved": lds / (ms * 1e-3) / 1e9, "peak": LDS_PEAK_GBS,
                         "unit": "GB/s", "frac": lds / (ms * 1e-3) / 1e9 / LDS_PEAK_GBS,
                         "bytes": lds}}


def feature_usage_by_trees(T, ens, Xd, cfg, sizes=(1, 10, 100, 1000)):
    """Table 4's shape on the ranking workload: the share of features examined per document as
    the ensemble grows (prefixes of the model, the first 10,000 documents)."""
    import torch
    x = Xd[:10_000].contiguous()
    out = {}
    for n in sizes:
        if n > ens.n_trees:
            continue
        with T.TreeEnsemble.from_ensemble(ens.take_trees(n)) as m:
            c, _ = m.feature_usage(x, want_masks=False)
            torch.cuda.synchronize()
            out[str(n)] = float(100.0 * c.float().mean().item() / cfg.n_features)
    return out


def multi_output(T, W, ens, Xd, cfg, scalar_ms, reps=10):
    """Vector-valued leaves and bagging on the ranking workload's trees and documents: 4 and 8
    outputs per leaf (one and two passes over the trees), and 4 averaged bags of 250 trees."""
    import torch
    out = {}
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)

    def timed(m):
        m.predict(Xd)
        torch.cuda.synchronize()
        ev0.record()
        for _ in range(reps):
            m.predict(Xd)
        ev1.record()
        torch.cuda.synchronize()
        return ev0.elapsed_time(ev1) / reps

    n = int(Xd.shape[0])
    for n_out in (4, 8):
        vals = W.make_leaf_vectors(ens, n_out, "dense", seed=n_out)
        with T.TreeEnsemble.from_ensemble(ens, leaf_values=vals) as m:
            ms = timed(m)
        out[f"outputs_{n_out}"] = {"ms": ms, "vs_scalar": ms / scalar_ms,
                                   "doc_tree_output_per_s": n * ens.n_trees * n_out / (ms * 1e-3)}
    with T.TreeEnsemble.from_ensemble(ens, n_bags=4) as m:
        ms = timed(m)
    out["bags_4"] = {"ms": ms, "vs_scalar": ms / scalar_ms}
    return out


def codegen(T, W, reps=10):
    """The model-specialised kernel (TREE_ENS_CODEGEN, the CodeGen form of Section 3) against
    the generic one on small models: the tiny workload, and prefixes of the ranking and the
    shallow workloads (compile time included in the record)."""
    import torch
    out = {}
    for name, wl, n_trees, n_docs in (("tiny_10x8", "tiny_10x8", None, None),
                                      ("rank_1kx32_200trees", "rank_1kx32", 200, None),
                                      ("shallow_20kx8_1000trees", "shallow_20kx8_1M", 1000, None)):
        cfg = W.WORKLOADS[wl]
        ens = W.make_ensemble(cfg, n_trees=n_trees)
        Xd = torch.from_numpy(W.make_docs(cfg, n_docs=n_docs)).to("cuda")
        rec = {"trees": ens.n_trees, "nodes": ens.n_nodes, "docs": int(Xd.shape[0])}
        for label, flags in (("generic", 0), ("codegen", T.TREE_ENS_CODEGEN)):
            t0 = time.perf_counter()
            h = T.tree_ens_create(ens.tree_offsets, ens.feature, ens.threshold, ens.left, ens.right,
                                  ens.value, flags)
            create_s = time.perf_counter() - t0
            with T.TreeEnsemble(h) as m:
                o = torch.empty(Xd.shape[0], dtype=torch.float32, device="cuda")
                for _ in range(3):
                    m.predict(Xd, o)
                torch.cuda.synchronize()
                e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
                e0.record()
                for _ in range(reps):
                    m.predict(Xd, o)
                e1.record()
                torch.cuda.synchronize()
                ms = e0.elapsed_time(e1) / reps
            rec[label] = {"ms": ms, "create_s": create_s,
                          "doc_tree_per_s": Xd.shape[0] * ens.n_trees / (ms * 1e-3)}
        out[name] = rec
        del Xd
        torch.cuda.empty_cache()
    return out


def cpu_baseline(W, wl, budget_s=10.0):
    import numpy as np
    import oracle
    cfg = W.WORKLOADS[wl]
    ens = W.make_ensemble(cfg)
    X = W.make_docs(cfg)
    # every host CPU the process may use, capped by the thread budget the machine's
    # environment grants (OMP_NUM_THREADS, set to one GPU's share of the host on shared boxes)
    host_cpus = os.cpu_count() or 1
    threads = min(host_cpus, len(os.sched_getaffinity(0)))
    if os.environ.get("OMP_NUM_THREADS", "").isdigit() and int(os.environ["OMP_NUM_THREADS"]) > 0:
        threads = min(threads, int(os.environ["OMP_NUM_THREADS"]))
    oracle.score(ens, X[:1000], threads=threads, want_leaves=False)
    runs = []
    t_start = time.perf_counter()
    while time.perf_counter() - t_start < budget_s and len(runs) < 50:
        t0 = time.perf_counter()
        oracle.score(ens, X, threads=threads, want_leaves=False)
        runs.append(time.perf_counter() - t0)
    sec = statistics.median(runs)
    n1 = min(cfg.n_docs, 10_000)
    t0 = time.perf_counter()
    oracle.score(ens, X[:n1], threads=1, want_leaves=False)
    single = time.perf_counter() - t0
    return {"value": cfg.n_docs * cfg.n_trees / sec, "unit": "doc·tree/s", "cores": threads, "kind": "oracle",
            "sample": f"{cfg.name}: all {cfg.n_docs} docs x {cfg.n_trees} trees, {len(runs)} runs "
                      f"(median), plain C oracle (branching walk, fp64 sum), OpenMP",
            "ns_per_doc": sec * 1e9 / cfg.n_docs,
            "single_thread_ns_per_doc_tree": single * 1e9 / (n1 * cfg.n_trees),
            "cpu_model": _cpu_model(), "host_cpus": host_cpus}


def pmc_probe(T, W, workload: str = HEADLINE) -> int:
    """Copy the workload's feature matrix once (reads and writes exactly its bytes: the
    calibration for the FETCH_SIZE / WRITE_SIZE counters), then score it three times."""
    import torch
    cfg = W.WORKLOADS[workload]
    ens = W.make_ensemble(cfg)
    Xd = torch.from_numpy(W.make_docs(cfg)).to("cuda")
    copy = torch.empty_like(Xd)
    torch.cuda.synchronize()
    copy.copy_(Xd)
    torch.cuda.synchronize()
    with T.TreeEnsemble.from_ensemble(ens) as m:
        out = torch.empty(cfg.n_docs, dtype=torch.float32, device="cuda")
        for _ in range(3):
            m.predict(Xd, out)
        torch.cuda.synchronize()
    log(f"pmc probe: copied {Xd.numel() * 4} bytes, scored {cfg.n_docs} docs x3")
    return 0


def write_traffic(fetch_csv: str, write_csv: str, workload: str = HEADLINE,
                  out_path: str = TRAFFIC_FILE) -> int:
    """Per-launch HBM traffic of the scoring kernel from two rocprofv3 --pmc runs of
    --pmc-probe WORKLOAD (FETCH_SIZE, then WRITE_SIZE; KiB per dispatch), each scaled by what
    the same counter reads for the probe's plain device copy of the feature matrix (a kernel
    that reads and writes exactly that many bytes). Runs on the host; adds the workload's entry
    to profiles/hbm_traffic.json (entries taken on another kernel source are dropped)."""
    import csv
    import workloads as W
    cfg = W.WORKLOADS[workload]
    copy_bytes = cfg.n_docs * cfg.n_features * 4

    def per_kernel(path, counter):
        copies, scores = [], []
        with open(path) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] != counter:
                    continue
                v = float(r["Counter_Value"])
                if "copyBuffer" in r["Kernel_Name"]:
                    copies.append(v)
                elif "score_kernel" in r["Kernel_Name"]:
                    scores.append(v)
        if not copies or not scores:
            raise SystemExit(f"{path}: no copy or scoring dispatch with {counter}")
        return max(copies), statistics.mean(scores), len(scores)

    f_copy, f_score, n_f = per_kernel(fetch_csv, "FETCH_SIZE")
    w_copy, w_score, n_w = per_kernel(write_csv, "WRITE_SIZE")
    f_factor = copy_bytes / 1024.0 / f_copy
    w_factor = copy_bytes / 1024.0 / w_copy
    read_b = f_score * 1024.0 * f_factor
    write_b = w_score * 1024.0 * w_factor
    fetch_dir, write_dir = os.path.dirname(fetch_csv), os.path.dirname(write_csv)
    try:
        with open(out_path) as fh:
            rec = json.load(fh)
    except (OSError, ValueError):
        rec = {}
    if rec.get("kernel_hash") != kernel_hash():
        rec = {"kernel_hash": kernel_hash(), "workloads": {}}
    rec["note"] = ("HBM bytes per launch of the scoring kernel, mean over the probe's dispatches; "
                   "FETCH_SIZE and WRITE_SIZE each scaled by their reading on a plain device copy "
                   "of the workload's feature matrix (a kernel that moves exactly its bytes).")
    rec["workloads"][cfg.name] = {
        "fetch_kib_raw": f_score, "write_kib_raw": w_score, "dispatches": [n_f, n_w],
        "calibration": {"copy_bytes": copy_bytes, "fetch_kib": f_copy, "write_kib": w_copy,
                        "fetch_factor": f_factor, "write_factor": w_factor},
        "hbm_read_bytes_per_launch": int(round(read_b)),
        "hbm_write_bytes_per_launch": int(round(write_b)),
        "hbm_bytes_per_launch": int(round(read_b + write_b)),
        "algorithmic_hbm_bytes": cfg.n_docs * cfg.n_features * 4 + cfg.n_docs * 4,
        "commands": [
            f"rocprofv3 --pmc FETCH_SIZE --output-format csv -d {fetch_dir} -o fetch -- python3 -u bench.py --pmc-probe {cfg.name}",
            f"rocprofv3 --pmc WRITE_SIZE --output-format csv -d {write_dir} -o write -- python3 -u bench.py --pmc-probe {cfg.name}",
            f"python bench.py --write-traffic {fetch_csv} {write_csv} {cfg.name}",
        ],
    }
    with open(out_path, "w") as fh:
        json.dump(rec, fh, indent=1)
    log(f"wrote {out_path}: {read_b / 1e6:.1f} MB read + {write_b / 1e6:.2f} MB written per launch")
    return 0


def _cpu_model() -> str:
    """The host CPU's model name as lscpu reports it (else /proc/cpuinfo)."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.strip().startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except (OSError, subprocess.SubprocessError):
        pass
    try:
        with open("/proc/cpuinfo") as fh:
            for line in fh:
                if line.startswith("model name"):
                    return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def main() -> int:
    ap = argparse.ArgumentParser(description=__doc__, formatter_class=argparse.RawDescriptionHelpFormatter)
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--no-cpu-baseline", action="store_true", help="skip the oracle timing")
    ap.add_argument("--no-extra", action="store_true", help="only the headline workload")
    ap.add_argument("--pmc-probe", nargs="?", const=HEADLINE, default=None, metavar="WORKLOAD",
                    help="for rocprofv3 --pmc runs: one device copy of the workload's feature "
                         "matrix (a kernel of known traffic, for calibration) followed by 3 "
                         "predicts of the whole workload (default: the headline one)")
    ap.add_argument("--write-traffic", nargs="+", metavar="ARG",
                    help="host only: FETCH_CSV WRITE_CSV [WORKLOAD]: turn the counter CSVs of the "
                         "two --pmc-probe runs of a workload into its entry of "
                         "profiles/hbm_traffic.json")
    args = ap.parse_args()
    if args.write_traffic:
        if len(args.write_traffic) not in (2, 3):
            ap.error("--write-traffic takes FETCH_CSV WRITE_CSV [WORKLOAD]")
        return write_traffic(*args.write_traffic)
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.gpus != 1 or world != 1:
        print("bench.py measures one GPU only: this scorer runs on a single MI355X and has no "
              "multi-GPU path (--gpus must be 1).", file=sys.stderr)
        return 2
    import torch
    import paper_1212_2287_amd as T
    import workloads as W
    T.load_library()
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2

    if args.pmc_probe:
        return pmc_probe(T, W, args.pmc_probe)
    rec, model, ens, Xd, out = measure_workload(T, W, HEADLINE, args.steps, args.warmup)
    lat = latency_100(model, Xd)
    log(f"100-doc batch: median {lat['median_us']:.1f} us, device {lat['device_us_per_call']:.1f} us/call")
    rr = rerank(T, W, model, Xd, W.WORKLOADS[HEADLINE])
    log(f"rerank top-{rr['k']} of {rr['queries']} queries: top-k kernel {rr['topk_us']:.1f} us, "
        f"score + top-k {rr['predict_topk_ms']:.3f} ms")
    mo = multi_output(T, W, ens, Xd, W.WORKLOADS[HEADLINE], rec["kernel_ms"])
    log("vector leaves / bags: " + ", ".join(f"{k} {v['ms']:.3f} ms" for k, v in mo.items()))
    fu = feature_usage(model, Xd, W.WORKLOADS[HEADLINE], rec["visits"])
    fu["pct_by_trees"] = feature_usage_by_trees(T, ens, Xd, W.WORKLOADS[HEADLINE])
    log(f"feature usage: {fu['avg_pct']:.1f}% of {fu['n_features']} features per document, "
        f"trace {fu['ms']:.3f} ms (LDS frac {fu['roofline']['frac']:.3f}); by trees {fu['pct_by_trees']}")
    model.close()
    del Xd, out
    torch.cuda.empty_cache()

    extra = {}
    cg = None
    if not args.no_extra:
        cg = codegen(T, W)
        log("codegen vs generic: " + ", ".join(
            f"{k} {v['codegen']['ms']:.3f} / {v['generic']['ms']:.3f} ms (compile {v['codegen']['create_s']:.1f} s)"
            for k, v in cg.items()))
        for wl, steps, samp in (("tiny_10x8", 20, None), ("wide_1kx64_f700", 10, None),
                                ("shallow_20kx8_1M", 5, None), ("large_5kx256_f700_1M", 3, 16384)):
            r, m, _, xd, o = measure_workload(T, W, wl, steps, 1, visits_sample=samp)
            r.pop("model", None)
            big = W.WORKLOADS[wl].n_docs >= 1_000_000
            r["feature_usage"] = feature_usage(m, xd, W.WORKLOADS[wl], r["visits"], reps=1 if big else 5)
            log(f"{wl} feature usage: {r['feature_usage']['avg_pct']:.1f}%, "
                f"trace {r['feature_usage']['ms']:.3f} ms")
            extra[wl] = r
            m.close()
            del xd, o
            torch.cuda.empty_cache()

    cpu = None if args.no_cpu_baseline else cpu_baseline(W, HEADLINE)
    cfg = W.WORKLOADS[HEADLINE]
    line = {
        "metric": METRIC, "value": rec["value"], "unit": "doc·tree/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": rec["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "accumulate": "f64", "data": "synthetic",
        "config": {"workload": f"{cfg.name}: {cfg.n_trees} trees x {cfg.n_leaves} leaves (depth <= "
                               f"{cfg.max_depth}), {cfg.n_features} features, {cfg.n_docs} docs",
                   "n_trees": cfg.n_trees, "n_docs": cfg.n_docs, "n_features": cfg.n_features,
                   "docs_per_block": rec["model"]["docs_per_block"]},
        "ns_per_doc": rec["ns_per_doc"], "kernel_ms": rec["kernel_ms"],
        "score_kernel_ms": rec["score_kernel_ms"], "step_stats": rec["step_stats"],
        "latency_100doc_us": lat, "rerank": rr, "feature_usage": fu,
        "multi_output": mo, "codegen": cg, "visits": rec["visits"],
        "roofline": rec["roofline"], "roofline_hbm": rec["roofline_hbm"],
        "roofline_lds_issue": rec["roofline_lds_issue"],
        "cpu_baseline": cpu, "workloads_extra": extra, "kernel_hash": kernel_hash(),
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
