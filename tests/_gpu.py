"""Helpers shared by the GPU tests: device upload, the score tolerance, oracle comparison."""
from __future__ import annotations

import numpy as np

RTOL = 1e-5  # |gpu - oracle| <= ATOL + RTOL * |oracle|, per document
ATOL = 1e-6


def dev(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a)).to("cuda")


def assert_scores_close(gpu: np.ndarray, ref: np.ndarray, what: str = "") -> None:
    gpu = np.asarray(gpu, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    err = np.abs(gpu - ref)
    bad = ~(err <= ATOL + RTOL * np.abs(ref))
    if bad.any():
        i = int(np.argmax(np.where(bad, err, -1)))
        raise AssertionError(f"{what}: {int(bad.sum())} of {gpu.size} scores out of tolerance; "
                             f"worst doc {i}: gpu {gpu[i]!r} oracle {ref[i]!r} err {err[i]:.3g}")


def assert_leaves_equal(gpu: np.ndarray, ref: np.ndarray, what: str = "") -> None:
    gpu = np.asarray(gpu)
    assert gpu.shape == ref.shape, (gpu.shape, ref.shape)
    if not np.array_equal(gpu, ref):
        d, t = np.argwhere(gpu != ref)[0]
        raise AssertionError(f"{what}: {int((gpu != ref).sum())} leaf ids differ; first doc {d} "
                             f"tree {t}: gpu {gpu[d, t]} oracle {ref[d, t]}")
