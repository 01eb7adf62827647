"""ctypes binding of ``libtreeens.so``: the C ABI of ``include/tree_ens.h`` under the same
names, plus a small ``TreeEnsemble`` owner class. Argument marshalling only -- every step of
scoring runs in the HIP kernels; torch supplies device memory and the current stream.

The library is loaded from this package's directory and never built here: if it is missing the
first call raises ``TreeEnsLibraryMissing`` (build it with ``__graft_entry__.build()``).
"""
from __future__ import annotations

import ctypes
import os
import re
from typing import Optional

import numpy as np

PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(PKG, "libtreeens.so")
HEADER = os.path.join(os.path.dirname(PKG), "include", "tree_ens.h")

TREE_ENS_OK = 0
TREE_ENS_E_ARG = -1
TREE_ENS_E_MODEL = -2
TREE_ENS_E_SHAPE = -3
TREE_ENS_E_DEVICE = -4
TREE_ENS_E_NOMEM = -5
TREE_ENS_RIGHT_IF_GE = 0
TREE_ENS_RIGHT_IF_GT = 1
TREE_ENS_CODEGEN = 2  # also compile a kernel specialised for the model (hiprtc)

_CODE_NAMES = {0: "OK", -1: "E_ARG", -2: "E_MODEL", -3: "E_SHAPE", -4: "E_DEVICE", -5: "E_NOMEM"}


class TreeEnsLibraryMissing(RuntimeError):
    pass


class TreeEnsError(RuntimeError):
    def __init__(self, code: int, where: str, message: str):
        super().__init__(f"{where}: {_CODE_NAMES.get(code, code)} ({code}): {message}")
        self.code = code
        self.message = message


_lib: Optional[ctypes.CDLL] = None


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load (once) and return the HIP library; raise if it has not been built."""
    global _lib
    if _lib is not None and path == LIB_PATH:
        return _lib
    # torch ships its own HIP runtime under the same soname (libamdhip64.so.7) as the system
    # one this library links against. Importing torch first makes the loader resolve this
    # library's dependency to the runtime torch already uses, so the process has one HIP
    # runtime and torch's streams and allocations are valid here.
    import torch  # noqa: F401
    if not os.path.exists(path):
        raise TreeEnsLibraryMissing(
            f"{path} is missing: the gfx950 HIP library must be built (__graft_entry__.build())")
    lib = ctypes.CDLL(path)
    P, i32, i64, u32 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32
    lib.tree_ens_create.restype = ctypes.c_int
    lib.tree_ens_create.argtypes = [ctypes.POINTER(P), i32, P, P, P, P, P, P, u32]
    lib.tree_ens_create_multi.restype = ctypes.c_int
    lib.tree_ens_create_multi.argtypes = [ctypes.POINTER(P), i32, P, P, P, P, P, P, i32, i32, u32]
    lib.tree_ens_codegen_source.restype = ctypes.c_int
    lib.tree_ens_codegen_source.argtypes = [i32, P, P, P, P, P, P, u32, P, i64, P]
    lib.tree_ens_outputs.restype = ctypes.c_int
    lib.tree_ens_outputs.argtypes = [P, P, P]
    lib.tree_ens_kernel_timing.restype = ctypes.c_int
    lib.tree_ens_kernel_timing.argtypes = [P, i32]
    lib.tree_ens_kernel_time.restype = ctypes.c_int
    lib.tree_ens_kernel_time.argtypes = [P, P, P]
    lib.tree_ens_predict.restype = ctypes.c_int
    lib.tree_ens_predict.argtypes = [P, P, P, i64, i32, P]
    lib.tree_ens_predict_noalloc.restype = ctypes.c_int
    lib.tree_ens_predict_noalloc.argtypes = [P, P, P, i64, i32, P]
    lib.tree_ens_predict_leaves.restype = ctypes.c_int
    lib.tree_ens_predict_leaves.argtypes = [P, P, P, i64, i32, P]
    lib.tree_ens_topk.restype = ctypes.c_int
    lib.tree_ens_feature_usage.restype = ctypes.c_int
    lib.tree_ens_feature_usage.argtypes = [P, P, P, i64, i32, P, P]
    lib.tree_ens_topk.argtypes = [P, P, i64, P, i64, i32, P, P]
    lib.tree_ens_predict_topk.restype = ctypes.c_int
    lib.tree_ens_predict_topk.argtypes = [P, P, P, i64, i32, P, i64, i32, P, P, P]
    lib.tree_ens_info.restype = ctypes.c_int
    lib.tree_ens_info.argtypes = [P, P, P, P, P, P, P]
    lib.tree_ens_destroy.restype = None
    lib.tree_ens_destroy.argtypes = [P]
    lib.tree_ens_last_error.restype = ctypes.c_char_p
    lib.tree_ens_last_error.argtypes = []
    if path == LIB_PATH:
        _lib = lib
    return lib


def header_functions(header: str = HEADER) -> list[str]:
    """Names of the functions ``include/tree_ens.h`` declares."""
    text = open(header).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(tree_ens_[a-z_]+)\s*\(", text)))


def tree_ens_last_error() -> str:
    return load_library().tree_ens_last_error().decode()


def _check(rc: int, where: str) -> None:
    if rc != TREE_ENS_OK:
        raise TreeEnsError(rc, where, tree_ens_last_error())


def _arr(a, dtype):
    return np.ascontiguousarray(np.asarray(a), dtype=dtype)


def _model_args(tree_offsets, feature, threshold, left, right, value, n_outputs=1):
    off = _arr(tree_offsets, np.int64)
    fe, th = _arr(feature, np.int32), _arr(threshold, np.float32)
    le, ri, va = _arr(left, np.int32), _arr(right, np.int32), _arr(value, np.float32)
    n_trees = int(off.shape[0]) - 1
    if n_trees < 0:
        raise ValueError("tree_offsets needs n_trees + 1 entries")
    n = int(off[-1]) if n_trees > 0 else 0
    for name, a in (("feature", fe), ("threshold", th), ("left", le), ("right", ri)):
        if a.shape[0] < n:
            raise ValueError(f"{name} has {a.shape[0]} entries; tree_offsets asks for {n}")
    if va.size < n * n_outputs:
        raise ValueError(f"value has {va.size} entries; {n} nodes x {n_outputs} outputs are needed")

    def ptr(a):
        return a.ctypes.data if a.size else None

    # the arrays are returned too: they must outlive the call
    return n_trees, [ptr(a) for a in (off, fe, th, le, ri, va)], (off, fe, th, le, ri, va)


def tree_ens_create(tree_offsets, feature, threshold, left, right, value,
                    flags: int = TREE_ENS_RIGHT_IF_GE) -> ctypes.c_void_p:
    """Validate, pack and upload an ensemble given as flat creation-order arrays (host)."""
    lib = load_library()
    n_trees, ptrs, _keep = _model_args(tree_offsets, feature, threshold, left, right, value)
    h = ctypes.c_void_p()
    rc = lib.tree_ens_create(ctypes.byref(h), n_trees, *ptrs, int(flags))
    _check(rc, "tree_ens_create")
    return h


def tree_ens_create_multi(tree_offsets, feature, threshold, left, right, value, n_outputs: int,
                          n_bags: int = 1, flags: int = TREE_ENS_RIGHT_IF_GE) -> ctypes.c_void_p:
    """tree_ens_create with leaf rows of ``n_outputs`` values (``value`` [n_nodes, n_outputs])
    and ``n_bags`` averaged bags."""
    lib = load_library()
    n_trees, ptrs, _keep = _model_args(tree_offsets, feature, threshold, left, right, value, n_outputs)
    h = ctypes.c_void_p()
    rc = lib.tree_ens_create_multi(ctypes.byref(h), n_trees, *ptrs, int(n_outputs), int(n_bags), int(flags))
    _check(rc, "tree_ens_create_multi")
    return h


def tree_ens_codegen_source(tree_offsets, feature, threshold, left, right, value,
                            flags: int = TREE_ENS_RIGHT_IF_GE) -> str:
    """The HIP source TREE_ENS_CODEGEN compiles for the model (host only)."""
    lib = load_library()
    n_trees, ptrs, _keep = _model_args(tree_offsets, feature, threshold, left, right, value)
    n = ctypes.c_int64()
    _check(lib.tree_ens_codegen_source(n_trees, *ptrs, int(flags), None, 0, ctypes.byref(n)),
           "tree_ens_codegen_source")
    buf = ctypes.create_string_buffer(n.value + 1)
    _check(lib.tree_ens_codegen_source(n_trees, *ptrs, int(flags), buf, n.value + 1, None),
           "tree_ens_codegen_source")
    return buf.value.decode()


def tree_ens_outputs(h) -> tuple[int, int]:
    """(n_outputs, n_bags) of a handle."""
    n_out, n_bags = ctypes.c_int32(), ctypes.c_int32()
    _check(load_library().tree_ens_outputs(h, ctypes.byref(n_out), ctypes.byref(n_bags)), "tree_ens_outputs")
    return n_out.value, n_bags.value


def tree_ens_kernel_timing(h, enable: bool) -> None:
    """Start (a new record) or stop timing the scoring launches of later predicts."""
    _check(load_library().tree_ens_kernel_timing(h, 1 if enable else 0), "tree_ens_kernel_timing")


def tree_ens_kernel_time(h) -> tuple[float, int]:
    """(total milliseconds, launches) of the scoring launches timed since the last start."""
    ms, n = ctypes.c_double(), ctypes.c_int32()
    _check(load_library().tree_ens_kernel_time(h, ctypes.byref(ms), ctypes.byref(n)), "tree_ens_kernel_time")
    return ms.value, n.value


def _stream_of(t, stream) -> Optional[int]:
    import torch
    if stream is None:
        # the raw handle of torch's current stream on X's device (cheaper than building a
        # Stream object per call)
        raw = getattr(torch._C, "_cuda_getCurrentRawStream", None)
        if raw is not None:
            return raw(t.device.index)
        return torch.cuda.current_stream(t.device).cuda_stream
    return int(getattr(stream, "cuda_stream", stream))


def _check_docs(X):
    import torch
    if not isinstance(X, torch.Tensor) or X.device.type != "cuda":
        raise TypeError("X must be a CUDA (HIP) torch tensor")
    if X.dtype != torch.float32 or X.dim() != 2 or not X.is_contiguous():
        raise TypeError("X must be a contiguous float32 [n_docs, n_features] tensor")


def tree_ens_predict(h, X, scores=None, stream=None, n_outputs=None, _noalloc=False):
    """Scores of the documents ``X`` (device float32 [n_docs, n_features]) as float32 [n_docs]
    (or [n_docs, n_outputs] for a handle with several outputs), enqueued on ``stream``
    (default: torch's current stream for X's device)."""
    import torch
    _check_docs(X)
    n_docs, n_feat = X.shape
    if n_outputs is None:
        n_outputs = tree_ens_outputs(h)[0]
    if scores is None:
        shape = (n_docs,) if n_outputs == 1 else (n_docs, n_outputs)
        scores = torch.empty(shape, dtype=torch.float32, device=X.device)
    elif scores.dtype != torch.float32 or scores.numel() < n_docs * n_outputs or \
            not scores.is_contiguous() or scores.device != X.device:
        raise TypeError("scores must be a contiguous float32 tensor of n_docs * n_outputs entries "
                        "on X's device")
    fn = "tree_ens_predict_noalloc" if _noalloc else "tree_ens_predict"
    rc = getattr(load_library(), fn)(h, _stream_of(X, stream), X.data_ptr() if n_docs else None,
                                     n_docs, n_feat, scores.data_ptr() if n_docs else None)
    _check(rc, fn)
    return scores


def tree_ens_predict_noalloc(h, X, scores, stream=None, n_outputs=None):
    """tree_ens_predict through the allocation-free entry point: ``scores`` must be given (a
    device float32 tensor of n_docs * n_outputs entries); the library allocates nothing."""
    if scores is None:
        raise TypeError("tree_ens_predict_noalloc needs a preallocated scores tensor")
    return tree_ens_predict(h, X, scores, stream, n_outputs, _noalloc=True)


def tree_ens_predict_leaves(h, X, leaf_ids=None, stream=None):
    """Leaf reached per (document, tree), int32 [n_docs, n_trees], tree-local input node ids."""
    import torch
    _check_docs(X)
    n_docs, n_feat = X.shape
    n_trees = tree_ens_info(h)["n_trees"]
    if leaf_ids is None:
        leaf_ids = torch.empty((n_docs, n_trees), dtype=torch.int32, device=X.device)
    elif leaf_ids.dtype != torch.int32 or leaf_ids.numel() < n_docs * n_trees or \
            not leaf_ids.is_contiguous() or leaf_ids.device != X.device:
        raise TypeError("leaf_ids must be a contiguous int32 tensor of n_docs*n_trees entries")
    rc = load_library().tree_ens_predict_leaves(h, _stream_of(X, stream), X.data_ptr() if n_docs else None,
                                                n_docs, n_feat,
                                                leaf_ids.data_ptr() if n_docs * n_trees else None)
    _check(rc, "tree_ens_predict_leaves")
    return leaf_ids


def tree_ens_feature_usage(h, X, counts=None, masks=None, want_masks: bool = True, stream=None):
    """Features examined per document over all trees: (counts int32 [n_docs], masks int32
    [n_docs, (n_features + 31) // 32] holding the uint32 bit patterns, or None when
    ``want_masks`` is false and no ``masks`` tensor is given)."""
    import torch
    _check_docs(X)
    n_docs, n_feat = X.shape
    words = (n_feat + 31) // 32
    if counts is None:
        counts = torch.empty(n_docs, dtype=torch.int32, device=X.device)
    elif counts.dtype != torch.int32 or counts.numel() < n_docs or not counts.is_contiguous() \
            or counts.device != X.device:
        raise TypeError("counts must be a contiguous int32 tensor of n_docs entries on X's device")
    if masks is None and want_masks:
        masks = torch.empty((n_docs, words), dtype=torch.int32, device=X.device)
    if masks is not None and (masks.dtype != torch.int32 or masks.numel() < n_docs * words or
                              not masks.is_contiguous() or masks.device != X.device):
        raise TypeError("masks must be a contiguous int32 tensor of n_docs*words entries on X's device")
    rc = load_library().tree_ens_feature_usage(
        h, _stream_of(X, stream), X.data_ptr() if n_docs else None, n_docs, n_feat,
        counts.data_ptr() if n_docs else None,
        masks.data_ptr() if masks is not None and n_docs else None)
    _check(rc, "tree_ens_feature_usage")
    return counts, masks


def _topk_outputs(device, n_groups, k, top_idx, top_scores):
    import torch
    if top_idx is None:
        top_idx = torch.empty((n_groups, k), dtype=torch.int32, device=device)
    elif top_idx.dtype != torch.int32 or top_idx.numel() < n_groups * k or not top_idx.is_contiguous() \
            or top_idx.device != device:
        raise TypeError("top_idx must be a contiguous int32 tensor of n_groups*k entries on the device")
    if top_scores is None:
        top_scores = torch.empty((n_groups, k), dtype=torch.float32, device=device)
    elif top_scores.dtype != torch.float32 or top_scores.numel() < n_groups * k or \
            not top_scores.is_contiguous() or top_scores.device != device:
        raise TypeError("top_scores must be a contiguous float32 tensor of n_groups*k entries")
    return top_idx, top_scores


def _check_offsets(group_offsets, device):
    import torch
    if not isinstance(group_offsets, torch.Tensor) or group_offsets.dtype != torch.int64 or \
            group_offsets.dim() != 1 or not group_offsets.is_contiguous() or \
            group_offsets.device != device or group_offsets.numel() < 1:
        raise TypeError("group_offsets must be a contiguous int64 [n_groups + 1] tensor on the device")
    return group_offsets.numel() - 1


def tree_ens_topk(scores, group_offsets, k: int, top_idx=None, top_scores=None, stream=None):
    """Per-group top-k of device float32 ``scores`` over the groups of ``group_offsets`` (device
    int64 [n_groups + 1]): (top_idx int32 [n_groups, k], top_scores float32 [n_groups, k])."""
    import torch
    if not isinstance(scores, torch.Tensor) or scores.device.type != "cuda" or \
            scores.dtype != torch.float32 or scores.dim() != 1 or not scores.is_contiguous():
        raise TypeError("scores must be a contiguous float32 CUDA (HIP) vector")
    n_groups = _check_offsets(group_offsets, scores.device)
    top_idx, top_scores = _topk_outputs(scores.device, n_groups, k, top_idx, top_scores)
    rc = load_library().tree_ens_topk(_stream_of(scores, stream), scores.data_ptr() if scores.numel() else None,
                                      scores.numel(), group_offsets.data_ptr(), n_groups, int(k),
                                      top_idx.data_ptr() if n_groups else None,
                                      top_scores.data_ptr() if n_groups else None)
    _check(rc, "tree_ens_topk")
    return top_idx, top_scores


def tree_ens_predict_topk(h, X, group_offsets, k: int, scores=None, top_idx=None, top_scores=None,
                          stream=None):
    """Scores of ``X`` and their per-group top-k in one call: (scores, top_idx, top_scores)."""
    import torch
    _check_docs(X)
    n_docs, n_feat = X.shape
    if scores is None:
        scores = torch.empty(n_docs, dtype=torch.float32, device=X.device)
    elif scores.dtype != torch.float32 or scores.numel() < n_docs or not scores.is_contiguous() \
            or scores.device != X.device:
        raise TypeError("scores must be a contiguous float32 tensor of n_docs entries on X's device")
    n_groups = _check_offsets(group_offsets, X.device)
    top_idx, top_scores = _topk_outputs(X.device, n_groups, k, top_idx, top_scores)
    rc = load_library().tree_ens_predict_topk(
        h, _stream_of(X, stream), X.data_ptr() if n_docs else None, n_docs, n_feat,
        group_offsets.data_ptr(), n_groups, int(k), scores.data_ptr() if n_docs else None,
        top_idx.data_ptr() if n_groups else None, top_scores.data_ptr() if n_groups else None)
    _check(rc, "tree_ens_predict_topk")
    return scores, top_idx, top_scores


def tree_ens_info(h) -> dict:
    lib = load_library()
    nt, mf, md, nt2, dpb = (ctypes.c_int32() for _ in range(5))
    pb = ctypes.c_int64()
    rc = lib.tree_ens_info(h, ctypes.byref(nt), ctypes.byref(mf), ctypes.byref(md), ctypes.byref(pb),
                           ctypes.byref(nt2), ctypes.byref(dpb))
    _check(rc, "tree_ens_info")
    return {"n_trees": nt.value, "min_features": mf.value, "max_depth": md.value,
            "packed_bytes": pb.value, "n_tiles": nt2.value, "docs_per_block": dpb.value}


def tree_ens_destroy(h) -> None:
    if h is not None:
        load_library().tree_ens_destroy(h)


class TreeEnsemble:
    """Owner of a packed model on the current device.

    ``TreeEnsemble.from_arrays(tree_offsets, feature, threshold, left, right, value, flags,
    n_outputs, n_bags)`` or ``TreeEnsemble.from_ensemble(ens, flags, leaf_values, n_bags)`` for
    any object with those attributes; ``TreeEnsemble(handle)`` adopts a handle from the
    module-level create functions. ``n_outputs`` and ``n_bags`` are read back from the handle;
    ``flags`` may include ``TREE_ENS_CODEGEN``."""

    def __init__(self, handle):
        self._h = handle
        self.n_outputs, self.n_bags = tree_ens_outputs(handle)

    @classmethod
    def from_arrays(cls, tree_offsets, feature, threshold, left, right, value,
                    flags: int = TREE_ENS_RIGHT_IF_GE, n_outputs: int = 1, n_bags: int = 1) -> "TreeEnsemble":
        if n_outputs == 1 and n_bags == 1:
            return cls(tree_ens_create(tree_offsets, feature, threshold, left, right, value, flags))
        return cls(tree_ens_create_multi(tree_offsets, feature, threshold, left, right, value,
                                         n_outputs, n_bags, flags))

    @classmethod
    def from_ensemble(cls, ens, flags: int = TREE_ENS_RIGHT_IF_GE, leaf_values=None,
                      n_bags: int = 1) -> "TreeEnsemble":
        """``leaf_values`` [n_nodes, n_outputs] replaces ``ens.value`` (vector-valued leaves)."""
        value, n_out = ens.value, 1
        if leaf_values is not None:
            value = np.ascontiguousarray(leaf_values, dtype=np.float32)
            if value.ndim != 2 or value.shape[0] != ens.n_nodes:
                raise ValueError("leaf_values must be [n_nodes, n_outputs]")
            n_out = value.shape[1]
        return cls.from_arrays(ens.tree_offsets, ens.feature, ens.threshold, ens.left, ens.right,
                               value, flags, n_out, n_bags)

    @property
    def handle(self):
        if self._h is None:
            raise ValueError("model was destroyed")
        return self._h

    def predict(self, X, out=None, stream=None):
        return tree_ens_predict(self.handle, X, out, stream, self.n_outputs)

    def predict_noalloc(self, X, out, stream=None):
        return tree_ens_predict_noalloc(self.handle, X, out, stream, self.n_outputs)

    def predict_leaves(self, X, out=None, stream=None):
        return tree_ens_predict_leaves(self.handle, X, out, stream)

    def feature_usage(self, X, want_masks: bool = True, stream=None):
        return tree_ens_feature_usage(self.handle, X, want_masks=want_masks, stream=stream)

    def predict_topk(self, X, group_offsets, k: int, stream=None):
        """(scores, top_idx, top_scores): scores of X and each query group's k best documents."""
        return tree_ens_predict_topk(self.handle, X, group_offsets, k, stream=stream)

    def info(self) -> dict:
        return tree_ens_info(self.handle)

    def kernel_timing(self, enable: bool) -> None:
        tree_ens_kernel_timing(self.handle, enable)

    def kernel_time(self) -> tuple[float, int]:
        return tree_ens_kernel_time(self.handle)

    def close(self) -> None:
        if self._h is not None:
            tree_ens_destroy(self._h)
            self._h = None

    def __enter__(self):
        return self

    def __exit__(self, *exc):
        self.close()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
