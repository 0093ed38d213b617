"""Python binding of libtod's C ABI (argument marshalling only).

Every function here has the name of the C entry point it calls and does no
arithmetic of its own: torch supplies device memory and the current HIP
stream; all work runs in the library's HIP kernels.  Importing this module
raises ImportError if ``libtod.so`` has not been built (there is no CPU or
PyTorch fallback).
"""
from __future__ import annotations

import ctypes
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libtod.so")

TOD_OK = 0
TOD_ERR_INVALID_ARG = 1
TOD_ERR_NONFINITE = 2
TOD_ERR_WORKSPACE = 3
TOD_ERR_UNSUPPORTED = 4
TOD_ERR_HIP = 5
TOD_ERR_INTERNAL = 6
TOD_ERR_CAPACITY = 7

PREC_AUTO, PREC_FP32, PREC_FP16, PREC_BF16 = 0, 1, 2, 3
PRECISIONS = {"auto": PREC_AUTO, "fp32": PREC_FP32, "fp16": PREC_FP16, "bf16": PREC_BF16}
PRECISION_NAMES = {v: k for k, v in PRECISIONS.items()}
SCORES = {"kth": 0, "largest": 0, "mean": 1, "median": 2, "sum": 3}

SYMBOLS = ("tod_default_options", "tod_workspace_size", "tod_knn", "tod_knn_noalloc",
           "tod_knn_score", "tod_lof", "tod_lof_ties_workspace_size", "tod_lof_ties",
           "tod_knn_decision", "tod_knn_classify", "tod_abod", "tod_cof", "tod_nwr_workspace_size",
           "tod_nwr", "tod_loci_workspace_size", "tod_loci",
           "tod_plan", "tod_plan_workspace",
           "tod_status_string", "tod_last_error")


class tod_options(ctypes.Structure):
    _fields_ = [
        ("struct_size", ctypes.c_uint32),
        ("precision", ctypes.c_int32),
        ("exclude_self", ctypes.c_int32),
        ("shortlist", ctypes.c_int32),
        ("query_block", ctypes.c_int64),
        ("ref_splits", ctypes.c_int32),
        ("margin_scale", ctypes.c_float),
        ("force_fallback", ctypes.c_int32),
        ("no_recheck", ctypes.c_int32),
        ("reorder", ctypes.c_int32),
        ("score", ctypes.c_int32),
        ("tail_parts", ctypes.c_int32),
    ]


class tod_stats(ctypes.Structure):
    _fields_ = [
        ("struct_size", ctypes.c_uint32),
        ("precision", ctypes.c_int32),
        ("kprime", ctypes.c_int32),
        ("ref_splits", ctypes.c_int32),
        ("query_block", ctypes.c_int64),
        ("blocks", ctypes.c_int64),
        ("rows_certified", ctypes.c_int64),
        ("rows_fallback", ctypes.c_int64),
        ("tile_launches", ctypes.c_int64),
        ("ms_prep", ctypes.c_float),
        ("ms_tile", ctypes.c_float),
        ("ms_recheck", ctypes.c_float),
        ("ms_fallback", ctypes.c_float),
        ("ms_score", ctypes.c_float),
        ("ms_total", ctypes.c_float),
        ("reordered", ctypes.c_int32),
        ("pairs_candidate", ctypes.c_int64),
        ("pairs_uncertain", ctypes.c_int64),
        ("pairs_in_range", ctypes.c_int64),
        ("tail_parts", ctypes.c_int32),
        ("tail_rows", ctypes.c_int64),
        ("list_runs", ctypes.c_int32),
    ]

    def as_dict(self) -> dict:
        out = {name: getattr(self, name) for name, _ in self._fields_ if name != "struct_size"}
        out["precision"] = PRECISION_NAMES.get(self.precision, self.precision)
        return out


class TodError(RuntimeError):
    def __init__(self, status: int, where: str, detail: str):
        self.status = status
        super().__init__("%s failed: %s (%s)" % (where, status_string(status), detail))


def _load():
    if not os.path.exists(LIB_PATH):
        raise ImportError(
            "libtod.so is not built (expected at %s); run __graft_entry__.build() or "
            "python paper_2110_14007_amd/build.py" % LIB_PATH)
    lib = ctypes.CDLL(LIB_PATH)
    vp, i64, i32, sz = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    opt_p, st_p = ctypes.POINTER(tod_options), ctypes.POINTER(tod_stats)
    lib.tod_default_options.argtypes = [opt_p]
    lib.tod_default_options.restype = None
    lib.tod_workspace_size.argtypes = [i64, i64, i64, i32, i32, opt_p]
    lib.tod_workspace_size.restype = sz
    lib.tod_knn.argtypes = [vp, i64, vp, i64, i64, i32, opt_p, vp, sz, vp, vp, vp, st_p]
    lib.tod_knn.restype = ctypes.c_int
    lib.tod_knn_noalloc.argtypes = [vp, i64, vp, i64, i64, i32, opt_p, vp, vp, vp, st_p]
    lib.tod_knn_noalloc.restype = ctypes.c_int
    lib.tod_knn_score.argtypes = [vp, i64, i64, i32, opt_p, vp, sz, vp, vp, vp, vp, st_p]
    lib.tod_knn_score.restype = ctypes.c_int
    lib.tod_lof.argtypes = [vp, i64, i64, i32, opt_p, vp, sz, vp, vp, vp, vp, vp, st_p]
    lib.tod_lof.restype = ctypes.c_int
    lib.tod_lof_ties_workspace_size.argtypes = [i64, i64, i32, i64, opt_p]
    lib.tod_lof_ties_workspace_size.restype = sz
    lib.tod_lof_ties.argtypes = [vp, i64, i64, i32, i64, opt_p, vp, sz, vp, vp, vp, st_p]
    lib.tod_lof_ties.restype = ctypes.c_int
    lib.tod_knn_decision.argtypes = [vp, i64, vp, i64, i64, i32, opt_p, vp, sz, vp, vp, vp, vp,
                                      st_p]
    lib.tod_knn_decision.restype = ctypes.c_int
    lib.tod_knn_classify.argtypes = [vp, i64, vp, i64, i64, i32, vp, i32, opt_p, vp, sz, vp, vp,
                                     st_p]
    lib.tod_knn_classify.restype = ctypes.c_int
    lib.tod_abod.argtypes = [vp, i64, i64, i32, opt_p, vp, sz, vp, vp, vp, vp, st_p]
    lib.tod_cof.argtypes = [vp, i64, i64, i32, opt_p, vp, sz, vp, vp, vp, vp, vp, st_p]
    lib.tod_cof.restype = ctypes.c_int
    lib.tod_abod.restype = ctypes.c_int
    lib.tod_nwr_workspace_size.argtypes = [i64, i64, i64, opt_p]
    lib.tod_nwr_workspace_size.restype = sz
    lib.tod_nwr.argtypes = [vp, i64, vp, i64, i64, ctypes.c_double, opt_p, vp, sz, vp, vp, i64, vp,
                            vp, ctypes.POINTER(i64), st_p]
    lib.tod_nwr.restype = ctypes.c_int
    dbl = ctypes.c_double
    lib.tod_loci_workspace_size.argtypes = [i64, i64, i32, i64, opt_p]
    lib.tod_loci_workspace_size.restype = sz
    lib.tod_loci.argtypes = [vp, i64, i64, ctypes.POINTER(dbl), i32, dbl, i32, dbl, i64, opt_p, vp,
                             sz, vp, vp, vp, vp, vp, vp, vp, st_p]
    lib.tod_loci.restype = ctypes.c_int
    lib.tod_plan.argtypes = [i64, i64, i64, i32, opt_p, st_p]
    lib.tod_plan.restype = ctypes.c_int
    lib.tod_plan_workspace.argtypes = [i64, i64, i64, i32, i32, opt_p, sz, st_p]
    lib.tod_plan_workspace.restype = ctypes.c_int
    lib.tod_status_string.argtypes = [ctypes.c_int]
    lib.tod_status_string.restype = ctypes.c_char_p
    lib.tod_last_error.argtypes = []
    lib.tod_last_error.restype = ctypes.c_char_p
    return lib


_lib = _load()


def status_string(status: int) -> str:
    return _lib.tod_status_string(int(status)).decode()


def last_error() -> str:
    return _lib.tod_last_error().decode()


def options(precision="auto", exclude_self=False, shortlist=0, query_block=0, ref_splits=0,
            margin_scale=1.0, force_fallback=False, no_recheck=False, reorder=0,
            score="kth", tail_parts=0) -> tod_options:
    o = tod_options()
    _lib.tod_default_options(ctypes.byref(o))
    o.precision = PRECISIONS[precision] if isinstance(precision, str) else int(precision)
    o.exclude_self = int(bool(exclude_self))
    o.shortlist = int(shortlist)
    o.query_block = int(query_block)
    o.ref_splits = int(ref_splits)
    o.margin_scale = float(margin_scale)
    o.force_fallback = int(bool(force_fallback))
    o.no_recheck = int(bool(no_recheck))
    o.reorder = int(reorder)
    o.score = SCORES[score] if isinstance(score, str) else int(score)
    o.tail_parts = int(tail_parts)
    return o


def new_stats() -> tod_stats:
    s = tod_stats()
    s.struct_size = ctypes.sizeof(tod_stats)
    return s


def _check(status: int, where: str):
    if status != TOD_OK:
        raise TodError(status, where, last_error())


def tod_workspace_size(nq: int, nr: int, d: int, k: int, mode: int = 0, opts=None) -> int:
    """mode 0: kNN / scores / decision, 1 (or True): LOF, 2: classifier."""
    return int(_lib.tod_workspace_size(int(nq), int(nr), int(d), int(k), int(mode),
                                       ctypes.byref(opts) if opts is not None else None))


def tod_plan_workspace(nq: int, nr: int, d: int, k: int, ws_bytes: int, mode: int = 0,
                       opts=None) -> dict:
    """Plan of a call with a workspace of ws_bytes (host only)."""
    s = new_stats()
    st = _lib.tod_plan_workspace(int(nq), int(nr), int(d), int(k), int(mode),
                                 ctypes.byref(opts) if opts is not None else None,
                                 ctypes.c_size_t(int(ws_bytes)), ctypes.byref(s))
    _check(st, "tod_plan_workspace")
    return {"precision": PRECISION_NAMES[s.precision], "kprime": s.kprime,
            "ref_splits": s.ref_splits, "query_block": s.query_block, "blocks": s.blocks,
            "reordered": s.reordered, "list_runs": s.list_runs}


def tod_plan(nq: int, nr: int, d: int, k: int, opts=None) -> dict:
    s = new_stats()
    _check(_lib.tod_plan(int(nq), int(nr), int(d), int(k),
                         ctypes.byref(opts) if opts is not None else None, ctypes.byref(s)),
           "tod_plan")
    return {"precision": PRECISION_NAMES[s.precision], "kprime": s.kprime,
            "ref_splits": s.ref_splits, "query_block": s.query_block, "blocks": s.blocks,
            "reordered": bool(s.reordered), "list_runs": s.list_runs}


# ---------------------------------------------------------------------------
# torch-facing wrappers
# ---------------------------------------------------------------------------

def _torch():
    import torch
    return torch


def _dev_matrix(x, name):
    torch = _torch()
    if not isinstance(x, torch.Tensor) or not x.is_cuda:
        raise TypeError("%s must be a CUDA (HIP) torch tensor" % name)
    if x.dtype != torch.float32 or x.dim() != 2 or not x.is_contiguous():
        raise TypeError("%s must be a contiguous 2-D float32 tensor" % name)
    return x


class Workspace:
    """Reusable device workspace (torch uint8 buffer, grown on demand)."""

    def __init__(self, device=None):
        self.buf = None
        self.device = device

    def get(self, nbytes: int, device):
        torch = _torch()
        if self.buf is None or self.buf.numel() < nbytes or self.buf.device != device:
            self.buf = torch.empty(max(nbytes, 256), dtype=torch.uint8, device=device)
        return self.buf


class FixedWorkspace:
    """A device workspace of a fixed size chosen by the caller.  The library
    plans its query blocks to fit it (automatic batching sized to memory);
    a workspace below the fixed buffers plus one 32-row block is an error."""

    def __init__(self, nbytes: int, device="cuda:0"):
        torch = _torch()
        self.buf = torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)

    def get(self, nbytes: int, device):
        return self.buf


def _ws(workspace, nbytes, device):
    """(buffer, pointer, size) of a workspace of at least nbytes.

    The caller must hold the returned buffer until the library call returns:
    a temporary workspace would otherwise go back to torch's caching
    allocator, which may hand the same memory to the next output tensor.
    """
    if workspace is None:
        workspace = Workspace()
    buf = workspace.get(nbytes, device)
    return buf, ctypes.c_void_p(buf.data_ptr()), ctypes.c_size_t(buf.numel())


def _stream(stream):
    torch = _torch()
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def _p(t):
    return ctypes.c_void_p(t.data_ptr()) if t is not None else None


def tod_knn(xq, xr, k: int, opts=None, workspace=None, stream=None, stats=None):
    """k nearest rows of xr for every row of xq -> (idx int64 [nq,k], dist fp32 [nq,k])."""
    torch = _torch()
    _dev_matrix(xq, "xq")
    _dev_matrix(xr, "xr")
    nq, d = xq.shape
    nr = xr.shape[0]
    if xr.shape[1] != d:
        raise ValueError("xq and xr must have the same number of columns")
    idx = torch.empty((nq, k), dtype=torch.int64, device=xq.device)
    dist = torch.empty((nq, k), dtype=torch.float32, device=xq.device)
    need = tod_workspace_size(nq, nr, d, k, False, opts)
    wsbuf, wsp, wsn = _ws(workspace, need, xq.device)
    st = _lib.tod_knn(_p(xq), nq, _p(xr), nr, d, int(k),
                      ctypes.byref(opts) if opts is not None else None, wsp, wsn,
                      _stream(stream), _p(idx), _p(dist),
                      ctypes.byref(stats) if stats is not None else None)
    _check(st, "tod_knn")
    return idx, dist


NOALLOC_SCRATCH_BYTES = 64 << 20  # TOD_NOALLOC_SCRATCH_BYTES of include/tod.h


def tod_knn_noalloc(xq, xr, k: int, opts=None, stream=None, stats=None, out=None):
    """tod_knn with the library's static scratch as its workspace (no device
    allocation inside the call) -> (idx int64 [nq,k], dist fp32 [nq,k]).
    out: optional preallocated (idx, dist) tensors, so that the caller's side
    allocates nothing either."""
    torch = _torch()
    _dev_matrix(xq, "xq")
    _dev_matrix(xr, "xr")
    nq, d = xq.shape
    nr = xr.shape[0]
    if xr.shape[1] != d:
        raise ValueError("xq and xr must have the same number of columns")
    if out is None:
        idx = torch.empty((nq, k), dtype=torch.int64, device=xq.device)
        dist = torch.empty((nq, k), dtype=torch.float32, device=xq.device)
    else:
        idx, dist = out
        if (tuple(idx.shape) != (nq, k) or idx.dtype != torch.int64 or not idx.is_contiguous()
                or tuple(dist.shape) != (nq, k) or dist.dtype != torch.float32
                or not dist.is_contiguous()):
            raise ValueError("out must be contiguous (int64 [nq,k], fp32 [nq,k]) tensors")
    st = _lib.tod_knn_noalloc(_p(xq), nq, _p(xr), nr, d, int(k),
                              ctypes.byref(opts) if opts is not None else None,
                              _stream(stream), _p(idx), _p(dist),
                              ctypes.byref(stats) if stats is not None else None)
    _check(st, "tod_knn_noalloc")
    return idx, dist


def tod_knn_score(x, k: int, opts=None, workspace=None, stream=None, stats=None,
                  return_lists: bool = False):
    """kNN-OD score of every row of x (self excluded); optionally the lists too."""
    torch = _torch()
    _dev_matrix(x, "x")
    n, d = x.shape
    score = torch.empty((n,), dtype=torch.float32, device=x.device)
    idx = dist = None
    if return_lists:
        idx = torch.empty((n, k), dtype=torch.int64, device=x.device)
        dist = torch.empty((n, k), dtype=torch.float32, device=x.device)
    need = tod_workspace_size(n, n, d, k, False, opts)
    wsbuf, wsp, wsn = _ws(workspace, need, x.device)
    st = _lib.tod_knn_score(_p(x), n, d, int(k), ctypes.byref(opts) if opts is not None else None,
                            wsp, wsn, _stream(stream), _p(score), _p(idx), _p(dist),
                            ctypes.byref(stats) if stats is not None else None)
    _check(st, "tod_knn_score")
    return (score, idx, dist) if return_lists else score


def tod_lof(x, k: int, opts=None, workspace=None, stream=None, stats=None,
            return_lists: bool = False, out=None):
    """LOF and kNN-OD scores of every row of x -> (lof fp32 [n], knn_score fp32 [n][, idx, dist])."""
    torch = _torch()
    _dev_matrix(x, "x")
    n, d = x.shape
    if out is None:
        lof = torch.empty((n,), dtype=torch.float32, device=x.device)
        score = torch.empty((n,), dtype=torch.float32, device=x.device)
    else:
        lof, score = out
    idx = dist = None
    if return_lists:
        idx = torch.empty((n, k), dtype=torch.int64, device=x.device)
        dist = torch.empty((n, k), dtype=torch.float32, device=x.device)
    need = tod_workspace_size(n, n, d, k, True, opts)
    wsbuf, wsp, wsn = _ws(workspace, need, x.device)
    st = _lib.tod_lof(_p(x), n, d, int(k), ctypes.byref(opts) if opts is not None else None,
                      wsp, wsn, _stream(stream), _p(lof), _p(score), _p(idx), _p(dist),
                      ctypes.byref(stats) if stats is not None else None)
    _check(st, "tod_lof")
    return (lof, score, idx, dist) if return_lists else (lof, score)


def tod_lof_ties_workspace_size(n: int, d: int, k: int, capacity: int, opts=None) -> int:
    return int(_lib.tod_lof_ties_workspace_size(int(n), int(d), int(k), int(capacity),
                                                ctypes.byref(opts) if opts is not None else None))


def tod_lof_ties(x, k: int, opts=None, capacity=None, grow: bool = True, workspace=None,
                 stream=None, stats=None):
    """LOF on tie-inclusive k-distance neighbourhoods -> (lof fp32 [n], count int32 [n]).

    ``capacity`` is the number of (point, neighbour) pairs the workspace is
    sized for (default n k + n + 2^16); if the neighbourhoods hold more and
    ``grow`` is set, the workspace is resized to the count the library
    reports and the call is made once more, else TodError(TOD_ERR_CAPACITY)
    is raised.
    """
    torch = _torch()
    _dev_matrix(x, "x")
    n, d = x.shape
    lof = torch.empty((n,), dtype=torch.float32, device=x.device)
    count = torch.empty((n,), dtype=torch.int32, device=x.device)
    st = stats if stats is not None else new_stats()
    optp = ctypes.byref(opts) if opts is not None else None
    cap = int(capacity) if capacity is not None else n * int(k) + n + (1 << 16)
    for _ in range(2):
        need = tod_lof_ties_workspace_size(n, d, k, cap, opts)
        if need == 0:  # arguments the size query rejects: let the call report why
            need = 256
        wsbuf, wsp, wsn = _ws(workspace, need, x.device)
        rc = _lib.tod_lof_ties(_p(x), n, d, int(k), cap, optp, wsp, wsn, _stream(stream),
                               _p(lof), _p(count), ctypes.byref(st))
        if rc != TOD_ERR_CAPACITY or not grow:
            break
        cap = int(st.pairs_in_range)
    _check(rc, "tod_lof_ties")
    del wsbuf
    return lof, count


def tod_knn_decision(xq, xr, k: int, opts=None, workspace=None, stream=None, stats=None,
                     return_lists: bool = False):
    """kNN-OD scores of new points xq against the fitted set xr (nothing excluded)."""
    torch = _torch()
    _dev_matrix(xq, "xq")
    _dev_matrix(xr, "xr")
    nq, d = xq.shape
    nr = xr.shape[0]
    if xr.shape[1] != d:
        raise ValueError("xq and xr must have the same number of columns")
    score = torch.empty((nq,), dtype=torch.float32, device=xq.device)
    idx = dist = None
    if return_lists:
        idx = torch.empty((nq, k), dtype=torch.int64, device=xq.device)
        dist = torch.empty((nq, k), dtype=torch.float32, device=xq.device)
    need = tod_workspace_size(nq, nr, d, k, 0, opts)
    wsbuf, wsp, wsn = _ws(workspace, need, xq.device)
    st = _lib.tod_knn_decision(_p(xq), nq, _p(xr), nr, d, int(k),
                               ctypes.byref(opts) if opts is not None else None, wsp, wsn,
                               _stream(stream), _p(score), _p(idx), _p(dist),
                               ctypes.byref(stats) if stats is not None else None)
    _check(st, "tod_knn_decision")
    return (score, idx, dist) if return_lists else score


def tod_knn_classify(xq, xr, labels_r, k: int, n_classes: int, opts=None, workspace=None,
                     stream=None, stats=None):
    """Majority-vote class of every row of xq among its k nearest rows of xr -> int32 [nq]."""
    torch = _torch()
    _dev_matrix(xq, "xq")
    _dev_matrix(xr, "xr")
    if (not isinstance(labels_r, torch.Tensor) or not labels_r.is_cuda
            or labels_r.dtype != torch.int32 or labels_r.dim() != 1
            or labels_r.shape[0] != xr.shape[0] or not labels_r.is_contiguous()):
        raise TypeError("labels_r must be a contiguous int32 CUDA tensor of length nr")
    nq, d = xq.shape
    nr = xr.shape[0]
    pred = torch.empty((nq,), dtype=torch.int32, device=xq.device)
    need = tod_workspace_size(nq, nr, d, k, 2, opts)
    wsbuf, wsp, wsn = _ws(workspace, need, xq.device)
    st = _lib.tod_knn_classify(_p(xq), nq, _p(xr), nr, d, int(k), _p(labels_r), int(n_classes),
                               ctypes.byref(opts) if opts is not None else None, wsp, wsn,
                               _stream(stream), _p(pred),
                               ctypes.byref(stats) if stats is not None else None)
    _check(st, "tod_knn_classify")
    return pred


def tod_abod(x, k: int, opts=None, workspace=None, stream=None, stats=None,
             return_lists: bool = False):
    """ABOD score (mean neighbour-pair cosine) of every row of x (self excluded)."""
    torch = _torch()
    _dev_matrix(x, "x")
    n, d = x.shape
    score = torch.empty((n,), dtype=torch.float32, device=x.device)
    idx = dist = None
    if return_lists:
        idx = torch.empty((n, k), dtype=torch.int64, device=x.device)
        dist = torch.empty((n, k), dtype=torch.float32, device=x.device)
    need = tod_workspace_size(n, n, d, k, 1, opts)
    wsbuf, wsp, wsn = _ws(workspace, need, x.device)
    st = _lib.tod_abod(_p(x), n, d, int(k), ctypes.byref(opts) if opts is not None else None,
                       wsp, wsn, _stream(stream), _p(score), _p(idx), _p(dist),
                       ctypes.byref(stats) if stats is not None else None)
    _check(st, "tod_abod")
    return (score, idx, dist) if return_lists else score


def tod_cof(x, k: int, opts=None, workspace=None, stream=None, stats=None,
            return_lists: bool = False):
    """COF of every row of x (self excluded) -> (cof fp32 [n], knn_score fp32 [n][, idx, dist])."""
    torch = _torch()
    _dev_matrix(x, "x")
    n, d = x.shape
    cof = torch.empty((n,), dtype=torch.float32, device=x.device)
    score = torch.empty((n,), dtype=torch.float32, device=x.device)
    idx = dist = None
    if return_lists:
        idx = torch.empty((n, k), dtype=torch.int64, device=x.device)
        dist = torch.empty((n, k), dtype=torch.float32, device=x.device)
    need = tod_workspace_size(n, n, d, k, 1, opts)
    wsbuf, wsp, wsn = _ws(workspace, need, x.device)
    st = _lib.tod_cof(_p(x), n, d, int(k), ctypes.byref(opts) if opts is not None else None,
                      wsp, wsn, _stream(stream), _p(cof), _p(score), _p(idx), _p(dist),
                      ctypes.byref(stats) if stats is not None else None)
    _check(st, "tod_cof")
    return (cof, score, idx, dist) if return_lists else (cof, score)


def tod_nwr_workspace_size(nq: int, nr: int, d: int, opts=None) -> int:
    return int(_lib.tod_nwr_workspace_size(int(nq), int(nr), int(d),
                                           ctypes.byref(opts) if opts is not None else None))


def tod_nwr(xq, xr, phi: float, opts=None, workspace=None, stream=None, stats=None,
            capacity=None, with_dist: bool = True, count_only: bool = False,
            workspace_bytes=None):
    """Neighbours within range phi -> (row_ptr int64 [nq+1], idx int64 [total], dist fp32 [total]).

    With count_only, only row_ptr is computed (idx and dist are None).  The
    outputs are allocated with ``capacity`` entries (default 64 per query
    row); if the pairs in range do not fit, they are reallocated to the
    total the library reports and the call is made once more.
    ``workspace_bytes`` overrides the workspace size (candidate room).
    """
    torch = _torch()
    _dev_matrix(xq, "xq")
    _dev_matrix(xr, "xr")
    nq, d = xq.shape
    nr = xr.shape[0]
    if xr.shape[1] != d:
        raise ValueError("xq and xr must have the same number of columns")
    need = int(workspace_bytes) if workspace_bytes is not None else \
        tod_nwr_workspace_size(nq, nr, d, opts)
    wsbuf, wsp, wsn = _ws(workspace, need, xq.device)
    row_ptr = torch.empty((nq + 1,), dtype=torch.int64, device=xq.device)
    total = ctypes.c_int64(0)
    optp = ctypes.byref(opts) if opts is not None else None
    stp = ctypes.byref(stats) if stats is not None else None
    if count_only:
        st = _lib.tod_nwr(_p(xq), nq, _p(xr), nr, d, float(phi), optp, wsp, wsn, _stream(stream),
                          _p(row_ptr), 0, None, None, ctypes.byref(total), stp)
        _check(st, "tod_nwr")
        return row_ptr, None, None
    cap = 64 * nq if capacity is None else int(capacity)
    for _ in range(2):
        idx = torch.empty((max(cap, 1),), dtype=torch.int64, device=xq.device)
        dist = torch.empty((max(cap, 1),), dtype=torch.float32, device=xq.device) \
            if with_dist else None
        st = _lib.tod_nwr(_p(xq), nq, _p(xr), nr, d, float(phi), optp, wsp, wsn, _stream(stream),
                          _p(row_ptr), cap, _p(idx), _p(dist), ctypes.byref(total), stp)
        if st != TOD_ERR_CAPACITY:
            break
        cap = int(total.value)
    _check(st, "tod_nwr")
    n = int(total.value)
    return row_ptr, idx[:n], (dist[:n] if dist is not None else None)


def tod_loci_workspace_size(n: int, d: int, n_radii: int, capacity: int, opts=None) -> int:
    return int(_lib.tod_loci_workspace_size(int(n), int(d), int(n_radii), int(capacity),
                                            ctypes.byref(opts) if opts is not None else None))


def tod_loci(x, radii, alpha: float = 0.5, n_min: int = 20, k_sigma: float = 3.0, opts=None,
             capacity=None, grow: bool = True, workspace=None, stream=None, stats=None,
             return_all: bool = False):
    """LOCI at the ladder of sampling radii -> (score fp64 [n], flag int32 [n]).

    With return_all, a third element holds n_alpha, n_r (int32 [n, L]), mdef
    and sigma_mdef (fp64 [n, L]).  ``capacity`` is the number of pairs within
    the largest radius (self pairs included) the workspace is sized for
    (default 64 per row); if more are in range and ``grow`` is set, the
    workspace is resized to the count the library reports and the call is
    made once more, else TodError(TOD_ERR_CAPACITY) is raised.
    """
    torch = _torch()
    _dev_matrix(x, "x")
    n, d = x.shape
    rad = [float(r) for r in radii]
    nl = len(rad)
    rarr = (ctypes.c_double * max(nl, 1))(*rad)
    dev = x.device
    score = torch.empty((n,), dtype=torch.float64, device=dev)
    flag = torch.empty((n,), dtype=torch.int32, device=dev)
    extra = None
    if return_all:
        extra = {"n_alpha": torch.empty((n, nl), dtype=torch.int32, device=dev),
                 "n_r": torch.empty((n, nl), dtype=torch.int32, device=dev),
                 "mdef": torch.empty((n, nl), dtype=torch.float64, device=dev),
                 "sigma_mdef": torch.empty((n, nl), dtype=torch.float64, device=dev)}
    st = stats if stats is not None else new_stats()
    optp = ctypes.byref(opts) if opts is not None else None
    cap = int(capacity) if capacity is not None else 64 * n
    for _ in range(2):
        need = tod_loci_workspace_size(n, d, nl, cap, opts)
        if need == 0:  # arguments the size query rejects: let the call report why
            need = 256
        wsbuf, wsp, wsn = _ws(workspace, need, dev)
        rc = _lib.tod_loci(_p(x), n, d, rarr, nl, float(alpha), int(n_min), float(k_sigma), cap,
                           optp, wsp, wsn, _stream(stream), _p(score), _p(flag),
                           _p(extra["n_alpha"]) if extra else None,
                           _p(extra["n_r"]) if extra else None,
                           _p(extra["mdef"]) if extra else None,
                           _p(extra["sigma_mdef"]) if extra else None, ctypes.byref(st))
        if rc != TOD_ERR_CAPACITY or not grow:
            break
        cap = int(st.pairs_in_range)
    _check(rc, "tod_loci")
    del wsbuf
    return (score, flag, extra) if return_all else (score, flag)


def raw_library():
    """The loaded ctypes library (for ABI tests)."""
    return _lib
