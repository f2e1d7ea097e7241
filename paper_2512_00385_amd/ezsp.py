"""Thin Python binding of the C ABI in ``include/ezsp.h`` (libezsp.so).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  Tensors must already live on the current HIP device; outputs and
the workspace are allocated with torch on that device, and the call is
enqueued on torch's current stream.  There is no fallback: when the
library is missing, loading raises.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np
import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libezsp.so")

OK = 0
ERR_INVALID_ARG = -1
ERR_NONFINITE = -2
ERR_RANGE = -3
ERR_WORKSPACE = -4
ERR_DEVICE = -5
ERR_NOT_CONVERGED = -6
F_ENERGY = 1
F_LINK_ISOLATED = 2

ENTRY_POINTS = (
    "ezsp_knn_workspace_size", "ezsp_knn",
    "ezsp_partition_workspace_size", "ezsp_partition",
    "ezsp_partition_from_knn",
    "ezsp_component_stats_workspace_size", "ezsp_component_stats",
    "ezsp_status_string", "ezsp_last_error",
    "ezsp_profile_enable", "ezsp_profile_read", "ezsp_profile_only",
    "ezsp_grid_subsample_workspace_size", "ezsp_grid_subsample",
    "ezsp_edge_loss_workspace_size", "ezsp_edge_loss",
    "ezsp_purity_workspace_size", "ezsp_purity",
    "ezsp_embed_mlp", "ezsp_sync_status", "ezsp_knn_noalloc",
    "ezsp_knn_walk_stats",
)


class Params(ctypes.Structure):
    """Mirror of ezsp_params."""
    _fields_ = [("k", ctypes.c_int32), ("n_levels", ctypes.c_int32),
                ("lambdas", ctypes.c_void_p), ("min_size", ctypes.c_void_p),
                ("max_rounds", ctypes.c_int32), ("flags", ctypes.c_uint32)]


class LossStats(ctypes.Structure):
    """Mirror of ezsp_loss_stats."""
    _fields_ = [("loss", ctypes.c_double), ("n_edges", ctypes.c_int64),
                ("n_intra", ctypes.c_int64), ("n_inter", ctypes.c_int64),
                ("n_intra_kept", ctypes.c_int64)]


class PurityStats(ctypes.Structure):
    """Mirror of ezsp_purity_stats."""
    _fields_ = [("miou", ctypes.c_double), ("purity", ctypes.c_double),
                ("n_present", ctypes.c_int64)]


class EzspError(RuntimeError):
    def __init__(self, code: int, where: str, detail: str):
        super().__init__(f"{where}: {status_string(code)} ({code}): {detail}")
        self.code = code


_lib = None


def load() -> ctypes.CDLL:
    """Load libezsp.so (built by ``paper_2512_00385_amd/build.py``)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(
            f"{LIB_PATH} is missing: build it with "
            "`python paper_2512_00385_amd/build.py` (or __graft_entry__.build())")
    lib = ctypes.CDLL(LIB_PATH)
    P, i32, i64, sz = (ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64,
                       ctypes.c_size_t)
    sig = {
        "ezsp_knn_workspace_size": (sz, [i64, i32]),
        "ezsp_knn": (ctypes.c_int, [P, i64, i32, P, P, P, sz, P]),
        "ezsp_partition_workspace_size": (sz, [i64, i32, P]),
        "ezsp_partition": (ctypes.c_int, [P, P, i64, i32, P, P, P, P, P, sz,
                                          P]),
        "ezsp_partition_from_knn": (ctypes.c_int, [P, P, i64, i32, P, P, P, P,
                                                   P, sz, P]),
        "ezsp_component_stats_workspace_size": (sz, [i64, i64, i32]),
        "ezsp_component_stats": (ctypes.c_int, [P, i64, i64, P, i32, P, P, P,
                                                P, P, sz, P]),
        "ezsp_status_string": (ctypes.c_char_p, [ctypes.c_int]),
        "ezsp_last_error": (ctypes.c_char_p, []),
        "ezsp_profile_enable": (ctypes.c_int, [ctypes.c_int]),
        "ezsp_profile_read": (ctypes.c_int, [ctypes.c_char_p, P, P, P]),
        "ezsp_profile_only": (ctypes.c_int, [ctypes.c_char_p]),
        "ezsp_grid_subsample_workspace_size": (sz, [i64]),
        "ezsp_grid_subsample": (ctypes.c_int, [P, i64, ctypes.c_float, P, P,
                                               P, sz, P]),
        "ezsp_edge_loss_workspace_size": (sz, [i64, i32]),
        "ezsp_edge_loss": (ctypes.c_int, [P, i64, i32, P, i32, P, P,
                                          ctypes.c_double, ctypes.c_double,
                                          P, P, P, P, P, sz, P]),
        "ezsp_purity_workspace_size": (sz, [i64, i64, i32]),
        "ezsp_purity": (ctypes.c_int, [P, i64, i64, P, i32, P, P, P, P, sz,
                                       P]),
        "ezsp_embed_mlp": (ctypes.c_int, [P, i64, i32, i32, i32, P, P, P, P,
                                          P, P, P, P]),
        "ezsp_sync_status": (ctypes.c_int, [P, sz, P]),
        "ezsp_knn_noalloc": (ctypes.c_int, [P, i64, i32, P, P, P]),
        "ezsp_knn_walk_stats": (ctypes.c_int, [P, i64, i32, P, P, P, P, sz,
                                               P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


def status_string(code: int) -> str:
    return load().ezsp_status_string(int(code)).decode()


def last_error() -> str:
    return load().ezsp_last_error().decode()


def profile_enable(on: bool = True):
    """Start (clearing the totals) or stop per-stage event timing."""
    load().ezsp_profile_enable(1 if on else 0)


def profile_only(stage=None):
    """Time only `stage` (None: every stage) while profiling is on."""
    load().ezsp_profile_only(stage.encode() if stage else None)


STAGES = ("morton_sort", "knn_query", "graph_build", "select", "union",
          "stats", "contract", "compose", "tail", "link")
EXTRA_STAGES = ("grid_subsample", "edge_loss", "purity", "embed_mlp")


def profile_read(stage: str):
    """(launches, total milliseconds, algorithmic bytes) of a stage."""
    n = ctypes.c_int64(0)
    ms = ctypes.c_double(0.0)
    nb = ctypes.c_double(0.0)
    load().ezsp_profile_read(stage.encode(), ctypes.byref(n), ctypes.byref(ms),
                             ctypes.byref(nb))
    return int(n.value), float(ms.value), float(nb.value)


def _check(code: int, where: str):
    if code != OK:
        raise EzspError(code, where, last_error())


def _ptr(t):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _dev_tensor(t, dtype, name, cols=None):
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a device tensor")
    if t.dtype != dtype:
        raise TypeError(f"{name} must be {dtype}, got {t.dtype}")
    if cols is not None and (t.dim() != 2 or t.shape[1] != cols):
        raise ValueError(f"{name} must have shape [n, {cols}]")
    return t.contiguous()


def _stream(device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _workspace(nbytes: int, device):
    if nbytes == 0:
        raise EzspError(ERR_INVALID_ARG, "workspace size", "invalid sizes")
    return torch.empty(nbytes, dtype=torch.uint8, device=device)


def _params(k, lambdas, min_size, max_rounds, energy, link=False):
    lam = np.ascontiguousarray(np.atleast_1d(np.asarray(lambdas, np.float64)))
    ms = None
    if min_size is not None:
        ms = np.ascontiguousarray(np.atleast_1d(np.asarray(min_size,
                                                           np.int64)))
        if ms.shape != lam.shape:
            raise ValueError("min_size needs one value per level")
    p = Params(int(k), int(lam.shape[0]), lam.ctypes.data,
               None if ms is None else ms.ctypes.data, int(max_rounds),
               (F_ENERGY if energy else 0) | (F_LINK_ISOLATED if link else 0))
    return p, lam, ms  # keep the arrays alive with the struct


class Pending:
    """The workspace of a stream-asynchronous call, kept alive until its
    device-detected errors have been checked (ezsp_sync_status)."""

    def __init__(self, ws, nbytes, device, where):
        self.ws, self.nbytes, self.device, self.where = ws, nbytes, device, where

    def check(self):
        """Synchronise the stream; raise EzspError for a device error."""
        _check(load().ezsp_sync_status(_ptr(self.ws), self.nbytes,
                                       _stream(self.device)), self.where)


def knn(xyz: torch.Tensor, k: int, want_d2: bool = False, sync: bool = True):
    """Exact kNN (ezsp_knn): nbr [n, k] int32 (and d2 [n, k] fp32).  With
    sync=False the call returns right after enqueuing, with a Pending whose
    check() reports device errors: (nbr, [d2,] pending)."""
    lib = load()
    xyz = _dev_tensor(xyz, torch.float32, "xyz", 3)
    n = xyz.shape[0]
    dev = xyz.device
    nbr = torch.empty((n, k), dtype=torch.int32, device=dev)
    d2 = torch.empty((n, k), dtype=torch.float32, device=dev) \
        if want_d2 else None
    nbytes = lib.ezsp_knn_workspace_size(n, k)
    ws = _workspace(nbytes, dev)
    _check(lib.ezsp_knn(_ptr(xyz), n, int(k), _ptr(nbr), _ptr(d2), _ptr(ws),
                        nbytes, _stream(dev)), "ezsp_knn")
    pending = Pending(ws, nbytes, dev, "ezsp_knn")
    if sync:
        pending.check()
        return (nbr, d2) if want_d2 else nbr
    return ((nbr, d2) if want_d2 else (nbr,)) + (pending,)


def knn_walk_stats(xyz: torch.Tensor, k: int):
    """ezsp_knn_walk_stats: (nbr [n, k] int32, 16-point buckets scanned and
    inner nodes entered per 64-point query group, each [ceil(n / 64)]
    int32)."""
    lib = load()
    xyz = _dev_tensor(xyz, torch.float32, "xyz", 3)
    n = xyz.shape[0]
    dev = xyz.device
    g = (n + 63) // 64
    nbr = torch.empty((n, k), dtype=torch.int32, device=dev)
    scans = torch.empty(g, dtype=torch.int32, device=dev)
    nodes = torch.empty(g, dtype=torch.int32, device=dev)
    nbytes = lib.ezsp_knn_workspace_size(n, k)
    ws = _workspace(nbytes, dev)
    _check(lib.ezsp_knn_walk_stats(_ptr(xyz), n, int(k), _ptr(nbr),
                                   _ptr(scans), _ptr(nodes), _ptr(ws), nbytes,
                                   _stream(dev)), "ezsp_knn_walk_stats")
    Pending(ws, nbytes, dev, "ezsp_knn_walk_stats").check()
    return nbr, scans, nodes


def partition_workspace_size(n: int, d: int, k: int, n_levels: int = 1):
    p, _, _ = _params(k, [0.0] * n_levels, None, 0, False)
    return load().ezsp_partition_workspace_size(n, d, ctypes.byref(p))


class Partitioner:
    """Reusable call state for ezsp_partition: the workspace is allocated
    once, so repeated calls on the same sizes allocate nothing new."""

    def __init__(self, n: int, d: int, k: int, lambdas, min_size=None,
                 max_rounds: int = 0, energy: bool = False, device=None,
                 link: bool = False):
        self.lib = load()
        self.n, self.d, self.k = int(n), int(d), int(k)
        self.device = torch.device(device or "cuda")
        self.params, self._lam, self._ms = _params(k, lambdas, min_size,
                                                   max_rounds, energy, link)
        self.L = int(self._lam.shape[0])
        self.nbytes = self.lib.ezsp_partition_workspace_size(
            self.n, self.d, ctypes.byref(self.params))
        self.ws = _workspace(self.nbytes, self.device)
        self.labels = torch.empty((self.L, self.n), dtype=torch.int32,
                                  device=self.device)
        self.n_comp = np.zeros(self.L, np.int64)
        self.energy = np.zeros(self.L, np.float64) if energy else None

    def __call__(self, xyz: torch.Tensor, emb: torch.Tensor):
        xyz = _dev_tensor(xyz, torch.float32, "xyz", 3)
        emb = _dev_tensor(emb, torch.float32, "emb", self.d)
        if xyz.shape[0] != self.n or emb.shape[0] != self.n:
            raise ValueError("xyz/emb do not have n rows")
        rc = self.lib.ezsp_partition(
            _ptr(xyz), _ptr(emb), self.n, self.d, ctypes.byref(self.params),
            _ptr(self.labels), self.n_comp.ctypes.data,
            None if self.energy is None else self.energy.ctypes.data,
            _ptr(self.ws), self.nbytes, _stream(self.device))
        _check(rc, "ezsp_partition")
        return self.labels, self.n_comp.copy(), \
            None if self.energy is None else self.energy.copy()


def partition(xyz: torch.Tensor, emb: torch.Tensor, k: int, lambdas,
              min_size=None, max_rounds: int = 0, energy: bool = False,
              link: bool = False):
    """kNN graph + merge ladder (ezsp_partition); link: prepare_graph's
    linking of isolated nodes (EZSP_F_LINK_ISOLATED).

    Returns (labels [L, n] int32 on the device, n_comp int64 numpy [L],
    energy float64 numpy [L] or None)."""
    emb = _dev_tensor(emb, torch.float32, "emb")
    if emb.dim() != 2:
        raise ValueError("emb must have shape [n, d]")
    part = Partitioner(xyz.shape[0], emb.shape[1], k, lambdas, min_size,
                       max_rounds, energy, xyz.device, link)
    labels, nc, en = part(xyz, emb)
    return labels, nc, en


def partition_from_knn(nbr: torch.Tensor, emb: torch.Tensor, lambdas,
                       min_size=None, max_rounds: int = 0,
                       energy: bool = False):
    """Merge ladder on a given neighbour table (ezsp_partition_from_knn)."""
    lib = load()
    nbr = _dev_tensor(nbr, torch.int32, "nbr")
    emb = _dev_tensor(emb, torch.float32, "emb")
    if nbr.dim() != 2 or emb.dim() != 2 or nbr.shape[0] != emb.shape[0]:
        raise ValueError("nbr [n, k] and emb [n, d] needed")
    n, k = nbr.shape
    d = emb.shape[1]
    dev = emb.device
    p, lam, ms = _params(k, lambdas, min_size, max_rounds, energy)
    L = lam.shape[0]
    # from_knn needs no kNN scratch; the xyz query is an upper bound
    nbytes = lib.ezsp_partition_workspace_size(n, d, ctypes.byref(p))
    ws = _workspace(nbytes, dev)
    labels = torch.empty((L, n), dtype=torch.int32, device=dev)
    n_comp = np.zeros(L, np.int64)
    en = np.zeros(L, np.float64) if energy else None
    rc = lib.ezsp_partition_from_knn(
        _ptr(nbr), _ptr(emb), n, d, ctypes.byref(p), _ptr(labels),
        n_comp.ctypes.data, None if en is None else en.ctypes.data, _ptr(ws),
        nbytes, _stream(dev))
    _check(rc, "ezsp_partition_from_knn")
    return labels, n_comp, en


def component_stats(labels: torch.Tensor, n_comp: int, emb: torch.Tensor,
                    xyz: torch.Tensor | None = None, sync: bool = True):
    """Size, mean embedding and centroid per superpoint.  With sync=False
    the call returns right after enqueuing: (size, mean, centroid,
    pending), pending.check() reporting device errors."""
    lib = load()
    labels = _dev_tensor(labels, torch.int32, "labels")
    emb = _dev_tensor(emb, torch.float32, "emb")
    n, d = emb.shape
    dev = emb.device
    if xyz is not None:
        xyz = _dev_tensor(xyz, torch.float32, "xyz", 3)
    size = torch.empty(n_comp, dtype=torch.int64, device=dev)
    mean = torch.empty((n_comp, d), dtype=torch.float32, device=dev)
    cen = torch.empty((n_comp, 3), dtype=torch.float32, device=dev) \
        if xyz is not None else None
    nbytes = lib.ezsp_component_stats_workspace_size(n, int(n_comp), d)
    ws = _workspace(nbytes, dev)
    _check(lib.ezsp_component_stats(_ptr(labels), n, int(n_comp), _ptr(emb),
                                    d, _ptr(xyz), _ptr(size), _ptr(mean),
                                    _ptr(cen), _ptr(ws), nbytes,
                                    _stream(dev)), "ezsp_component_stats")
    pending = Pending(ws, nbytes, dev, "ezsp_component_stats")
    if sync:
        pending.check()
        return size, mean, cen
    return size, mean, cen, pending


def grid_subsample(xyz: torch.Tensor, h: float) -> torch.Tensor:
    """Indices (increasing, int32) of the point kept in every occupied cell
    of a regular grid of spacing h: the cell's smallest point index."""
    lib = load()
    xyz = _dev_tensor(xyz, torch.float32, "xyz", 3)
    n = xyz.shape[0]
    keep = torch.empty(n, dtype=torch.int32, device=xyz.device)
    n_keep = ctypes.c_int64(0)
    nbytes = lib.ezsp_grid_subsample_workspace_size(n)
    ws = _workspace(nbytes, xyz.device)
    _check(lib.ezsp_grid_subsample(_ptr(xyz), n, float(h), _ptr(keep),
                                   ctypes.byref(n_keep), _ptr(ws), nbytes,
                                   _stream(xyz.device)),
           "ezsp_grid_subsample")
    return keep[:n_keep.value]


def edge_loss(emb: torch.Tensor, nbr: torch.Tensor, cls: torch.Tensor,
              word: torch.Tensor, tau: float, rho: float,
              want_affinity: bool = True, want_grad: bool = True,
              want_sampled: bool = True):
    """Affinity and contrastive edge loss over the kNN pairs.  Returns
    (stats dict, affinity [n,k] fp32 or None, grad [n,d] fp32 or None,
    sampled [n,k] uint8 or None)."""
    lib = load()
    emb = _dev_tensor(emb, torch.float32, "emb")
    n, d = emb.shape
    nbr = _dev_tensor(nbr, torch.int32, "nbr")
    if nbr.dim() != 2 or nbr.shape[0] != n:
        raise ValueError("nbr must have shape [n, k]")
    k = nbr.shape[1]
    cls = _dev_tensor(cls, torch.int32, "cls")
    if isinstance(word, torch.Tensor) and word.dtype == torch.uint32:
        word = word.view(torch.int32)
    word = _dev_tensor(word, torch.int32, "word (uint32 or its int32 bits)")
    if cls.shape != (n,) or word.shape != (n, k):
        raise ValueError("cls must be [n] and word [n, k]")
    dev = emb.device
    aff = torch.empty((n, k), dtype=torch.float32, device=dev) \
        if want_affinity else None
    grad = torch.empty((n, d), dtype=torch.float32, device=dev) \
        if want_grad else None
    smp = torch.empty((n, k), dtype=torch.uint8, device=dev) \
        if want_sampled else None
    out = LossStats()
    nbytes = lib.ezsp_edge_loss_workspace_size(n, k)
    ws = _workspace(nbytes, dev)
    _check(lib.ezsp_edge_loss(_ptr(emb), n, d, _ptr(nbr), k, _ptr(cls),
                              _ptr(word), float(tau), float(rho), _ptr(aff),
                              _ptr(grad), _ptr(smp), ctypes.byref(out),
                              _ptr(ws), nbytes, _stream(dev)),
           "ezsp_edge_loss")
    stats = {f: getattr(out, f) for f, _ in LossStats._fields_}
    return stats, aff, grad, smp


def purity(labels: torch.Tensor, n_comp: int, cls: torch.Tensor, n_cls: int):
    """Majority class per superpoint, per-class IoU, mIoU and purity.
    Returns (stats dict, majority [n_comp] int32, iou [n_cls] fp64)."""
    lib = load()
    labels = _dev_tensor(labels, torch.int32, "labels")
    cls = _dev_tensor(cls, torch.int32, "cls")
    n = labels.shape[0]
    if cls.shape != labels.shape:
        raise ValueError("labels and cls must have the same shape")
    dev = labels.device
    maj = torch.empty(int(n_comp), dtype=torch.int32, device=dev)
    iou = torch.empty(int(n_cls), dtype=torch.float64, device=dev)
    out = PurityStats()
    nbytes = lib.ezsp_purity_workspace_size(n, int(n_comp), int(n_cls))
    ws = _workspace(nbytes, dev)
    _check(lib.ezsp_purity(_ptr(labels), n, int(n_comp), _ptr(cls),
                           int(n_cls), _ptr(maj), _ptr(iou), ctypes.byref(out),
                           _ptr(ws), nbytes, _stream(dev)), "ezsp_purity")
    stats = {f: getattr(out, f) for f, _ in PurityStats._fields_}
    return stats, maj, iou


def embed_mlp(x_bits: torch.Tensor, w1, b1, w2, b2, w3, b3) -> torch.Tensor:
    """Per-point MLP d_in -> 32 -> 32 -> d_out on the matrix cores.  x_bits
    and the weights are bfloat16 tensors (or int16 tensors of their bits) on
    the device, weights as [fan_in, fan_out]; biases fp32.  Returns
    [n, d_out] fp32, computed in stream order (the call does not wait)."""
    lib = load()

    def bits(t, name):
        if not isinstance(t, torch.Tensor) or not t.is_cuda:
            raise TypeError(f"{name} must be a device tensor")
        if t.dtype == torch.bfloat16:
            t = t.view(torch.int16)
        if t.dtype != torch.int16:
            raise TypeError(f"{name} must be bfloat16 (or its int16 bits)")
        return t.contiguous()
    x = bits(x_bits, "x")
    w1, w2, w3 = bits(w1, "w1"), bits(w2, "w2"), bits(w3, "w3")
    b1 = _dev_tensor(b1, torch.float32, "b1")
    b2 = _dev_tensor(b2, torch.float32, "b2")
    b3 = _dev_tensor(b3, torch.float32, "b3")
    n, d_in = x.shape
    d_hid, d_out = w1.shape[1], w3.shape[1]
    if w1.shape[0] != d_in or w2.shape != (d_hid, d_hid) or \
            w3.shape[0] != d_hid:
        raise ValueError("weight shapes do not chain")
    out = torch.empty((n, d_out), dtype=torch.float32, device=x.device)
    _check(lib.ezsp_embed_mlp(_ptr(x), n, d_in, d_hid, d_out, _ptr(w1),
                              _ptr(b1), _ptr(w2), _ptr(b2), _ptr(w3),
                              _ptr(b3), _ptr(out), _stream(x.device)),
           "ezsp_embed_mlp")
    return out
