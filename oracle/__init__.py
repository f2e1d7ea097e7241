"""Plain sequential CPU oracle for the EZ-SP partition step (arXiv 2512.00385).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import this package.  It shares no
code with the HIP path (``paper_2512_00385_amd``) and never imports it.

The arithmetic lives in ``ezsp_oracle.c`` (single-threaded C, no implicit
FMA: the kNN's fused steps are explicit ``fmaf`` calls); this
module only loads it with ctypes and moves numpy arrays in and out.  Every
function cites the passage of the paper it follows in the C header.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "ezsp_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")

# gcc flags: no contraction into FMA, no fast-math, round-to-nearest default.
CFLAGS = ["-O2", "-std=c11", "-ffp-contract=off", "-fno-fast-math", "-fPIC",
          "-shared", "-Wall", "-Wextra", "-Wno-unused-parameter"]

_lib = None


def build(force: bool = False) -> str:
    """Compile liboracle.so with gcc (built here for the tests, never shipped)."""
    if force or not os.path.exists(_LIB) or \
            os.path.getmtime(_LIB) < max(os.path.getmtime(_SRC),
                                         os.path.getmtime(_SRC[:-2] + ".h")):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", *CFLAGS, _SRC, "-o", tmp, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


class RoundLog(ctypes.Structure):
    _fields_ = [("level", ctypes.c_int32), ("round", ctypes.c_int32),
                ("n_nodes", ctypes.c_int64), ("n_edges", ctypes.c_int64),
                ("n_choosing", ctypes.c_int64), ("n_comp", ctypes.c_int64),
                ("min_gap", ctypes.c_double), ("min_sign", ctypes.c_double)]


def _load():
    global _lib
    if _lib is not None:
        return _lib
    build()
    lib = ctypes.CDLL(_LIB)
    P = ctypes.c_void_p
    i32, i64, dbl = ctypes.c_int32, ctypes.c_int64, ctypes.c_double
    sig = {
        "or_knn_brute": (ctypes.c_int, [P, i64, i32, P, P]),
        "or_knn_one": (ctypes.c_int, [P, i64, i32, i64, P, P]),
        "or_knn_kdtree": (ctypes.c_int, [P, i64, i32, P, P]),
        "or_graph": (i64, [P, i64, i32, P, P, P]),
        "or_fixed_shift": (ctypes.c_int, [P, i64, i32]),
        "or_quantize": (None, [P, i64, i32, i32, P]),
        "or_gains": (None, [i64, P, P, P, P, P, i32, i32, dbl, P]),
        "or_select": (None, [i64, i64, P, P, P, P, i64, P]),
        "or_components": (i64, [i64, P, P]),
        "or_contract": (i64, [i64, i64, P, P, P, P, P, i32, P, i64, P, P, P,
                              P, P]),
        "or_partition": (ctypes.c_int, [P, i64, i32, i64, P, P, P, i32, P, P,
                                        i32, P, P, P, P, i64, P]),
        "or_partition_linked": (ctypes.c_int, [P, P, i64, i32, i64, P, P, P,
                                               i32, P, P, i32, i32, P, P, P,
                                               P, i64, P]),
        "or_link_isolated": (i64, [i64, i64, P, P, P, P, i32, P, P]),
        "or_energy": (dbl, [P, i64, i32, i32, P, i64, i64, P, P, P, dbl]),
        "or_component_stats": (ctypes.c_int, [P, i64, i64, P, i32, P, P, P,
                                              P]),
        "or_grid_subsample": (i64, [P, i64, ctypes.c_float, P]),
        "or_edge_loss": (ctypes.c_int, [P, i64, i32, P, i32, P, P, dbl, dbl,
                                        P, P, P, P]),
        "or_purity": (ctypes.c_int, [P, i64, i64, P, i32, P, P, P]),
        "or_round_bf16": (dbl, [dbl]),
        "or_embed_mlp": (ctypes.c_int, [P, i64, i32, i32, i32, P, P, P, P, P,
                                        P, P]),
    }
    for name, (res, args) in sig.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _lib = lib
    return lib


class LossOut(ctypes.Structure):
    _fields_ = [("loss", ctypes.c_double), ("n_edges", ctypes.c_int64),
                ("n_intra", ctypes.c_int64), ("n_inter", ctypes.c_int64),
                ("n_intra_kept", ctypes.c_int64)]


class PurityOut(ctypes.Structure):
    _fields_ = [("miou", ctypes.c_double), ("purity", ctypes.c_double),
                ("n_present", ctypes.c_int64)]


class OracleError(RuntimeError):
    def __init__(self, code: int, where: str):
        super().__init__(f"{where} failed with code {code}")
        self.code = code


def _p(a):
    return None if a is None else a.ctypes.data


def _c(a, dtype):
    return np.ascontiguousarray(a, dtype=dtype)


# --------------------------------------------------------------------------
# kNN and graph (Sec. 3.1, Sec. 4.1)
# --------------------------------------------------------------------------

def knn(xyz, k: int, method: str = "kdtree"):
    """Exact kNN: (nbr int32 [n,k], d2 fp32 [n,k]); -1 / inf padding."""
    lib = _load()
    xyz = _c(xyz, np.float32).reshape(-1, 3)
    n = xyz.shape[0]
    nbr = np.empty((n, k), np.int32)
    d2 = np.empty((n, k), np.float32)
    fn = lib.or_knn_kdtree if method == "kdtree" else lib.or_knn_brute
    rc = fn(_p(xyz), n, k, _p(nbr), _p(d2))
    if rc:
        raise OracleError(rc, "knn")
    return nbr, d2


def knn_one(xyz, k: int, p: int):
    """Brute-force neighbours of the single point p."""
    lib = _load()
    xyz = _c(xyz, np.float32).reshape(-1, 3)
    nbr = np.empty(k, np.int32)
    d2 = np.empty(k, np.float32)
    rc = lib.or_knn_one(_p(xyz), xyz.shape[0], k, int(p), _p(nbr), _p(d2))
    if rc:
        raise OracleError(rc, "knn_one")
    return nbr, d2


def graph(nbr):
    """Unique undirected kNN edges sorted by (lo, hi) with w = 1."""
    lib = _load()
    nbr = _c(nbr, np.int32)
    n, k = nbr.shape
    lo = np.empty(n * k, np.int32)
    hi = np.empty(n * k, np.int32)
    w = np.empty(n * k, np.int64)
    m = lib.or_graph(_p(nbr), n, k, _p(lo), _p(hi), _p(w))
    if m < 0:
        raise OracleError(m, "graph")
    return lo[:m].copy(), hi[:m].copy(), w[:m].copy()


# --------------------------------------------------------------------------
# fixed point and one round, step by step (Prop. 1; Steps 1-4)
# --------------------------------------------------------------------------

def fixed_shift(emb) -> int:
    emb = _c(emb, np.float32)
    n = emb.shape[0]
    d = emb.shape[1] if emb.ndim == 2 else 1
    F = _load().or_fixed_shift(_p(emb), n, d)
    if F < 0:
        raise OracleError(F, "fixed_shift")
    return F


def quantize(emb, F: int):
    emb = _c(emb, np.float32)
    if emb.ndim == 1:
        emb = emb[:, None]
    S = np.empty(emb.shape, np.int64)
    _load().or_quantize(_p(emb), emb.shape[0], emb.shape[1], F, _p(S))
    return S


def gains(lo, hi, w, size, S, F: int, lam: float):
    lo, hi = _c(lo, np.int32), _c(hi, np.int32)
    w, size, S = _c(w, np.int64), _c(size, np.int64), _c(S, np.int64)
    if S.ndim == 1:
        S = S[:, None]
    delta = np.empty(lo.shape[0], np.float64)
    _load().or_gains(lo.shape[0], _p(lo), _p(hi), _p(w), _p(size), _p(S),
                     S.shape[1], F, float(lam), _p(delta))
    return delta


def select(nn: int, lo, hi, delta, size, min_size: int = 0):
    lo, hi = _c(lo, np.int32), _c(hi, np.int32)
    delta, size = _c(delta, np.float64), _c(size, np.int64)
    target = np.empty(nn, np.int32)
    _load().or_select(nn, lo.shape[0], _p(lo), _p(hi), _p(delta), _p(size),
                      int(min_size), _p(target))
    return target


def components(target):
    target = _c(target, np.int32)
    label = np.empty(target.shape[0], np.int32)
    nc = _load().or_components(target.shape[0], _p(target), _p(label))
    return label, int(nc)


def contract(lo, hi, w, size, S, label, nc: int):
    lo, hi = _c(lo, np.int32), _c(hi, np.int32)
    w, size, S = _c(w, np.int64), _c(size, np.int64), _c(S, np.int64)
    label = _c(label, np.int32)
    if S.ndim == 1:
        S = S[:, None]
    d = S.shape[1]
    ne = lo.shape[0]
    size_o = np.empty(nc, np.int64)
    S_o = np.empty((nc, d), np.int64)
    lo_o = np.empty(max(ne, 1), np.int32)
    hi_o = np.empty(max(ne, 1), np.int32)
    w_o = np.empty(max(ne, 1), np.int64)
    m = _load().or_contract(size.shape[0], ne, _p(lo), _p(hi), _p(w),
                            _p(size), _p(S), d, _p(label), nc, _p(size_o),
                            _p(S_o), _p(lo_o), _p(hi_o), _p(w_o))
    return size_o, S_o, lo_o[:m].copy(), hi_o[:m].copy(), w_o[:m].copy()


# --------------------------------------------------------------------------
# the ladder and the energy (Sec. 3.2; Alg. A-2; Eq. gmpp)
# --------------------------------------------------------------------------

def partition_graph(emb, lo, hi, w, lambdas, min_size=None, max_rounds=0,
                    want_log=False, want_energy=True, xyz=None, link_k=0):
    """Round-synchronous merge ladder on a given graph; with link_k > 0 and
    positions xyz, isolated nodes are linked first in every round.

    Returns (labels [L,n] int32, n_comp [L] int64, energy [L] or None,
    log list of dicts or None)."""
    lib = _load()
    emb = _c(emb, np.float32)
    if emb.ndim == 1:
        emb = emb[:, None]
    n, d = emb.shape
    lo, hi, w = _c(lo, np.int32), _c(hi, np.int32), _c(w, np.int64)
    lam = _c(np.atleast_1d(lambdas), np.float64)
    L = lam.shape[0]
    ms = None if min_size is None else _c(np.atleast_1d(min_size), np.int64)
    labels = np.empty((L, n), np.int32)
    n_comp = np.empty(L, np.int64)
    energy = np.empty(L, np.float64) if want_energy else None
    cap = 4096 if want_log else 0
    log = (RoundLog * max(cap, 1))()
    log_len = ctypes.c_int64(0)
    if link_k:
        xyz = _c(xyz, np.float32).reshape(-1, 3)
        rc = lib.or_partition_linked(
            _p(emb), _p(xyz), n, d, lo.shape[0], _p(lo), _p(hi), _p(w), L,
            _p(lam), _p(ms), int(link_k), int(max_rounds), _p(labels),
            _p(n_comp), _p(energy),
            ctypes.addressof(log) if want_log else None, cap,
            ctypes.addressof(log_len))
    else:
        rc = lib.or_partition(_p(emb), n, d, lo.shape[0], _p(lo), _p(hi),
                              _p(w), L, _p(lam), _p(ms), int(max_rounds),
                              _p(labels), _p(n_comp), _p(energy),
                              ctypes.addressof(log) if want_log else None,
                              cap, ctypes.addressof(log_len))
    if rc:
        raise OracleError(rc, "partition")
    rounds = None
    if want_log:
        rounds = [{f: getattr(log[i], f) for f, _ in RoundLog._fields_}
                  for i in range(log_len.value)]
    return labels, n_comp, energy, rounds


def partition(xyz, emb, k: int, lambdas, min_size=None, max_rounds=0,
              want_log=False, want_energy=True, knn_method="kdtree",
              link=False):
    """kNN graph, then the ladder: the whole path the GPU library computes
    (link: prepare_graph's linking of isolated nodes with the same k)."""
    nbr, _ = knn(xyz, k, knn_method)
    lo, hi, w = graph(nbr)
    return partition_graph(emb, lo, hi, w, lambdas, min_size, max_rounds,
                           want_log, want_energy, xyz=xyz,
                           link_k=k if link else 0)


def link_isolated(lo, hi, size, Sx, k: int):
    """One linking step: the new (lo, hi) pairs for the isolated nodes."""
    lo, hi = _c(lo, np.int32), _c(hi, np.int32)
    size, Sx = _c(size, np.int64), _c(Sx, np.int64).reshape(-1, 3)
    nn = size.shape[0]
    lo_o = np.empty(max(nn * k, 1), np.int32)
    hi_o = np.empty(max(nn * k, 1), np.int32)
    m = _load().or_link_isolated(nn, lo.shape[0], _p(lo), _p(hi), _p(size),
                                 _p(Sx), int(k), _p(lo_o), _p(hi_o))
    if m < 0:
        raise OracleError(m, "link_isolated")
    return lo_o[:m].copy(), hi_o[:m].copy()


def energy(emb, label, lo, hi, w, lam: float, F: int | None = None):
    lib = _load()
    emb = _c(emb, np.float32)
    if emb.ndim == 1:
        emb = emb[:, None]
    n, d = emb.shape
    if F is None:
        F = fixed_shift(emb)
    label = _c(label, np.int32)
    lo, hi, w = _c(lo, np.int32), _c(hi, np.int32), _c(w, np.int64)
    nc = int(label.max()) + 1
    return lib.or_energy(_p(emb), n, d, F, _p(label), nc, lo.shape[0], _p(lo),
                         _p(hi), _p(w), float(lam))


def component_stats(label, n_comp: int, emb, xyz=None):
    lib = _load()
    label = _c(label, np.int32)
    emb = _c(emb, np.float32)
    if emb.ndim == 1:
        emb = emb[:, None]
    n, d = emb.shape
    size = np.empty(n_comp, np.int64)
    mean = np.empty((n_comp, d), np.float32)
    cen = None
    if xyz is not None:
        xyz = _c(xyz, np.float32).reshape(-1, 3)
        cen = np.empty((n_comp, 3), np.float32)
    rc = lib.or_component_stats(_p(label), n, n_comp, _p(emb), d, _p(xyz),
                                _p(size), _p(mean), _p(cen))
    if rc:
        raise OracleError(rc, "component_stats")
    return size, mean, cen


# --------------------------------------------------------------------------
# grid subsampling (Sec. 4.1), contrastive edge loss (Sec. 3.1), purity and
# oracle mIoU (Sec. 4.2 "Metrics")
# --------------------------------------------------------------------------

def grid_subsample(xyz, h: float):
    """Indices (increasing) of the smallest-index point of every grid cell."""
    xyz = _c(xyz, np.float32).reshape(-1, 3)
    keep = np.empty(max(xyz.shape[0], 1), np.int32)
    m = _load().or_grid_subsample(_p(xyz), xyz.shape[0], float(h), _p(keep))
    if m < 0:
        raise OracleError(m, "grid_subsample")
    return keep[:m].copy()


def edge_loss(emb, nbr, cls, word, tau: float, rho: float,
              want_affinity=True, want_grad=True):
    """Eq. loss over the sampled kNN pairs.  Returns (dict of the sums and
    counts, affinity [n,k] fp64 or None, grad [n,d] fp64 or None,
    sampled [n,k] uint8: 1 where the slot owns a sampled edge)."""
    emb = _c(emb, np.float32)
    if emb.ndim == 1:
        emb = emb[:, None]
    n, d = emb.shape
    nbr = _c(nbr, np.int32).reshape(n, -1)
    k = nbr.shape[1]
    cls = _c(cls, np.int32)
    word = _c(word, np.uint32).reshape(n, k)
    aff = np.empty((n, k), np.float64) if want_affinity else None
    grad = np.empty((n, d), np.float64) if want_grad else None
    sampled = np.empty((n, k), np.uint8)
    out = LossOut()
    rc = _load().or_edge_loss(_p(emb), n, d, _p(nbr), k, _p(cls), _p(word),
                              float(tau), float(rho), _p(aff), _p(grad),
                              _p(sampled), ctypes.byref(out))
    if rc:
        raise OracleError(rc, "edge_loss")
    res = {f: getattr(out, f) for f, _ in LossOut._fields_}
    return res, aff, grad, sampled


def purity(label, n_comp: int, cls, n_cls: int):
    """Majority class per component, per-class IoU, mIoU and purity."""
    label, cls = _c(label, np.int32), _c(cls, np.int32)
    n = label.shape[0]
    maj = np.empty(n_comp, np.int32)
    iou = np.empty(n_cls, np.float64)
    out = PurityOut()
    rc = _load().or_purity(_p(label), n, int(n_comp), _p(cls), int(n_cls),
                           _p(maj), _p(iou), ctypes.byref(out))
    if rc:
        raise OracleError(rc, "purity")
    return ({"miou": out.miou, "purity": out.purity,
             "n_present": out.n_present}, maj, iou)


# --------------------------------------------------------------------------
# point-embedding MLP (stand-in for the embedding network of Sec. 3.1)
# --------------------------------------------------------------------------

def round_bf16(v: float) -> float:
    return _load().or_round_bf16(float(v))


def embed_mlp(x_bits, w1_bits, b1, w2_bits, b2, w3_bits, b3):
    """The MLP on bfloat16 bit patterns (uint16 arrays): fp64 output [n,
    d_out] (exact last-layer sums)."""
    x = _c(x_bits, np.uint16)
    n, d_in = x.shape
    w1, w2, w3 = (_c(w, np.uint16) for w in (w1_bits, w2_bits, w3_bits))
    b1, b2, b3 = (_c(b, np.float32) for b in (b1, b2, b3))
    d_hid, d_out = w1.shape[1], w3.shape[1]
    out = np.empty((n, d_out), np.float64)
    rc = _load().or_embed_mlp(_p(x), n, d_in, d_hid, d_out, _p(w1), _p(b1),
                              _p(w2), _p(b2), _p(w3), _p(b3), _p(out))
    if rc:
        raise OracleError(rc, "embed_mlp")
    return out
