"""A second, independent statement of the merge procedure, used only to pin
the oracle.

It follows the paper's recursive formulation (App. Alg. A-2 for one level,
App. Alg. A-1 for the weakly connected components) rather than the oracle's
structure: embeddings are plain float64 means (no fixed point), components
come from max-propagation of random node ids until nothing changes, and the
graph is re-contracted after every round.  It shares no code with the
oracle.  Ties are not resolved here, so callers use inputs whose decisions
have clear margins.
"""
from __future__ import annotations

import numpy as np


def canonical(labels):
    """Renumber labels by first occurrence (smallest member first)."""
    labels = np.asarray(labels)
    _, first = np.unique(labels, return_index=True)
    order = np.argsort(first)
    remap = np.empty(order.shape[0], np.int64)
    remap[order] = np.arange(order.shape[0])
    _, inv = np.unique(labels, return_inverse=True)
    return remap[inv]


def wcc_max_prop(n, src, dst, rng):
    """Alg. A-1: random ids, max over neighbours until stable, then
    consecutive ids."""
    ids = rng.permutation(n)
    while True:
        nxt = ids.copy()
        np.maximum.at(nxt, src, ids[dst])
        np.maximum.at(nxt, dst, ids[src])
        if np.array_equal(nxt, ids):
            break
        ids = nxt
    _, comp = np.unique(ids, return_inverse=True)
    return comp


def merge_level(feat, size, lo, hi, w, lam, s_min=0, rng=None, max_rounds=10_000):
    """One level of Alg. A-2 (recursion unrolled into a loop).  Returns the
    component of every input node."""
    rng = rng or np.random.default_rng(0)
    feat = np.asarray(feat, np.float64).copy()
    if feat.ndim == 1:
        feat = feat[:, None]
    size = np.asarray(size, np.float64).copy()
    n = feat.shape[0]
    assign = np.arange(n)
    lo = np.asarray(lo, np.int64)
    hi = np.asarray(hi, np.int64)
    w = np.asarray(w, np.float64)
    for _ in range(max_rounds):
        # prepare_graph: no self loops, one edge per pair, summed weights
        keep = lo != hi
        a, b = np.minimum(lo[keep], hi[keep]), np.maximum(lo[keep], hi[keep])
        if a.size == 0:
            break
        key = a * feat.shape[0] + b
        uk, inv = np.unique(key, return_inverse=True)
        w = np.bincount(inv, weights=w[keep])
        lo, hi = uk // feat.shape[0], uk % feat.shape[0]
        # edge_merge_energy, Eq. delta
        f = size[lo] * size[hi] / (size[lo] + size[hi])
        gain = lam * w - f * ((feat[lo] - feat[hi]) ** 2).sum(1)
        # keep_valid_merges: directed candidates, best outgoing per source
        src = np.concatenate([lo, hi])
        dst = np.concatenate([hi, lo])
        g2 = np.concatenate([gain, gain])
        ok = (g2 > 0) | (size[src] < s_min)
        if not ok.any():
            break
        src, dst, g2 = src[ok], dst[ok], g2[ok]
        order = np.lexsort((-g2, src))
        first = np.ones(order.shape[0], bool)
        first[1:] = src[order][1:] != src[order][:-1]
        sel = order[first]
        comp = wcc_max_prop(feat.shape[0], src[sel], dst[sel], rng)
        assign = comp[assign]
        nc = comp.max() + 1
        if nc == 1:
            break
        # component_attributes and component_graph
        ns = np.bincount(comp, weights=size, minlength=nc)
        nf = np.zeros((nc, feat.shape[1]))
        np.add.at(nf, comp, feat * size[:, None])
        feat = nf / ns[:, None]
        size = ns
        lo, hi = comp[lo], comp[hi]
    return assign
