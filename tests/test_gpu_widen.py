"""GPU parity of the grid subsampling, the contrastive edge loss and the
purity / oracle mIoU against the CPU oracle, through the C ABI.

Bars: kept indices, pair counts, the sampled-slot mask, majorities, IoUs,
mIoU and purity are bit-identical (integer work, and fp64 divisions of the
same integers in the same order).  Affinities, the loss and the gradient are
fp32 arithmetic against the oracle's fp64: each distance carries a relative
error of a few fp32 ulps, so affinities must agree to 2e-6 absolute, the fp64
sum of the loss terms to 1e-5 relative, and every gradient element (fp32
atomics over the ~2k pairs touching a point) to 1e-4 relative plus 1e-5 of
the largest gradient element."""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_00385_amd import ezsp, scenes

pytestmark = pytest.mark.gpu

AFF_ATOL = 2e-6
LOSS_RTOL = 1e-5
GRAD_RTOL, GRAD_ATOL_REL = 1e-4, 1e-5


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ezsp.load()
    yield


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


# --------------------------------------------------------------------------
# grid subsampling
# --------------------------------------------------------------------------

def grid_clouds():
    rng = np.random.default_rng(11)
    lat = np.stack(np.meshgrid(np.arange(9), np.arange(7), np.arange(5),
                               indexing="ij"), -1).reshape(-1, 3)
    lat = ((lat + 0.5) * 0.25).astype(np.float32)
    return {
        "uniform": (rng.random((20000, 3)) * 3 - 1).astype(np.float32),
        "lattice_x3": lat[rng.permutation(np.repeat(np.arange(len(lat)), 3))],
        "single": np.array([[1.0, -2.0, 3.0]], np.float32),
        "identical": np.ones((777, 3), np.float32),
        "planar": np.concatenate([rng.random((5000, 2), dtype=np.float32),
                                  np.zeros((5000, 1), np.float32)], 1),
        "cells_on_edges": (rng.integers(0, 40, (30000, 3)) * 0.125)
        .astype(np.float32),
    }


@pytest.mark.parametrize("name", list(grid_clouds().keys()))
@pytest.mark.parametrize("h", [0.01, 0.125, 0.3, 50.0])
def test_grid_clouds(name, h):
    xyz = grid_clouds()[name]
    ref = oracle.grid_subsample(xyz, h)
    got = ezsp.grid_subsample(dev(xyz), h).cpu().numpy()
    assert np.array_equal(got, ref), (name, h, got.size, ref.size)


@pytest.mark.parametrize("name,h", [("room-1m", 0.03), ("driving-3m", 0.10)])
def test_grid_scene_full(name, h):
    xyz = scenes.load(name).xyz
    ref = oracle.grid_subsample(xyz, h)
    got = ezsp.grid_subsample(dev(xyz), h).cpu().numpy()
    assert 0 < ref.size < xyz.shape[0]
    assert np.array_equal(got, ref)


def test_grid_errors():
    with pytest.raises(ezsp.EzspError) as e:
        ezsp.grid_subsample(dev(np.array([[0, 0, 0], [3000, 0, 0]],
                                         np.float32)), 1e-3)
    assert e.value.code == ezsp.ERR_RANGE
    bad = np.zeros((100, 3), np.float32)
    bad[17, 1] = np.nan
    with pytest.raises(ezsp.EzspError) as e:
        ezsp.grid_subsample(dev(bad), 0.1)
    assert e.value.code == ezsp.ERR_NONFINITE


# --------------------------------------------------------------------------
# affinity and contrastive loss
# --------------------------------------------------------------------------

def loss_case(n, d, k, n_cls, seed, word_range=1 << 32, messy=False):
    rng = np.random.default_rng(seed)
    xyz = rng.random((n, 3), dtype=np.float32)
    nbr, _ = oracle.knn(xyz, k, "brute" if n <= 3000 else "kdtree")
    if messy:  # empty slots, self slots and repeats inside a row
        nbr = nbr.copy()
        nbr[rng.random(nbr.shape) < 0.05] = -1
        rows = rng.integers(0, n, n // 20)
        nbr[rows, -1] = rows
        if k >= 2:
            rows = rng.integers(0, n, n // 20)
            nbr[rows, -2] = nbr[rows, 0]
    cls = (xyz[:, 0] * n_cls).astype(np.int32)  # spatially coherent classes
    emb = (rng.standard_normal((n_cls, d))[cls] +
           0.3 * rng.standard_normal((n, d))).astype(np.float32)
    word = rng.integers(0, word_range, (n, k), dtype=np.uint64).astype(np.uint32)
    return emb, nbr, cls, word


def check_loss(emb, nbr, cls, word, tau, rho):
    ref, raff, rgrad, rsmp = oracle.edge_loss(emb, nbr, cls, word, tau, rho)
    st, aff, grad, smp = ezsp.edge_loss(dev(emb), dev(nbr), dev(cls),
                                        dev(word.view(np.int32)), tau, rho)
    for key in ("n_edges", "n_intra", "n_inter", "n_intra_kept"):
        assert st[key] == ref[key], key
    assert np.array_equal(smp.cpu().numpy(), rsmp)
    np.testing.assert_allclose(aff.cpu().numpy(), raff, rtol=0, atol=AFF_ATOL)
    assert st["loss"] == pytest.approx(ref["loss"], rel=LOSS_RTOL, abs=1e-12)
    g = grad.cpu().numpy().astype(np.float64)
    scale = max(np.abs(rgrad).max(), 1e-30)
    np.testing.assert_allclose(g, rgrad, rtol=GRAD_RTOL,
                               atol=GRAD_ATOL_REL * scale)
    return ref


@pytest.mark.parametrize("d", [1, 5, 8, 32])
@pytest.mark.parametrize("rho", [0.0, 0.1, 0.3, 1.0])
def test_loss_random(d, rho):
    emb, nbr, cls, word = loss_case(2500, d, 8, 6, seed=d)
    ref = check_loss(emb, nbr, cls, word, 1.0, rho)
    assert ref["n_inter"] > 0 and ref["n_intra"] > 0


@pytest.mark.parametrize("k", [1, 3, 10, 16, 64])
def test_loss_messy_tables_and_ties(k):
    # words from a range of 16: the (word, slot) order decides most draws
    emb, nbr, cls, word = loss_case(3000, 12, k, 4, seed=100 + k,
                                    word_range=16, messy=True)
    check_loss(emb, nbr, cls, word, 0.5, 0.2)


def test_loss_degenerate():
    # one point, an empty row
    emb = np.zeros((1, 4), np.float32)
    r = check_loss(emb, -np.ones((1, 2), np.int32), np.zeros(1, np.int32),
                   np.zeros((1, 2), np.uint32), 1.0, 0.5)
    assert r["n_edges"] == 0 and r["loss"] == 0.0
    # one class, rho < 1: no inter pair, so every intra pair is dropped
    emb, nbr, cls, word = loss_case(500, 8, 6, 1, seed=9)
    r = check_loss(emb, nbr, cls, word, 1.0, 0.3)
    assert r["n_inter"] == 0 and r["n_intra_kept"] == 0
    # coincident embeddings on intra pairs
    emb = np.ones((400, 8), np.float32)
    _, nbr, cls, word = loss_case(400, 8, 5, 3, seed=10)
    check_loss(emb, nbr, np.zeros(400, np.int32), word, 2.0, 1.0)


def test_loss_bad_neighbour():
    emb, nbr, cls, word = loss_case(300, 8, 4, 3, seed=12)
    nbr = nbr.copy()
    nbr[5, 2] = 300
    with pytest.raises(ezsp.EzspError) as e:
        ezsp.edge_loss(dev(emb), dev(nbr), dev(cls), dev(word.view(np.int32)),
                       1.0, 0.3)
    assert e.value.code == ezsp.ERR_INVALID_ARG


def test_loss_paper_settings_full():
    # D = 32, k = 8, tau = 1, rho_intra = 0.3 on the 3M-point driving tile,
    # primitive ids as classes, the GPU kNN table (bit-exact elsewhere)
    sc = scenes.load("driving-3m-paper")
    nbr = ezsp.knn(dev(sc.xyz), 8)
    word = np.random.default_rng(2024).integers(
        0, 1 << 32, (sc.n, 8), dtype=np.uint64).astype(np.uint32)
    ref = check_loss(sc.emb, nbr.cpu().numpy(), sc.obj.astype(np.int32), word,
                     1.0, 0.3)
    assert ref["n_intra_kept"] < ref["n_intra"]


# --------------------------------------------------------------------------
# purity and oracle mIoU
# --------------------------------------------------------------------------

def check_purity(label, nc, cls, n_cls):
    ref, rmaj, riou = oracle.purity(label, nc, cls, n_cls)
    st, maj, iou = ezsp.purity(dev(label), nc, dev(cls), n_cls)
    assert np.array_equal(maj.cpu().numpy(), rmaj)
    assert np.array_equal(iou.cpu().numpy(), riou, equal_nan=True)
    assert st["miou"] == ref["miou"] and st["purity"] == ref["purity"]
    assert st["n_present"] == ref["n_present"]
    return ref


@pytest.mark.parametrize("n,nc,n_cls", [(1, 1, 1), (1000, 37, 5),
                                        (50000, 3000, 13), (20000, 50, 5000),
                                        (200000, 200000, 40)])
def test_purity_random(n, nc, n_cls):
    rng = np.random.default_rng(n + nc)
    label = rng.integers(0, nc, n).astype(np.int32)
    cls = ((label * 7 + (rng.random(n) < 0.4) * rng.integers(0, n_cls, n))
           % n_cls).astype(np.int32)
    check_purity(label, nc, cls, n_cls)


def test_purity_empty_components_and_ties():
    label = np.array([0, 0, 2, 2, 5, 5, 5, 5], np.int32)
    cls = np.array([1, 0, 3, 3, 2, 0, 2, 0], np.int32)
    ref = check_purity(label, 8, cls, 4)
    assert ref["n_present"] == 4


def test_purity_of_gpu_partition():
    # the partition of the room scene scored against its primitive ids
    for name in ("room-20k-paper", "driving-3m-paper"):
        sc = scenes.load(name)
        labels, n_comp, _ = ezsp.partition(dev(sc.xyz), dev(sc.emb), sc.k,
                                           sc.lambdas, min_size=sc.min_size)
        n_cls = int(sc.obj.max()) + 1
        for lvl in range(len(sc.lambdas)):
            lab = labels[lvl].cpu().numpy()
            r = check_purity(lab, int(n_comp[lvl]), sc.obj.astype(np.int32),
                             n_cls)
            assert 0.0 < r["miou"] <= 1.0


def test_purity_bad_label():
    label = np.zeros(100, np.int32)
    label[3] = 9
    with pytest.raises(ezsp.EzspError) as e:
        ezsp.purity(dev(label), 5, dev(np.zeros(100, np.int32)), 2)
    assert e.value.code == ezsp.ERR_INVALID_ARG
