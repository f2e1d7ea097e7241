"""GPU parity of prepare_graph's linking of isolated nodes
(EZSP_F_LINK_ISOLATED) against the oracle's linked ladder: labels of every
level and superpoint counts bit-exact, the energy (cut term on the input
graph) within 1e-9 relative.  Linking only acts when a whole connected
component of the kNN graph has become one node, so the inputs are clouds of
separated clusters, the paper's settings on the driving tile (whose kNN graph
has three components), and a connected cloud where nothing may change."""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_00385_amd import ezsp, scenes

pytestmark = pytest.mark.gpu

ENERGY_RTOL = 1e-9


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ezsp.load()
    yield


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def check_linked(xyz, emb, k, lambdas, min_size=None):
    labels, nc, en = ezsp.partition(dev(xyz), dev(emb), k, lambdas, min_size,
                                    energy=True, link=True)
    rl, rnc, ren, _ = oracle.partition(xyz, emb, k, lambdas, min_size,
                                       link=True)
    labels = labels.cpu().numpy()
    assert np.array_equal(nc, rnc), (nc, rnc)
    for l in range(len(lambdas)):
        assert np.array_equal(labels[l], rl[l]), l
    np.testing.assert_allclose(en, ren, rtol=ENERGY_RTOL, atol=0)
    return labels, nc


def clusters(n_clusters, d, seed, size_lo=2, size_hi=40, sigma=0.05):
    """Separated blobs (radius 0.3, centres 5 apart on a jittered grid) of
    random sizes; each blob's embedding is a constant N(0, I) vector plus
    N(0, sigma^2) noise."""
    rng = np.random.default_rng(seed)
    side = int(np.ceil(n_clusters ** (1 / 3)))
    xyz, emb = [], []
    for c in range(n_clusters):
        g = np.array([c % side, (c // side) % side, c // (side * side)])
        centre = 5.0 * g + rng.uniform(-1, 1, 3)
        m = int(rng.integers(size_lo, size_hi + 1))
        xyz.append(centre + rng.uniform(-0.3, 0.3, (m, 3)))
        emb.append(rng.standard_normal(d) + sigma * rng.standard_normal((m, d)))
    xyz = np.concatenate(xyz).astype(np.float32)
    emb = np.concatenate(emb).astype(np.float32)
    perm = rng.permutation(xyz.shape[0])
    return xyz[perm], emb[perm]


def test_link_two_clusters():
    a = np.array([[0, 0, 0], [0.1, 0, 0], [0, 0.1, 0]], np.float32)
    g = np.stack(np.meshgrid(np.arange(4), np.arange(3), [0],
                             indexing="ij"), -1).reshape(-1, 3)
    b = (np.array([10.0, 0, 0]) + 0.1 * g).astype(np.float32)
    xyz = np.concatenate([a, b])
    emb = np.concatenate([np.zeros((3, 1)),
                          np.full((12, 1), 10.0)]).astype(np.float32)
    _, nc = check_linked(xyz, emb, 2, [0.1, 0.1], [0, 5])
    assert nc.tolist() == [2, 1]


@pytest.mark.parametrize("seed", range(4))
@pytest.mark.parametrize("k", [2, 4, 8])
def test_link_cluster_clouds(seed, k):
    xyz, emb = clusters(60 + 20 * seed, 4, seed)
    check_linked(xyz, emb, k, [0.05, 0.5, 2.0], [3, 15, 40])


def test_link_many_isolated_at_once():
    # 300 tight blobs of k+1..k+3 points: every blob closes on itself, so
    # hundreds of nodes become isolated in the same round
    xyz, emb = clusters(300, 8, 7, size_lo=9, size_hi=11, sigma=0.01)
    check_linked(xyz, emb, 8, [0.5, 0.5, 5.0], [5, 30, 90])


def test_link_connected_cloud_unchanged():
    sc = scenes.random_cloud(3000, 6, seed=4, sigma=0.3)
    la, nca = check_linked(sc.xyz, sc.emb, 8, [0.01, 0.05, 0.05],
                           [5, 30, 90])
    lb, ncb, _ = ezsp.partition(dev(sc.xyz), dev(sc.emb), 8,
                                [0.01, 0.05, 0.05], [5, 30, 90])
    assert np.array_equal(la, lb.cpu().numpy()) and np.array_equal(nca, ncb)


def test_link_paper_settings_driving_full():
    # D = 32, k = 8, lambda 0.02, s_min [5, 30, 90] on the 3M-point tile
    sc = scenes.load("driving-3m-paper")
    check_linked(sc.xyz, sc.emb, sc.k, sc.lambdas, sc.min_size)


def test_link_large_k():
    # k = 64 nearest nodes per isolated node: the largest per-thread lists
    xyz, emb = clusters(120, 4, 21, size_lo=66, size_hi=80)
    check_linked(xyz, emb, 64, [0.05, 0.5], [3, 200])
