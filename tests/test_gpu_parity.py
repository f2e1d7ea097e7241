"""GPU parity: the HIP path (called through the C ABI) against the CPU oracle
on the same seeded inputs.  kNN indices and distances, per-level labels,
superpoint counts and statistics must be bit-identical; the energy, a sum
whose order differs between the two sides, must agree to 1e-9 relative
(the stated bar is 1e-5)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_00385_amd import ezsp, scenes
from tests.alg_steps import canonical

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


def clouds():
    rng = np.random.default_rng(1)
    return {
        "uniform": rng.random((700, 3), dtype=np.float32),
        "lattice": np.stack(np.meshgrid(np.arange(8), np.arange(8),
                                        np.arange(6), indexing="ij"),
                            -1).reshape(-1, 3).astype(np.float32),
        "duplicates": np.repeat(rng.random((60, 3), dtype=np.float32), 7, 0),
        "clusters": scenes.random_cloud(900, 4, seed=3).xyz,
        "planar": np.concatenate([rng.random((400, 2), dtype=np.float32),
                                  np.zeros((400, 1), np.float32)], 1),
        "line": np.stack([np.arange(300, dtype=np.float32) * 0.5,
                          np.zeros(300, np.float32),
                          np.zeros(300, np.float32)], 1),
    }


# --------------------------------------------------------------------------
# kNN
# --------------------------------------------------------------------------

@pytest.mark.parametrize("name", ["uniform", "clusters", "line"])
@pytest.mark.parametrize("k", [1, 10, 64])
def test_knn_walk_stats(name, k):
    """The kNN with its walk statistics: the same table as ezsp_knn and the
    oracle; every 64-point group scans at least its own buckets and at most
    every bucket."""
    xyz = clouds()[name]
    n = xyz.shape[0]
    nbr, scans, nodes = ezsp.knn_walk_stats(dev(xyz), k)
    ref, _ = oracle.knn(xyz, k, "brute")
    assert np.array_equal(nbr.cpu().numpy(), ref)
    assert np.array_equal(nbr.cpu().numpy(), ezsp.knn(dev(xyz), k).cpu().numpy())
    g, nb = (n + 63) // 64, (n + 15) // 16
    own = np.minimum(4, nb - 4 * np.arange(g))
    scans, nodes = scans.cpu().numpy(), nodes.cpu().numpy()
    assert scans.shape == (g,) and nodes.shape == (g,)
    assert (scans >= own).all() and (scans <= nb).all()
    assert (nodes >= 0).all()


@pytest.mark.parametrize("n,want", [(1, [1]), (16, [1]), (17, [2]),
                                    (32, [2]), (49, [4]), (64, [4])])
def test_knn_walk_stats_small(n, want):
    """Up to four buckets, one group: it scans its own buckets, and the walk
    then finds every bucket already taken; no inner node is entered."""
    xyz = np.random.default_rng(n).random((n, 3), dtype=np.float32)
    _, scans, nodes = ezsp.knn_walk_stats(dev(xyz), min(4, max(n - 1, 1)))
    assert scans.cpu().numpy().tolist() == want
    assert nodes.cpu().numpy().tolist() == [0] * len(want)


@pytest.mark.parametrize("name", list(clouds().keys()))
@pytest.mark.parametrize("k", [1, 8, 10, 33, 64])
def test_knn_clouds(name, k):
    xyz = clouds()[name]
    ref, rd = oracle.knn(xyz, k, "brute")
    nbr, d2 = ezsp.knn(dev(xyz), k, want_d2=True)
    assert np.array_equal(nbr.cpu().numpy(), ref)
    assert np.array_equal(d2.cpu().numpy(), rd)


@pytest.mark.parametrize("n", [1, 2, 5, 11, 33, 65, 97])
def test_knn_tiny_and_ragged(n):
    xyz = np.random.default_rng(n).random((n, 3), dtype=np.float32)
    for k in (1, 10, 64):
        ref, rd = oracle.knn(xyz, k, "brute")
        nbr, d2 = ezsp.knn(dev(xyz), k, want_d2=True)
        assert np.array_equal(nbr.cpu().numpy(), ref), (n, k)
        assert np.array_equal(d2.cpu().numpy(), rd), (n, k)


@pytest.mark.parametrize("n", [7, 20, 37])
def test_knn_overflowing_distances(n):
    """Coordinates near 1e20: most squared distances overflow to +inf, and
    ties at +inf go to the smaller index, ahead of the padding that fills
    the last bucket (n not a multiple of 16; with k >= n every real point
    is listed and the rest is -1)."""
    rng = np.random.default_rng(n)
    xyz = ((rng.random((n, 3)) - 0.5) * 2e20).astype(np.float32)
    xyz[: n // 3] *= np.float32(1e-19)  # a few finite distances as well
    for k in (3, 10, 40):
        ref, rd = oracle.knn(xyz, k, "brute")
        nbr, d2 = ezsp.knn(dev(xyz), k, want_d2=True)
        assert np.isinf(rd).any()
        assert np.array_equal(nbr.cpu().numpy(), ref), (n, k)
        assert np.array_equal(d2.cpu().numpy(), rd), (n, k)


def test_knn_room_full():
    sc = scenes.load("room-20k")
    ref, rd = oracle.knn(sc.xyz, sc.k)
    nbr, d2 = ezsp.knn(dev(sc.xyz), sc.k, want_d2=True)
    assert np.array_equal(nbr.cpu().numpy(), ref)
    assert np.array_equal(d2.cpu().numpy(), rd)


def test_knn_driving_tile_sampled():
    """Full 3M-point driving tile, the benchmark's launch configuration;
    200 sampled rows are recomputed by the oracle's brute force."""
    sc = scenes.load("driving-3m")
    nbr, d2 = ezsp.knn(dev(sc.xyz), sc.k, want_d2=True)
    nbr, d2 = nbr.cpu().numpy(), d2.cpu().numpy()
    rng = np.random.default_rng(0)
    # sample near the sensor (densest), far away, and uniformly
    r = np.hypot(sc.xyz[:, 0], sc.xyz[:, 1])
    idx = np.concatenate([np.argsort(r)[:50], np.argsort(r)[-50:],
                          rng.integers(0, sc.n, 100)])
    for p in idx:
        one, d1 = oracle.knn_one(sc.xyz, sc.k, int(p))
        assert np.array_equal(one, nbr[p]), p
        assert np.array_equal(d1, d2[p]), p
    # properties at any size: sorted rows, no self, valid ids
    assert (nbr >= 0).all() and (nbr < sc.n).all()
    assert (nbr != np.arange(sc.n)[:, None]).all()
    assert (np.diff(d2, axis=1) >= 0).all()


def test_knn_nonfinite():
    xyz = np.random.default_rng(0).random((100, 3), dtype=np.float32)
    xyz[17, 1] = np.nan
    with pytest.raises(ezsp.EzspError) as e:
        ezsp.knn(dev(xyz), 5)
    assert e.value.code == ezsp.ERR_NONFINITE


# --------------------------------------------------------------------------
# partition
# --------------------------------------------------------------------------

def check_against_oracle(xyz, emb, k, lambdas, min_size=None, max_rounds=0):
    labels, nc, en = ezsp.partition(dev(xyz), dev(emb), k, lambdas, min_size,
                                    max_rounds, energy=True)
    rl, rnc, ren, _ = oracle.partition(xyz, emb, k, lambdas, min_size,
                                       max_rounds)
    labels = labels.cpu().numpy()
    assert np.array_equal(nc, rnc), (nc, rnc)
    for l in range(len(lambdas)):
        assert np.array_equal(labels[l], rl[l]), l
    np.testing.assert_allclose(en, ren, rtol=ENERGY_RTOL, atol=0)
    return labels, nc


@pytest.fixture(params=["tail", "no-tail"])
def tail_mode(request, monkeypatch):
    """Small graphs finish in the single-block tail kernel; "no-tail" keeps
    every round on the multi-kernel path (EZSP_TAIL_NODES=0)."""
    if request.param == "no-tail":
        monkeypatch.setenv("EZSP_TAIL_NODES", "0")
    else:
        monkeypatch.delenv("EZSP_TAIL_NODES", raising=False)
    return request.param


def test_partition_room_full(tail_mode):
    sc = scenes.load("room-20k")
    check_against_oracle(sc.xyz, sc.emb, sc.k, sc.lambdas)


def test_partition_room_ladder(tail_mode):
    sc = scenes.load("room-20k")
    check_against_oracle(sc.xyz, sc.emb, sc.k, [0.02, 0.05, 0.2, 0.8, 3.2])


_FULL = {}


def _oracle_full(name):
    """The oracle's own kNN, graph and ladder on a whole workload (computed
    once per module)."""
    if name not in _FULL:
        sc = scenes.load(name)
        rl, rnc, ren, _ = oracle.partition(sc.xyz, sc.emb, sc.k, sc.lambdas,
                                           sc.min_size)
        _FULL[name] = (sc, rl, rnc, ren)
    return _FULL[name]


@pytest.mark.parametrize("name", ["room-20k-paper", "room-1m", "driving-3m",
                                  "room-1m-paper", "driving-3m-paper"])
def test_partition_full_size(name, tail_mode):
    """Whole workloads in the benchmark's launch configuration (a reused
    Partitioner workspace, no energy pass): the 1M-point room and the
    3M-point driving tile with the benchmark ladder and with the paper's own
    settings (D = 32, k = 8, lambda = 0.02, s_min ladder [5, 30, 90]), every
    label of every level against the oracle's own full run; then the energy
    through ezsp.partition."""
    sc, rl, rnc, ren = _oracle_full(name)
    part = ezsp.Partitioner(sc.n, sc.d, sc.k, sc.lambdas, sc.min_size,
                            device=torch.device("cuda:0"))
    xyz, emb = dev(sc.xyz), dev(sc.emb)
    for _ in range(2):  # the second call reuses the workspace
        labels, nc, _ = part(xyz, emb)
        assert np.array_equal(nc, rnc), (nc, rnc)
        labels = labels.cpu().numpy()
        for l in range(len(sc.lambdas)):
            assert np.array_equal(labels[l], rl[l]), l
    _, _, en = ezsp.partition(xyz, emb, sc.k, sc.lambdas, sc.min_size,
                              energy=True)
    np.testing.assert_allclose(en, ren, rtol=ENERGY_RTOL, atol=0)


@pytest.mark.parametrize("seed", range(6))
@pytest.mark.parametrize("lambdas", [[0.1], [0.05, 0.2, 0.8], [0.8, 0.2],
                                     [0.01, 0.03, 0.1, 0.3, 1.0, 3.0]])
def test_partition_random_clouds(seed, lambdas, tail_mode):
    sc = scenes.random_cloud(3000 + 137 * seed, 1 + 5 * seed, seed=seed,
                             sigma=0.05 * (1 + seed % 3))
    check_against_oracle(sc.xyz, sc.emb, 10, lambdas)


@pytest.mark.parametrize("case", ["room", "ladder", "clouds", "smin",
                                  "ties"])
def test_partition_tail_rebuild_every_round(case, monkeypatch):
    """The tail kernel with every round taking the path of a full table
    (every live row rebuilt into the other buffer, EZSP_TAIL_REBUILD=1)."""
    monkeypatch.delenv("EZSP_TAIL_NODES", raising=False)
    monkeypatch.setenv("EZSP_TAIL_REBUILD", "1")
    if case == "room":
        sc = scenes.load("room-20k")
        check_against_oracle(sc.xyz, sc.emb, sc.k, sc.lambdas)
    elif case == "ladder":
        sc = scenes.load("room-20k")
        check_against_oracle(sc.xyz, sc.emb, sc.k, [0.02, 0.05, 0.2, 0.8, 3.2])
    elif case == "clouds":
        for seed in range(3):
            sc = scenes.random_cloud(3000 + 137 * seed, 1 + 5 * seed,
                                     seed=seed, sigma=0.05 * (1 + seed))
            check_against_oracle(sc.xyz, sc.emb, 10, [0.05, 0.2, 0.8])
    elif case == "smin":
        sc = scenes.random_cloud(3000, 6, seed=4, sigma=0.3)
        check_against_oracle(sc.xyz, sc.emb, 8, [0.01, 0.05, 0.05],
                             min_size=[5, 30, 90])
    else:
        sc = scenes.random_cloud(1500, 3, seed=5)
        check_against_oracle(sc.xyz, np.ones_like(sc.emb), 10, [0.5, 2.0])


@pytest.mark.parametrize("k", [1, 4, 16])
def test_partition_k(k):
    sc = scenes.random_cloud(2500, 8, seed=11)
    check_against_oracle(sc.xyz, sc.emb, k, [0.05, 0.4])


def test_partition_min_size(tail_mode):
    sc = scenes.random_cloud(3000, 6, seed=4, sigma=0.3)
    check_against_oracle(sc.xyz, sc.emb, 8, [0.01, 0.05, 0.05],
                         min_size=[5, 30, 90])


def test_partition_lambda_zero_and_huge():
    sc = scenes.random_cloud(2000, 4, seed=7)
    labels, nc = check_against_oracle(sc.xyz, sc.emb, 10, [0.0, 1e30])
    assert nc[0] == sc.n and (labels[0] == np.arange(sc.n)).all()


def test_partition_constant_embeddings_ties(tail_mode):
    """Every gain equal: conflict removal is decided by the tie rule alone."""
    sc = scenes.random_cloud(2000, 3, seed=8)
    emb = np.ones_like(sc.emb) * 0.25
    check_against_oracle(sc.xyz, emb, 10, [0.1, 0.3])
    lat = clouds()["lattice"]
    check_against_oracle(lat, np.zeros((lat.shape[0], 2), np.float32), 6,
                         [0.5])


def test_partition_duplicate_points():
    xyz = clouds()["duplicates"]
    emb = np.random.default_rng(3).standard_normal(
        (xyz.shape[0], 4)).astype(np.float32) * 0.1
    check_against_oracle(xyz, emb, 10, [0.05, 0.5])


@pytest.mark.parametrize("d", [1, 2, 64])
def test_partition_dims(d, tail_mode):
    sc = scenes.random_cloud(1500, d, seed=20 + d)
    check_against_oracle(sc.xyz, sc.emb, 10, [0.02 * d, 0.2 * d])


@pytest.mark.parametrize("n", [1, 2, 3, 11, 64, 65])
def test_partition_tiny(n):
    rng = np.random.default_rng(n)
    xyz = rng.random((n, 3), dtype=np.float32)
    emb = rng.standard_normal((n, 3)).astype(np.float32)
    check_against_oracle(xyz, emb, 10, [0.5, 2.0, 8.0])


def test_partition_max_rounds(tail_mode):
    sc = scenes.random_cloud(2000, 4, seed=9)
    with pytest.raises(oracle.OracleError):
        oracle.partition(sc.xyz, sc.emb, 10, [0.2], max_rounds=1)
    with pytest.raises(ezsp.EzspError) as e:
        ezsp.partition(dev(sc.xyz), dev(sc.emb), 10, [0.2], max_rounds=1)
    assert e.value.code == ezsp.ERR_NOT_CONVERGED
    # a cap that the oracle accepts is accepted too
    rl, rnc, _, log = oracle.partition(sc.xyz, sc.emb, 10, [0.2],
                                       want_log=True)
    cap = len(log)
    labels, nc, _ = ezsp.partition(dev(sc.xyz), dev(sc.emb), 10, [0.2],
                                   max_rounds=cap)
    assert np.array_equal(labels.cpu().numpy(), rl)


def test_partition_errors():
    sc = scenes.random_cloud(500, 4, seed=1)
    bad = sc.emb.copy()
    bad[3, 2] = np.inf
    with pytest.raises(ezsp.EzspError) as e:
        ezsp.partition(dev(sc.xyz), dev(bad), 10, [0.1])
    assert e.value.code == ezsp.ERR_NONFINITE
    huge = sc.emb * np.float32(2.0 ** 40)
    with pytest.raises(ezsp.EzspError) as e:
        ezsp.partition(dev(sc.xyz), dev(huge), 10, [0.1])
    assert e.value.code == ezsp.ERR_RANGE
    xbad = sc.xyz.copy()
    xbad[0, 0] = np.nan
    with pytest.raises(ezsp.EzspError) as e:
        ezsp.partition(dev(xbad), dev(sc.emb), 10, [0.1])
    assert e.value.code == ezsp.ERR_NONFINITE


def test_partition_deterministic():
    sc = scenes.random_cloud(20000, 8, seed=12)
    a = ezsp.partition(dev(sc.xyz), dev(sc.emb), 10, [0.05, 0.2])
    b = ezsp.partition(dev(sc.xyz), dev(sc.emb), 10, [0.05, 0.2])
    assert torch.equal(a[0], b[0]) and np.array_equal(a[1], b[1])


# --------------------------------------------------------------------------
# partition on a given neighbour table
# --------------------------------------------------------------------------

def test_from_knn_matches_graph_oracle(tail_mode):
    sc = scenes.random_cloud(3000, 5, seed=13)
    nbr, _ = oracle.knn(sc.xyz, 8)
    lo, hi, w = oracle.graph(nbr)
    rl, rnc, ren, _ = oracle.partition_graph(sc.emb, lo, hi, w,
                                             [0.05, 0.3])
    labels, nc, en = ezsp.partition_from_knn(dev(nbr), dev(sc.emb),
                                             [0.05, 0.3], energy=True)
    assert np.array_equal(labels.cpu().numpy(), rl)
    assert np.array_equal(nc, rnc)
    np.testing.assert_allclose(en, ren, rtol=ENERGY_RTOL)


def test_from_knn_irregular_table():
    """-1 padding, self entries and repeats in a row are ignored."""
    rng = np.random.default_rng(14)
    n, k = 800, 9
    nbr = rng.integers(-1, n, (n, k)).astype(np.int32)
    nbr[::7, 3] = np.arange(0, n, 7)          # self entries
    nbr[::5, 4] = nbr[::5, 2]                 # repeats
    emb = rng.standard_normal((n, 3)).astype(np.float32)
    lo, hi, w = oracle.graph(nbr)
    rl, rnc, ren, _ = oracle.partition_graph(emb, lo, hi, w, [0.8, 3.0])
    labels, nc, en = ezsp.partition_from_knn(dev(nbr), dev(emb), [0.8, 3.0],
                                             energy=True)
    assert np.array_equal(labels.cpu().numpy(), rl)
    assert np.array_equal(nc, rnc)
    np.testing.assert_allclose(en, ren, rtol=ENERGY_RTOL)
    bad = nbr.copy()
    bad[5, 5] = n
    with pytest.raises(ezsp.EzspError) as e:
        ezsp.partition_from_knn(dev(bad), dev(emb), [0.8])
    assert e.value.code == ezsp.ERR_INVALID_ARG


# --------------------------------------------------------------------------
# component statistics
# --------------------------------------------------------------------------

def test_component_stats():
    rng = np.random.default_rng(0)
    n, nc = 50_000, 3001
    lab = rng.integers(0, nc, n).astype(np.int32)
    lab[lab == 17] = 18  # one empty superpoint
    emb = rng.standard_normal((n, 12)).astype(np.float32)
    xyz = (rng.random((n, 3)) * 100).astype(np.float32)
    size, mean, cen = ezsp.component_stats(dev(lab), nc, dev(emb), dev(xyz))
    rs, rm, rc = oracle.component_stats(lab, nc, emb, xyz)
    assert np.array_equal(size.cpu().numpy(), rs)
    assert np.array_equal(mean.cpu().numpy(), rm)
    assert np.array_equal(cen.cpu().numpy(), rc)
    bad = lab.copy()
    bad[10] = nc
    with pytest.raises(ezsp.EzspError) as e:
        ezsp.component_stats(dev(bad), nc, dev(emb))
    assert e.value.code == ezsp.ERR_INVALID_ARG


def test_component_stats_of_partition():
    sc = scenes.load("room-20k")
    labels, nc, _ = ezsp.partition(dev(sc.xyz), dev(sc.emb), 10, [0.1])
    size, mean, cen = ezsp.component_stats(labels[0], int(nc[0]),
                                           dev(sc.emb), dev(sc.xyz))
    rs, rm, rc = oracle.component_stats(labels[0].cpu().numpy(), int(nc[0]),
                                        sc.emb, sc.xyz)
    assert np.array_equal(size.cpu().numpy(), rs)
    assert np.array_equal(mean.cpu().numpy(), rm)
    assert np.array_equal(cen.cpu().numpy(), rc)
