"""GPU parity on spatially ordered inputs whose merge forests are deep.

When gains tie, every node keeps the neighbour with the smaller smallest
point index (the tie rule of Step 2).  Points stored in scan order along a
line then each pick their predecessor, so one round's merge forest is a
chain as long as the line (App. Alg. A-1 still gives one component).  The
shuffled scenes never build such forests; these inputs do, and the GPU's
pointer jumping must still reach every root and give the oracle's labels.
"""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_00385_amd import ezsp

pytestmark = pytest.mark.gpu

ENERGY_RTOL = 1e-9


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ezsp.load()
    yield


@pytest.fixture(params=["tail", "no-tail"])
def tail_mode(request, monkeypatch):
    if request.param == "no-tail":
        monkeypatch.setenv("EZSP_TAIL_NODES", "0")
    else:
        monkeypatch.delenv("EZSP_TAIL_NODES", raising=False)
    return request.param


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def line(n, spacing=0.5):
    """n points on the x axis in index order, exactly representable."""
    x = np.arange(n, dtype=np.float32) * np.float32(spacing)
    z = np.zeros(n, np.float32)
    return np.stack([x, z, z], 1)


def check(xyz, emb, k, lambdas, min_size=None):
    labels, nc, en = ezsp.partition(dev(xyz), dev(emb), k, lambdas, min_size,
                                    energy=True)
    rl, rnc, ren, _ = oracle.partition(xyz, emb, k, lambdas, min_size)
    assert np.array_equal(nc, rnc), (nc, rnc)
    labels = labels.cpu().numpy()
    for l in range(len(lambdas)):
        assert np.array_equal(labels[l], rl[l]), l
    np.testing.assert_allclose(en, ren, rtol=ENERGY_RTOL, atol=0)
    return labels, nc


def test_line_one_chain_200k(tail_mode):
    """200,000 collinear points in index order, one constant embedding,
    k = 2: every gain is lambda, each point picks its predecessor, and the
    first round's forest is a single chain of 200,000 nodes."""
    n = 200_000
    xyz = line(n)
    emb = np.full((n, 4), 0.25, np.float32)
    labels, nc = check(xyz, emb, 2, [0.1])
    assert nc.tolist() == [1] and not labels.any()


def test_line_segments(tail_mode):
    """A line of 60 segments of 3000 points each with its own embedding:
    chains of 3000 nodes in every segment in the first round, then merges
    between segments at the higher lambdas."""
    n, seg = 180_000, 3000
    rng = np.random.default_rng(5)
    xyz = line(n)
    vals = rng.standard_normal((n // seg, 3)).astype(np.float32) * 0.3
    emb = np.repeat(vals, seg, 0)
    check(xyz, emb, 2, [0.05, 200.0, 2000.0])


def test_scan_grid(tail_mode):
    """A 2-D grid stored row by row (the order of a scanning sensor), tied
    embeddings per block of rows, k = 4 and 8."""
    nx, ny = 1500, 60
    gx, gy = np.meshgrid(np.arange(nx, dtype=np.float32),
                         np.arange(ny, dtype=np.float32) * np.float32(1.5),
                         indexing="xy")
    xyz = np.stack([gx.ravel(), gy.ravel(), np.zeros(nx * ny, np.float32)], 1)
    emb = np.repeat(np.arange(ny // 10, dtype=np.float32), 10 * nx)[:, None]
    emb = np.concatenate([emb, np.ones_like(emb)], 1) * np.float32(0.5)
    for k in (4, 8):
        check(xyz, emb, k, [0.1, 1.0])


def test_from_knn_line_table(tail_mode):
    """The same chain through a caller-supplied table (both neighbours of
    each point, in index order), 100,000 nodes."""
    n = 100_000
    i = np.arange(n, dtype=np.int32)
    nbr = np.stack([i - 1, i + 1], 1).astype(np.int32)
    nbr[0, 0] = -1
    nbr[-1, 1] = -1
    emb = np.zeros((n, 2), np.float32)
    lo, hi, w = oracle.graph(nbr)
    rl, rnc, ren, _ = oracle.partition_graph(emb, lo, hi, w, [0.3])
    labels, nc, en = ezsp.partition_from_knn(dev(nbr), dev(emb), [0.3],
                                             energy=True)
    assert np.array_equal(nc, rnc) and rnc.tolist() == [1]
    assert np.array_equal(labels.cpu().numpy(), rl)
    np.testing.assert_allclose(en, ren, rtol=ENERGY_RTOL)
