"""GPU parity on the streaming workload: ray-cast 64-beam LiDAR sweeps of the
street scene (64 rings x 20,000 azimuths, ring-major order), embedded on the
GPU by the random-weight MLP, then partitioned.

The oracle partitions the GPU's own embeddings (the MLP's fp32 accumulation
order is the matrix unit's, so its outputs are compared separately, within
their bound, in test_gpu_mlp.py); labels, superpoint counts and the full kNN
table must then be bit-identical.  The sweeps are spatially ordered inputs:
points along a ring are neighbours in index order."""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_00385_amd import ezsp, scenes

pytestmark = pytest.mark.gpu

LAMBDAS = [0.05, 0.2, 0.8]
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


def to_dev(a):
    a = np.ascontiguousarray(a)
    if a.dtype == np.uint16:
        a = a.view(np.int16)
    return torch.from_numpy(a).cuda()


_EMB = {}
_REF = {}


def sweep_and_embedding(index):
    """The sweep and its GPU MLP embedding (once per module)."""
    if index not in _EMB:
        xyz, feat, obj = scenes.sweep(0, index)
        w = [to_dev(a) for a in scenes.mlp_weights(0)]
        emb = ezsp.embed_mlp(to_dev(feat), *w)
        torch.cuda.synchronize()
        _EMB[index] = (xyz, emb)
    return _EMB[index]


def test_sweep_shape():
    """64 rings x 20,000 azimuths, misses dropped, ring-major order."""
    xyz, obj, ring, rng_m, sensor = scenes.lidar_sweep(0, 0)
    n = xyz.shape[0]
    assert 1_200_000 <= n <= 64 * 20_000
    assert (np.diff(ring) >= 0).all() and ring.min() == 0 and \
        ring.max() == 63
    assert rng_m.max() <= 120.0
    assert len(np.unique(obj)) > 50


@pytest.mark.parametrize("index", [0, 1])
def test_sweep_knn_full_table(index):
    """Every row of the kNN table of a whole sweep, k = 10."""
    xyz, _ = sweep_and_embedding(index)
    nbr, d2 = ezsp.knn(to_dev(xyz), 10, want_d2=True)
    ref, rd = oracle.knn(xyz, 10)
    assert np.array_equal(nbr.cpu().numpy(), ref)
    assert np.array_equal(d2.cpu().numpy(), rd)


@pytest.mark.parametrize("index", [0, 1])
def test_sweep_mlp_partition(index, tail_mode):
    """GPU MLP -> ezsp.Partitioner (the benchmark's launch configuration,
    the workspace reused) against the oracle's kNN, graph and ladder on the
    GPU's embeddings; then the energy."""
    xyz, emb = sweep_and_embedding(index)
    if index not in _REF:
        _REF[index] = oracle.partition(xyz, emb.cpu().numpy(), 10, LAMBDAS)
    rl, rnc, ren, _ = _REF[index]
    part = ezsp.Partitioner(xyz.shape[0], 16, 10, LAMBDAS,
                            device=torch.device("cuda:0"))
    x = to_dev(xyz)
    for _ in range(2):
        labels, nc, _ = part(x, emb)
        assert np.array_equal(nc, rnc), (nc, rnc)
        labels = labels.cpu().numpy()
        for l in range(len(LAMBDAS)):
            assert np.array_equal(labels[l], rl[l]), l
    _, _, en = ezsp.partition(x, emb, 10, LAMBDAS, energy=True)
    np.testing.assert_allclose(en, ren, rtol=ENERGY_RTOL, atol=0)
