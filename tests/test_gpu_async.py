"""The stream-asynchronous entry points (ezsp_knn, ezsp_component_stats,
ezsp_embed_mlp): work enqueued back to back on one stream with no host
synchronisation in between gives the same results as the oracle, and
errors the device detects surface through ezsp_sync_status."""
import numpy as np
import pytest
import torch

import oracle
from paper_2512_00385_amd import ezsp, scenes

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    ezsp.load()
    yield


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def test_knn_then_stats_without_sync():
    """kNN -> labels derived from its table by stream-ordered torch ops ->
    component statistics, one host synchronisation at the end."""
    sc = scenes.random_cloud(50_000, 12, seed=21)
    nc = 997
    x, e = dev(sc.xyz), dev(sc.emb)
    torch.cuda.synchronize()
    nbr, p1 = ezsp.knn(x, 10, sync=False)
    lab = (nbr[:, 3].to(torch.int64) * 7919 % nc).to(torch.int32)
    size, mean, cen, p2 = ezsp.component_stats(lab, nc, e, x, sync=False)
    p1.check()
    p2.check()
    ref_nbr, _ = oracle.knn(sc.xyz, 10)
    assert np.array_equal(nbr.cpu().numpy(), ref_nbr)
    ref_lab = (ref_nbr[:, 3].astype(np.int64) * 7919 % nc).astype(np.int32)
    rs, rm, rc = oracle.component_stats(ref_lab, nc, sc.emb, sc.xyz)
    assert np.array_equal(size.cpu().numpy(), rs)
    assert np.array_equal(mean.cpu().numpy(), rm)
    assert np.array_equal(cen.cpu().numpy(), rc)


def test_mlp_then_partition_without_sync():
    """The embedding MLP's output feeds the partition on the same stream."""
    xyz, feat, _ = scenes.sweep(0, 0)
    xyz, feat = xyz[:200_000], feat[:200_000]
    w = [dev(a.view(np.int16) if a.dtype == np.uint16 else a)
         for a in scenes.mlp_weights(0)]
    x = dev(xyz)
    emb = ezsp.embed_mlp(dev(feat.view(np.int16)), *w)
    labels, nc, _ = ezsp.partition(x, emb, 10, [0.05, 0.2])
    rl, rnc, _, _ = oracle.partition(xyz, emb.cpu().numpy(), 10, [0.05, 0.2])
    assert np.array_equal(nc, rnc)
    assert np.array_equal(labels.cpu().numpy(), rl)


def test_async_errors_surface_at_status():
    xyz = np.random.default_rng(0).random((5000, 3), dtype=np.float32)
    xyz[4321, 2] = np.inf
    nbr, pending = ezsp.knn(dev(xyz), 8, sync=False)  # returns: enqueued
    with pytest.raises(ezsp.EzspError) as e:
        pending.check()
    assert e.value.code == ezsp.ERR_NONFINITE
    lab = np.zeros(5000, np.int32)
    lab[17] = 40
    emb = np.ones((5000, 3), np.float32)
    out = ezsp.component_stats(dev(lab), 40, dev(emb), sync=False)
    with pytest.raises(ezsp.EzspError) as e:
        out[-1].check()
    assert e.value.code == ezsp.ERR_INVALID_ARG
    # a later call on a fresh workspace is unaffected
    good = np.random.default_rng(1).random((300, 3), dtype=np.float32)
    ref, _ = oracle.knn(good, 8)
    assert np.array_equal(ezsp.knn(dev(good), 8).cpu().numpy(), ref)
