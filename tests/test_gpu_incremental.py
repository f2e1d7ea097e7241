"""GPU parity of the incremental rounds (opt-in, EZSP_INCREMENTAL): in a
level whose rounds merge few nodes, node ids stay fixed and a round touches
only its worklist, the merged components and the rows that listed them; ids
are renumbered at the level end, before the tail, and when the table fills.
Every case runs with incremental rounds off (the default), on with their
default switch (graphs of 32768 nodes and more), forced on small graphs
(EZSP_INCREMENTAL=64), with renumbering forced after every second
incremental round (EZSP_INCR_COMPACT_EVERY=2), and forced without the tail
kernel; labels, counts and energy against the oracle."""
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


MODES = {
    "default": {},
    "on": {"EZSP_INCREMENTAL": "1"},
    "forced": {"EZSP_INCREMENTAL": "64"},
    "forced-renumber": {"EZSP_INCREMENTAL": "64",
                        "EZSP_INCR_COMPACT_EVERY": "2"},
    "forced-no-tail": {"EZSP_INCREMENTAL": "64", "EZSP_TAIL_NODES": "0"},
}


@pytest.fixture(params=list(MODES))
def mode(request, monkeypatch):
    for k in ("EZSP_INCREMENTAL", "EZSP_INCR_COMPACT_EVERY",
              "EZSP_TAIL_NODES"):
        monkeypatch.delenv(k, raising=False)
    for k, v in MODES[request.param].items():
        monkeypatch.setenv(k, v)
    return request.param


def dev(a):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


_REF = {}


def check(key, xyz, emb, k, lambdas, min_size=None):
    if key not in _REF:
        _REF[key] = oracle.partition(xyz, emb, k, lambdas, min_size)
    rl, rnc, ren, _ = _REF[key]
    labels, nc, en = ezsp.partition(dev(xyz), dev(emb), k, lambdas, min_size,
                                    energy=True)
    assert np.array_equal(nc, rnc), (nc, rnc)
    labels = labels.cpu().numpy()
    for l in range(len(lambdas)):
        assert np.array_equal(labels[l], rl[l]), l
    np.testing.assert_allclose(en, ren, rtol=ENERGY_RTOL, atol=0)


CLOUDS = [(60000, 4, 0.3, 0.05), (60000, 8, 0.2, 0.05), (100000, 4, 0.5, 0.1),
          (50000, 2, 0.3, 0.02)]


@pytest.mark.parametrize("case", range(len(CLOUDS)))
def test_slow_levels(case, mode):
    """Noisy clouds whose first levels keep 84-99 % of their nodes per
    round for a dozen rounds."""
    n, d, sigma, lam = CLOUDS[case]
    sc = scenes.random_cloud(n, d, seed=3, sigma=sigma)
    check(("cloud", case), sc.xyz, sc.emb, 10, [lam, 4 * lam, 16 * lam])


def test_min_size_ladder(mode):
    """s_min ladder: small components merge along their best edge whatever
    its gain."""
    sc = scenes.random_cloud(80000, 6, seed=9, sigma=0.4)
    check("smin", sc.xyz, sc.emb, 8, [0.01, 0.01, 0.01], [5, 30, 90])


def test_room_paper(mode):
    sc = scenes.load("room-20k-paper")
    check("room-20k-paper", sc.xyz, sc.emb, sc.k, sc.lambdas, sc.min_size)


def test_line_chains(mode):
    """Scan-ordered segments with tied gains inside each (chains)."""
    n, seg = 120_000, 500
    rng = np.random.default_rng(11)
    x = np.arange(n, dtype=np.float32) * np.float32(0.5)
    z = np.zeros(n, np.float32)
    xyz = np.stack([x, z, z], 1)
    vals = rng.standard_normal((n // seg, 3)).astype(np.float32)
    emb = np.repeat(vals, seg, 0) + \
        (rng.standard_normal((n, 3)) * 0.3).astype(np.float32)
    check("line", xyz, emb, 2, [0.05, 0.5, 5.0])
