"""CPU-side checks of the C ABI: the library loads without a GPU, exports
every function that include/ezsp.h declares, and rejects bad arguments on
the host before anything reaches the device."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2512_00385_amd import ezsp

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "ezsp.h")

pytestmark = pytest.mark.skipif(not os.path.exists(ezsp.LIB_PATH),
                                reason="libezsp.so not built")

FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: validation fails first


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(ezsp_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_symbol():
    lib = ezsp.load()
    names = declared_functions()
    assert len(names) >= 9
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(ezsp.ENTRY_POINTS)


def test_knn_noalloc_rejects_sizes_beyond_its_scratch():
    lib = ezsp.load()
    assert lib.ezsp_knn_noalloc(FAKE, 3_000_000, 10, FAKE, None, None) == \
        ezsp.ERR_INVALID_ARG
    assert "static scratch" in ezsp.last_error()
    assert lib.ezsp_knn_noalloc(FAKE, 0, 10, FAKE, None, None) == \
        ezsp.ERR_INVALID_ARG
    assert lib.ezsp_knn_noalloc(None, 100, 10, FAKE, None, None) == \
        ezsp.ERR_INVALID_ARG


def test_sync_status_rejects_bad_workspace():
    lib = ezsp.load()
    assert lib.ezsp_sync_status(None, 1 << 20, None) == ezsp.ERR_INVALID_ARG
    assert lib.ezsp_sync_status(FAKE, 16, None) == ezsp.ERR_INVALID_ARG


def test_status_strings():
    for code in range(0, -7, -1):
        assert ezsp.status_string(code) != "unknown status"
    assert ezsp.status_string(-99) == "unknown status"


def test_workspace_queries():
    lib = ezsp.load()
    assert lib.ezsp_knn_workspace_size(1000, 10) > 1000 * 10 * 4
    assert lib.ezsp_knn_workspace_size(0, 10) == 0
    assert lib.ezsp_knn_workspace_size(10, 0) == 0
    assert lib.ezsp_knn_workspace_size(10, 65) == 0
    p, _, _ = ezsp._params(10, [0.1, 0.2], None, 0, False)
    big = lib.ezsp_partition_workspace_size(3_000_000, 16, ctypes.byref(p))
    small = lib.ezsp_partition_workspace_size(1000, 16, ctypes.byref(p))
    assert big > small > 0
    assert lib.ezsp_partition_workspace_size(1000, 65, ctypes.byref(p)) == 0
    assert lib.ezsp_partition_workspace_size(2 ** 31, 16, ctypes.byref(p)) == 0
    assert lib.ezsp_component_stats_workspace_size(1000, 10, 8) > 0
    assert lib.ezsp_component_stats_workspace_size(1000, 0, 8) == 0


def call_knn(n=100, k=10, xyz=FAKE, nbr=FAKE, ws=FAKE, ws_bytes=1 << 30):
    return ezsp.load().ezsp_knn(xyz, n, k, nbr, None, ws, ws_bytes, None)


def test_knn_rejects_bad_arguments():
    assert call_knn(n=0) == ezsp.ERR_INVALID_ARG
    assert call_knn(n=2 ** 31) == ezsp.ERR_INVALID_ARG
    assert call_knn(k=0) == ezsp.ERR_INVALID_ARG
    assert call_knn(k=65) == ezsp.ERR_INVALID_ARG
    assert call_knn(xyz=None) == ezsp.ERR_INVALID_ARG
    assert call_knn(nbr=None) == ezsp.ERR_INVALID_ARG
    assert call_knn(ws=None) == ezsp.ERR_INVALID_ARG
    assert call_knn(ws_bytes=16) == ezsp.ERR_WORKSPACE
    assert "workspace" in ezsp.last_error()


def test_knn_walk_stats_rejects_bad_arguments():
    lib = ezsp.load()

    def call(n=100, k=10, xyz=FAKE, nbr=FAKE, scans=FAKE, nodes=FAKE,
             ws=FAKE, ws_bytes=1 << 40):
        return lib.ezsp_knn_walk_stats(xyz, n, k, nbr, scans, nodes, ws,
                                       ws_bytes, None)
    assert call(n=0) == ezsp.ERR_INVALID_ARG
    assert call(k=65) == ezsp.ERR_INVALID_ARG
    assert call(scans=None) == ezsp.ERR_INVALID_ARG
    assert call(nodes=None) == ezsp.ERR_INVALID_ARG
    assert call(ws_bytes=16) == ezsp.ERR_WORKSPACE


def call_partition(n=100, d=8, k=10, lambdas=(0.1,), min_size=None,
                   max_rounds=0, flags=0, ws_bytes=1 << 40, xyz=FAKE,
                   labels=FAKE, n_comp=FAKE, params="ok"):
    lam = np.asarray(lambdas, np.float64)
    ms = None if min_size is None else np.asarray(min_size, np.int64)
    p = ezsp.Params(k, len(lam), lam.ctypes.data if len(lam) else None,
                    None if ms is None else ms.ctypes.data, max_rounds, flags)
    pp = ctypes.byref(p) if params == "ok" else None
    return ezsp.load().ezsp_partition(xyz, FAKE, n, d, pp, labels, n_comp,
                                      None, FAKE, ws_bytes, None)


def test_partition_rejects_bad_arguments():
    E = ezsp.ERR_INVALID_ARG
    assert call_partition(params=None) == E
    assert call_partition(n=0) == E
    assert call_partition(d=0) == E
    assert call_partition(d=65) == E
    assert call_partition(k=0) == E
    assert call_partition(k=65) == E
    assert call_partition(lambdas=()) == E
    assert call_partition(lambdas=[0.1] * 17) == E
    assert call_partition(lambdas=(-0.1,)) == E
    assert call_partition(lambdas=(float("nan"),)) == E
    assert call_partition(lambdas=(float("inf"),)) == E
    assert call_partition(max_rounds=-1) == E
    assert call_partition(flags=4) == E  # unknown bit
    assert call_partition(xyz=None) == E
    assert call_partition(labels=None) == E
    assert call_partition(n_comp=None) == E
    # 4*k*n must stay below 2^31 (int32 table indices)
    assert call_partition(n=60_000_000, k=10) == E
    assert call_partition(ws_bytes=1024) == ezsp.ERR_WORKSPACE


def test_from_knn_and_stats_reject_bad_arguments():
    lib = ezsp.load()
    lam = np.array([0.1])
    p = ezsp.Params(10, 1, lam.ctypes.data, None, 0, 0)
    assert lib.ezsp_partition_from_knn(None, FAKE, 10, 4, ctypes.byref(p),
                                       FAKE, FAKE, None, FAKE, 1 << 40,
                                       None) == ezsp.ERR_INVALID_ARG
    assert lib.ezsp_partition_from_knn(FAKE, FAKE, 10, 4, ctypes.byref(p),
                                       FAKE, FAKE, None, FAKE, 10,
                                       None) == ezsp.ERR_WORKSPACE
    # linking isolated nodes needs positions: not with a given table
    pl = ezsp.Params(10, 1, lam.ctypes.data, None, 0, ezsp.F_LINK_ISOLATED)
    assert lib.ezsp_partition_from_knn(FAKE, FAKE, 10, 4, ctypes.byref(pl),
                                       FAKE, FAKE, None, FAKE, 1 << 40,
                                       None) == ezsp.ERR_INVALID_ARG
    # and its workspace is larger
    assert lib.ezsp_partition_workspace_size(1000, 8, ctypes.byref(pl)) > \
        lib.ezsp_partition_workspace_size(1000, 8, ctypes.byref(p))
    cs = lib.ezsp_component_stats
    assert cs(FAKE, 10, 0, FAKE, 4, None, FAKE, FAKE, None, FAKE, 1 << 40,
              None) == ezsp.ERR_INVALID_ARG
    assert cs(FAKE, 10, 3, FAKE, 0, None, FAKE, FAKE, None, FAKE, 1 << 40,
              None) == ezsp.ERR_INVALID_ARG
    # xyz without a centroid output
    assert cs(FAKE, 10, 3, FAKE, 4, FAKE, FAKE, FAKE, None, FAKE, 1 << 40,
              None) == ezsp.ERR_INVALID_ARG
    assert cs(FAKE, 10, 3, FAKE, 4, None, FAKE, FAKE, None, FAKE, 8,
              None) == ezsp.ERR_WORKSPACE


def test_params_struct_layout():
    # ezsp_params: int32 k, int32 n_levels, 2 pointers, int32, uint32
    assert ctypes.sizeof(ezsp.Params) == 32
    assert ezsp.Params.lambdas.offset == 8
    assert ezsp.Params.min_size.offset == 16
    assert ezsp.Params.max_rounds.offset == 24
    assert ezsp.Params.flags.offset == 28


def test_grid_loss_purity_reject_bad_arguments():
    lib = ezsp.load()
    E, W = ezsp.ERR_INVALID_ARG, ezsp.ERR_WORKSPACE
    nk = ctypes.byref(ctypes.c_int64(0))
    assert lib.ezsp_grid_subsample_workspace_size(1000) > 1000 * 4
    assert lib.ezsp_grid_subsample_workspace_size(0) == 0
    gs = lib.ezsp_grid_subsample
    assert gs(None, 10, 0.1, FAKE, nk, FAKE, 1 << 40, None) == E
    assert gs(FAKE, 10, 0.1, None, nk, FAKE, 1 << 40, None) == E
    assert gs(FAKE, 10, 0.1, FAKE, None, FAKE, 1 << 40, None) == E
    assert gs(FAKE, 0, 0.1, FAKE, nk, FAKE, 1 << 40, None) == E
    assert gs(FAKE, 10, 0.0, FAKE, nk, FAKE, 1 << 40, None) == E
    assert gs(FAKE, 10, -1.0, FAKE, nk, FAKE, 1 << 40, None) == E
    assert gs(FAKE, 10, float("inf"), FAKE, nk, FAKE, 1 << 40, None) == E
    assert gs(FAKE, 10, float("nan"), FAKE, nk, FAKE, 1 << 40, None) == E
    assert gs(FAKE, 10, 0.1, FAKE, nk, FAKE, 8, None) == W

    assert lib.ezsp_edge_loss_workspace_size(1000, 8) > 1000 * 8
    assert lib.ezsp_edge_loss_workspace_size(1000, 0) == 0
    st = ctypes.byref(ezsp.LossStats())

    def loss(n=100, d=8, k=8, tau=1.0, rho=0.3, emb=FAKE, out=st,
             ws_bytes=1 << 40):
        return lib.ezsp_edge_loss(emb, n, d, FAKE, k, FAKE, FAKE, tau, rho,
                                  None, None, None, out, FAKE, ws_bytes, None)
    assert loss(emb=None) == E
    assert loss(out=None) == E
    assert loss(n=0) == E
    assert loss(d=0) == E
    assert loss(d=1025) == E
    assert loss(k=0) == E
    assert loss(k=65) == E
    assert loss(n=300_000_000, k=8) == E
    assert loss(tau=0.0) == E
    assert loss(tau=float("inf")) == E
    assert loss(rho=-0.1) == E
    assert loss(rho=1.5) == E
    assert loss(rho=float("nan")) == E
    assert loss(ws_bytes=8) == W

    assert lib.ezsp_purity_workspace_size(1000, 10, 5) > 0
    assert lib.ezsp_purity_workspace_size(1000, 0, 5) == 0
    assert lib.ezsp_purity_workspace_size(1000, 10, 0) == 0
    ps = ctypes.byref(ezsp.PurityStats())
    pu = lib.ezsp_purity
    assert pu(None, 10, 3, FAKE, 2, None, None, ps, FAKE, 1 << 40, None) == E
    assert pu(FAKE, 10, 3, FAKE, 2, None, None, None, FAKE, 1 << 40, None) == E
    assert pu(FAKE, 10, 0, FAKE, 2, None, None, ps, FAKE, 1 << 40, None) == E
    assert pu(FAKE, 10, 3, FAKE, 0, None, None, ps, FAKE, 1 << 40, None) == E
    assert pu(FAKE, 10, 3, FAKE, 2, None, None, ps, FAKE, 8, None) == W


def test_result_struct_layouts():
    assert ctypes.sizeof(ezsp.LossStats) == 40
    assert ctypes.sizeof(ezsp.PurityStats) == 24
    assert ezsp.PurityStats.n_present.offset == 16


def test_embed_mlp_rejects_bad_arguments():
    lib = ezsp.load()
    E = ezsp.ERR_INVALID_ARG

    def mlp(n=10, d_in=6, d_hid=32, d_out=16, x=FAKE, out=FAKE):
        return lib.ezsp_embed_mlp(x, n, d_in, d_hid, d_out, FAKE, FAKE, FAKE,
                                  FAKE, FAKE, FAKE, out, None)
    assert mlp(x=None) == E
    assert mlp(out=None) == E
    assert mlp(n=0) == E
    assert mlp(d_in=0) == E
    assert mlp(d_in=9) == E
    assert mlp(d_hid=16) == E
    assert mlp(d_out=0) == E
    assert mlp(d_out=33) == E
    assert mlp(n=2 ** 31) == E
