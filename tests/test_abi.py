"""The C-ABI library loads without a GPU, exports every declared symbol, and
rejects invalid arguments on the host before launching anything."""
import ctypes as C
import os
import re

import pytest

from paper_2606_17081_amd import rkroute as rk

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    names = set()
    for f in os.listdir(os.path.join(ROOT, "include")):
        if f.endswith(".h"):
            src = open(os.path.join(ROOT, "include", f)).read()
            src = re.sub(r"/\*.*?\*/", "", src, flags=re.S)
            names |= set(re.findall(r"\b(rk_[a-z_0-9]+)\s*\(", src))
    return names


def test_library_exports_every_declared_symbol():
    if not rk.library_available():
        pytest.skip("librkroute.so not built")
    L = rk.lib()
    declared = _declared()
    assert declared, "no declarations found"
    assert declared == set(rk.EXPORTED)
    for name in declared:
        assert hasattr(L, name), name


def test_status_strings_and_host_validation():
    if not rk.library_available():
        pytest.skip("librkroute.so not built")
    L = rk.lib()
    assert L.rk_status_string(0) == b"ok"
    assert L.rk_status_string(-4) == b"table full"
    p = rk.CostParams(1.0, 0.5, 4.0, 512)
    assert L.rk_route_score_batch(4, 0, None, None, None, 12, None, p, 0, None, None, None, None) == rk.RK_EINVAL
    assert b"W outside" in L.rk_last_error()
    bad = rk.CostParams(-1.0, 0.5, 4.0, 512)
    assert L.rk_route_score_batch(4, 2, None, None, None, 12, None, bad, 0, None, None, None, None) == rk.RK_EINVAL
    assert L.rk_route_score_batch(4, 2, None, None, None, 3, None, p, 0, None, None, None, None) == rk.RK_EINVAL
    assert L.rk_route_score_batch(4, 2, None, None, None, 12, None, p, 7, None, None, None, None) == rk.RK_EINVAL
    assert L.rk_route_score_batch(0, 2, None, None, None, 12, None, p, 0, None, None, None, None) == rk.RK_OK
    assert L.rk_hash_chains(-1, None, None, None, None, None) == rk.RK_EINVAL
    assert L.rk_hash_chains(0, None, None, None, None, None) == rk.RK_OK
    import numpy as np
    koff = np.array([0, 10, 5], np.int64)
    assert L.rk_table_build(2, None, C.c_void_p(koff.ctypes.data), C.c_void_p(8), 8, None) == rk.RK_EINVAL
    koff = np.array([0, 200], np.int64)
    assert L.rk_table_build(1, None, C.c_void_p(koff.ctypes.data), C.c_void_p(8), 8, None) == rk.RK_ETABLEFULL


def test_episode_and_poa_host_validation():
    if not rk.library_available():
        pytest.skip("librkroute.so not built")
    L = rk.lib()
    b = rk.EpisodeBatch(1, 65, 16, 8, 4, 8, 2, 1, 0, 0, 4, 0, 0, 0, None, None, None, None, None)
    o = rk.EpisodeOutputs()
    assert L.rk_simulate_episodes(C.byref(b), C.byref(o), None, 0, None) == rk.RK_EUNSUPPORTED
    b = rk.EpisodeBatch(1, 4, 16, 8, 4, 8, 2, 1, 3, 0, 4, 0, 0, 0, None, None, None, None, None)
    assert L.rk_simulate_episodes(C.byref(b), C.byref(o), None, 0, None) == rk.RK_EINVAL
    b = rk.EpisodeBatch(0, 4, 16, 8, 4, 8, 2, 1, 0, 0, 4, 0, 0, 0, None, None, None, None, None)
    assert L.rk_simulate_episodes(C.byref(b), C.byref(o), None, 0, None) == rk.RK_OK
    b = rk.EpisodeBatch(2, 4, 16, 8, 4, 8, 2, 1, 0, 0, 4, 0, 0, 0, C.c_void_p(8), C.c_void_p(8), C.c_void_p(8),
                        C.c_void_p(8), C.c_void_p(8))
    assert L.rk_simulate_episodes(C.byref(b), C.byref(o), C.c_void_p(8), 16, None) == rk.RK_ENOMEM
    need = rk.simulate_workspace_size(2, 4, 16, 8, 4, 10)
    assert need > 0 and need == 2 * rk.simulate_workspace_size(1, 4, 16, 8, 4, 10)
    # flags: none is defined
    b = rk.EpisodeBatch(2, 4, 16, 8, 4, 8, 2, 1, 0, 0, 4, 1, 0, 0, C.c_void_p(8), C.c_void_p(8), C.c_void_p(8),
                        C.c_void_p(8), C.c_void_p(8))
    assert L.rk_simulate_episodes(C.byref(b), C.byref(o), C.c_void_p(8), need, None) == rk.RK_EINVAL
    assert b"flags" in L.rk_last_error()
    # workspace slots: fewer workspaces than episodes need less memory; negative counts or a
    # nonzero pad are rejected
    b.flags = 0
    one = rk.simulate_workspace_size(1, 4, 16, 8, 4, 4)
    b.ws_slots = -1
    assert L.rk_simulate_episodes(C.byref(b), C.byref(o), C.c_void_p(8), need, None) == rk.RK_EINVAL
    assert b"ws_slots" in L.rk_last_error()
    b.ws_slots, b.ws_pad = 1, 7
    assert L.rk_simulate_episodes(C.byref(b), C.byref(o), C.c_void_p(8), need, None) == rk.RK_EINVAL
    b.ws_pad = 0
    assert L.rk_simulate_episodes(C.byref(b), C.byref(o), C.c_void_p(8), one - 1, None) == rk.RK_ENOMEM
    assert b"needed" in L.rk_last_error()
    pp = rk.PoaParams(0.005, 0.02, 0.01, 2, 64, 0.015, 0)
    assert L.rk_poa_estimate(1, None, 0, None, 8, 8, 65, None, None, None, pp, None, None, None, None, 0,
                             None) == rk.RK_EUNSUPPORTED
    assert L.rk_poa_estimate(0, None, 0, None, 0, 8, 4, None, None, None, pp, None, None, None, None, 0,
                             None) == rk.RK_OK
    bad = rk.PoaParams(0.005, 0.02, 0.01, 0, 64, 0.015, 0)
    assert L.rk_poa_estimate(1, None, 0, None, 8, 8, 4, None, None, None, bad, None, None, None, None, 0,
                             None) == rk.RK_EINVAL


def test_index_host_validation():
    if not rk.library_available():
        pytest.skip("librkroute.so not built")
    import numpy as np
    L = rk.lib()
    p = rk.CostParams(1.0, 0.5, 4.0, 512)
    koff = np.zeros(66, np.int64)
    assert L.rk_index_build(65, None, C.c_void_p(koff.ctypes.data), C.c_void_p(16), 8, None) == rk.RK_EUNSUPPORTED
    assert L.rk_index_build(2, None, C.c_void_p(koff.ctypes.data), C.c_void_p(16), 3, None) == rk.RK_EINVAL
    koff = np.array([0, 10, 5], np.int64)
    assert L.rk_index_build(2, None, C.c_void_p(koff.ctypes.data), C.c_void_p(16), 8, None) == rk.RK_EINVAL
    koff = np.array([0, 100, 129], np.int64)     # 129 keys for 256 slots: above load 0.5
    assert L.rk_index_build(2, None, C.c_void_p(koff.ctypes.data), C.c_void_p(16), 8, None) == rk.RK_ETABLEFULL
    assert L.rk_route_score_index(4, 65, None, None, None, 12, None, p, 0, None, None, None,
                                  None) == rk.RK_EUNSUPPORTED
    assert L.rk_route_score_index(4, 2, None, None, None, 32, None, p, 0, None, None, None, None) == rk.RK_EINVAL
    assert L.rk_route_score_index(4, 2, None, None, None, 12, None, p, 5, None, None, None, None) == rk.RK_EINVAL
    bad = rk.CostParams(1.0, 0.5, 4.0, 0)
    assert L.rk_route_score_index(4, 2, None, None, None, 12, None, bad, 0, None, None, None, None) == rk.RK_EINVAL
    assert L.rk_route_score_index(0, 2, None, None, None, 12, None, p, 0, None, None, None, None) == rk.RK_OK
    assert L.rk_route_score_index(3, 2, None, None, None, 12, None, p, 0, None, None, None, None) == rk.RK_EINVAL
