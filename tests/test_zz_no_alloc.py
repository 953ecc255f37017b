"""rk_poa_estimate_noalloc (the PoA-hat estimate on the library's static device
buffer, for callers that cannot allocate) against rk_poa_estimate with a
caller workspace: identical window sums and ratios on two calls in a row, the
second on a smaller input, through the C ABI."""
import ctypes as C

import numpy as np
import pytest

from paper_2606_17081_amd import workload as wl

pytestmark = pytest.mark.gpu


def _poa_both(torch, rk, r):
    outs = []
    for noalloc in (False, True):
        sel = torch.full((max(r.n_windows, 1),), -1.0, dtype=torch.float64, device="cuda")
        coo = torch.full_like(sel, -1.0)
        hat = torch.full((len(r.episodes),), -1.0, dtype=torch.float64, device="cuda")
        args = (r.win_off, r.ep_win_off, r.n_rows, r.max_window, r.W, r.route_worker, r.overlap, r.route_blocks,
                r.poa_params, sel, coo, hat)
        if noalloc:
            rk.poa_estimate_noalloc(*args)
        else:
            rk.poa_estimate(*args, r.poa_ws)
        torch.cuda.synchronize()
        assert rk.device_status(reset=True) == 0
        outs.append([t.cpu().numpy() for t in (sel, coo, hat)])
    return outs


def test_noalloc_matches_workspace_twice():
    import torch
    assert torch.cuda.is_available(), "GPU tests need an MI355X"
    from paper_2606_17081_amd import rkroute as rk
    from paper_2606_17081_amd.episodes import EpisodeRunner
    big = wl.sweep70b_workload()                 # 1.31 M rows: most of the static buffer
    small = wl.tiny_workload()
    sizes = []
    for w in (big, small):
        r = EpisodeRunner(w)
        r.hash()
        r.simulate()
        torch.cuda.synchronize()
        need = rk.poa_workspace_size(r.n_rows, r.W)
        assert need <= rk.RK_POA_NOALLOC_BYTES
        sizes.append(r.n_rows)
        print("episodes", len(w.episodes), "rows", r.n_rows, "windows", r.n_windows, flush=True)
        ws_out, na_out = _poa_both(torch, rk, r)
        for a, b in zip(ws_out, na_out):
            assert np.array_equal(a.view(np.uint64), b.view(np.uint64))
        assert np.all(na_out[2] > 0)
    assert sizes[1] < sizes[0]


def test_noalloc_rejects_oversized_shapes():
    from paper_2606_17081_amd import rkroute as rk
    L = rk.lib()
    pp = rk.PoaParams(0.005, 0.02, 0.01, 2, 64, 0.015, 0)
    rows = rk.RK_POA_NOALLOC_BYTES // (64 * 4) + 1           # the matrix alone is larger than the buffer
    p8 = C.c_void_p(8)
    rc = L.rk_poa_estimate_noalloc(1, p8, 0, None, rows, 64, 64, p8, p8, p8, pp, p8, p8, None, None)
    assert rc == rk.RK_EUNSUPPORTED
    assert b"static buffer" in L.rk_last_error()
