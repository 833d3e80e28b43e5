"""pack_select_static (the selection with the library's static scratch, for
callers that cannot allocate) against pack_select with a caller workspace:
two calls in a row through the C ABI, the second with a smaller input, each
must give the same picks, count and score bit for bit."""
import ctypes

import numpy as np
import pytest

from paper_2607_05380_amd import configs, tabpack
from select_cases import screened_cases

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _with_workspace(pk, cand, y, m_ens):
    C, Nv = cand.shape
    n = ctypes.c_size_t()
    assert pk.lib.pack_select_workspace_size(C, Nv, ctypes.byref(n)) == 0
    ws = torch.empty(n.value, dtype=torch.uint8, device="cuda")
    sel = torch.full((m_ens,), -1, dtype=torch.int32, device="cuda")
    nsel = torch.zeros(1, dtype=torch.int32, device="cuda")
    score = torch.zeros(1, dtype=torch.float64, device="cuda")
    rc = pk.lib.pack_select(pk.h, cand.data_ptr(), y.data_ptr(), C, Nv, m_ens, ws.data_ptr(), ws.numel(),
                            sel.data_ptr(), nsel.data_ptr(), score.data_ptr(), None)
    assert rc == 0, pk.lib.pack_last_error()
    torch.cuda.synchronize()
    return sel.cpu().numpy(), int(nsel.item()), score.item()


def _static(pk, cand, y, m_ens):
    C, Nv = cand.shape
    sel = torch.full((m_ens,), -1, dtype=torch.int32, device="cuda")
    nsel = torch.zeros(1, dtype=torch.int32, device="cuda")
    score = torch.zeros(1, dtype=torch.float64, device="cuda")
    torch.cuda.synchronize()
    rc = pk.lib.pack_select_static(pk.h, cand.data_ptr(), y.data_ptr(), C, Nv, m_ens, sel.data_ptr(),
                                   nsel.data_ptr(), score.data_ptr(), None)
    assert rc == 0, pk.lib.pack_last_error()
    torch.cuda.synchronize()
    return sel.cpu().numpy(), int(nsel.item()), score.item()


@pytest.mark.parametrize("task", ["reg", "multi"])
def test_static_selection_matches_workspace_selection(task):
    cfg = configs.workload({"reg": "regression_onehot", "multi": "multiclass_lognormal"}[task], K=2)
    pk = tabpack.Pack(cfg)
    # the larger case first, then a smaller one: the second call must not see
    # anything the first left in the shared array
    for C, Nv, m_ens in ((96, 20_000, 32), (7, 1_500, 5)):
        (cand, y, gap), = screened_cases(task, C, Nv, m_ens, seeds=range(C * 7 + Nv, C * 7 + Nv + 40))
        print(f"[no_alloc] {task} C={C} Nv={Nv} m_ens={m_ens} gap {gap:.1e}", flush=True)
        c_d, y_d = torch.from_numpy(cand).cuda(), torch.from_numpy(y).cuda()
        sel_w, n_w, s_w = _with_workspace(pk, c_d, y_d, m_ens)
        sel_s, n_s, s_s = _static(pk, c_d, y_d, m_ens)
        assert n_s == n_w >= 1
        np.testing.assert_array_equal(sel_s[:n_s], sel_w[:n_w])
        assert s_s == s_w


def test_static_selection_rejects_inputs_beyond_its_array():
    pk = tabpack.Pack(configs.workload("regression_onehot", K=2))
    n = ctypes.c_size_t()
    C, Nv = 96, 600_000
    assert pk.lib.pack_select_workspace_size(C, Nv, ctypes.byref(n)) == 0
    assert n.value > 4 << 20
    # rejected by the size check before any pointer is used
    dummy = torch.zeros(4, dtype=torch.float64, device="cuda")
    rc = pk.lib.pack_select_static(pk.h, dummy.data_ptr(), dummy.data_ptr(), C, Nv, 8, dummy.data_ptr(),
                                   dummy.data_ptr(), dummy.data_ptr(), None)
    assert rc == -1  # PACK_EINVAL
    assert b"PACK_SELECT_STATIC_BYTES" in pk.lib.pack_last_error()
