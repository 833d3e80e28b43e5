"""Degenerate inputs through the C ABI: a single validation or prediction row
(one ragged chunk of the padded batch), empty inputs rejected with PACK_EINVAL
before any launch, and the greedy selection's degenerate cases (no picks
asked for, a single candidate)."""
import ctypes
import math

import numpy as np
import pytest

from oracle.greedy import greedy_select
from oracle.pack import OraclePack
from paper_2607_05380_amd import configs, tabpack
from parity import TOL, check_tensor, make_inputs, oracle_cfg, oracle_hparams, to_dev

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

PACK_EINVAL = -1


@pytest.mark.parametrize("name", ["binary_small", "multiclass_lognormal"])
def test_single_row_eval_and_predict(name):
    cfg = configs.workload(name, K=3, B=256)
    tol = TOL[cfg["precision"]]
    _, _, Xva, yva, _, _ = make_inputs(cfg, 600, 5)
    Xva, yva = Xva[:1].copy(), yva[:1].copy()
    pk = tabpack.Pack(cfg).bind()
    op = OraclePack(oracle_cfg(cfg), hparams=oracle_hparams(cfg),
                    precision="bf16" if cfg["precision"] == "bf16" else "fp64")
    Xv, yv = to_dev(Xva, yva)
    pred, score = pk.eval_members(Xv, yv)
    out = pk.predict(Xv)
    torch.cuda.synchronize()
    pr, sr = op.eval_members(Xva, yva)
    check_tensor("pred", pred.cpu().numpy(), pr, tol)
    check_tensor("score", score.cpu().numpy(), sr, tol)
    for k in range(3):
        check_tensor(f"predict m{k}", out[k].cpu().numpy(), op.predict_values(k, Xva), tol)


def test_empty_inputs_rejected():
    cfg = configs.workload("regression_onehot", K=2, B=256)
    _, _, Xva, yva, _, _ = make_inputs(cfg, 600, 8)
    pk = tabpack.Pack(cfg).bind()
    lib = pk.lib
    Xv, yv = to_dev(Xva, yva)
    pred = torch.zeros((2, 8), dtype=torch.float32, device="cuda")
    score = torch.zeros(2, dtype=torch.float64, device="cuda")
    assert lib.pack_eval_members(pk.h, Xv.data_ptr(), yv.data_ptr(), 0, pred.data_ptr(), score.data_ptr(),
                                 None) == PACK_EINVAL
    assert b"Nv" in lib.pack_last_error()
    assert lib.pack_predict(pk.h, Xv.data_ptr(), 0, 0, pred.data_ptr(), None) == PACK_EINVAL
    n = ctypes.c_size_t()
    assert lib.pack_select_workspace_size(0, 8, ctypes.byref(n)) == PACK_EINVAL
    assert lib.pack_select_workspace_size(2, 0, ctypes.byref(n)) == PACK_EINVAL
    assert lib.pack_select_workspace_size(2, 8, ctypes.byref(n)) == 0 and n.value > 0
    ws = torch.empty(n.value, dtype=torch.uint8, device="cuda")
    sel = torch.zeros(4, dtype=torch.int32, device="cuda")
    nsel = torch.zeros(1, dtype=torch.int32, device="cuda")
    sc = torch.zeros(1, dtype=torch.float64, device="cuda")
    for C, Nv, m in ((0, 8, 2), (2, 0, 2), (2, 8, -1)):
        assert lib.pack_select(pk.h, pred.data_ptr(), yv.data_ptr(), C, Nv, m, ws.data_ptr(), ws.numel(),
                               sel.data_ptr(), nsel.data_ptr(), sc.data_ptr(), None) == PACK_EINVAL
    torch.cuda.synchronize()
    # nothing was launched: the outputs keep their values
    assert (pred == 0).all() and (nsel == 0).all()


def test_select_degenerate_cases():
    cfg = configs.workload("regression_onehot", K=2)
    pk = tabpack.Pack(cfg)
    rng = np.random.default_rng(4)
    y = rng.standard_normal(50).astype(np.float32)
    cand = (y[None, :] + rng.standard_normal((3, 50))).astype(np.float32)
    c_d, y_d = to_dev(cand, y)
    # no picks asked for: an empty ensemble with score +inf
    sel, s = pk.select(c_d, y_d, 0)
    assert sel == [] and s == math.inf
    # a single candidate is always taken (any finite score improves on +inf)
    sel, s = pk.select(c_d[:1].contiguous(), y_d, 5)
    sel_o, s_o = greedy_select(cand[:1].astype(np.float64), y, "reg", 5)
    assert sel == sel_o == [0]
    assert s == pytest.approx(s_o, rel=1e-12)
    # m_ens larger than the pool: every candidate at most once
    sel, s = pk.select(c_d, y_d, 10)
    sel_o, s_o = greedy_select(cand.astype(np.float64), y, "reg", 10)
    assert sel == sel_o and len(set(sel)) == len(sel) <= 3
    assert s == pytest.approx(s_o, rel=1e-12)


def test_out_of_range_batch_indices_are_flagged_and_never_read():
    # entries outside [0, N) read row 0 instead and raise the status flag: the
    # step equals (bit for bit) the step with those entries set to 0
    cfg = configs.workload("regression_onehot", K=3, B=200)
    Xtr, ytr, _, _, _, idx = make_inputs(cfg, 1000, 10)
    bad = idx.copy()
    bad[0, 5], bad[1, 0], bad[2, -1] = -1, 1000, np.iinfo(np.int32).max
    fixed = np.where((bad < 0) | (bad >= 1000), 0, bad).astype(np.int32)
    X, y, bad_d, fixed_d = to_dev(Xtr, ytr, bad, fixed)
    runs = []
    for ix in (bad_d, fixed_d):
        pk = tabpack.Pack(cfg).bind()
        assert pk.status() == 0
        loss = pk.train_step(X, y, ix, 1).cpu().numpy()
        runs.append((loss, pk.status(), [pk.get_params(k) for k in range(3)]))
        assert pk.status() == 0  # cleared by the read
    (l1, s1, p1), (l2, s2, p2) = runs
    assert s1 == tabpack.STATUS_IDX_RANGE and s2 == 0
    np.testing.assert_array_equal(l1, l2)
    for a, b in zip(p1, p2):
        for (W1, b1), (W2, b2) in zip(a, b):
            np.testing.assert_array_equal(W1, W2)
            np.testing.assert_array_equal(b1, b2)


def test_stream_copy_copies_exactly():
    src = torch.arange(1 << 20, dtype=torch.float32, device="cuda") * 0.5 - 7.0
    dst = torch.zeros_like(src)
    tabpack.stream_copy(src, dst)
    torch.cuda.synchronize()
    assert torch.equal(src, dst)
    # a ragged size: fewer vectors than one round of the grid
    s2, d2 = src[:4 * 37].clone(), torch.zeros(4 * 37, device="cuda")
    tabpack.stream_copy(s2, d2)
    torch.cuda.synchronize()
    assert torch.equal(s2, d2)
