"""Full-size parity in the launch configuration bench.py times: the whole pack
runs on the GPU at the workload's real shape (K = 64), and the oracle recomputes
a sample of members one by one -- members are independent (Section 3.6), so a
member's oracle step needs only its own base batch."""
import numpy as np
import pytest

from oracle.greedy import greedy_select
from oracle.pack import OraclePack
from paper_2607_05380_amd import configs, synth, tabpack
from parity import TOL, check_tensor, compare_member, oracle_cfg, oracle_hparams

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _sample_members(hp, extra=()):
    widths = [h["width"] for h in hp]
    picks = {0, int(np.argmin(widths)), int(np.argmax(widths)), len(hp) - 1, *extra}
    return sorted(picks)


@pytest.mark.parametrize("name", ["regression_large", "binary_wide"])
def test_fullsize_step_sampled_members(name):
    cfg = configs.workload(name)
    print(f"[fullsize] {name}: generating {cfg['n_train']} x {cfg['d_in']} on the device", flush=True)
    Xtr, ytr, _, _ = synth.make_data_device(cfg, "cuda", n_val=16)
    orders = synth.epoch_orders_device(cfg, 0, cfg["n_train"])
    idx = orders[:, :cfg["B"]].contiguous()
    pk = tabpack.Pack(cfg).bind()
    loss = pk.train_step(Xtr, ytr, idx, 1)
    torch.cuda.synchronize()
    hp = oracle_hparams(cfg)
    sample = _sample_members(hp)
    print(f"[fullsize] {name}: oracle on members {sample}", flush=True)
    op = OraclePack(oracle_cfg(cfg), hparams=hp, precision="bf16", members=sample)
    p0 = {k: [(W.copy(), b.copy()) for W, b in op.params[k]] for k in sample}
    lg = loss.cpu().numpy()
    idx_h = idx.cpu().numpy()
    tol = TOL["bf16"]
    for k in sample:
        rows = idx_h[k].astype(np.int64)
        Xk = Xtr[torch.from_numpy(rows).cuda()].cpu().numpy()
        yk = ytr[torch.from_numpy(rows).cuda()].cpu().numpy()
        lo, grads = op.member_step(k, Xk, yk, np.arange(cfg["B"]), 1)
        if op.last_grads is None:
            op.last_grads = [None] * cfg["K"]
        op.last_grads[k] = grads
        check_tensor(f"loss{k}", lg[k:k + 1], np.array([lo]), tol)
        compare_member(pk, op, k, p0[k], tol, prefix=f"{name}.")
    assert np.isfinite(lg).all()


def test_fullsize_eval_sampled_members():
    cfg = configs.workload("regression_large")
    _, _, Xva, yva = synth.make_data_device(cfg, "cuda", n_train=1024)
    pk = tabpack.Pack(cfg).bind()
    pred, score = pk.eval_members(Xva, yva)
    torch.cuda.synchronize()
    hp = oracle_hparams(cfg)
    sample = _sample_members(hp)
    op = OraclePack(oracle_cfg(cfg), hparams=hp, precision="bf16", members=sample)
    Xh, yh = Xva.cpu().numpy(), yva.cpu().numpy()
    pr, sr = op.eval_members(Xh, yh, members=sample)
    check_tensor("pred", pred.cpu().numpy()[sample], pr[sample], TOL["bf16"])
    check_tensor("score", score.cpu().numpy()[sample], sr[sample], TOL["bf16"])


def test_fullsize_select():
    # the online pool at its largest: 64 current members + 32 previous picks,
    # 70,000 validation rows, m_ens = 32
    C, Nv = 96, 70_000
    rng = np.random.default_rng(5)
    y = rng.standard_normal(Nv).astype(np.float32)
    cand = (y[None, :] * rng.uniform(0.2, 1.0, (C, 1)) + rng.standard_normal((C, Nv)) * rng.uniform(0.3, 1.5, (C, 1))
            ).astype(np.float32)
    pk = tabpack.Pack(configs.workload("regression_large", K=2))
    sel, s = pk.select(torch.from_numpy(cand).cuda(), torch.from_numpy(y).cuda(), 32)
    sel_o, s_o = greedy_select(cand, y, "reg", 32)
    assert sel == sel_o and s == pytest.approx(s_o, rel=1e-12)
