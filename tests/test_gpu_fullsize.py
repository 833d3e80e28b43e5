"""Full-size parity in the launch configuration bench.py times: the whole pack
runs on the GPU at the workload's real shape, and the oracle recomputes a
sample of members one by one -- members are independent (Section 3.6), so a
member's oracle step needs only its own base batch."""
import numpy as np
import pytest

from oracle.greedy import greedy_select
from oracle.pack import OraclePack
from paper_2607_05380_amd import configs, synth, tabpack
from parity import (TOL, check_decisions, check_tensor, compare_member, compare_member_fp64, gpu_hints, oracle_cfg,
                    oracle_hparams)
from test_gpu_embed import EMB, _compare as compare_embedded, _gpu as embedded_tensors, randomize_embeddings
from test_gpu_muon import MUON, _compare as compare_muon
from select_cases import screened_cases

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _sample_members(hp, extra=()):
    widths = [h["width"] for h in hp]
    picks = {0, int(np.argmin(widths)), int(np.argmax(widths)), len(hp) - 1, *extra}
    return sorted(picks)


def _fullsize_step(cfg, precisions=("bf16",), setup=None, rows="stream"):
    """One packed step at the workload's real shape on the GPU, and oracle packs
    (one per precision policy) holding only the sampled members, stepped on
    the same base batches.  ``setup(pk, ops, sample)`` may change initial
    parameters on both sides; it returns the sampled members' initial values
    (default: the layer parameters).  rows="stream": the first layer reads its
    rows straight from the data where the pack allows it, as bench.py runs it;
    "gather": the batch is gathered first."""
    name = cfg["name"]
    print(f"[fullsize] {name}: generating {cfg['n_train']} x {cfg['d_in']} on the device", flush=True)
    Xtr, ytr, _, _ = synth.make_data_device(cfg, "cuda", n_val=16)
    orders = synth.epoch_orders_device(cfg, 0, cfg["n_train"])
    idx = orders[:, :cfg["B"]].contiguous()
    pk = tabpack.Pack(cfg).bind()
    if rows == "stream" and pk.can_bind_data():
        pk.bind_data(Xtr)
        print(f"[fullsize] {name}: first-layer rows streamed from the data", flush=True)
    hp = oracle_hparams(cfg)
    sample = _sample_members(hp)
    ops = [OraclePack(oracle_cfg(cfg), hparams=hp, precision=p, members=sample) for p in precisions]
    if setup is not None:
        p0 = setup(pk, ops, sample)
    else:
        p0 = {k: [(W.copy(), b.copy()) for W, b in ops[0].params[k]] for k in sample}
    loss = pk.train_step(Xtr, ytr, idx, 1)
    torch.cuda.synchronize()
    print(f"[fullsize] {name}: oracle on members {sample}", flush=True)
    lg = loss.cpu().numpy()
    idx_h = idx.cpu().numpy()
    for op in ops:
        op.last_grads = [None] * cfg["K"]
        op.last_emb_grads = [None] * cfg["K"]
    for k in sample:
        rows = torch.from_numpy(idx_h[k].astype(np.int64)).cuda()
        Xk, yk = Xtr[rows].cpu().numpy(), ytr[rows].cpu().numpy()
        hints = gpu_hints(pk, k, cfg, 1)
        for op in ops:
            # the bf16-policy oracle takes the GPU's ReLU decisions within its
            # window around 0; the exact fp64 oracle takes its own everywhere
            policy = op.rnd is not None
            lo, op.last_grads[k] = op.member_step(k, Xk, yk, np.arange(cfg["B"]), 1, hints if policy else None)
            tag = "bf16" if policy else "fp64"
            check_tensor(f"{name}.loss{k}.{tag}", lg[k:k + 1], np.array([lo]), TOL["bf16"])
            if policy:
                check_decisions(op, k, f"{name}.m{k}")
    assert np.isfinite(lg).all()
    return pk, ops, sample, p0


@pytest.mark.parametrize("name,rows", [("regression_onehot", "stream"), ("multiclass_lognormal", "stream"),
                                       ("binary_wide", "stream"), ("regression_large", "stream"),
                                       ("regression_large", "gather")])
def test_fullsize_step_sampled_members(name, rows):
    cfg = configs.workload(name)
    pk, (op, op64), sample, p0 = _fullsize_step(cfg, ("bf16", "fp64"), rows=rows)
    for k in sample:
        compare_member(pk, op, k, p0[k], TOL["bf16"], prefix=f"{name}.")
        w64 = compare_member_fp64(pk, op64, k, p0[k], prefix=f"{name}.")
        print(f"[fullsize] {name} member {k}: gradient frob vs the exact fp64 oracle {w64:.4f}", flush=True)


def test_fullsize_muon_step_sampled_members():
    # the regression_large pack with Muon for the hidden weights at K = 64
    cfg = configs.workload("regression_large", **MUON)
    pk, (op,), sample, p0 = _fullsize_step(cfg)
    report = []
    compare_muon(pk, op, p0, TOL["bf16"], 1, 0.05, report, members=sample, prefix="fullsize.")
    print(f"[fullsize] muon worst update frob {max(r[1] for r in report if r[0].endswith('.frob')):.3e}",
          flush=True)


def test_fullsize_embedded_step_sampled_members():
    # the regression_large pack with periodic embeddings at K = 64; the sampled
    # members start from non-zero b, alpha, beta so that every embedding
    # gradient is exercised at the first step
    cfg = configs.workload("regression_large", **EMB)

    def setup(pk, ops, sample):
        randomize_embeddings(pk, ops[0], sample, cfg["seed"])
        return {k: [(n, np.array(a, np.float64)) for n, a, _, _, _ in embedded_tensors(pk, k)] for k in sample}

    pk, (op,), sample, p0 = _fullsize_step(cfg, setup=setup)
    compare_embedded(pk, op, p0, TOL["bf16"], 1, members=sample, prefix="fullsize.")


@pytest.mark.parametrize("name,over,nv", [("regression_large", {}, None), ("multiclass_lognormal", {}, None),
                                          ("regression_large", EMB, 3000)])
def test_fullsize_eval_sampled_members(name, over, nv):
    # evaluation over the whole validation set (the embedded pack over 3,000
    # rows: its first layer launch runs the tall tiles on every 1,024-row chunk)
    cfg = configs.workload(name, **over)
    _, _, Xva, yva = synth.make_data_device(cfg, "cuda", n_train=1024)
    if nv is not None:
        Xva, yva = Xva[:nv].contiguous(), yva[:nv].contiguous()
    pk = tabpack.Pack(cfg).bind()
    pred, score = pk.eval_members(Xva, yva)
    torch.cuda.synchronize()
    hp = oracle_hparams(cfg)
    sample = _sample_members(hp)
    print(f"[fullsize] eval {name} {len(yva)} rows, members {sample}", flush=True)
    op = OraclePack(oracle_cfg(cfg), hparams=hp, precision="bf16", members=sample)
    Xh, yh = Xva.cpu().numpy(), yva.cpu().numpy()
    pr, sr = op.eval_members(Xh, yh, members=sample)
    check_tensor(f"{name}.pred", pred.cpu().numpy()[sample], pr[sample], TOL["bf16"])
    check_tensor(f"{name}.score", score.cpu().numpy()[sample], sr[sample], TOL["bf16"])


def test_fullsize_select():
    # the online pool at its largest: 64 current members + 32 previous picks,
    # 70,000 validation rows, m_ens = 32; the case is screened for near-ties
    (cand, y, gap), = screened_cases("reg", 96, 70_000, 32, seeds=range(5, 50), count=1)
    print(f"[fullsize] select: smallest relative gap between best and runner-up {gap:.2e}", flush=True)
    pk = tabpack.Pack(configs.workload("regression_large", K=2))
    sel, s = pk.select(torch.from_numpy(cand).cuda(), torch.from_numpy(y).cuda(), 32)
    sel_o, s_o = greedy_select(cand, y, "reg", 32)
    assert sel == sel_o and s == pytest.approx(s_o, rel=1e-12)
