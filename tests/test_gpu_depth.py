"""GPU parity of packs whose members have different depths (App. F samples the
number of layers per base model): every layer-l launch holds only the members
with at least l hidden blocks, and each member's head reads its own last
layer.  Compared with the fp64 oracle, whose members simply have their own
number of Linear-ReLU-Dropout blocks."""
import numpy as np
import pytest

from oracle.pack import OraclePack
from paper_2607_05380_amd import configs, synth, tabpack
from parity import TOL, check_tensor, compare_member, make_inputs, oracle_cfg, oracle_hparams, to_dev
from test_gpu_parity import run_step

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

CASES = {
    "fp32-L3": ("binary_small", dict(K=6, L=3, depth_lo=1, depth_hi=3)),
    "bf16-L3": ("regression_onehot", dict(K=8, B=300, depth_lo=1, depth_hi=3)),
    "bf16-L4-ce": ("multiclass_lognormal", dict(K=6, B=260, L=4, depth_lo=1, depth_hi=4)),
}


@pytest.mark.parametrize("case", list(CASES))
def test_variable_depth_step_parity(case):
    name, over = CASES[case]
    cfg = configs.workload(name, **over)
    depths = [h["depth"] for h in tabpack.Pack(cfg).hparams()]
    print(f"[depth] {case} depths {depths}", flush=True)
    assert len(set(depths)) >= 2 and min(depths) >= 1 and max(depths) <= cfg["L"]
    tol = TOL[cfg["precision"]]
    steps = 3 if cfg["precision"] == "fp32" else 1
    pk, op, losses, _ = run_step(cfg, steps=steps)
    for lg, lo, _ in losses:
        check_tensor("loss", lg, lo, tol)
    for k in range(cfg["K"]):
        assert len(pk.get_params(k)) == depths[k] + 1
        compare_member(pk, op, k, run_step.p0[k], tol, steps=steps, prefix=f"d{depths[k]}.")


def test_variable_depth_eval_and_predict():
    cfg = configs.workload("regression_onehot", K=7, B=256, depth_lo=1, depth_hi=3)
    Xtr, ytr, Xva, yva, _, idx = make_inputs(cfg, 2000, 900)
    X, y, idx_d, Xv, yv = to_dev(Xtr, ytr, idx, Xva, yva)
    pk = tabpack.Pack(cfg).bind()
    pk.train_step(X, y, idx_d, 1)
    op = OraclePack(oracle_cfg(cfg), hparams=oracle_hparams(cfg), precision="bf16")
    op.train_step(Xtr, ytr, idx, 1)
    pred, score = pk.eval_members(Xv, yv)
    pr, sr = op.eval_members(Xva, yva)
    check_tensor("pred", pred.cpu().numpy(), pr, TOL["bf16"])
    check_tensor("score", score.cpu().numpy(), sr, TOL["bf16"])
    mem = pk.predict(Xv).cpu().numpy()
    for k in range(cfg["K"]):
        check_tensor(f"predict {k}", mem[k], op.predict_values(k, Xva), TOL["bf16"])


def test_member_depth_independent_of_pack():
    # a member's step is bit-identical whether its pack-mates are deeper or shallower
    cfg = configs.workload("regression_onehot", K=4, B=300, depth_lo=1, depth_hi=3)
    # no dropout and the big pack's initial parameters copied over: the masks and
    # initial values depend on the member's index, which differs between packs
    members = [dict(width=w, dropout=0.0, lr=2e-3, wd=1e-3, depth=d)
               for w, d in ((160, 1), (200, 3), (96, 2), (300, 3))]
    Xtr, ytr, _, _, orders, _ = make_inputs(cfg, 3000, 10)
    X, y = to_dev(Xtr, ytr)
    packs = [tabpack.Pack(cfg, members=members).bind()]
    for k in range(4):
        one = tabpack.Pack(dict(cfg, K=1), members=[members[k]]).bind()
        one.set_params(0, packs[0].get_params(k))
        packs.append(one)
    for s in range(2):
        (idx,) = to_dev(synth.batch_indices(orders, s, cfg["B"]))
        packs[0].train_step(X, y, idx, s + 1)
        for k in range(4):
            packs[k + 1].train_step(X, y, idx[k:k + 1].contiguous(), s + 1)
    for k in range(4):
        a, b = packs[0].get_params(k), packs[k + 1].get_params(0)
        assert len(a) == members[k]["depth"] + 1
        for (W1, b1), (W2, b2) in zip(a, b):
            np.testing.assert_array_equal(W1, W2)
            np.testing.assert_array_equal(b1, b2)
