"""GPU tests of the online-training additions: removing members from the pack
(pack_set_active), predictions of members and of the ensemble (pack_predict),
and the whole online loop (paper_2607_05380_amd.online) against the oracle's
loop (Sections 3.5 and 3.6)."""
import math

import numpy as np
import pytest

from oracle.online import ensemble_predict, run_online
from oracle.pack import OraclePack
from paper_2607_05380_amd import configs, synth, tabpack
from paper_2607_05380_amd.online import OnlineTrainer, Snapshot
from parity import TOL, check_tensor, check_update, make_inputs, oracle_cfg, oracle_hparams, record, to_dev

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

# fp32 online loop against the fp64 oracle loop over several epochs: relative
# difference of the per-member and ensemble validation scores
ONLINE_SCORE_REL = 1e-4  # measured 4.8e-5

MEMBERS = [dict(width=w, dropout=p, lr=2e-3, wd=1e-3)
           for w, p in ((96, 0.1), (200, 0.0), (257, 0.3), (40, 0.2), (300, 0.4), (130, 0.1))]


def _state(pk, k):
    return pk.get_params(k), pk.get_moments(k)


def _assert_same(a, b, msg):
    (p1, (m1, v1)), (p2, (m2, v2)) = a, b
    for x1, x2 in ((p1, p2), (m1, m2), (v1, v2)):
        for (W1, b1), (W2, b2) in zip(x1, x2):
            np.testing.assert_array_equal(W1, W2, err_msg=msg)
            np.testing.assert_array_equal(b1, b2, err_msg=msg)


def test_inactive_members_are_frozen_and_others_unchanged():
    # removing members from the pack must leave every other member's step
    # bit-identical (members are independent) and the removed ones untouched
    cfg = configs.workload("regression_onehot", K=6, B=300)
    Xtr, ytr, _, _, orders, _ = make_inputs(cfg, 3000, 10)
    X, y = to_dev(Xtr, ytr)
    idx = [to_dev(synth.batch_indices(orders, s, cfg["B"]))[0] for s in range(3)]
    full = tabpack.Pack(cfg, members=MEMBERS).bind()
    loss_full = [full.train_step(X, y, idx[s], s + 1).cpu().numpy() for s in range(3)]
    part = tabpack.Pack(cfg, members=MEMBERS)
    init = [part.get_params(k) for k in range(6)]
    part.set_active([1, 0, 1, 1, 0, 1])          # before binding
    part.bind()
    losses = []
    for s in range(3):
        out = torch.full((6,), -7.0, device="cuda")
        losses.append(part.train_step(X, y, idx[s], s + 1, out).cpu().numpy())
    for k in range(6):
        if k in (1, 4):
            p, (m, v) = _state(part, k)
            for (W, b), (Wi, bi) in zip(p, init[k]):
                np.testing.assert_array_equal(W, Wi)
                np.testing.assert_array_equal(b, bi)
            assert all((W == 0).all() and (b == 0).all() for W, b in m + v)
            assert all(l[k] == -7.0 for l in losses)
        else:
            _assert_same(_state(part, k), _state(full, k), f"member {k}")
            assert all(l[k] == lf[k] for l, lf in zip(losses, loss_full))


def test_member_removed_and_readmitted_matches_oracle():
    # member 2 sits out step 2 (removed after step 1, back for step 3): its state
    # is frozen meanwhile, and its third step uses the global step counter 3
    cfg = configs.workload("binary_small", K=4)
    members = MEMBERS[:4]
    Xtr, ytr, _, _, orders, _ = make_inputs(cfg, 2048, 10)
    X, y = to_dev(Xtr, ytr)
    pk = tabpack.Pack(cfg, members=members).bind()
    ref = tabpack.Pack(cfg, members=members).bind()
    p0 = pk.get_params(2)
    op = OraclePack(oracle_cfg(cfg), hparams=oracle_hparams(cfg, members))
    sets = ([1, 1, 1, 1], [1, 1, 0, 1], [1, 1, 1, 1])
    for s, act in enumerate(sets):
        idx = synth.batch_indices(orders, s, cfg["B"])
        (idx_d,) = to_dev(idx)
        pk.set_active(act)
        before = _state(pk, 2)
        pk.train_step(X, y, idx_d, s + 1)
        ref.train_step(X, y, idx_d, s + 1)
        op.train_step(Xtr, ytr, idx, s + 1, members=[k for k in range(4) if act[k]])
        if not act[2]:
            _assert_same(_state(pk, 2), before, "frozen member 2")
    for k in range(4):
        if k != 2:
            _assert_same(_state(pk, k), _state(ref, k), f"member {k}")
    # two AdamW steps (t = 1 and t = 3) against the oracle's, as in the step parity tests
    lr = members[2]["lr"]
    for l, ((W, b), (Wr, br), (W0, b0)) in enumerate(zip(pk.get_params(2), op.params[2], p0)):
        check_update(f"W{l}", W, Wr, W0, None, None, lr, TOL["fp32"], steps=2)
        check_update(f"b{l}", b, br, b0, None, None, lr, TOL["fp32"], steps=2)


@pytest.mark.parametrize("name,over", [("binary_small", {}), ("regression_onehot", dict(K=5, B=300)),
                                       ("multiclass_lognormal", dict(K=4, B=300))])
def test_predict_members_and_ensemble_match_oracle(name, over):
    cfg = configs.workload(name, **over)
    Xtr, ytr, Xva, yva, orders, idx = make_inputs(cfg, 3000, 700)  # 700 rows: several row chunks, ragged
    X, y, idx_d, Xv = to_dev(Xtr, ytr, idx, Xva)
    pk = tabpack.Pack(cfg).bind()
    pk.train_step(X, y, idx_d, 1)
    prec = "bf16" if cfg["precision"] == "bf16" else "fp64"
    op = OraclePack(oracle_cfg(cfg), hparams=oracle_hparams(cfg), precision=prec)
    op.train_step(Xtr, ytr, idx, 1)
    K = cfg["K"]
    tol = TOL["bf16"] if cfg["precision"] == "bf16" else dict(TOL["fp32"], atol=1e-6)
    for active in ([True] * K, [k % 2 == 1 for k in range(K)]):
        pk.set_active(active)
        mem = pk.predict(Xv).cpu().numpy()
        ens = pk.predict(Xv, ensemble=True).cpu().numpy()
        ids = [k for k in range(K) if active[k]]
        assert mem.shape == (len(ids), len(Xva), cfg["d_out"]) and ens.shape == (len(Xva), cfg["d_out"])
        refs = [op.predict_values(k, Xva) for k in ids]
        for i, k in enumerate(ids):
            check_tensor(f"{name} member {k}", mem[i], refs[i], tol)
        if cfg["task"] == "multi":
            np.testing.assert_allclose(mem.sum(axis=2), 1.0, rtol=0, atol=1e-5)
        check_tensor(f"{name} ensemble", ens, np.mean(refs, axis=0), tol)
        np.testing.assert_allclose(ens, mem.astype(np.float64).mean(axis=0), rtol=1e-6, atol=1e-7)


def _oracle_loop(cfg, Xtr, ytr, Xva, yva, p_base, p_ens, m_ens, epochs, precision):
    op = OraclePack(oracle_cfg(cfg), hparams=oracle_hparams(cfg), precision=precision)
    n, B = len(Xtr), cfg["B"]
    t = [0]

    def epoch_fn(e, members):
        orders = synth.epoch_orders(cfg, e, n)
        for s in range(n // B):
            t[0] += 1
            op.train_step(Xtr, ytr, synth.batch_indices(orders, s, B), t[0], members=members)
        preds, scores = op.eval_members(Xva, yva, members=members)
        return {k: preds[k] for k in members}, {k: scores[k] for k in members}

    def snapshot(k):
        layers = [(W.copy(), b.copy()) for W, b in op.params[k]]
        if op.use_emb:
            return {n: a.copy() for n, a in op.emb[k].items()}, layers
        return layers

    return op, run_online(epoch_fn, snapshot, cfg["K"], yva, cfg["task"], p_base, p_ens, m_ens, epochs)


EMB_ONLINE = dict(emb_lo=8, emb_hi=16, emb_step=4, sigma_lo=0.1, sigma_hi=3.0)


def test_online_loop_matches_oracle_fp32():
    # learning rates from [3e-3, 2e-2] so that members overfit within a few
    # epochs: the run removes members and stops on the ensemble's patience
    cfg = configs.workload("binary_small", lr_lo=3e-3, lr_hi=2e-2)
    Xtr, ytr, Xva, yva = synth.make_data(cfg)
    p_base, p_ens, m_ens, epochs = 1, 2, 3, 10
    op, (ens, s, hist) = _oracle_loop(cfg, Xtr, ytr, Xva, yva, p_base, p_ens, m_ens, epochs, "fp64")
    X, y, Xv, yv = to_dev(Xtr, ytr, Xva, yva)
    tr = OnlineTrainer(cfg, p_base=p_base, p_ens=p_ens, m_ens=m_ens, max_epochs=epochs)
    tr.fit(X, y, Xv, yv, orders=lambda e: to_dev(synth.epoch_orders(cfg, e, len(Xtr)).astype(np.int32))[0])
    assert sum(len(h["removed"]) for h in hist) >= 2 and len(hist) < epochs, "removal and stopping exercised"
    assert len(tr.history) == len(hist)
    for a, b in zip(tr.history, hist):
        assert a["members"] == b["members"], (a, b)
        rel = [abs(a["scores"][k] - b["scores"][k]) / abs(b["scores"][k]) for k in a["members"]]
        record(f"online.epoch{a['epoch']}.scores", "online_score", n=len(rel), max_rel=max(rel),
               ens_rel=abs(a["score"] - b["score"]) / abs(b["score"]))
        for k in a["members"]:
            assert a["scores"][k] == pytest.approx(b["scores"][k], rel=ONLINE_SCORE_REL), (a["epoch"], k)
        assert a["ensemble"] == b["ensemble"], (a, b)
        assert a["removed"] == b["removed"]
        assert a["score"] == pytest.approx(b["score"], rel=ONLINE_SCORE_REL)
    assert [x.key for x in tr.ensemble] == [x.key for x in ens]
    # the final ensemble's prediction on fresh rows vs the oracle's snapshots
    Xte, _, _, _ = synth.make_data(dict(cfg, seed=cfg["seed"] + 99), n_train=900, n_val=1)
    got = tr.predict(to_dev(Xte)[0]).cpu().numpy()
    hp = oracle_hparams(cfg)

    def predict(inst):
        one = OraclePack(dict(oracle_cfg(cfg), K=1), hparams=[hp[inst.member]], params=[inst.params])
        return one.predict_values(0, Xte)

    ref = ensemble_predict(ens, predict)
    # the snapshots are up to 72 AdamW steps (lr up to 2e-2) into fp32 and fp64
    # trajectories that drift apart slowly: probabilities within 2e-3, and a
    # relative Frobenius error of the whole prediction within 1e-3
    err = np.abs(got - ref)
    frob = np.linalg.norm(got - ref) / np.linalg.norm(ref)
    record("online.final_prediction", "online_predict", n=err.size, max_abs=err.max(), frob=frob)
    assert err.max() <= 2e-3, err.max()
    assert frob <= 1e-3, frob


def test_embedded_inference_pack_matches_oracle():
    # The final ensemble of a pack with periodic embeddings (the paper's default
    # backbone): snapshots taken from the oracle's own loop at several epochs,
    # each with its member's embedding, are loaded into the trainer's inference
    # pack, whose ensemble prediction on fresh rows must match the oracle's mean
    # over the same snapshots.  The GPU's own embedded loop is checked against
    # the selection and patience rules on its own scores
    # (test_online_loop_bf16_decisions_follow_the_rules): compared with the
    # fp64 oracle's trajectory, a single ReLU decision within rounding noise of
    # 0 changes the sign-like first AdamW steps of the embedding after a dozen
    # fp32 steps, and the two trajectories part.
    cfg = configs.workload("binary_small", lr_lo=3e-3, lr_hi=2e-2, **EMB_ONLINE)
    Xtr, ytr, Xva, yva = synth.make_data(cfg)
    op, (ens, s, hist) = _oracle_loop(cfg, Xtr, ytr, Xva, yva, 1, 2, 3, 10, "fp64")
    assert len({x.member for x in ens}) >= 2 and len({x.epoch for x in ens}) >= 2
    tr = OnlineTrainer(cfg, p_base=1, p_ens=2, m_ens=3, max_epochs=1)
    assert all(h["d_emb"] > 0 for h in tr.hp)
    tr.ensemble = [Snapshot(x.member, x.epoch, tr.hp[x.member], [x.params[0]] + list(x.params[1]), None)
                   for x in ens]
    Xte, _, _, _ = synth.make_data(dict(cfg, seed=cfg["seed"] + 99), n_train=900, n_val=1)
    got = tr.predict(to_dev(Xte)[0]).cpu().numpy()
    hp = oracle_hparams(cfg)

    def predict(inst):
        emb_p, layers = inst.params
        one = OraclePack(dict(oracle_cfg(cfg), K=1), hparams=[hp[inst.member]], params=[layers])
        one.emb[0] = emb_p
        return one.predict_values(0, Xte)

    ref = ensemble_predict(ens, predict)
    check_tensor("embedded ensemble prediction", got, ref, dict(TOL["fp32"], atol=1e-6))


@pytest.mark.parametrize("emb", [{}, EMB_ONLINE], ids=["plain", "embeddings"])
def test_online_loop_bf16_decisions_follow_the_rules(emb):
    # bf16 run on the GPU; its own per-epoch validation values, replayed through
    # the oracle's loop, must give the same removals, ensembles and stop; with
    # periodic embeddings the final ensemble's inference pack is rebuilt with
    # every snapshot's embedding
    cfg = configs.workload("regression_onehot", K=6, B=256, **emb)
    Xtr, ytr, Xva, yva = synth.make_data(cfg, n_train=2048, n_val=600)
    X, y, Xv, yv = to_dev(Xtr, ytr, Xva, yva)
    tr = OnlineTrainer(cfg, p_base=1, p_ens=1, m_ens=4, max_epochs=8)
    seen = []
    real_eval = tr.pack.eval_members

    def recording_eval(Xv_, yv_):
        pred, score = real_eval(Xv_, yv_)
        seen.append((pred.cpu().numpy().astype(np.float64), score.cpu().numpy()))
        return pred, score

    tr.pack.eval_members = recording_eval
    tr.fit(X, y, Xv, yv)

    def epoch_fn(e, members):
        pred, score = seen[e]
        return {k: pred[k] for k in members}, {k: float(score[k]) for k in members}

    ens, s, hist = run_online(epoch_fn, lambda k: None, cfg["K"], yva, cfg["task"], 1, 1, 4, 8)
    assert len(hist) == len(tr.history)
    for a, b in zip(tr.history, hist):
        assert (a["members"], a["ensemble"], a["removed"]) == (b["members"], b["ensemble"], b["removed"])
        assert a["score"] == pytest.approx(b["score"], rel=1e-9, abs=1e-12)
    assert [x.key for x in tr.ensemble] == [x.key for x in ens]
    got = tr.predict(Xv).cpu().numpy()[:, 0]
    # the inference pack rebuilt from the snapshots reproduces their validation values
    mean = np.mean([seen[e][0][k] for k, e in (x.key for x in ens)], axis=0)
    np.testing.assert_allclose(got, mean, rtol=1e-5, atol=1e-6)
    assert math.isfinite(tr.ensemble_score)
