"""CPU tests of the online training loop (Sections 3.5 and 3.6 of the paper):
the oracle's loop against a hand-worked run and closed forms of its stopping
rules, and the library's driver (paper_2607_05380_amd.online) against the
oracle's loop on scripted validation values through a stand-in pack."""
import math
import os

import numpy as np
import pytest
import torch
from hypothesis import given, settings, strategies as st

from oracle.greedy import greedy_select
from oracle.online import run_online
from oracle.pack import score
from paper_2607_05380_amd.online import OnlineTrainer

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "online_hand.txt")


def _golden():
    d = {}
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        k, *v = line.split()
        d[k] = v
    return d


def _keys(tokens):
    return [tuple(int(x) for x in t.split(":")) for t in tokens]


def test_oracle_online_hand_example():
    g = _golden()
    K = int(g["K"][0])
    yv = np.array([float(g["y"][0])])
    trained = []

    def epoch_fn(e, members):
        trained.append(list(members))
        vals = [float(x) for x in g[f"epoch{e}"]]
        preds = {k: np.array([vals[k]]) for k in members}
        return preds, {k: score(preds[k], yv, "reg") for k in members}

    ens, s, hist = run_online(epoch_fn, lambda k: ("params", k), K, yv, g["task"][0], int(g["p_base"][0]),
                              int(g["p_ens"][0]), int(g["m_ens"][0]), max_epochs=10)
    assert len(hist) == int(g["epochs"][0])
    for e, h in enumerate(hist):
        assert trained[e] == [int(x) for x in g[f"members{e}"]]
        assert h["ensemble"] == _keys(g[f"ensemble{e}"])
        assert h["removed"] == [int(x) for x in g.get(f"removed{e}", [])]
    assert [inst.key for inst in ens] == _keys(g["final"])
    assert s == float(g["final_score"][0])


def _first_stop(seq, patience):
    """First index e at which none of seq[e-patience .. e] is a strict new minimum
    of the sequence so far (non-finite values never are), or None."""
    for e in range(patience, len(seq)):
        before = [x for x in seq[:e - patience] if math.isfinite(x)]
        prior = min(before) if before else math.inf
        window = [x for x in seq[e - patience:e + 1] if math.isfinite(x)]
        if not window or min(window) >= prior:
            return e
    return None


@settings(max_examples=80, deadline=None)
@given(st.integers(1, 5), st.integers(0, 2), st.integers(0, 2), st.integers(1, 4), st.integers(0, 2 ** 31))
def test_oracle_online_stopping_rules_closed_form(K, p_base, p_ens, m_ens, seed):
    rng = np.random.default_rng(seed)
    E, Nv = 9, 3
    yv = rng.normal(size=Nv)
    vals = rng.normal(size=(E, K, Nv)).round(1)  # coarse values: ties and repeats happen
    vals[rng.random((E, K)) < 0.1] = np.nan       # some epochs score +inf
    trained = []

    def epoch_fn(e, members):
        trained.append(list(members))
        preds = {k: vals[e, k] for k in members}
        return preds, {k: score(preds[k], yv, "reg") for k in members}

    ens, s, hist = run_online(epoch_fn, lambda k: k, K, yv, "reg", p_base, p_ens, m_ens, max_epochs=E)
    # a member leaves exactly at the first epoch whose last p_base + 1 scores hold no new best
    for k in range(K):
        seq = [hist[e]["scores"][k] for e in range(len(hist)) if k in hist[e]["members"]]
        rem = [e for e, h in enumerate(hist) if k in h["removed"]]
        stop = _first_stop(seq, p_base)
        if stop is None:
            assert rem == [] and len(seq) == len(hist)
        else:
            assert rem == [stop] and len(seq) == stop + 1
    # training ends at the first epoch whose last p_ens + 1 ensemble scores hold no new best
    # (or when no member is left, or after E epochs)
    ens_scores = [h["score"] for h in hist]
    stop = _first_stop(ens_scores, p_ens)
    left = [e for e, h in enumerate(hist) if len(h["removed"]) == len(h["members"])]  # nobody left after e
    ends = [x for x in (stop, left[0] if left else None) if x is not None]
    assert len(hist) == (min(ends) + 1 if ends else E)
    # the result is the ensemble of the (first) epoch with the best score
    finite = [(sc, e) for e, sc in enumerate(ens_scores) if math.isfinite(sc)]
    if finite:
        best, e_best = min(finite)
        assert s == best and [i.key for i in ens] == hist[e_best]["ensemble"]
    else:
        assert ens == [] and s == math.inf
    # every ensemble member is a distinct (member, epoch) snapshot from the pool of its epoch
    for e, h in enumerate(hist):
        assert len(set(h["ensemble"])) == len(h["ensemble"]) <= m_ens
        prev = set(hist[e - 1]["ensemble"]) if e else set()
        assert all((k == e and m in h["members"]) or (m, k) in prev for m, k in h["ensemble"])


class ScriptedPack:
    """Stands in for tabpack.Pack: validation values come from a script, the
    selection from the oracle's greedy; records what the driver asks for."""

    def __init__(self, vals, yv, task):
        self.vals, self.yv, self.task = vals, yv, task
        self.K, self.B = vals.shape[1], 4
        self.active = [True] * self.K
        self.epoch = 0
        self.steps = []
        self.trained = []

    def hparams(self):
        return [dict(width=8, dropout=0.0, lr=1e-3, wd=0.0)] * self.K

    def can_bind_data(self):  # the driver then trains without a data copy
        return False

    def train_step(self, X, y, idx, t, loss):
        self.steps.append(t)
        if len(self.trained) <= self.epoch:
            self.trained.append([k for k in range(self.K) if self.active[k]])

    def eval_members(self, Xv, yv):
        e = self.epoch
        pred = torch.full((self.K, len(self.yv)), float("nan"), dtype=torch.float32)
        sc = torch.full((self.K,), float("nan"), dtype=torch.float64)
        for k in range(self.K):
            if self.active[k]:
                pred[k] = torch.from_numpy(self.vals[e, k].astype(np.float32))
                sc[k] = score(pred[k].double().numpy(), self.yv, self.task)
        self.epoch += 1
        return pred, sc

    def select(self, cand, yv, m_ens):
        return greedy_select(cand.double().numpy(), self.yv, self.task, m_ens)

    def get_params(self, k):
        return ("params", k, self.epoch - 1)

    def set_active(self, active):
        self.active = list(active)


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 6), st.integers(0, 2), st.integers(0, 2), st.integers(1, 4),
       st.sampled_from(["reg", "bin"]), st.integers(0, 2 ** 31))
def test_driver_decisions_match_oracle_loop(K, p_base, p_ens, m_ens, task, seed):
    rng = np.random.default_rng(seed)
    E, Nv, N = 8, 5, 12
    if task == "reg":
        yv = rng.normal(size=Nv)
        vals = rng.normal(size=(E, K, Nv)).round(1)
    else:
        yv = (rng.random(Nv) < 0.5).astype(np.float64)
        vals = rng.random(size=(E, K, Nv)).round(1).clip(0.05, 0.95)
    vals = vals.astype(np.float32).astype(np.float64)

    def epoch_fn(e, members):
        preds = {k: vals[e, k] for k in members}
        return preds, {k: score(preds[k], yv, task) for k in members}

    ens, s, hist = run_online(epoch_fn, lambda k: None, K, yv, task, p_base, p_ens, m_ens, max_epochs=E)

    pk = ScriptedPack(vals, yv, task)
    tr = OnlineTrainer.__new__(OnlineTrainer)
    tr.cfg, tr.p_base, tr.p_ens, tr.m_ens, tr.max_epochs = {}, p_base, p_ens, m_ens, E
    tr.pack, tr.hp, tr._infer = pk, pk.hparams(), None
    X = torch.zeros((N, 2))
    tr.fit(X, torch.zeros(N), torch.zeros((Nv, 2)), torch.from_numpy(yv),
           orders=lambda e: torch.zeros((K, N), dtype=torch.int32))
    assert len(tr.history) == len(hist)
    for a, b in zip(tr.history, hist):
        assert a["members"] == b["members"]
        assert a["picks"] == b["picks"]
        assert a["ensemble"] == b["ensemble"]
        assert a["removed"] == b["removed"]
        assert a["improved"] == b["improved"]
        assert a["score"] == b["score"] or (math.isinf(a["score"]) and math.isinf(b["score"]))
    assert pk.trained == [h["members"] for h in hist]
    assert pk.steps == list(range(1, len(hist) * (N // pk.B) + 1))  # global step counter across epochs
    assert [snap.key for snap in tr.ensemble] == [inst.key for inst in ens]
    assert all(snap.params == ("params",) + snap.key for snap in tr.ensemble)
    assert tr.ensemble_score == s


@pytest.mark.parametrize("over", [dict(emb_lo=8, emb_hi=32, emb_step=4), dict(depth_lo=1, depth_hi=3, optimizer="muon"),
                                  dict()])
def test_inference_pack_spec_keeps_every_member_hyperparameter(over):
    # the final-ensemble pack is rebuilt from snapshots (pack_init alone, no
    # device): with periodic embeddings its members need their d_emb and sigma,
    # or the layout (and pack_init's range check) would not match the snapshots
    from paper_2607_05380_amd import configs, tabpack
    from paper_2607_05380_amd.online import Snapshot, inference_spec
    cfg = configs.workload("regression_onehot", K=5, B=256, **over)
    src = tabpack.Pack(cfg)
    hp = src.hparams()
    snaps = [Snapshot(k, 3, hp[k], src.get_params(k), None) for k in (4, 1, 1, 3)]
    icfg, members = inference_spec(cfg, snaps)
    pk = tabpack.Pack(icfg, members=members)
    got = pk.hparams()
    for i, s in enumerate(snaps):
        for key in ("width", "depth", "dropout", "lr", "wd", "d_emb", "sigma", "muon_lr", "t"):
            assert got[i][key] == hp[s.member][key], (key, i)
        assert pk.param_count(i) == src.param_count(s.member)
        pk.set_params(i, s.params)
        for a, b in zip(pk.get_params(i), s.params):
            if isinstance(a, dict):
                for n in a:
                    np.testing.assert_array_equal(a[n], b[n])
            else:
                np.testing.assert_array_equal(a[0], b[0])
                np.testing.assert_array_equal(a[1], b[1])
