"""Pins of the oracle's hyperparameter sampler and greedy selection (CPU only)."""
import itertools
import os

import numpy as np
import pytest
from hypothesis import given, settings, strategies as st
from scipy.stats import kstest

from oracle.greedy import greedy_select
from oracle.pack import score
from oracle.sampling import sample_hparams

CFG = dict(seed=2607053805, K=4000, width_lo=256, width_hi=1024, dropout_lo=0.0, dropout_hi=0.5,
           lr_lo=1e-4, lr_hi=3e-3, wd_lo=1e-5, wd_hi=1e-2)


def test_sampler_ranges_and_distributions():
    hp = sample_hparams(CFG)
    w = np.array([h["width"] for h in hp])
    assert w.min() >= 256 and w.max() <= 1024 and len(np.unique(w)) > 600
    assert kstest((w - 256 + 0.5) / 769, "uniform").pvalue > 1e-4
    p = np.array([h["dropout"] for h in hp])
    assert kstest(p / 0.5, "uniform").pvalue > 1e-4
    for key, lo, hi in (("lr", 1e-4, 3e-3), ("wd", 1e-5, 1e-2)):
        v = np.array([h[key] for h in hp])
        assert v.min() >= lo and v.max() <= hi
        assert kstest((np.log(v) - np.log(lo)) / (np.log(hi) - np.log(lo)), "uniform").pvalue > 1e-4
    for h in hp[:50]:
        assert h["t"] == int(np.floor(h["dropout"] * 2 ** 16)) and h["s"] == 1 / (1 - h["dropout"])
    assert sample_hparams(dict(CFG, K=5)) == hp[:5]
    assert sample_hparams(dict(CFG, K=5, seed=1)) != hp[:5]


def test_sampler_depths():
    # depth ~ UniformInt[lo, hi]: every value in range, counts within 5 sigma of
    # the binomial; the other draws do not change when a depth range is added
    hp = sample_hparams(dict(CFG, L=4, depth_lo=2, depth_hi=4))
    d = np.array([h["depth"] for h in hp])
    assert d.min() == 2 and d.max() == 4
    n, p = len(d), 1.0 / 3.0
    for v in (2, 3, 4):
        assert abs((d == v).sum() - n * p) <= 5 * np.sqrt(n * p * (1 - p))
    base = sample_hparams(dict(CFG, L=4))
    assert all(h["depth"] == 4 for h in base)
    assert [{k: h[k] for k in ("width", "dropout", "lr", "wd")} for h in hp] == \
        [{k: h[k] for k in ("width", "dropout", "lr", "wd")} for h in base]
    one = sample_hparams(dict(CFG, K=50, L=3, depth_lo=3, depth_hi=3))
    assert all(h["depth"] == 3 for h in one)


def test_degenerate_ranges():
    hp = sample_hparams(dict(CFG, K=20, width_lo=64, width_hi=64, dropout_lo=0.0, dropout_hi=0.0,
                             lr_lo=1e-3, lr_hi=1e-3))
    assert all(h["width"] == 64 and h["dropout"] == 0.0 and h["t"] == 0 and h["lr"] == 1e-3 for h in hp)


def _golden():
    d = {}
    for line in open(os.path.join(os.path.dirname(__file__), "golden", "greedy_hand.txt")):
        if line.startswith("#") or not line.strip():
            continue
        k, *v = line.split()
        d[k] = v
    return d


def test_greedy_hand_example():
    g = _golden()
    cand = np.array([float(x) for x in g["cand"]])[:, None]
    sel, s = greedy_select(cand, np.array([float(g["y"][0])]), g["task"][0], int(g["m_ens"][0]))
    assert sel == [int(x) for x in g["selected"]]
    assert s == float(g["score"][0])


def _brute(cand, y, task, m_ens):
    # Enumerate every (ensemble-so-far + one candidate) subset and score its mean from scratch.
    S, best = [], np.inf
    for _ in range(min(m_ens, len(cand))):
        trials = [(score(np.mean(cand[S + [c]], axis=0), y, task), c)
                  for c in range(len(cand)) if c not in S]
        s, c = min(trials, key=lambda t: (t[0], t[1]))
        if not np.isfinite(s) or (S and s >= best):
            break
        S.append(c)
        best = s
    return S, best


@settings(max_examples=60, deadline=None)
@given(st.integers(1, 8), st.integers(1, 40), st.integers(1, 10), st.sampled_from(["reg", "bin", "multi"]),
       st.integers(0, 2 ** 31))
def test_greedy_matches_brute_force(C, N, m_ens, task, seed):
    rng = np.random.default_rng(seed)
    if task == "reg":
        cand, y = rng.standard_normal((C, N)), rng.standard_normal(N)
    elif task == "bin":
        cand, y = rng.random((C, N)), (rng.random(N) < 0.5).astype(float)
    else:
        cand, y = rng.random((C, N)), rng.integers(0, 3, N)
    sel, s = greedy_select(cand, y, task, m_ens)
    sel_b, s_b = _brute(cand, y, task, m_ens)
    assert sel == sel_b
    assert s == pytest.approx(s_b, rel=1e-12)
    # invariants: first pick is the best single model; no repeats; size bound; strict improvement
    singles = [score(c, y, task) for c in cand]
    assert sel[0] == int(np.argmin(singles))
    assert len(set(sel)) == len(sel) <= m_ens
    prev = np.inf
    for i in range(1, len(sel) + 1):
        cur = score(np.mean(cand[sel[:i]], axis=0), y, task)
        assert cur < prev
        prev = cur


def test_greedy_skips_non_finite_candidates():
    y = np.zeros(3)
    cand = np.array([[np.nan, 0, 0], [0.5, 0.5, 0.5], [np.inf, 1, 1]])
    assert greedy_select(cand, y, "reg", 3) == ([1], 0.5)
    assert greedy_select(cand[[0, 2]], y, "reg", 3) == ([], float("inf"))


def test_greedy_single_pick_equals_argmin_of_library_scores():
    from sklearn.metrics import mean_squared_error
    rng = np.random.default_rng(8)
    cand, y = rng.standard_normal((12, 30)), rng.standard_normal(30)
    sel, s = greedy_select(cand, y, "reg", 1)
    lib = [np.sqrt(mean_squared_error(y, c)) for c in cand]
    assert sel == [int(np.argmin(lib))] and s == pytest.approx(min(lib), rel=1e-13)
