"""Seeded candidate matrices for the selection parity tests, screened for
near-ties: the greedy rule (Section 3.5, Ensemble) compares fp64 scores, and
the GPU sums them in another order than the oracle, so a case is kept only if
at every iteration the best candidate beats the runner-up, and the stop test
(best against the current ensemble score) is decided, by at least 1e-9 of
|best|.  Selected indices must then agree exactly."""
import numpy as np

from oracle.pack import score

NEAR_TIE = 1e-9


def greedy_margins(cand, y, task, m_ens):
    """The oracle's greedy iterations with their decision margins: returns the
    smallest relative gap over the iterations, between the best and the
    runner-up candidate and between the best and the ensemble score it must
    improve (inf when a choice is uncontested)."""
    cand = np.asarray(cand, dtype=np.float64)
    C = cand.shape[0]
    chosen, total, best, gap = [], np.zeros(cand.shape[1]), np.inf, np.inf
    while len(chosen) < min(m_ens, C):
        n = len(chosen)
        trial = np.array([score((total + cand[c]) / (n + 1), y, task) if c not in chosen else np.inf
                          for c in range(C)])
        order = np.argsort(trial, kind="stable")
        s = trial[order[0]]
        if not np.isfinite(s):
            break
        scale = max(abs(s), 1e-300)
        if len(order) > 1 and np.isfinite(trial[order[1]]):
            gap = min(gap, (trial[order[1]] - s) / scale)
        if n > 0:
            gap = min(gap, abs(best - s) / scale)
            if s >= best:
                break
        chosen.append(int(order[0]))
        total = total + cand[order[0]]
        best = s
    return gap


def make_case(task, C, Nv, seed):
    """Candidate predictions [C, Nv] (fp32) and labels for one task."""
    rng = np.random.default_rng(seed)
    if task == "reg":
        y = rng.standard_normal(Nv).astype(np.float32)
        cand = (y[None, :] * rng.uniform(0.2, 1.0, (C, 1))
                + rng.standard_normal((C, Nv)) * rng.uniform(0.3, 1.5, (C, 1))).astype(np.float32)
    elif task == "bin":
        y = (rng.random(Nv) < 0.4).astype(np.float32)
        cand = np.clip(0.5 * y[None, :] + 0.5 * rng.random((C, Nv)), 0, 1).astype(np.float32)
    else:
        y = rng.integers(0, 10, Nv).astype(np.int32)
        cand = rng.uniform(0.02, 0.9, (C, Nv)).astype(np.float32)
    return cand, y


def screened_cases(task, C, Nv, m_ens, seeds, count=1):
    """The first ``count`` cases over ``seeds`` whose greedy run has no near-tie:
    [(cand, y, smallest relative gap)]."""
    out = []
    for seed in seeds:
        cand, y = make_case(task, C, Nv, seed)
        gap = greedy_margins(cand, y, task, m_ens)
        if gap >= NEAR_TIE:
            out.append((cand, y, gap))
            if len(out) == count:
                return out
    raise RuntimeError(f"no near-tie-free case among the seeds for {task} C={C} Nv={Nv}")
