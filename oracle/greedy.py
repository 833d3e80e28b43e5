"""Greedy ensemble selection, step by step as §3.5 (Ensemble) describes it.

1. The first member is the single candidate with the best ensemble score on
   the validation set.
2. Each further iteration adds the candidate (not yet in the ensemble -- no
   replacement) whose addition gives the best score of the averaged ensemble;
   the candidates' own scores play no part.
3. Stop once m_ens members are in, or when the best addition does not improve
   the score.

Readings where the text is silent: ties go to the lowest candidate index;
"improve" means a strict decrease; a non-finite score counts as +inf; the
first pick must have a finite score (if none has, nothing is selected).
Ensemble predictions are plain averages of the candidates' per-row values
(probabilities for classification), scored with ``pack.score``.
"""
import numpy as np

from .pack import score


def greedy_select(cand, yv, task, m_ens):
    """Returns (selected indices in pick order, ensemble score)."""
    cand = np.asarray(cand, dtype=np.float64)
    C = cand.shape[0]
    chosen = []
    total = np.zeros(cand.shape[1])
    best = float("inf")
    while len(chosen) < min(m_ens, C):
        n = len(chosen)
        trial = np.full(C, np.inf)
        for c in range(C):
            if c not in chosen:
                trial[c] = score((total + cand[c]) / (n + 1), yv, task)
        c_star = int(np.argmin(trial))
        s = trial[c_star]
        if not np.isfinite(s) or (n > 0 and s >= best):
            break
        chosen.append(c_star)
        total = total + cand[c_star]
        best = s
    return chosen, best
