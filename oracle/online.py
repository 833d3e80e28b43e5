"""The online training loop around the packed step, as §3.5 and §3.6 describe it.

TEST INFRASTRUCTURE ONLY (see the package header): written from the paper,
independently of the library's driver.

Per epoch (§3.6 Training, §3.5 Online ensemble):

1. Every member still in the pack trains one epoch on its own batch sequence.
2. Every such member is scored on the validation set.
3. The candidate pool is the latest state of every member still in the pack
   (in increasing member order) followed by the previous epoch's ensemble
   members (in their pick order); the ensemble is rebuilt from scratch by
   greedy selection over that pool.  Instances of one member from different
   epochs are distinct candidates.
4. Early stopping of base models: a member whose validation score has not
   improved for p_base + 1 consecutive epochs is removed from the pack.
5. Early stopping of the ensemble: training stops after p_ens + 1 consecutive
   epochs without improvement of the ensemble's validation score.

Readings where the text is silent (the same in the library's driver):
* "improve" is a strict decrease; a non-finite score never improves;
* a member's patience counts epochs since its best score so far (the first
  finite score is an improvement over "no score");
* selection (step 3) sees this epoch's states of every member in the pack,
  including members that step 4 then removes -- their state at removal stays
  in the pool only through the ensemble;
* the result is the ensemble of the epoch with the best ensemble score;
* training also ends when no member is left or after max_epochs epochs.
"""
import numpy as np

from .greedy import greedy_select


class Instance:
    """One selected snapshot of a member: (member, epoch), its validation
    values and its parameters at that epoch."""

    def __init__(self, member, epoch, pred, params):
        self.member, self.epoch = member, epoch
        self.pred = np.asarray(pred, dtype=np.float64)
        self.params = params

    @property
    def key(self):
        return (self.member, self.epoch)


def run_online(epoch_fn, snapshot_fn, K, yv, task, p_base, p_ens, m_ens, max_epochs):
    """Runs the loop.

    epoch_fn(epoch, members) trains the listed members for one epoch and
    returns (preds, scores): preds[k] the validation values of member k (the
    per-row values ensembles average), scores[k] its validation score.
    snapshot_fn(k) returns member k's current parameters.

    Returns (best ensemble as a list of Instance, its score, history), history
    holding one dict per epoch.
    """
    active = [True] * K
    best = [float("inf")] * K
    bad = [0] * K
    prev = []
    best_ens, best_score, bad_ens = [], float("inf"), 0
    history = []
    for e in range(max_epochs):
        members = [k for k in range(K) if active[k]]
        preds, scores = epoch_fn(e, members)
        cand = [np.asarray(preds[k], dtype=np.float64) for k in members] + [inst.pred for inst in prev]
        picks, ens_score = greedy_select(np.stack(cand), yv, task, m_ens)
        ens = []
        for i in picks:
            if i < len(members):
                k = members[i]
                ens.append(Instance(k, e, preds[k], snapshot_fn(k)))
            else:
                ens.append(prev[i - len(members)])
        removed = []
        for k in members:
            s = scores[k]
            if np.isfinite(s) and s < best[k]:
                best[k], bad[k] = s, 0
            else:
                bad[k] += 1
            if bad[k] > p_base:
                active[k] = False
                removed.append(k)
        improved = bool(np.isfinite(ens_score) and ens_score < best_score)
        if improved:
            best_ens, best_score, bad_ens = ens, ens_score, 0
        else:
            bad_ens += 1
        history.append(dict(epoch=e, members=members, scores={k: scores[k] for k in members},
                            picks=list(picks), ensemble=[inst.key for inst in ens], score=ens_score,
                            removed=removed, improved=improved))
        prev = ens
        if bad_ens > p_ens or not any(active):
            break
    return best_ens, best_score, history


def ensemble_predict(instances, predict_fn):
    """Mean of predict_fn(instance) ([N, d_out] each) over the ensemble's instances."""
    vals = [np.asarray(predict_fn(inst), dtype=np.float64) for inst in instances]
    return np.mean(np.stack(vals), axis=0)
