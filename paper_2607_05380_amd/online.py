"""Online training of a pack around the packed step (arXiv 2607.05380,
Sections 3.5 and 3.6): per-epoch validation of every member, early stopping
of base models (removal from the pack), the online greedy ensemble rebuilt
each epoch from the members' latest states plus the previous ensemble, early
stopping of the ensemble, a store of the selected members' snapshots and the
final ensemble's prediction.

The driver keeps only control state -- patience counters, which snapshots
form the ensemble -- and moves data between device buffers.  Every number
comes from the library's kernels: the training steps, the validation values
and scores (pack_eval_members), the greedy selection (pack_select) and the
ensemble prediction (pack_predict on a pack rebuilt from the snapshots).

Rules (the paper leaves the details open; these are the readings taken):
* an epoch trains every member still in the pack on its own permutation of
  the training rows, drop-last batches of B, with the global AdamW step
  counter continuing across epochs;
* the pool is the latest states of the members still in the pack (increasing
  member index) followed by the previous ensemble's snapshots (pick order);
  a member's snapshots from different epochs are different candidates;
* "improves" means a strict decrease of the score; a non-finite score never
  improves; a member's first finite score is an improvement;
* after the selection, a member without improvement for p_base + 1
  consecutive epochs leaves the pack (pack_set_active);
* training stops after p_ens + 1 consecutive epochs without improvement of
  the ensemble score, when no member is left, or after max_epochs;
* the final ensemble is the one of the epoch with the best ensemble score.
"""
import math

from . import synth, tabpack


class Snapshot:
    """A member's state at the end of one epoch, kept while it is in an
    ensemble: its hyperparameters, parameters (host, dense layout) and its
    validation values (device fp32 [Nv])."""

    def __init__(self, member, epoch, hp, params, val):
        self.member, self.epoch, self.hp, self.params, self.val = member, epoch, hp, params, val

    @property
    def key(self):
        return (self.member, self.epoch)


def inference_spec(cfg, snapshots):
    """(config, explicit member hyperparameters) of a pack holding one member per
    snapshot, in order: every sampled hyperparameter of the snapshot's member is
    kept, the embedding's d_emb and sigma included, so that the pack's layout
    matches the snapshots' parameters."""
    out = dict(cfg, K=len(snapshots), keep_grads=0)
    hps = []
    for s in snapshots:
        hp = dict(width=s.hp["width"], dropout=s.hp["dropout"], lr=s.hp["lr"], wd=s.hp["wd"], depth=s.hp["depth"],
                  muon_lr=s.hp.get("muon_lr", 0.0))
        if s.hp.get("d_emb"):
            hp["d_emb"], hp["sigma"] = s.hp["d_emb"], s.hp["sigma"]
        hps.append(hp)
    return out, hps


class OnlineTrainer:
    def __init__(self, cfg, p_base=16, p_ens=32, m_ens=32, max_epochs=1000, members=None, device="cuda"):
        self.cfg = dict(cfg)
        self.p_base, self.p_ens, self.m_ens, self.max_epochs = p_base, p_ens, m_ens, max_epochs
        self.device = device
        self.pack = tabpack.Pack(self.cfg, members=members).bind(device)
        self.hp = self.pack.hparams()
        self.history = []
        self.ensemble = []
        self.ensemble_score = math.inf
        self._infer = None

    def fit(self, X, y, Xv, yv, orders=None):
        """X, y: training rows (device); Xv, yv: validation rows (device).
        orders(epoch) -> device int32 [K, N] per-member row permutations
        (default: the seeded device generator of ``synth``)."""
        import torch
        K, B = self.pack.K, self.pack.B
        N = X.shape[0]
        steps = N // B
        if steps < 1:
            raise ValueError(f"{N} training rows give no full batch of {B}")
        if orders is None:
            def orders(e):
                return synth.epoch_orders_device(self.cfg, e, N, X.device)
        if self.pack.can_bind_data():  # the first layer reads its rows straight from X
            self.pack.bind_data(X)
        active = [True] * K
        best = [math.inf] * K
        bad = [0] * K
        prev = []
        best_ens, best_score, bad_ens = [], math.inf, 0
        loss = torch.empty(K, dtype=torch.float32, device=X.device)
        t = 0
        self.history = []
        for e in range(self.max_epochs):
            members = [k for k in range(K) if active[k]]
            order = orders(e)
            for s in range(steps):
                t += 1
                idx = order[:, s * B:(s + 1) * B].contiguous()
                self.pack.train_step(X, y, idx, t, loss)
            pred, score = self.pack.eval_members(Xv, yv)
            scores = score.cpu().tolist()
            rows = torch.tensor(members, dtype=torch.long, device=pred.device)
            cand = torch.cat([pred.index_select(0, rows)] + [snap.val[None] for snap in prev]).contiguous()
            picks, ens_score = self.pack.select(cand, yv, self.m_ens)
            ens = []
            for i in picks:
                if i < len(members):
                    k = members[i]
                    ens.append(Snapshot(k, e, self.hp[k], self.pack.get_params(k), pred[k].clone()))
                else:
                    ens.append(prev[i - len(members)])
            removed = []
            for k in members:
                sk = scores[k]
                if math.isfinite(sk) and sk < best[k]:
                    best[k], bad[k] = sk, 0
                else:
                    bad[k] += 1
                if bad[k] > self.p_base:
                    active[k] = False
                    removed.append(k)
            if removed:
                self.pack.set_active(active)
            improved = math.isfinite(ens_score) and ens_score < best_score
            if improved:
                best_ens, best_score, bad_ens = ens, ens_score, 0
            else:
                bad_ens += 1
            self.history.append(dict(epoch=e, members=members, scores={k: scores[k] for k in members},
                                     picks=list(picks), ensemble=[snap.key for snap in ens], score=ens_score,
                                     removed=removed, improved=improved, steps=steps))
            prev = ens
            if bad_ens > self.p_ens or not any(active):
                break
        self.ensemble, self.ensemble_score = best_ens, best_score
        self._infer = None
        return self

    def inference_pack(self):
        """A pack holding exactly the final ensemble's snapshots (one member each)."""
        if not self.ensemble:
            raise RuntimeError("no ensemble: fit() selected nothing")
        if self._infer is None:
            cfg, hps = inference_spec(self.cfg, self.ensemble)
            pk = tabpack.Pack(cfg, members=hps).bind(self.device)
            for i, snap in enumerate(self.ensemble):
                pk.set_params(i, snap.params)
            self._infer = pk
        return self._infer

    def predict(self, X):
        """The final ensemble's prediction on X (device fp32 [N, d_in]): the mean
        of its snapshots' outputs / P(class 1) / class probabilities, [N, d_out]."""
        return self.inference_pack().predict(X, ensemble=True)
