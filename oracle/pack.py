"""The pack: K independent base models, one Python loop iteration each.

§3.3 Model Pack: packing must reproduce the original base models exactly, so
the reference result of a packed step is simply K separate MLP steps.
§3.6 Training: member k trains on its own base batch X[idx[k]], and the pack's
objective is the *sum* of the members' batch-mean losses (losses aggregated,
predictions not), which gives every member exactly its standalone gradient.
§3.4 Optimizer Pack: member k is updated by its own AdamW with (lr_k, wd_k).
"""
import numpy as np

from . import embed, mlp, muon
from .sampling import init_member, member_depth, sample_hparams


class OraclePack:
    """Holds fp64 parameters and AdamW moments of K members.

    precision "fp64" is the exact definition; "bf16" applies the bf16
    mixed-precision rounding policy described in ``mlp`` to the matrix-product
    operands (parameters, moments and updates stay float64).
    """

    def __init__(self, cfg, hparams=None, params=None, precision="fp64", members=None):
        """``members``: optional subset of member indices to materialise (the
        others stay None and must not be stepped)."""
        self.cfg = dict(cfg)
        self.rnd = mlp.to_bf16 if precision == "bf16" else None
        self.hp = hparams if hparams is not None else sample_hparams(cfg)
        keep = set(range(len(self.hp)) if members is None else members)
        # periodic feature embeddings (App. F) when the members have d_emb
        self.use_emb = bool(self.hp) and "d_emb" in self.hp[0]
        self.emb = [embed.init_embedding(cfg, k, h["d_emb"], h["sigma"]) if self.use_emb and k in keep else None
                    for k, h in enumerate(self.hp)]
        if params is None:
            params = [init_member(cfg, k, h["width"], member_depth(cfg, h),
                                  cfg["d_in"] * h["d_emb"] if self.use_emb else None) if k in keep else None
                      for k, h in enumerate(self.hp)]
        self.params = [None if p is None else [(W.copy(), b.copy()) for W, b in p] for p in params]
        self.m = [None if p is None else [(np.zeros_like(W), np.zeros_like(b)) for W, b in p] for p in self.params]
        self.v = [None if p is None else [(np.zeros_like(W), np.zeros_like(b)) for W, b in p] for p in self.params]
        self.emb_m = [None if e is None else {n: np.zeros_like(a) for n, a in e.items()} for e in self.emb]
        self.emb_v = [None if e is None else {n: np.zeros_like(a) for n, a in e.items()} for e in self.emb]
        self.t = 0
        self.last_grads = None
        self.last_emb_grads = None
        self.last_hint_stats = None

    def masks(self, k, step):
        c, h = self.cfg, self.hp[k]
        return [mlp.dropout_mask(c["seed"], k, step, l + 1, c["B"], h["width"], h["t"])
                for l in range(member_depth(c, h))]

    def member_step(self, k, X, y, idx_k, step, hints=None):
        """Forward, loss, backward and the optimizer step for member k; returns
        (loss, grads).  With cfg["optimizer"] == "muon" the hidden weights take a
        Muon step (learning rate hp["muon_lr"], momentum buffer in ``m``) and
        every other parameter an AdamW step; otherwise everything is AdamW.
        hints: optional per-layer ReLU decisions of another implementation
        (``mlp.relu_derivative``); the counts land in last_hint_stats[k]."""
        c, h = self.cfg, self.hp[k]
        use_muon = c.get("optimizer", "adamw") == "muon"
        depth = len(self.params[k]) - 1
        rows = np.asarray(idx_k, dtype=np.int64)
        masks = self.masks(k, step)
        H0 = X[rows]
        if self.use_emb:
            H0, ecache = embed.embed(H0, self.emb[k])
        Y, cache = mlp.forward(self.params[k], H0, masks, h["s"], rnd=self.rnd)
        loss, dY = mlp.loss_and_dy(Y, y[rows], c["task"])
        stats = {}
        if self.last_hint_stats is None:
            self.last_hint_stats = [None] * len(self.hp)
        self.last_hint_stats[k] = stats
        if self.use_emb:
            grads, dE = mlp.backward(self.params[k], cache, dY, masks, h["s"], input_grad=True, hints=hints,
                                     stats=stats)
            eg = embed.embed_backward(dE, ecache, self.emb[k])
            self.last_emb_grads[k] = eg
            args = (step, h["lr"], h["wd"], c["beta1"], c["beta2"], c["eps"])
            for n in ("w", "b", "alpha", "beta"):  # AdamW, decayed like the weights
                self.emb[k][n], self.emb_m[k][n], self.emb_v[k][n] = mlp.adamw_step(
                    self.emb[k][n], eg[n], self.emb_m[k][n], self.emb_v[k][n], *args)
        else:
            grads = mlp.backward(self.params[k], cache, dY, masks, h["s"], hints=hints, stats=stats)
        new_p, new_m, new_v = [], [], []
        for i, ((W, b), (gW, gb), (mW, mb), (vW, vb)) in enumerate(
                zip(self.params[k], grads, self.m[k], self.v[k])):
            args = (step, h["lr"], h["wd"], c["beta1"], c["beta2"], c["eps"])
            if use_muon and i < depth:
                W2, mW2 = muon.muon_step(W, gW, mW, h["muon_lr"], h["wd"], c.get("muon_momentum", 0.95),
                                         bool(c.get("muon_nesterov", 1)), int(c.get("ns_steps", 5)),
                                         rnd=self.rnd)
                vW2 = vW
            else:
                W2, mW2, vW2 = mlp.adamw_step(W, gW, mW, vW, *args)
            b2, mb2, vb2 = mlp.adamw_step(b, gb, mb, vb, *args, decay=bool(c["decay_bias"]))
            new_p.append((W2, b2))
            new_m.append((mW2, mb2))
            new_v.append((vW2, vb2))
        self.params[k], self.m[k], self.v[k] = new_p, new_m, new_v
        return loss, grads

    def train_step(self, X, y, idx, step, members=None, hints=None):
        """One step for every member (or for ``members`` only); returns losses [K].

        ``step`` is the 1-based AdamW step t, also the dropout counter.
        Members left out keep their state; their loss is reported as NaN.
        hints: optional {member: per-layer ReLU decisions} (``member_step``).
        """
        K = self.cfg["K"]
        X = np.asarray(X, dtype=np.float64)
        losses = np.full(K, np.nan)
        self.last_grads = [None] * K
        self.last_emb_grads = [None] * K
        self.last_hint_stats = [None] * K
        for k in (range(K) if members is None else members):
            losses[k], self.last_grads[k] = self.member_step(k, X, y, idx[k], step,
                                                             None if hints is None else hints.get(k))
        self.t = step
        return losses

    def predict(self, k, Xv):
        """Output of member k on Xv (no dropout)."""
        H0 = np.asarray(Xv, dtype=np.float64)
        if self.use_emb:
            H0, _ = embed.embed(H0, self.emb[k])
        Y, _ = mlp.forward(self.params[k], H0, rnd=self.rnd)
        return Y

    def predict_values(self, k, X):
        """Member k's prediction values on X, [N, d_out] (see ``prediction_values``)."""
        return prediction_values(self.predict(k, X), self.cfg["task"])

    def eval_members(self, Xv, yv, members=None):
        """(pred [K, Nv], score [K]) as in ``prediction`` and ``score``."""
        K = self.cfg["K"]
        preds = np.full((K, len(yv)), np.nan)
        scores = np.full(K, np.nan)
        for k in (range(K) if members is None else members):
            preds[k] = prediction(self.predict(k, Xv), yv, self.cfg["task"])
            scores[k] = score(preds[k], yv, self.cfg["task"])
        return preds, scores


def prediction_values(Y, task):
    """All prediction values of one member, [N, d_out]: the outputs (regression),
    P(class 1) (binary) or the softmax probabilities (multiclass).  The final
    ensemble averages these across its members (§3.5: ensembles average
    predictions; probabilities for classification)."""
    Y = np.asarray(Y, dtype=np.float64)
    if task == mlp.TASK_REG:
        return Y
    if task == mlp.TASK_BIN:
        return 1.0 / (1.0 + np.exp(-Y))
    mx = Y.max(axis=1, keepdims=True)
    P = np.exp(Y - mx)
    return P / P.sum(axis=1, keepdims=True)


def prediction(Y, yv, task):
    """Per-row candidate value used for scoring and ensembling.

    Regression: the output itself.  Binary: the probability of class 1.
    Multiclass: the probability assigned to the true class (ensembles average
    probabilities, and the cross-entropy of an average needs only that column).
    """
    if task == mlp.TASK_REG:
        return Y[:, 0]
    if task == mlp.TASK_BIN:
        return 1.0 / (1.0 + np.exp(-Y[:, 0]))
    mx = Y.max(axis=1, keepdims=True)
    P = np.exp(Y - mx)
    P /= P.sum(axis=1, keepdims=True)
    return P[np.arange(len(yv)), np.asarray(yv, dtype=np.int64)]


PROB_CLIP = 1e-15


def score(pred, yv, task):
    """Validation score (lower is better): RMSE, binary CE, or multiclass CE.

    Probabilities are clipped to [1e-15, 1 - 1e-15] before the logarithm.  A
    non-finite result is reported as +inf.
    """
    p = np.asarray(pred, dtype=np.float64)
    if task == mlp.TASK_REG:
        d = p - np.asarray(yv, dtype=np.float64)
        s = np.sqrt(np.mean(d * d))
    elif task == mlp.TASK_BIN:
        y = np.asarray(yv, dtype=np.float64)
        q = np.clip(p, PROB_CLIP, 1.0 - PROB_CLIP)
        s = np.mean(-y * np.log(q) - (1.0 - y) * np.log1p(-q))
    else:
        s = np.mean(-np.log(np.clip(p, PROB_CLIP, 1.0)))
    return float(s) if np.isfinite(s) else float("inf")
