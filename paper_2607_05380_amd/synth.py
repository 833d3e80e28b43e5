"""Seeded synthetic tabular data and batch orders.

Holds no arithmetic of the packed method: it only makes inputs (features,
targets, per-member batch index lists) that both the HIP library and the CPU
oracle consume.  Random numbers come from numpy Generator(Philox(key=[seed,
stream])) with stream 0 = data and stream 4 = batch order.

Recipes (per workload, see ``configs``):
  normal              d_in columns ~ N(0, 1)
  onehot              (d_in - 16) columns ~ N(0,1) followed by 4 categorical
                      features uniform over 4 levels, one-hot encoded (16 cols)
  lognormal_rankgauss exp(N(0,1)) columns mapped by the rank-Gauss transform
                      Phi^-1((rank + 0.5) / N_train) fitted on the training
                      rows and applied to validation rows by interpolation
  zero_inflated       N(0,1) columns; a seeded 20% of the columns have each
                      entry set to exactly 0 with probability 0.5
  block_correlated    blocks of 30 columns, x = sqrt(.6) z_block + sqrt(.4) e
Teacher: a tanh MLP with 32 hidden units, W ~ N(0, 1/fan_in), zero biases.
Labels: 'sign' -> 1[teacher > 0]; 'argmax' -> argmax of d_out teacher logits;
'teacher_noise' -> teacher + N(0, 0.1^2), standardised on train;
'teacher_t3' -> unit-variance teacher + 0.1 * Student-t(3), standardised.
"""
import numpy as np
from scipy.special import ndtri


def _rng(seed, stream):
    return np.random.Generator(np.random.Philox(key=np.array([seed, stream], dtype=np.uint64)))


def _features(cfg, rng, n):
    d = cfg["d_in"]
    kind = cfg["features"]
    if kind in ("normal", "lognormal_rankgauss", "zero_inflated"):
        X = rng.standard_normal((n, d), dtype=np.float32)
        if kind == "lognormal_rankgauss":
            np.exp(X, out=X)
        elif kind == "zero_inflated":
            cols = rng.choice(d, size=max(1, int(round(0.2 * d))), replace=False)
            for c in np.sort(cols):
                X[rng.random(n) < 0.5, c] = 0.0
        return X
    if kind == "onehot":
        n_num = d - 16
        X = np.zeros((n, d), dtype=np.float32)
        X[:, :n_num] = rng.standard_normal((n, n_num), dtype=np.float32)
        for j in range(4):
            lev = rng.integers(0, 4, size=n)
            X[np.arange(n), n_num + 4 * j + lev] = 1.0
        return X
    if kind == "block_correlated":
        X = np.empty((n, d), dtype=np.float32)
        nb = (d + 29) // 30
        chunk = 65536
        for r0 in range(0, n, chunk):
            r1 = min(n, r0 + chunk)
            z = rng.standard_normal((r1 - r0, nb), dtype=np.float32)
            e = rng.standard_normal((r1 - r0, d), dtype=np.float32)
            zb = np.repeat(z, 30, axis=1)[:, :d]
            X[r0:r1] = np.float32(np.sqrt(0.6)) * zb + np.float32(np.sqrt(0.4)) * e
        return X
    raise ValueError(kind)


def _rank_gauss(Xtr, Xva):
    n = Xtr.shape[0]
    out_tr = np.empty_like(Xtr)
    out_va = np.empty_like(Xva)
    q = ndtri((np.arange(n) + 0.5) / n)
    for j in range(Xtr.shape[1]):
        order = np.argsort(Xtr[:, j], kind="stable")
        col = np.empty(n)
        col[order] = q
        out_tr[:, j] = col
        out_va[:, j] = np.interp(Xva[:, j], Xtr[order, j], q)
    return out_tr, out_va


def _teacher(rng, X, d_out):
    d = X.shape[1]
    W1 = rng.standard_normal((d, 32)) / np.sqrt(d)
    W2 = rng.standard_normal((32, d_out)) / np.sqrt(32)
    out = np.empty((X.shape[0], d_out))
    for r0 in range(0, X.shape[0], 65536):
        out[r0:r0 + 65536] = np.tanh(X[r0:r0 + 65536] @ W1) @ W2
    return out


def make_data(cfg, n_train=None, n_val=None):
    """(X_train fp32 [Ntr, d_in], y_train, X_val, y_val); y is fp32 or int32 labels."""
    n_tr = cfg["n_train"] if n_train is None else n_train
    n_va = cfg["n_val"] if n_val is None else n_val
    rng = _rng(cfg["seed"], 0)
    X = _features(cfg, rng, n_tr + n_va)
    Xtr, Xva = X[:n_tr], X[n_tr:]
    if cfg["features"] == "lognormal_rankgauss":
        Xtr, Xva = _rank_gauss(Xtr, Xva)
    Xtr = np.ascontiguousarray(Xtr, dtype=np.float32)
    Xva = np.ascontiguousarray(Xva, dtype=np.float32)
    lab = cfg["label"]
    T = _teacher(rng, np.concatenate([Xtr, Xva]), cfg["d_out"])
    if lab == "sign":
        y = (T[:, 0] > 0).astype(np.float32)
    elif lab == "argmax":
        y = np.argmax(T, axis=1).astype(np.int32)
    else:
        t = T[:, 0]
        if lab == "teacher_noise":
            t = t + 0.1 * rng.standard_normal(len(t))
        else:
            t = t / max(np.std(t[:n_tr]), 1e-12) + 0.1 * rng.standard_t(3, size=len(t))
        mu, sd = t[:n_tr].mean(), t[:n_tr].std()
        y = ((t - mu) / max(sd, 1e-12)).astype(np.float32)
    return Xtr, y[:n_tr], Xva, y[n_tr:]


def epoch_orders(cfg, epoch, n_train):
    """Per-member permutations of the training rows for one epoch: int64 [K, n_train]."""
    rng = _rng(cfg["seed"], 4 + (int(epoch) << 8))
    return np.stack([rng.permutation(n_train) for _ in range(cfg["K"])])


def batch_indices(orders, step_in_epoch, B):
    """idx [K, B] int32 of one step (drop-last batching of each member's order)."""
    s = int(step_in_epoch)
    return np.ascontiguousarray(orders[:, s * B:(s + 1) * B], dtype=np.int32)


# ----------------------------------------------------------------------------
# Device-side generator for full-size workloads (same recipes, torch's seeded
# generator on the GPU instead of numpy's; the values differ from make_data's).
# ----------------------------------------------------------------------------
def make_data_device(cfg, device="cuda", n_train=None, n_val=None, chunk=131072):
    """(X_train, y_train, X_val, y_val) as device tensors, generated on ``device``."""
    import torch
    n_tr = cfg["n_train"] if n_train is None else n_train
    n_va = cfg["n_val"] if n_val is None else n_val
    n = n_tr + n_va
    d = cfg["d_in"]
    g = torch.Generator(device=device)
    g.manual_seed(int(cfg["seed"]) * 16 + 0)
    X = torch.empty((n, d), dtype=torch.float32, device=device)
    kind = cfg["features"]
    for r0 in range(0, n, chunk):
        r1 = min(n, r0 + chunk)
        if kind == "block_correlated":
            nb = (d + 29) // 30
            z = torch.randn((r1 - r0, nb), generator=g, device=device)
            e = torch.randn((r1 - r0, d), generator=g, device=device)
            X[r0:r1] = (0.6 ** 0.5) * z.repeat_interleave(30, dim=1)[:, :d] + (0.4 ** 0.5) * e
        elif kind == "onehot":
            n_num = d - 16
            X[r0:r1, :n_num] = torch.randn((r1 - r0, n_num), generator=g, device=device)
            X[r0:r1, n_num:] = 0
            for j in range(4):
                lev = torch.randint(0, 4, (r1 - r0,), generator=g, device=device)
                X[torch.arange(r0, r1, device=device), n_num + 4 * j + lev] = 1.0
        else:
            X[r0:r1] = torch.randn((r1 - r0, d), generator=g, device=device)
            if kind == "lognormal_rankgauss":
                X[r0:r1].exp_()
    if kind == "zero_inflated":
        cols = torch.randperm(d, generator=g, device=device)[:max(1, int(round(0.2 * d)))]
        for c in cols.tolist():
            X[:, c].masked_fill_(torch.rand(n, generator=g, device=device) < 0.5, 0.0)
    if kind == "lognormal_rankgauss":
        q = torch.special.ndtri((torch.arange(n_tr, device=device, dtype=torch.float64) + 0.5) / n_tr).float()
        for j in range(d):
            col = X[:n_tr, j]
            srt, order = torch.sort(col)
            ranks = torch.empty_like(order)
            ranks[order] = torch.arange(n_tr, device=device)
            va = X[n_tr:, j]
            pos = torch.searchsorted(srt, va).clamp(1, n_tr - 1)
            lo, hi = srt[pos - 1], srt[pos]
            w = ((va - lo) / (hi - lo).clamp_min(1e-30)).clamp(0, 1)
            X[n_tr:, j] = q[pos - 1] + w * (q[pos] - q[pos - 1])
            X[:n_tr, j] = q[ranks]
    W1 = torch.randn((d, 32), generator=g, device=device) / d ** 0.5
    W2 = torch.randn((32, cfg["d_out"]), generator=g, device=device) / 32 ** 0.5
    T = torch.empty((n, cfg["d_out"]), dtype=torch.float32, device=device)
    for r0 in range(0, n, chunk):
        T[r0:r0 + chunk] = torch.tanh(X[r0:r0 + chunk] @ W1) @ W2
    lab = cfg["label"]
    if lab == "sign":
        y = (T[:, 0] > 0).float()
    elif lab == "argmax":
        y = T.argmax(dim=1).to(torch.int32)
    else:
        t = T[:, 0].double()
        if lab == "teacher_noise":
            t = t + 0.1 * torch.randn(n, generator=g, device=device, dtype=torch.float64)
        else:
            t = t / t[:n_tr].std().clamp_min(1e-12)
            z = torch.randn(n, generator=g, device=device, dtype=torch.float64)
            chi2 = (torch.randn((n, 3), generator=g, device=device, dtype=torch.float64) ** 2).sum(dim=1)
            t = t + 0.1 * z / torch.sqrt(chi2 / 3.0)  # Student-t with 3 degrees of freedom
        y = ((t - t[:n_tr].mean()) / t[:n_tr].std().clamp_min(1e-12)).float()
    return X[:n_tr], y[:n_tr].contiguous(), X[n_tr:], y[n_tr:].contiguous()


def epoch_orders_device(cfg, epoch, n_train, device="cuda"):
    """Per-member permutations of the training rows on the device: int32 [K, n_train]."""
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(int(cfg["seed"]) * 16 + 4 + 256 * int(epoch))
    return torch.stack([torch.randperm(n_train, generator=g, device=device, dtype=torch.int64)
                        for _ in range(cfg["K"])]).to(torch.int32)
