"""Pins of the oracle's periodic feature embeddings (CPU): the embedded member's
loss and gradients against torch float64 autograd and central finite
differences, the initial values against their definition (Box-Muller pairs,
N(0, sigma) statistics, zeros), the hyperparameter draws, and the first AdamW
step of the embedding parameters against its closed form."""
import math

import numpy as np
import pytest
import torch
from scipy.stats import kstest

from oracle import embed, mlp
from oracle.pack import OraclePack
from oracle.sampling import TAG_INIT, sample_hparams, stream_key
from oracle.philox import philox4x32_10

CFG = dict(seed=23, K=3, d_in=4, d_out=1, L=2, B=7, task=mlp.TASK_REG, beta1=0.9, beta2=0.999, eps=1e-8,
           decay_bias=1, width_lo=5, width_hi=7, dropout_lo=0.0, dropout_hi=0.3, lr_lo=1e-3, lr_hi=3e-3,
           wd_lo=1e-3, wd_hi=1e-2, emb_lo=8, emb_hi=16, emb_step=4, sigma_lo=0.1, sigma_hi=2.0)


def _random_emb(rng, d_in, d_emb):
    return dict(w=rng.standard_normal((d_in, d_emb - 1)), b=rng.standard_normal((d_in, d_emb - 1)),
                alpha=rng.standard_normal((d_in, d_emb)), beta=rng.standard_normal((d_in, d_emb)))


def _torch_embedded_loss(emb, params, X, y, masks, s, task):
    t = {n: torch.tensor(a, dtype=torch.float64, requires_grad=True) for n, a in emb.items()}
    Ws = [(torch.tensor(W, requires_grad=True), torch.tensor(b, requires_grad=True)) for W, b in params]
    x = torch.from_numpy(X)
    phi = x[:, :, None] * t["w"][None] + t["b"][None]
    feats = torch.cat([x[:, :, None], torch.cos(phi)], dim=2)
    H = (feats * t["alpha"][None] + t["beta"][None]).reshape(X.shape[0], -1)
    for l, (W, b) in enumerate(Ws[:-1]):
        H = torch.relu(H @ W.T + b) * torch.from_numpy(masks[l].astype(np.float64)) * s
    Y = H @ Ws[-1][0].T + Ws[-1][1]
    yt = torch.from_numpy(np.asarray(y, np.float64))
    loss = torch.nn.functional.mse_loss(Y[:, 0], yt) if task == mlp.TASK_REG else \
        torch.nn.functional.binary_cross_entropy_with_logits(Y[:, 0], yt)
    loss.backward()
    return loss.item(), {n: a.grad.numpy() for n, a in t.items()}, [(W.grad.numpy(), b.grad.numpy()) for W, b in Ws]


@pytest.mark.parametrize("task", [mlp.TASK_REG, mlp.TASK_BIN])
def test_embedded_member_matches_torch_autograd(task):
    rng = np.random.default_rng(5)
    d_in, d_emb, B, widths = 4, 6, 9, (7, 5)
    emb = _random_emb(rng, d_in, d_emb)
    dims = [d_in * d_emb] + list(widths) + [1]
    params = [(rng.standard_normal((dims[i + 1], dims[i])) / 3, rng.standard_normal(dims[i + 1]))
              for i in range(len(dims) - 1)]
    X = rng.standard_normal((B, d_in))
    y = rng.standard_normal(B) if task == mlp.TASK_REG else (rng.random(B) < 0.5).astype(np.float64)
    masks = [rng.random((B, w)) > 0.25 for w in widths]
    s = 1 / 0.75
    E, cache = embed.embed(X, emb)
    Y, mc = mlp.forward(params, E, masks, s)
    loss, dY = mlp.loss_and_dy(Y, y, task)
    grads, dE = mlp.backward(params, mc, dY, masks, s, input_grad=True)
    eg = embed.embed_backward(dE, cache, emb)
    tl, teg, tg = _torch_embedded_loss(emb, params, X, y, masks, s, task)
    assert abs(tl - loss) <= 1e-12 * max(1.0, abs(loss))
    for n in ("w", "b", "alpha", "beta"):
        np.testing.assert_allclose(eg[n], teg[n], rtol=1e-10, atol=1e-13, err_msg=n)
    for (gW, gb), (tW, tb) in zip(grads, tg):
        np.testing.assert_allclose(gW, tW, rtol=1e-10, atol=1e-13)
        np.testing.assert_allclose(gb, tb, rtol=1e-10, atol=1e-13)


def test_embedding_gradients_finite_differences():
    rng = np.random.default_rng(8)
    d_in, d_emb, N = 3, 5, 6
    emb = _random_emb(rng, d_in, d_emb)
    X = rng.standard_normal((N, d_in))
    G = rng.standard_normal((N, d_in * d_emb))  # loss = sum(G * E)
    E, cache = embed.embed(X, emb)
    eg = embed.embed_backward(G, cache, emb)
    h = 1e-6
    for n in ("w", "b", "alpha", "beta"):
        fd = np.zeros_like(emb[n])
        for idx in np.ndindex(*emb[n].shape):
            p = {m: a.copy() for m, a in emb.items()}
            p[n][idx] += h
            up = (G * embed.embed(X, p)[0]).sum()
            p[n][idx] -= 2 * h
            dn = (G * embed.embed(X, p)[0]).sum()
            fd[idx] = (up - dn) / (2 * h)
        np.testing.assert_allclose(eg[n], fd, rtol=1e-6, atol=1e-8, err_msg=n)


def test_embedding_values_and_layout():
    # column i * d_emb + j: j = 0 is alpha x + beta, j >= 1 alpha cos(w x + b) + beta
    rng = np.random.default_rng(9)
    emb = _random_emb(rng, 3, 4)
    X = rng.standard_normal((5, 3))
    E, _ = embed.embed(X, emb)
    for r in range(5):
        for i in range(3):
            assert E[r, i * 4] == pytest.approx(emb["alpha"][i, 0] * X[r, i] + emb["beta"][i, 0], rel=1e-14)
            for j in range(1, 4):
                ref = emb["alpha"][i, j] * math.cos(emb["w"][i, j - 1] * X[r, i] + emb["b"][i, j - 1]) + \
                    emb["beta"][i, j]
                assert E[r, i * 4 + j] == pytest.approx(ref, rel=1e-13, abs=1e-15)


def test_embedding_init():
    cfg = dict(CFG, d_in=300)
    sigma = 0.7
    e = embed.init_embedding(cfg, 2, 12, sigma)
    assert (e["b"] == 0).all() and (e["alpha"] == 0).all() and (e["beta"] == 0).all()
    w = e["w"].ravel()
    assert kstest(w / sigma, "norm").pvalue > 1e-4
    # Box-Muller pairs: elements 2m and 2m+1 share the radius sqrt(-2 ln u1) of block m
    k0, k1 = stream_key(cfg["seed"], TAG_INIT)
    for m in (0, 7, 1234):
        a = int(philox4x32_10(m, 0, embed.TENSOR_W, 2, k0, k1)[0])
        u1 = ((a >> 8) + 1) * 2.0 ** -24
        assert (w[2 * m] ** 2 + w[2 * m + 1] ** 2) == pytest.approx(-2 * math.log(u1) * sigma ** 2, rel=1e-6)
    # float32 values, deterministic, member-specific
    assert (w.astype(np.float32).astype(np.float64) == w).all()
    np.testing.assert_array_equal(embed.init_embedding(cfg, 2, 12, sigma)["w"], e["w"])
    assert not np.array_equal(embed.init_embedding(cfg, 3, 12, sigma)["w"], e["w"])


def test_embedding_hparam_draws():
    cfg = dict(CFG, K=3000, emb_lo=8, emb_hi=32, emb_step=4, sigma_lo=1e-2, sigma_hi=10.0)
    hp = sample_hparams(cfg)
    d = np.array([h["d_emb"] for h in hp])
    assert set(d.tolist()) == {8, 12, 16, 20, 24, 28, 32}
    for v in range(8, 33, 4):
        n, p = len(d), 1 / 7
        assert abs((d == v).sum() - n * p) <= 5 * math.sqrt(n * p * (1 - p))
    s = np.array([h["sigma"] for h in hp])
    assert kstest((np.log(s) - np.log(1e-2)) / (np.log(10) - np.log(1e-2)), "uniform").pvalue > 1e-4
    base = sample_hparams(dict(cfg, emb_lo=0))
    assert [h["width"] for h in base] == [h["width"] for h in hp] and "d_emb" not in base[0]


def test_pack_with_embeddings_first_step():
    # the first layer reads d_in * d_emb columns; the embedding parameters take
    # AdamW steps: at t = 1, theta (1 - lr wd) - lr g / (|g| + eps)
    hp = sample_hparams(CFG)
    op = OraclePack(CFG, hparams=hp)
    rng = np.random.default_rng(2)
    for k in range(3):
        # non-zero alpha so that every embedding parameter has a gradient
        op.emb[k]["alpha"] = rng.standard_normal(op.emb[k]["alpha"].shape)
        assert op.params[k][0][0].shape == (hp[k]["width"], CFG["d_in"] * hp[k]["d_emb"])
    e0 = [{n: a.copy() for n, a in e.items()} for e in op.emb]
    X, y = rng.standard_normal((30, 4)), rng.standard_normal(30)
    idx = np.stack([rng.permutation(30)[:7] for _ in range(3)])
    op.train_step(X, y, idx, 1)
    for k in range(3):
        lr, wd = hp[k]["lr"], hp[k]["wd"]
        for n in ("w", "b", "alpha", "beta"):
            g = op.last_emb_grads[k][n]
            assert np.abs(g).max() > 0, n
            np.testing.assert_allclose(op.emb[k][n], e0[k][n] * (1 - lr * wd) - lr * g / (np.abs(g) + 1e-8),
                                       rtol=1e-12, atol=1e-15)
