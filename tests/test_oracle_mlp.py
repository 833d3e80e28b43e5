"""Pins of the oracle's single-member arithmetic against independent references (CPU)."""
import numpy as np
import pytest
import torch

from oracle import mlp
from oracle.pack import OraclePack, prediction, score
from oracle.sampling import init_member, member_hparams

TASKS = [(mlp.TASK_REG, 1), (mlp.TASK_BIN, 1), (mlp.TASK_MULTI, 4)]


def _tiny(task, d_out, seed, d_in=3, widths=(5, 6), B=5):
    rng = np.random.default_rng(seed)
    dims = [d_in] + list(widths) + [d_out]
    params = [(rng.standard_normal((dims[i + 1], dims[i])), rng.standard_normal(dims[i + 1]))
              for i in range(len(dims) - 1)]
    X = rng.standard_normal((B, d_in))
    if task == mlp.TASK_REG:
        y = rng.standard_normal(B)
    elif task == mlp.TASK_BIN:
        y = (rng.random(B) < 0.5).astype(np.float64)
    else:
        y = rng.integers(0, d_out, B)
    masks = [rng.random((B, w)) > 0.3 for w in widths]
    return params, X, y, masks


def _loss(params, X, y, masks, s, task):
    Y, _ = mlp.forward(params, X, masks, s)
    return mlp.loss_and_dy(Y, y, task)[0]


@pytest.mark.parametrize("task,d_out", TASKS)
def test_finite_differences(task, d_out):
    # Central differences in fp64 on a tiny net; draws near the ReLU kink are rejected.
    for seed in range(40):
        params, X, y, masks = _tiny(task, d_out, seed)
        Y, cache = mlp.forward(params, X, masks, 1.25)
        if min(np.abs(Z).min() for Z in cache["Z"]) > 1e-4:
            break
    _, dY = mlp.loss_and_dy(Y, y, task)
    grads = mlp.backward(params, cache, dY, masks, 1.25)
    h = 1e-6
    for li, (W, b) in enumerate(params):
        for arr, g in ((W, grads[li][0]), (b, grads[li][1])):
            fd = np.zeros_like(arr)
            for idx in np.ndindex(arr.shape):
                old = arr[idx]
                arr[idx] = old + h
                lp = _loss(params, X, y, masks, 1.25, task)
                arr[idx] = old - h
                lm = _loss(params, X, y, masks, 1.25, task)
                arr[idx] = old
                fd[idx] = (lp - lm) / (2 * h)
            err = np.linalg.norm(fd - g) / max(np.linalg.norm(g), 1e-30)
            assert err < 1e-6, (li, err)


def _torch_member(params, masks, s):
    layers = []
    for W, b in params:
        lin = torch.nn.Linear(W.shape[1], W.shape[0], dtype=torch.float64)
        with torch.no_grad():
            lin.weight.copy_(torch.from_numpy(W))
            lin.bias.copy_(torch.from_numpy(b))
        layers.append(lin)

    def fwd(X):
        H = torch.from_numpy(X)
        for l, lin in enumerate(layers[:-1]):
            H = torch.relu(lin(H)) * torch.from_numpy(masks[l].astype(np.float64)) * s
        return layers[-1](H)
    return layers, fwd


def _torch_loss(Y, y, task):
    if task == mlp.TASK_REG:
        return torch.nn.functional.mse_loss(Y[:, 0], torch.from_numpy(np.asarray(y, np.float64)))
    if task == mlp.TASK_BIN:
        return torch.nn.functional.binary_cross_entropy_with_logits(
            Y[:, 0], torch.from_numpy(np.asarray(y, np.float64)))
    return torch.nn.functional.cross_entropy(Y, torch.from_numpy(np.asarray(y, np.int64)))


@pytest.mark.parametrize("task,d_out", TASKS)
def test_member_step_matches_torch_autograd_and_adamw(task, d_out):
    # Forward, loss, backward and three AdamW steps against torch float64 autograd
    # and torch.optim.AdamW with the member's (lr, wd).
    params, X, y, masks = _tiny(task, d_out, 3, d_in=7, widths=(11, 9), B=13)
    s, lr, wd = 1.0 / (1 - 0.2), 3e-3, 2e-2
    layers, fwd = _torch_member(params, masks, s)
    opt = torch.optim.AdamW([p for l in layers for p in (l.weight, l.bias)], lr=lr,
                            betas=(0.9, 0.999), eps=1e-8, weight_decay=wd)
    th = [(W.copy(), b.copy()) for W, b in params]
    mm = [(np.zeros_like(W), np.zeros_like(b)) for W, b in params]
    vv = [(np.zeros_like(W), np.zeros_like(b)) for W, b in params]
    for t in range(1, 4):
        Y, cache = mlp.forward(th, X, masks, s)
        loss, dY = mlp.loss_and_dy(Y, y, task)
        grads = mlp.backward(th, cache, dY, masks, s)
        opt.zero_grad()
        tl = _torch_loss(fwd(X), y, task)
        tl.backward()
        assert abs(tl.item() - loss) <= 1e-12 * max(1.0, abs(loss))
        for l, lin in enumerate(layers):
            np.testing.assert_allclose(grads[l][0], lin.weight.grad.numpy(), rtol=1e-10, atol=1e-13)
            np.testing.assert_allclose(grads[l][1], lin.bias.grad.numpy(), rtol=1e-10, atol=1e-13)
        opt.step()
        new = []
        for l in range(len(th)):
            Wn, mW, vW = mlp.adamw_step(th[l][0], grads[l][0], mm[l][0], vv[l][0], t, lr, wd, 0.9, 0.999, 1e-8)
            bn, mb, vb = mlp.adamw_step(th[l][1], grads[l][1], mm[l][1], vv[l][1], t, lr, wd, 0.9, 0.999, 1e-8)
            new.append((Wn, bn))
            mm[l], vv[l] = (mW, mb), (vW, vb)
        th = new
        for l, lin in enumerate(layers):
            np.testing.assert_allclose(th[l][0], lin.weight.detach().numpy(), rtol=1e-12, atol=1e-15)
            np.testing.assert_allclose(th[l][1], lin.bias.detach().numpy(), rtol=1e-12, atol=1e-15)


def test_adamw_first_step_closed_form():
    rng = np.random.default_rng(1)
    th, g = rng.standard_normal(50), rng.standard_normal(50)
    lr, wd = 2e-3, 1e-2
    new, m, v = mlp.adamw_step(th, g, 0 * g, 0 * g, 1, lr, wd, 0.9, 0.999, 1e-8)
    np.testing.assert_allclose(new, th * (1 - lr * wd) - lr * g / (np.abs(g) + 1e-8), rtol=1e-12)
    np.testing.assert_allclose(m, 0.1 * g)
    np.testing.assert_allclose(v, 0.001 * g * g)


def test_affine_closed_form():
    # With p = 0 and positive weights/inputs every unit is active: the net is affine.
    rng = np.random.default_rng(2)
    dims = [4, 6, 5, 1]
    params = [(rng.random((dims[i + 1], dims[i])), rng.random(dims[i + 1])) for i in range(3)]
    X = rng.random((7, 4))
    Y, _ = mlp.forward(params, X, [np.ones((7, 6), bool), np.ones((7, 5), bool)], 1.0)
    A = params[0][0].T @ params[1][0].T @ params[2][0].T
    c = (params[0][1] @ params[1][0].T + params[1][1]) @ params[2][0].T + params[2][1]
    np.testing.assert_allclose(Y, X @ A + c, rtol=1e-13)


def test_prediction_and_scores_against_sklearn():
    from sklearn.metrics import log_loss, mean_squared_error
    rng = np.random.default_rng(4)
    Yr = rng.standard_normal((40, 1))
    yr = rng.standard_normal(40)
    assert score(prediction(Yr, yr, "reg"), yr, "reg") == pytest.approx(
        np.sqrt(mean_squared_error(yr, Yr[:, 0])), rel=1e-13)
    yb = (rng.random(40) < 0.4).astype(np.float64)
    pb = prediction(Yr, yb, "bin")
    assert score(pb, yb, "bin") == pytest.approx(log_loss(yb, pb), rel=1e-12)
    Ym = rng.standard_normal((40, 5))
    ym = rng.integers(0, 5, 40)
    Pm = torch.softmax(torch.from_numpy(Ym), dim=1).numpy()
    pm = prediction(Ym, ym, "multi")
    np.testing.assert_allclose(pm, Pm[np.arange(40), ym], rtol=1e-13)
    assert score(pm, ym, "multi") == pytest.approx(log_loss(ym, Pm, labels=range(5)), rel=1e-12)


def test_init_statistics_and_layout():
    from scipy.stats import kstest
    cfg = dict(seed=99, d_in=300, d_out=3, L=2)
    p = init_member(cfg, 5, 200)
    assert [w.shape for w, _ in p] == [(200, 300), (200, 200), (3, 200)]
    for (W, b), fan in zip(p, (300, 200, 200)):
        bound = 1 / np.sqrt(fan)
        assert np.abs(W).max() <= bound and np.abs(b).max() <= bound
        assert kstest(W.ravel() / bound, "uniform", args=(-1, 2)).pvalue > 1e-4
        assert np.all(W.astype(np.float32) == W)
    q = init_member(cfg, 6, 200)
    assert not np.array_equal(p[0][0], q[0][0])
    np.testing.assert_array_equal(p[1][0], init_member(cfg, 5, 200)[1][0])


def test_pack_members_match_standalone_and_are_independent():
    cfg = dict(seed=11, K=3, d_in=6, d_out=1, L=2, B=8, task="reg", beta1=0.9, beta2=0.999,
               eps=1e-8, decay_bias=1, width_lo=4, width_hi=9, dropout_lo=0.0, dropout_hi=0.4,
               lr_lo=1e-4, lr_hi=3e-3, wd_lo=1e-5, wd_hi=1e-2)
    rng = np.random.default_rng(5)
    X, y = rng.standard_normal((30, 6)), rng.standard_normal(30)
    idx = np.stack([rng.permutation(30)[:8] for _ in range(3)])
    pack = OraclePack(cfg)
    base = [[(W.copy(), b.copy()) for W, b in p] for p in pack.params]
    losses = pack.train_step(X, y, idx, 1)
    # member k alone, written directly with mlp functions and torch's AdamW semantics
    for k in range(3):
        h = pack.hp[k]
        masks = pack.masks(k, 1)
        Y, cache = mlp.forward(base[k], X[idx[k]], masks, h["s"])
        loss, dY = mlp.loss_and_dy(Y, y[idx[k]], "reg")
        assert loss == losses[k]
        g = mlp.backward(base[k], cache, dY, masks, h["s"])
        for l in range(3):
            W1, _, _ = mlp.adamw_step(base[k][l][0], g[l][0], 0, 0, 1, h["lr"], h["wd"], .9, .999, 1e-8)
            np.testing.assert_array_equal(W1, pack.params[k][l][0])
    # perturb member 1's parameters and batch: members 0 and 2 are bit-identical
    pack2 = OraclePack(cfg, params=base)
    pack2.params[1][0][0][0, 0] += 1.0
    idx2 = idx.copy()
    idx2[1] = rng.permutation(30)[:8]
    losses2 = pack2.train_step(X, y, idx2, 1)
    for k in (0, 2):
        assert losses2[k] == losses[k]
        for l in range(3):
            np.testing.assert_array_equal(pack2.params[k][l][0], pack.params[k][l][0])
            np.testing.assert_array_equal(pack2.last_grads[k][l][1], pack.last_grads[k][l][1])
    assert losses2[1] != losses[1]


def test_to_bf16_matches_torch_rounding():
    rng = np.random.default_rng(9)
    x = np.concatenate([rng.standard_normal(20000) * 10 ** rng.uniform(-30, 30, 20000),
                        # exact ties between two bf16 neighbours, both parities
                        (np.arange(1, 2001, dtype=np.float64) * 2 ** -7 + 2 ** -16) * 3.0,
                        [0.0, -0.0, 1.0, -2.5, 3.0e38]])
    ref = torch.from_numpy(x.astype(np.float32)).to(torch.bfloat16).to(torch.float64).numpy()
    np.testing.assert_array_equal(mlp.to_bf16(x), ref)


class _RoundFwd(torch.autograd.Function):
    """bf16 rounding of a value, gradient passed straight through."""
    @staticmethod
    def forward(ctx, x):
        return x.float().to(torch.bfloat16).to(torch.float64)

    @staticmethod
    def backward(ctx, g):
        return g


class _RoundGrad(torch.autograd.Function):
    """Identity forward, bf16 rounding of the incoming gradient."""
    @staticmethod
    def forward(ctx, x):
        return x.clone()

    @staticmethod
    def backward(ctx, g):
        return g.float().to(torch.bfloat16).to(torch.float64)


@pytest.mark.parametrize("task,d_out", TASKS)
def test_bf16_policy_matches_torch_straight_through(task, d_out):
    # The bf16 policy built independently in torch: bf16 operands of every hidden
    # matrix product (straight-through), rounded dZ for dW/dH but not for db.
    params, X, y, masks = _tiny(task, d_out, 7, d_in=9, widths=(12, 10), B=17)
    s = 1.0 / (1 - 0.3)
    Y, cache = mlp.forward(params, X, masks, s, rnd=mlp.to_bf16)
    loss, dY = mlp.loss_and_dy(Y, y, task)
    grads = mlp.backward(params, cache, dY, masks, s)
    tW = [torch.tensor(W, requires_grad=True) for W, _ in params]
    tb = [torch.tensor(b, requires_grad=True) for _, b in params]
    H = _RoundFwd.apply(torch.from_numpy(X))
    for l in range(2):
        Z = _RoundGrad.apply(H @ _RoundFwd.apply(tW[l]).T) + tb[l]
        H = _RoundFwd.apply(torch.relu(Z) * torch.from_numpy(masks[l].astype(np.float64)) * s)
    Yt = H @ tW[2].T + tb[2]
    lt = _torch_loss(Yt, y, task)
    lt.backward()
    assert lt.item() == pytest.approx(loss, rel=1e-12)
    for l in range(3):
        np.testing.assert_allclose(grads[l][0], tW[l].grad.numpy(), rtol=1e-10, atol=1e-14)
        np.testing.assert_allclose(grads[l][1], tb[l].grad.numpy(), rtol=1e-10, atol=1e-14)


@pytest.mark.parametrize("depths", [(1, 3, 2), (4, 1, 1)])
def test_pack_members_of_different_depths_match_torch_autograd(depths):
    # a pack whose members have their own number of hidden blocks: each member's
    # loss and gradients equal torch float64 autograd of a network of that depth
    cfg = dict(seed=11, K=len(depths), d_in=4, d_out=1, L=max(depths), B=9, task=mlp.TASK_REG,
               beta1=0.9, beta2=0.999, eps=1e-8, decay_bias=1)
    hp = [member_hparams(6 + k, 0.25, 1e-3, 1e-2, d) for k, d in enumerate(depths)]
    op = OraclePack(cfg, hparams=hp)
    rng = np.random.default_rng(5)
    X = rng.standard_normal((30, 4))
    y = rng.standard_normal(30)
    idx = np.stack([rng.permutation(30)[:9] for _ in depths])
    p0 = [[(W.copy(), b.copy()) for W, b in p] for p in op.params]
    losses = op.train_step(X, y, idx, 1)
    for k, d in enumerate(depths):
        assert len(p0[k]) == d + 1 and len(op.masks(k, 1)) == d
        layers, fwd = _torch_member(p0[k], op.masks(k, 1), hp[k]["s"])
        tl = _torch_loss(fwd(X[idx[k]]), y[idx[k]], mlp.TASK_REG)
        tl.backward()
        assert abs(tl.item() - losses[k]) <= 1e-12 * max(1.0, abs(losses[k]))
        for l, lin in enumerate(layers):
            np.testing.assert_allclose(op.last_grads[k][l][0], lin.weight.grad.numpy(), rtol=1e-10, atol=1e-13)
            np.testing.assert_allclose(op.last_grads[k][l][1], lin.bias.grad.numpy(), rtol=1e-10, atol=1e-13)


def test_relu_decision_hints():
    # The backward pass may take another implementation's ReLU decisions for
    # pre-activations within window * rms(Z) of 0 (both branches correct up to
    # accumulation rounding).  Pinned against torch autograd of a network whose
    # ReLU derivative is set explicitly (value max(z, 0), derivative d).
    task, d_out = mlp.TASK_REG, 1
    params, X, y, masks = _tiny(task, d_out, 11, d_in=4, widths=(9, 7), B=12)
    s = 1.25
    Y, cache = mlp.forward(params, X, masks, s)
    _, dY = mlp.loss_and_dy(Y, y, task)
    plain = mlp.backward(params, cache, dY, masks, s)

    def same(a, b):
        for (x1, y1), (x2, y2) in zip(a, b):
            np.testing.assert_array_equal(x1, x2)
            np.testing.assert_array_equal(y1, y2)

    own = [(Z > 0).astype(np.int8) for Z in cache["Z"]]
    st = {}
    same(plain, mlp.backward(params, cache, dY, masks, s, hints=own, stats=st))
    assert st["taken"] == 0 and st["outside"] == 0
    # flip the decision of the smallest |Z| of each layer
    hints, rel = [], []
    for Z, o in zip(cache["Z"], own):
        h = o.copy()
        i = np.unravel_index(np.argmin(np.abs(Z)), Z.shape)
        h[i] = 1 - h[i]
        hints.append(h)
        rel.append(abs(Z[i]) / np.sqrt(np.mean(Z * Z)))
    # a window that holds them: the flips are taken
    window = max(rel) * 1.0001
    st = {}
    got = mlp.backward(params, cache, dY, masks, s, hints=hints, stats=st, window=window)
    assert st["taken"] == len(hints) and st["outside"] == 0
    d_eff = [np.where(np.abs(Z) <= window * np.sqrt(np.mean(Z * Z)), h == 1, Z > 0)
             for Z, h in zip(cache["Z"], hints)]
    tp = [(torch.tensor(W, requires_grad=True), torch.tensor(b, requires_grad=True)) for W, b in params]
    H = torch.tensor(X)
    for l, (W, b) in enumerate(tp[:-1]):
        Z = H @ W.T + b
        d = torch.tensor(d_eff[l].astype(np.float64))
        H = (torch.relu(Z).detach() + (Z - Z.detach()) * d) * torch.tensor(masks[l].astype(np.float64)) * s
    Yt = H @ tp[-1][0].T + tp[-1][1]
    torch.mean((Yt[:, 0] - torch.tensor(y)) ** 2).backward()
    for (gW, gb), (W, b) in zip(got, tp):
        np.testing.assert_allclose(gW, W.grad.numpy(), rtol=1e-10, atol=1e-13)
        np.testing.assert_allclose(gb, b.grad.numpy(), rtol=1e-10, atol=1e-13)
    assert any(not np.allclose(a[0], b[0]) for a, b in zip(got, plain))
    # a window that excludes them: the own decisions, and the disagreements counted
    st = {}
    same(plain, mlp.backward(params, cache, dY, masks, s, hints=hints, stats=st, window=min(rel) * 0.999))
    assert st["outside"] == len(hints) and st["taken"] == 0
    # unknown hints (-1) keep the own decisions whatever the window
    unk = [np.full(Z.shape, -1, np.int8) for Z in cache["Z"]]
    same(plain, mlp.backward(params, cache, dY, masks, s, hints=unk, window=1e9))
