"""GPU parity of packs with periodic feature embeddings (App. "Feature
Embeddings"): each member embeds every feature into d_emb values
alpha * [x, cos(w x + b)] + beta of its own, its first layer reads the
d_in * d_emb embedded columns, and the embedding parameters take AdamW steps.
Compared with the oracle (fp64, or its bf16 policy) on the same inputs."""
import numpy as np
import pytest

from oracle.pack import OraclePack
from paper_2607_05380_amd import configs, synth, tabpack
from parity import TOL, check_decisions, check_tensor, check_update, gpu_hints, make_inputs, oracle_cfg, oracle_hparams, to_dev

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

EMB = dict(emb_lo=8, emb_hi=32, emb_step=4, sigma_lo=1e-2, sigma_hi=10.0)
NAMES = ("w", "b", "alpha", "beta")


def _tensors(params, grads, m, v):
    """[(name, param, grad, m, v)] over the embedding and layer tensors of one member
    (GPU: dict first; oracle: passed as (emb dict, layer list))."""
    out = []
    emb, layers = params
    gemb, glayers = grads
    for n in NAMES:
        out.append((n, emb[n], gemb[n], m[0][n] if m else None, v[0][n] if v else None))
    for l, (W, b) in enumerate(layers):
        out.append((f"W{l}", W, glayers[l][0], m[1][l][0] if m else None, v[1][l][0] if v else None))
        out.append((f"b{l}", b, glayers[l][1], m[1][l][1] if m else None, v[1][l][1] if v else None))
    return out


def _gpu(pk, k):
    p, g = pk.get_params(k), pk.get_grads(k)
    m, v = pk.get_moments(k)
    return _tensors((p[0], p[1:]), (g[0], g[1:]), (m[0], m[1:]), (v[0], v[1:]))


def _ref(op, k):
    return _tensors((op.emb[k], op.params[k]), (op.last_emb_grads[k], op.last_grads[k]),
                    (op.emb_m[k], op.m[k]), (op.emb_v[k], op.v[k]))


def randomize_embeddings(pk, op, members, seed):
    """Non-zero b, alpha, beta (the same fp32 values on both sides), so that every
    embedding parameter has a gradient at the first step."""
    rng = np.random.default_rng(seed)
    for k in members:
        emb = op.emb[k]
        for n in ("b", "alpha", "beta"):
            emb[n] = rng.uniform(-1, 1, emb[n].shape).astype(np.float32).astype(np.float64)
        params = pk.get_params(k)
        params[0] = {n: emb[n] for n in NAMES}
        pk.set_params(k, params)


def _run(cfg, steps, n_train=3000, random_emb=False):
    Xtr, ytr, _, _, orders, _ = make_inputs(cfg, n_train, 10)
    X, y = to_dev(Xtr, ytr)
    pk = tabpack.Pack(cfg).bind()
    op = OraclePack(oracle_cfg(cfg), hparams=oracle_hparams(cfg),
                    precision="bf16" if cfg["precision"] == "bf16" else "fp64")
    if random_emb:
        randomize_embeddings(pk, op, range(cfg["K"]), cfg["seed"])
    p0 = [[(n, np.array(a, np.float64)) for n, a, _, _, _ in _gpu(pk, k)] for k in range(cfg["K"])]
    for s in range(steps):
        idx = synth.batch_indices(orders, s, cfg["B"])
        (idx_d,) = to_dev(idx)
        lg = pk.train_step(X, y, idx_d, s + 1).cpu().numpy()
        hints = {k: gpu_hints(pk, k, cfg, s + 1) for k in range(cfg["K"])}
        lo = op.train_step(Xtr, ytr, idx, s + 1, hints=hints)
        for k in range(cfg["K"]):
            check_decisions(op, k, f"step{s + 1}.m{k}")
        check_tensor(f"loss step {s + 1}", lg, lo, TOL[cfg["precision"]])
    return pk, op, p0


def _compare(pk, op, p0, tol, steps, members=None, prefix=""):
    for k in (range(op.cfg["K"]) if members is None else members):
        lr = op.hp[k]["lr"]
        for (n, p, g, m, v), (_, pr, gr, mr, vr), (_, a0) in zip(_gpu(pk, k), _ref(op, k), p0[k]):
            tag = f"{prefix}m{k}.{n}"
            kind = "emb" if n in NAMES else "layer"
            check_tensor(tag + ".grad", g, gr, tol, grad=True, kind=kind + "_grad")
            # w and b get their first non-zero gradient at step 2 (it is
            # proportional to alpha, which starts at zero and is about lr after
            # one step): those small sums with cancellations can flip the sign
            # of AdamW's first, sign-like step on a few elements of these small
            # tensors, each still within the 2 t lr bound
            frac = 0.1 if n in ("w", "b") and steps > 1 else None  # measured 4 of 88 elements (fp32)
            check_update(tag, p, pr, a0, g if steps == 1 else None, gr, lr, tol, steps, upd_frac=frac,
                         kind=kind + "_update")
            check_tensor(tag + ".m", m, mr, tol, grad=True, kind=kind + "_m")


def test_embedding_fp32_three_steps():
    # alpha starts at zero, so w and b receive their first gradients at step 2
    cfg = configs.workload("binary_small", emb_lo=8, emb_hi=16, emb_step=4, sigma_lo=0.1, sigma_hi=3.0)
    pk, op, p0 = _run(cfg, 3)
    print(f"[embed] d_emb {[h['d_emb'] for h in pk.hparams()]}", flush=True)
    _compare(pk, op, p0, TOL["fp32"], 3)
    for k in range(cfg["K"]):
        assert np.abs(pk.get_grads(k)[0]["w"]).max() > 0


@pytest.mark.parametrize("name,over", [("regression_large", dict(K=4, B=300)),
                                       ("multiclass_lognormal", dict(K=3, B=260, depth_lo=1, depth_hi=3))])
def test_embedding_bf16_step(name, over):
    # one step from non-zero alpha: after a bf16 step the embedding gradients of
    # w and b are proportional to alpha, whose first AdamW step is sign-like and
    # legitimately flips where its gradient is tiny, so a second step would
    # compare those flips rather than the kernels
    cfg = configs.workload(name, **over, **EMB)
    print(f"[embed] {name} d_emb {[h['d_emb'] for h in tabpack.Pack(cfg).hparams()]}", flush=True)
    pk, op, p0 = _run(cfg, 1, random_emb=True)
    _compare(pk, op, p0, TOL["bf16"], 1)


def test_embedding_eval_predict_and_muon():
    cfg = configs.workload("regression_onehot", K=4, B=256, optimizer="muon", **EMB)
    Xtr, ytr, Xva, yva, _, idx = make_inputs(cfg, 2000, 700)
    X, y, idx_d, Xv, yv = to_dev(Xtr, ytr, idx, Xva, yva)
    pk = tabpack.Pack(cfg).bind()
    pk.train_step(X, y, idx_d, 1)
    op = OraclePack(oracle_cfg(cfg), hparams=oracle_hparams(cfg), precision="bf16")
    op.train_step(Xtr, ytr, idx, 1)
    pred, score = pk.eval_members(Xv, yv)
    pr, sr = op.eval_members(Xva, yva)
    check_tensor("pred", pred.cpu().numpy(), pr, TOL["bf16"])
    check_tensor("score", score.cpu().numpy(), sr, TOL["bf16"])
    mem = pk.predict(Xv).cpu().numpy()
    for k in range(cfg["K"]):
        check_tensor(f"predict {k}", mem[k], op.predict_values(k, Xva), TOL["bf16"])


def test_embedded_tile_sets_and_streams_are_bit_identical(monkeypatch):
    # The embedded forward's 8-wave tiles (128 x 256, a last strip of at most
    # 128 columns on 256 x 128 tiles) reduce every output element over the
    # full depth in the small tiles' order, and the epilogue is the same per
    # element: training steps, states and evaluation predictions must be
    # bit-identical to the small tiles', and to another split over streams.
    # Padded widths 96, 256, 320, 416, 544, 1024: last strips of 96 (no wide
    # tile), 0, 64, 160 (a wide tile with masked waves), 32 and 0 columns.
    cfg = configs.workload("regression_large", K=6, B=300, **EMB)
    members = [dict(width=w, dropout=p, lr=2e-3, wd=1e-3, d_emb=e, sigma=1.0)
               for w, p, e in ((96, 0.1, 8), (256, 0.0, 12), (300, 0.3, 16), (416, 0.2, 20), (520, 0.4, 24),
                               (1000, 0.1, 32))]
    Xtr, ytr, Xva, yva, _, idx = make_inputs(cfg, 3000, 700)
    X, y, idx_d, Xv, yv = to_dev(Xtr, ytr, idx, Xva, yva)
    runs = {}
    for tiles, streams in (("small", "2"), ("wide", "2"), ("wide", "1")):
        if tiles == "small":
            monkeypatch.setenv("TABPACK_EMB_TILES", "small")
        else:
            monkeypatch.delenv("TABPACK_EMB_TILES", raising=False)
        monkeypatch.setenv("TABPACK_STREAMS", streams)
        pk = tabpack.Pack(cfg, members=members).bind()
        losses = [pk.train_step(X, y, idx_d, s).cpu().numpy() for s in (1, 2)]
        pred, score = pk.eval_members(Xv, yv)
        states = [(pk.get_params(k), pk.get_moments(k)) for k in range(cfg["K"])]
        runs[(tiles, streams)] = (losses, pred.cpu().numpy(), score.cpu().numpy(), states)
    ref = runs[("small", "2")]
    for key, got in runs.items():
        msg = str(key)
        for a, b in zip(ref[0], got[0]):
            np.testing.assert_array_equal(a, b, err_msg=msg)
        np.testing.assert_array_equal(ref[1], got[1], err_msg=msg)
        np.testing.assert_array_equal(ref[2], got[2], err_msg=msg)
        for (p1, m1), (p2, m2) in zip(ref[3], got[3]):
            for n in NAMES:
                np.testing.assert_array_equal(p1[0][n], p2[0][n], err_msg=msg)
            for (W1, b1), (W2, b2) in zip(p1[1:], p2[1:]):
                np.testing.assert_array_equal(W1, W2, err_msg=msg)
                np.testing.assert_array_equal(b1, b2, err_msg=msg)
            for x1, x2 in zip(m1, m2):
                for n in NAMES:
                    np.testing.assert_array_equal(x1[0][n], x2[0][n], err_msg=msg)
                for (W1, b1), (W2, b2) in zip(x1[1:], x2[1:]):
                    np.testing.assert_array_equal(W1, W2, err_msg=msg)
                    np.testing.assert_array_equal(b1, b2, err_msg=msg)
