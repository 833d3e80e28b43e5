"""Pins of the oracle's Muon step (CPU): the Newton-Schulz iteration against the
singular-value form of the same polynomial (numpy's SVD), padding and
orientation invariance, the momentum / Nesterov / update closed forms, the
split of parameters between Muon and AdamW in a pack, and the learning-rate
draw."""
import numpy as np
import pytest
from scipy.stats import kstest

from oracle import mlp
from oracle.muon import NS_COEFFS, NS_EPS, muon_step, newton_schulz
from oracle.pack import OraclePack
from oracle.sampling import sample_hparams


def _ns_svd(U, steps=5):
    # X0 = P S Q^T; every iteration maps each singular value s to a s + b s^3 + c s^5
    a, b, c = NS_COEFFS
    X0 = U / (np.linalg.norm(U) + NS_EPS)
    P, S, Qt = np.linalg.svd(X0, full_matrices=False)
    for _ in range(steps):
        S = a * S + b * S ** 3 + c * S ** 5
    return (P * S) @ Qt


@pytest.mark.parametrize("shape", [(7, 19), (19, 7), (12, 12), (1, 9), (9, 1)])
@pytest.mark.parametrize("steps", [1, 5])
def test_newton_schulz_matches_singular_value_polynomial(shape, steps):
    rng = np.random.default_rng(shape[0] * 100 + shape[1] + steps)
    U = rng.standard_normal(shape)
    O = newton_schulz(U, steps)
    ref = _ns_svd(U, steps)
    assert O.shape == shape
    np.testing.assert_allclose(O, ref, rtol=0, atol=1e-12 * max(1.0, np.abs(ref).max()))
    # five steps push every singular value into the band the coefficients aim at
    if steps == 5 and min(shape) > 1:
        sv = np.linalg.svd(O, compute_uv=False)
        assert sv.min() > 0.5 and sv.max() < 1.3


def test_newton_schulz_orientation_and_padding():
    rng = np.random.default_rng(3)
    U = rng.standard_normal((6, 11))
    np.testing.assert_allclose(newton_schulz(U.T), newton_schulz(U).T, rtol=0, atol=1e-14)
    P = np.zeros((8, 16))
    P[:6, :11] = U  # zero rows and columns, as in the pack's padded storage
    O = newton_schulz(P)
    np.testing.assert_allclose(O[:6, :11], newton_schulz(U), rtol=0, atol=1e-14)
    assert (O[6:] == 0).all() and (O[:, 11:] == 0).all()


def test_newton_schulz_scale_invariant_and_zero():
    rng = np.random.default_rng(4)
    U = rng.standard_normal((5, 9))
    # up to the 1e-7 added to the norm, which weighs 1e-7 / ||U|| relative
    np.testing.assert_allclose(newton_schulz(1e3 * U), newton_schulz(U), rtol=0, atol=1e-6)
    assert (newton_schulz(np.zeros((4, 6))) == 0).all()


@pytest.mark.parametrize("shape", [(5, 9), (9, 5)])
def test_muon_step_closed_form(shape):
    # two steps by hand: buf1 = G1, U1 = (1 + mu) G1; buf2 = mu G1 + G2, U2 = G2 + mu buf2
    rng = np.random.default_rng(7)
    W0 = rng.standard_normal(shape)
    G1, G2 = rng.standard_normal(shape), rng.standard_normal(shape)
    lr, wd, mu = 0.02, 0.1, 0.95
    scale = max(1.0, shape[0] / shape[1]) ** 0.5
    W1, b1 = muon_step(W0, G1, np.zeros(shape), lr, wd, mu)
    np.testing.assert_allclose(b1, G1, rtol=0, atol=0)
    np.testing.assert_allclose(W1, W0 * (1 - lr * wd) - lr * scale * _ns_svd((1 + mu) * G1), rtol=0, atol=1e-12)
    W2, b2 = muon_step(W1, G2, b1, lr, wd, mu)
    np.testing.assert_allclose(b2, mu * G1 + G2, rtol=0, atol=1e-15)
    U2 = G2 + mu * (mu * G1 + G2)
    np.testing.assert_allclose(W2, W1 * (1 - lr * wd) - lr * scale * _ns_svd(U2), rtol=0, atol=1e-12)
    # without Nesterov the direction is the buffer itself
    W2b, _ = muon_step(W1, G2, b1, lr, wd, mu, nesterov=False)
    np.testing.assert_allclose(W2b, W1 * (1 - lr * wd) - lr * scale * _ns_svd(mu * G1 + G2), rtol=0, atol=1e-12)


CFG = dict(seed=17, K=3, d_in=5, d_out=1, L=2, B=12, task=mlp.TASK_REG, beta1=0.9, beta2=0.999, eps=1e-8,
           decay_bias=1, width_lo=6, width_hi=9, dropout_lo=0.0, dropout_hi=0.2, lr_lo=1e-3, lr_hi=3e-3,
           wd_lo=1e-3, wd_hi=1e-2)


def test_pack_uses_muon_for_hidden_weights_and_adamw_for_the_rest():
    cfg_m = dict(CFG, optimizer="muon", muon_lr_lo=1e-2, muon_lr_hi=5e-2)
    hp = sample_hparams(cfg_m)
    assert all(1e-2 <= h["muon_lr"] <= 5e-2 for h in hp)
    rng = np.random.default_rng(1)
    X, y = rng.standard_normal((40, 5)), rng.standard_normal(40)
    idx = np.stack([rng.permutation(40)[:12] for _ in range(3)])
    om, oa = OraclePack(cfg_m, hparams=hp), OraclePack(CFG, hparams=hp)
    p0 = [[(W.copy(), b.copy()) for W, b in p] for p in om.params]
    om.train_step(X, y, idx, 1)
    oa.train_step(X, y, idx, 1)
    for k in range(3):
        h = hp[k]
        for l in range(3):
            (Wm, bm), (Wa, ba) = om.params[k][l], oa.params[k][l]
            gW = om.last_grads[k][l][0]
            np.testing.assert_array_equal(bm, ba)          # biases: AdamW in both
            if l == 2:
                np.testing.assert_array_equal(Wm, Wa)      # head: AdamW in both
                continue
            W0 = p0[k][l][0]
            sc = max(1.0, W0.shape[0] / W0.shape[1]) ** 0.5
            ref = W0 * (1 - h["muon_lr"] * h["wd"]) - h["muon_lr"] * sc * _ns_svd(1.95 * gW)
            np.testing.assert_allclose(Wm, ref, rtol=0, atol=1e-12)
            np.testing.assert_array_equal(om.m[k][l][0], gW)   # the momentum buffer after one step
            assert (om.v[k][l][0] == 0).all()


def test_muon_lr_draw_is_log_uniform():
    cfg = dict(CFG, K=4000, optimizer="muon", muon_lr_lo=1e-3, muon_lr_hi=1e-1)
    v = np.array([h["muon_lr"] for h in sample_hparams(cfg)])
    assert v.min() >= 1e-3 and v.max() <= 1e-1
    assert kstest((np.log(v) - np.log(1e-3)) / (np.log(1e-1) - np.log(1e-3)), "uniform").pvalue > 1e-4
    base = sample_hparams(dict(CFG, K=4000))
    assert [h["lr"] for h in base] == [h["lr"] for h in sample_hparams(cfg)]
