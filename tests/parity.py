"""Helpers shared by the GPU parity tests: run the HIP library and the fp64 oracle
on the same seeded inputs and compare them element by element.

Element test: |gpu - ref| <= atol + rtol * |ref|.

bf16 GEMMs (fp32 master weights).  The reference is the oracle's bf16 policy
(bf16 operands of the hidden matrix products, see oracle.mlp), so that the
ReLU/dropout decisions rest on the same rounded forward values as the kernels'.
Losses and outputs: rtol 2e-2, atol 1e-3.  Against the exact fp64 oracle about
0.1-0.5% of the ReLU decisions legitimately flip (|Z| below the bf16 rounding
noise) and each flip moves a whole dZ element, so there gradients are held to a
relative Frobenius error of FP64_GRAD_FROB.
fp32 MFMA mode: rtol 1e-4 everywhere.

Gradients meet three conditions: every element within the literal tolerance
(bf16 2e-2 rel / 1e-3 abs; fp32 1e-4 rel / 1e-5 abs), at most ``frac`` of the
elements outside the strict per-tensor band (rtol, gfloor * max|g|), and a
relative Frobenius error <= frob.  The strict band can be missed by a few
elements because an fp32-accumulated Z a hair from zero may take the other ReLU
branch than the fp64-accumulated one; one such flip moves a single term of a
whole weight-gradient row.

Parameters after t steps are checked through their update d = theta_t -
theta_0 (theta_0 is the bit-identical initial value on both sides):
  * |d_gpu - d_ref| <= 2 t lr (1 + 1e-6) + 1e-7 for every element (an AdamW
    step moves an element by at most about lr);
  * |d_gpu - d_ref| <= upd * lr for all but a share upd_frac of the elements
    (the first step is about -lr sign(g), so this pins lr_k, wd_k and the
    update rule per member);
  * after one step, theta within the literal tolerance wherever the two
    gradients agree to half the oracle's magnitude and that magnitude is well
    above AdamW's eps (>= 1e-5): the first step -lr g / (|g| + eps) is then the
    same on both sides.  Elsewhere -- gradients so small or so perturbed by
    legitimate ReLU-decision flips that sign(g) or |g| / (|g| + eps) differ --
    only the 2 lr bound and the upd_frac share apply.
"""
import numpy as np

from oracle.sampling import member_hparams, sample_hparams
from paper_2607_05380_amd import synth

TOL = {"bf16": dict(rtol=2e-2, atol=1e-3, gfloor=1e-3, frob=2e-2, lit_rtol=2e-2, lit_atol=1e-3, frac=0.25,
                   upd=2e-2, upd_frac=0.05),
       "fp32": dict(rtol=1e-4, atol=1e-6, gfloor=1e-4, frob=1e-4, lit_rtol=1e-4, lit_atol=1e-5, frac=0.01,
                    upd=1e-3, upd_frac=1e-3)}

FP64_GRAD_FROB = 0.25

ORACLE_KEYS = ("seed", "K", "d_in", "d_out", "L", "B", "task", "beta1", "beta2", "eps", "decay_bias",
               "width_lo", "width_hi", "dropout_lo", "dropout_hi", "lr_lo", "lr_hi", "wd_lo", "wd_hi")


def oracle_cfg(cfg):
    out = {k: cfg[k] for k in ORACLE_KEYS}
    out["depth_lo"], out["depth_hi"] = cfg.get("depth_lo", 0), cfg.get("depth_hi", 0)
    for k, v in (("optimizer", "adamw"), ("muon_lr_lo", 1e-3), ("muon_lr_hi", 1e-1), ("muon_momentum", 0.95),
                 ("muon_nesterov", 1), ("ns_steps", 5), ("emb_lo", 0), ("emb_hi", 0), ("emb_step", 4),
                 ("sigma_lo", 1e-2), ("sigma_hi", 10.0)):
        out[k] = cfg.get(k, v)
    return out


def oracle_hparams(cfg, members=None):
    if members is None:
        return sample_hparams(oracle_cfg(cfg))
    out = [member_hparams(m["width"], m["dropout"], m["lr"], m["wd"], m.get("depth"), m.get("muon_lr"))
           for m in members]
    for h, m in zip(out, members):
        if m.get("d_emb"):
            h["d_emb"], h["sigma"] = int(m["d_emb"]), float(m["sigma"])
    return out


def close_mask(gpu, ref, rtol, atol):
    return np.abs(np.asarray(gpu, np.float64) - ref) <= atol + rtol * np.abs(ref)


def check_tensor(name, gpu, ref, tol, grad=False, report=None):
    gpu = np.asarray(gpu, np.float64)
    ref = np.asarray(ref, np.float64)
    assert gpu.shape == ref.shape, (name, gpu.shape, ref.shape)
    assert np.isfinite(gpu).all(), name
    mx = np.abs(ref).max() if ref.size else 0.0
    frob = np.linalg.norm(gpu - ref) / max(np.linalg.norm(ref), 1e-30)
    if not grad:
        ok = close_mask(gpu, ref, tol["rtol"], tol["atol"])
        if report is not None:
            report.append((name, float(frob), int((~ok).sum())))
        assert ok.all(), f"{name}: {(~ok).sum()} of {ok.size} elements out of tolerance; worst " \
                         f"{np.abs(gpu - ref)[~ok].max():.3e} (max|ref| {mx:.3e}), frob {frob:.2e}"
        return frob
    strict = close_mask(gpu, ref, tol["rtol"], tol["gfloor"] * mx)
    literal = close_mask(gpu, ref, tol["lit_rtol"], tol["lit_atol"])
    if report is not None:
        report.append((name, float(frob), int((~strict).sum())))
    assert literal.all(), f"{name}: {(~literal).sum()} of {ok_size(gpu)} elements outside the literal " \
                          f"tolerance; worst {np.abs(gpu - ref)[~literal].max():.3e}"
    assert (~strict).mean() <= tol["frac"], f"{name}: {(~strict).sum()} of {gpu.size} elements outside " \
                                            f"the strict band (max|ref| {mx:.3e}), frob {frob:.2e}"
    if mx > 0:
        assert frob <= tol["frob"], f"{name}: relative Frobenius error {frob:.3e}"
    return frob


def ok_size(a):
    return np.asarray(a).size


def check_update(name, p_gpu, p_ref, p0, g_gpu, g_ref, lr, tol, steps=1, upd_frac=None, report=None):
    """Parameter check after ``steps`` AdamW steps (see the module notes)."""
    p_gpu = np.asarray(p_gpu, np.float64)
    d_gpu, d_ref = p_gpu - p0, p_ref - p0
    err = np.abs(d_gpu - d_ref)
    assert (err <= 2 * steps * lr * (1 + 1e-6) + 1e-7).all(), \
        f"{name}: update differs by {err.max():.3e} > 2 t lr ({2 * steps * lr:.3e})"
    off = float((err > tol["upd"] * lr + 1e-7).mean())
    if report is not None:
        report.append((name, off, int((err > tol["upd"] * lr + 1e-7).sum())))
    lim = tol["upd_frac"] if upd_frac is None else upd_frac
    assert off <= lim, f"{name}: {off:.2%} of the updates differ by more than {tol['upd']} lr"
    if steps == 1 and g_gpu is not None:
        lit = close_mask(p_gpu, p_ref, tol["lit_rtol"], tol["lit_atol"])
        g_gpu = np.asarray(g_gpu, np.float64)
        same = (np.abs(g_gpu - g_ref) <= 0.5 * np.abs(g_ref)) & (np.abs(g_ref) >= 1e-5)
        bad = ~lit & same
        if bad.any():
            i = np.flatnonzero(bad.ravel())[:6]
            detail = "; ".join(f"g_ref {np.ravel(g_ref)[j]:.3e} g_gpu {np.ravel(g_gpu)[j]:.3e} d_ref "
                               f"{d_ref.ravel()[j]:.3e} d_gpu {d_gpu.ravel()[j]:.3e}" for j in i)
            raise AssertionError(f"{name}: {bad.sum()} parameters outside the literal tolerance (lr {lr:.3e}): "
                                 f"{detail}")
    return off


def make_inputs(cfg, n_train, n_val, epoch=0, step_in_epoch=0):
    Xtr, ytr, Xva, yva = synth.make_data(cfg, n_train=n_train, n_val=n_val)
    orders = synth.epoch_orders(cfg, epoch, n_train)
    idx = synth.batch_indices(orders, step_in_epoch, cfg["B"])
    return Xtr, ytr, Xva, yva, orders, idx


def to_dev(*arrays):
    import torch
    return [torch.from_numpy(np.ascontiguousarray(a)).cuda() for a in arrays]


def compare_member(pk, op, k, p0, tol, steps=1, report=None, prefix=""):
    """Compare member k of the GPU pack with member k of the oracle pack after
    ``steps`` steps; p0 = the member's initial parameters."""
    lr = op.hp[k]["lr"]
    g_gpu = pk.get_grads(k)
    p_gpu = pk.get_params(k)
    m_gpu, v_gpu = pk.get_moments(k)
    names = [f"W{l+1}" for l in range(len(op.params[k]) - 1)] + ["Wout"]
    for l, nm in enumerate(names):
        gW, gb = op.last_grads[k][l]
        tag = f"{prefix}m{k}.{nm}"
        check_tensor(tag + ".grad", g_gpu[l][0], gW, tol, grad=True, report=report)
        check_tensor(tag + ".bgrad", g_gpu[l][1], gb, tol, grad=True, report=report)
        check_update(tag, p_gpu[l][0], op.params[k][l][0], p0[l][0], g_gpu[l][0], gW, lr, tol, steps, report=report)
        check_update(tag + ".b", p_gpu[l][1], op.params[k][l][1], p0[l][1], g_gpu[l][1], gb, lr, tol, steps,
                     report=report)
        check_tensor(tag + ".m", m_gpu[l][0], op.m[k][l][0], tol, grad=True, report=report)
        # v = sum of (1-b2) b2^i g^2: compare sqrt(v), which scales like |g|
        check_tensor(tag + ".sqrtv", np.sqrt(v_gpu[l][0]), np.sqrt(op.v[k][l][0]), tol, grad=True,
                     report=report)


def compare_member_fp64(pk, op64, k, p0, report=None, prefix=""):
    """bf16 GPU member vs the exact fp64 oracle: gradient Frobenius error bounded
    by FP64_GRAD_FROB; updates as in check_update with up to 10% of the first
    step's signs reversed by the bf16 ReLU-decision flips."""
    tol = TOL["bf16"]
    lr = op64.hp[k]["lr"]
    g_gpu = pk.get_grads(k)
    p_gpu = pk.get_params(k)
    worst = 0.0
    for l in range(len(op64.params[k])):
        gW, gb = op64.last_grads[k][l]
        for i, (nm, r) in enumerate((("W", gW), ("b", gb))):
            g = np.asarray(g_gpu[l][i], np.float64)
            frob = np.linalg.norm(g - r) / max(np.linalg.norm(r), 1e-30)
            worst = max(worst, frob)
            assert frob <= FP64_GRAD_FROB, f"{prefix}m{k}.{nm}{l}: grad frob vs fp64 {frob:.3f}"
            check_update(f"{prefix}m{k}.{nm}{l}", p_gpu[l][i], op64.params[k][l][i], p0[l][i], g, r, lr, tol,
                         upd_frac=0.10, report=report)
    return worst
