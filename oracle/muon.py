"""Muon for the hidden weights of a member, plain float64 numpy.

TEST INFRASTRUCTURE ONLY (see the package header).

The paper trains the main rectangular weights of the backbone's linear layers
with Muon and every other parameter (biases, the output head) with AdamW
(§3.7 "Optimizer family", App. F).  It cites Muon (Jordan et al., 2024, "Muon:
An optimizer for hidden layers in neural networks") without restating it; the
steps below are that published algorithm, written out:

    momentum     B <- mu B + G
    direction    U = G + mu B  (Nesterov; U = B without it)
    orthogonal   O = NS(U): X = U / (||U||_F + 1e-7), taken transposed when U
                 has more rows than columns; then, `steps` times,
                     A = X X^T,  B = b A + c A A,  X = a X + B X
                 with (a, b, c) = (3.4445, -4.7750, 2.0315); transposed back.
    update       W <- W (1 - lr wd) - lr max(1, rows / cols)^(1/2) O

rows and cols are the member's true dimensions ([out, in] of the weight), not
any padded storage: the step does not depend on how a pack lays members out
(the paper notes that varying widths needs exactly this care).

Precision.  ``rnd`` (e.g. ``mlp.to_bf16``) rounds every matrix the iteration
stores -- X after the normalisation, A, B and each new X -- as the bf16
kernels do; the arithmetic between roundings stays float64.
"""
import numpy as np

NS_COEFFS = (3.4445, -4.7750, 2.0315)
NS_EPS = 1e-7


def _same(x):
    return x


def newton_schulz(U, steps=5, rnd=None):
    """O = NS(U) as above (U: [rows, cols])."""
    rnd = rnd or _same
    a, b, c = NS_COEFFS
    U = np.asarray(U, dtype=np.float64)
    tall = U.shape[0] > U.shape[1]
    X = U.T if tall else U
    X = rnd(X / (np.linalg.norm(X) + NS_EPS))
    for _ in range(steps):
        A = rnd(X @ X.T)
        B = rnd(b * A + c * (A @ A))
        X = rnd(a * X + B @ X)
    return X.T if tall else X


def muon_step(W, G, buf, lr, wd, momentum=0.95, nesterov=True, steps=5, rnd=None):
    """One Muon step of a weight W [rows, cols] with gradient G; returns (W', buf')."""
    W = np.asarray(W, dtype=np.float64)
    G = np.asarray(G, dtype=np.float64)
    buf = momentum * np.asarray(buf, dtype=np.float64) + G
    U = G + momentum * buf if nesterov else buf
    O = newton_schulz(U, steps, rnd)
    scale = max(1.0, W.shape[0] / W.shape[1]) ** 0.5
    return W * (1.0 - lr * wd) - lr * scale * O, buf
