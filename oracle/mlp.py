"""One base model: forward, loss, backward, AdamW -- plain float64 numpy.

§3.3 Model Pack defines the base model as a sequence of Linear-ReLU-Dropout
blocks; the output head is a plain Linear layer with no activation or dropout.
Parameters use nn.Linear's layout: W is [out, in], b is [out], so a layer maps
H -> H @ W.T + b.

Losses (App. F, training of DL models): cross-entropy for classification
(binary cross-entropy with logits for two classes) and mean squared error for
regression, each averaged over the member's base batch of B rows.

Precision.  By default everything is float64 (the exact definition).  With
``rnd=to_bf16`` the same steps follow a bf16 mixed-precision policy: the
operands of every hidden-layer matrix product are bfloat16 values -- the
network input X, the hidden weights W_1..W_L, the stored activations H_l (after
bias, ReLU, dropout and scaling) and the stored pre-activation gradients dZ_l
-- while the head weights, biases, bias gradients (summed from dZ before it is
rounded), losses and all accumulations stay in high precision.  Rounding is
round-to-nearest-even of the float32 value.  The ReLU/dropout decisions of
the backward pass are then taken on the same bf16-rounded forward values the
bf16 kernels use, which is what makes an element-wise comparison meaningful.
"""
import numpy as np

from .philox import philox4x32_10
from .sampling import TAG_DROPOUT, stream_key

TASK_REG, TASK_BIN, TASK_MULTI = "reg", "bin", "multi"


def dropout_mask(seed, k, step, layer, B, width, t):
    """Keep mask (bool [B, width]) of member k, hidden layer ``layer`` (1-based).

    Element (r, c) reads the 16-bit half (r & 1) (0: low, 1: high bits) of
    word ((r >> 1) & 3) of the Philox4x32-10 block with counter
    (r >> 3, c, (k << 8) | layer, step mod 2**32) under the dropout stream key,
    and is kept iff that half >= t (t = floor(p * 2**16)); p = 0 keeps all.
    """
    k0, k1 = stream_key(seed, TAG_DROPOUT)
    r = np.arange(B, dtype=np.uint64)[:, None]
    c = np.arange(width, dtype=np.uint64)[None, :]
    words = philox4x32_10(r >> np.uint64(3), c, (int(k) << 8) | int(layer),
                          int(step) & 0xFFFFFFFF, k0, k1)
    sel = np.broadcast_to(((r >> np.uint64(1)) & np.uint64(3)).astype(np.int64), (B, width))
    shift = np.broadcast_to((r & np.uint64(1)) * np.uint64(16), (B, width)).astype(np.uint32)
    half = (np.choose(sel, words) >> shift) & np.uint32(0xFFFF)
    return half >= np.uint32(t)


def to_bf16(x):
    """Round to the nearest bfloat16 value (ties to even) via float32; float64 result."""
    u = np.asarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    u = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) & np.uint64(0xFFFF0000)
    return u.astype(np.uint32).view(np.float32).astype(np.float64)


def _same(x):
    return x


def forward(params, X, masks=None, scale=1.0, rnd=None):
    """Returns (Y, cache).  masks[l] is the keep mask of hidden layer l+1 or None."""
    rnd = rnd or _same
    H = rnd(np.asarray(X, dtype=np.float64))
    cache = {"H": [H], "Z": [], "rnd": rnd}
    L = len(params) - 1
    for l in range(L):
        W, b = params[l]
        Z = H @ rnd(W).T + b
        H = np.maximum(Z, 0.0)
        if masks is not None:
            H = H * masks[l] * scale
        H = rnd(H)
        cache["Z"].append(Z)
        cache["H"].append(H)
    Wo, bo = params[L]
    return H @ Wo.T + bo, cache


def loss_and_dy(Y, y, task):
    """Batch-mean loss and dLoss/dY for one member."""
    B = Y.shape[0]
    if task == TASK_REG:
        diff = Y[:, 0] - np.asarray(y, dtype=np.float64)
        return float(np.mean(diff * diff)), (2.0 * diff / B)[:, None]
    if task == TASK_BIN:
        z = Y[:, 0]
        t = np.asarray(y, dtype=np.float64)
        loss = np.maximum(z, 0.0) - z * t + np.log1p(np.exp(-np.abs(z)))
        sig = 1.0 / (1.0 + np.exp(-z))
        return float(np.mean(loss)), ((sig - t) / B)[:, None]
    if task == TASK_MULTI:
        lab = np.asarray(y, dtype=np.int64)
        mx = Y.max(axis=1, keepdims=True)
        lse = mx[:, 0] + np.log(np.exp(Y - mx).sum(axis=1))
        loss = lse - Y[np.arange(B), lab]
        P = np.exp(Y - lse[:, None])
        P[np.arange(B), lab] -= 1.0
        return float(np.mean(loss)), P / B
    raise ValueError(task)


# Decisions within this fraction of rms(Z) of the ReLU threshold may take
# either branch in an implementation that accumulates Z in another order or
# precision and rounds upstream activations at other points (see
# ``relu_derivative``): a bf16 activation that rounds the other way moves every
# pre-activation of its row in the next layer by up to one bf16 step of that
# term, and such moves compound over the layers.
HINT_WINDOW = 2e-2


def relu_derivative(Z, hint=None, window=HINT_WINDOW, stats=None):
    """The ReLU derivative [Z > 0] (0 at 0).

    ``hint`` (int8 array like Z: 1 positive, 0 not positive, -1 unknown) gives
    another implementation's decisions.  Where |Z| <= window * rms(Z) both
    branches are correct up to that implementation's accumulation rounding, so
    the hint's decision is taken there; everywhere else the decision is this
    function's own.  ``stats`` (a dict) receives the counts: elements inside
    the window, hints taken there that differ from [Z > 0], known hints
    outside the window that differ from it (a disagreement the window does not
    excuse), all known hints, and the largest |Z| / rms(Z) of a differing
    hint."""
    own = Z > 0.0
    if hint is None:
        return own
    hint = np.asarray(hint)
    assert hint.shape == Z.shape, (hint.shape, Z.shape)
    rms = np.sqrt(np.mean(Z * Z)) if Z.size else 0.0
    inside = np.abs(Z) <= window * rms
    known = hint >= 0
    differ = known & (own != (hint == 1))
    if stats is not None:
        stats["window"] = stats.get("window", 0) + int(inside.sum())
        stats["taken"] = stats.get("taken", 0) + int((differ & inside).sum())
        stats["outside"] = stats.get("outside", 0) + int((differ & ~inside).sum())
        stats["decisions"] = stats.get("decisions", 0) + int(known.sum())
        if differ.any() and rms > 0:
            # how far from the threshold the furthest disagreement lies, in rms(Z)
            stats["max_ratio"] = max(stats.get("max_ratio", 0.0), float(np.abs(Z[differ]).max() / rms))
    return np.where(inside & known, hint == 1, own)


def backward(params, cache, dY, masks=None, scale=1.0, input_grad=False, hints=None, stats=None,
             window=HINT_WINDOW):
    """Gradients [(dW, db), ...] in the layout of ``params``; with input_grad
    also dLoss/dH_0 (the gradient of the network's input), as a second value.
    hints[l]: optional decisions for hidden layer l + 1 (``relu_derivative``)."""
    L = len(params) - 1
    rnd = cache.get("rnd", _same)
    grads = [None] * (L + 1)
    H = cache["H"]
    Wo, _ = params[L]
    grads[L] = (dY.T @ H[L], dY.sum(axis=0))
    dH = dY @ Wo
    for l in range(L - 1, -1, -1):
        dZ = dH * relu_derivative(cache["Z"][l], None if hints is None else hints[l], window, stats)
        if masks is not None:
            dZ = dZ * masks[l] * scale
        db = dZ.sum(axis=0)
        dZ = rnd(dZ)
        W, _ = params[l]
        grads[l] = (dZ.T @ H[l], db)
        if l > 0 or input_grad:
            dH = dZ @ rnd(W)
    return (grads, dH) if input_grad else grads


def adamw_step(theta, g, m, v, t, lr, wd, beta1, beta2, eps, decay=True):
    """One decoupled-weight-decay Adam step (Loshchilov & Hutter), torch order.

    theta <- theta * (1 - lr*wd); m <- b1 m + (1-b1) g; v <- b2 v + (1-b2) g^2;
    theta <- theta - lr/(1-b1^t) * m / (sqrt(v)/sqrt(1-b2^t) + eps).
    Returns new (theta, m, v).
    """
    if decay:
        theta = theta * (1.0 - lr * wd)
    m = beta1 * m + (1.0 - beta1) * g
    v = beta2 * v + (1.0 - beta2) * g * g
    bc1 = 1.0 - beta1 ** t
    bc2 = 1.0 - beta2 ** t
    denom = np.sqrt(v) / np.sqrt(bc2) + eps
    return theta - (lr / bc1) * m / denom, m, v
