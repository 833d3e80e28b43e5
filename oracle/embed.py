"""Periodic feature embeddings of one member, plain float64 numpy.

TEST INFRASTRUCTURE ONLY (see the package header).

The paper's periodic embedding (App. "Feature Embeddings") maps each feature
x_i on its own to d_emb values,

    f(x_i) = alpha_i * [x_i, cos(w_i x_i + b_i)] + beta_i,

with w_i, b_i of length d_emb - 1 and alpha_i, beta_i of length d_emb (element-
wise products and sums, [.] a concatenation).  The backbone's input is every
feature's embedding concatenated, feature-major: column i * d_emb + j.
Initialisation as the paper states it: w_i ~ N(0, sigma) (sigma the standard
deviation), b_i = 0, alpha_i = 0, beta_i = 0.  The embedding parameters are
trained with AdamW (App. F: AdamW for everything but the main weights).
Per member, d_emb ~ UniformInt[8, 32] in steps of 4 and sigma ~
LogUniform[1e-2, 10] (App. F table).

Normal draws for w: element e (row-major [d_in, d_emb - 1]) of member k takes
block (e >> 1, 0, 100, k) of the init stream (tensor id 100); u1 = (word0 >> 8
+ 1) 2^-24 in (0, 1], u2 = (word1 >> 8) 2^-24; the Box-Muller pair
sqrt(-2 ln u1) (cos, sin)(2 pi u2) gives the cosine for even e and the sine for
odd e (Box and Muller, 1958); the value is float32(sigma z), computed in double
with the C library's log, cos and sin.
"""
import math

import numpy as np

from .philox import philox4x32_10
from .sampling import TAG_INIT, stream_key

TENSOR_W, TENSOR_B, TENSOR_ALPHA, TENSOR_BETA = 100, 101, 102, 103


def init_embedding(cfg, k, d_emb, sigma):
    """Initial embedding parameters of member k: dict of w, b [d_in, d_emb-1] and
    alpha, beta [d_in, d_emb] (float32 values in float64 arrays)."""
    d_in = int(cfg["d_in"])
    k0, k1 = stream_key(cfg["seed"], TAG_INIT)
    n = d_in * (d_emb - 1)
    blocks = np.arange((n + 1) // 2, dtype=np.uint64)
    words = philox4x32_10(blocks, 0, TENSOR_W, k, k0, k1)
    w = np.empty(n)
    for e in range(n):
        a, b = int(words[0][e >> 1]), int(words[1][e >> 1])
        u1 = ((a >> 8) + 1) * (2.0 ** -24)
        u2 = (b >> 8) * (2.0 ** -24)
        r = math.sqrt(-2.0 * math.log(u1))
        z = r * (math.cos(2.0 * math.pi * u2) if e % 2 == 0 else math.sin(2.0 * math.pi * u2))
        w[e] = float(np.float32(sigma * z))
    return dict(w=w.reshape(d_in, d_emb - 1), b=np.zeros((d_in, d_emb - 1)),
                alpha=np.zeros((d_in, d_emb)), beta=np.zeros((d_in, d_emb)))


def embed(X, emb):
    """E [N, d_in * d_emb] and the cache for ``embed_backward``."""
    X = np.asarray(X, dtype=np.float64)
    phi = X[:, :, None] * emb["w"][None] + emb["b"][None]                  # [N, d_in, d_emb-1]
    feats = np.concatenate([X[:, :, None], np.cos(phi)], axis=2)            # [N, d_in, d_emb]
    E = feats * emb["alpha"][None] + emb["beta"][None]
    return E.reshape(X.shape[0], -1), (X, phi, feats)


def embed_backward(dE, cache, emb):
    """Gradients (dict like ``emb``) from dLoss/dE [N, d_in * d_emb]."""
    X, phi, feats = cache
    N, d_in, d_emb = feats.shape
    dE = np.asarray(dE, dtype=np.float64).reshape(N, d_in, d_emb)
    dphi = -np.sin(phi) * dE[:, :, 1:] * emb["alpha"][None, :, 1:]
    return dict(w=(dphi * X[:, :, None]).sum(axis=0), b=dphi.sum(axis=0),
                alpha=(dE * feats).sum(axis=0), beta=dE.sum(axis=0))
