"""Per-member hyperparameter draws and initial parameters.

§3.7 Hyperparameters: every base model's hyperparameters are drawn at random
from user-given ranges.  The space used here has one hidden width per member
(shared by all of its hidden layers, as the paper's space lists a single
"Width (hidden size)" entry), a dropout rate, an AdamW learning rate and a
weight decay:

    width   ~ UniformInt[width_lo, width_hi]
    dropout ~ Uniform[dropout_lo, dropout_hi]
    lr      ~ LogUniform[lr_lo, lr_hi]
    wd      ~ LogUniform[wd_lo, wd_hi]
    depth   ~ UniformInt[depth_lo, depth_hi]   (App. F: "# layers"; only when a
              depth range is given, otherwise every member has L hidden blocks)
    muon_lr ~ LogUniform[muon_lr_lo, muon_lr_hi]  (App. F: "Muon learning rate";
              only with the Muon optimizer)
    d_emb   ~ emb_lo + emb_step UniformInt[0, (emb_hi - emb_lo) / emb_step],
    sigma   ~ LogUniform[sigma_lo, sigma_hi]      (App. F: periodic embeddings;
              only when emb_lo > 0)

Random words come from Philox4x32-10 (``oracle.philox``) with the stream tag
folded into the key:  key = (seed mod 2**32, (seed >> 32) XOR (tag << 28)),
tag 1 = hyperparameters, 2 = initial parameters, 3 = dropout.

* hyperparameters of member k: block (k, 0, 0, 0) gives two doubles u0, u1
  (width, dropout); block (k, 1, 0, 0) gives u2, u3 (lr, wd); block
  (k, 2, 0, 0) gives u4 (depth; its last two words are unused); block
  (k, 3, 0, 0) gives u5 (the Muon learning rate; last two words unused);
  block (k, 4, 0, 0) gives u6 (d_emb) and u7 (sigma).  A double is
  built from two words (a, b) as ((a >> 5) * 2**26 + (b >> 6)) * 2**-53.
* initial parameters follow torch.nn.Linear's default: W and b uniform on
  [-1/sqrt(fan_in), 1/sqrt(fan_in)], fan_in = the member's true input width.
  Element e (row-major [out][in]) of tensor t of member k takes word (e & 3) of
  block (e >> 2 mod 2**32, e >> 34, t, k); u = (word >> 8) * 2**-24 and the
  value is float32((2u - 1) * bound), evaluated in float64.  Tensor ids:
  W_l -> 2(l-1), b_l -> 2(l-1)+1 for hidden layers l = 1..L_k (the member's
  depth), W_out -> 2 L_k, b_out -> 2 L_k + 1.

Dropout: t_k = floor(p_k * 2**16) is the integer keep threshold of a 16-bit
draw and s_k = 1/(1 - p_k) the inverted-dropout scale (see
``mlp.dropout_mask``).  The drop probability realised is t_k / 2**16, within
2**-16 of p_k.
"""
import math

import numpy as np

from .philox import philox4x32_10

TAG_HPARAM, TAG_INIT, TAG_DROPOUT = 1, 2, 3


def stream_key(seed, tag):
    seed = int(seed)
    return (seed & 0xFFFFFFFF, ((seed >> 32) ^ (tag << 28)) & 0xFFFFFFFF)


def _u53(a, b):
    return ((int(a) >> 5) * 67108864.0 + (int(b) >> 6)) * (1.0 / 9007199254740992.0)


def _log_uniform(lo, hi, u):
    if lo == hi:
        return float(lo)
    return math.exp(math.log(lo) + u * (math.log(hi) - math.log(lo)))


def sample_hparams(cfg):
    """List of K dicts {width, dropout, lr, wd, depth, t, s} for cfg (a plain
    dict; a depth range is given by depth_lo, depth_hi, absent or 0 for none)."""
    k0, k1 = stream_key(cfg["seed"], TAG_HPARAM)
    dlo, dhi = int(cfg.get("depth_lo", 0) or 0), int(cfg.get("depth_hi", 0) or 0)
    out = []
    for k in range(cfg["K"]):
        w = [int(x) for x in philox4x32_10(k, 0, 0, 0, k0, k1)]
        u0, u1 = _u53(w[0], w[1]), _u53(w[2], w[3])
        w = [int(x) for x in philox4x32_10(k, 1, 0, 0, k0, k1)]
        u2, u3 = _u53(w[0], w[1]), _u53(w[2], w[3])
        lo, hi = cfg["width_lo"], cfg["width_hi"]
        width = lo + int(math.floor(u0 * (hi - lo + 1)))
        p = cfg["dropout_lo"] + u1 * (cfg["dropout_hi"] - cfg["dropout_lo"])
        depth = cfg.get("L")
        if dlo > 0:
            w = [int(x) for x in philox4x32_10(k, 2, 0, 0, k0, k1)]
            depth = dlo + int(math.floor(_u53(w[0], w[1]) * (dhi - dlo + 1)))
        hp = member_hparams(width, p, _log_uniform(cfg["lr_lo"], cfg["lr_hi"], u2),
                            _log_uniform(cfg["wd_lo"], cfg["wd_hi"], u3), depth)
        if cfg.get("optimizer", "adamw") == "muon":
            w = [int(x) for x in philox4x32_10(k, 3, 0, 0, k0, k1)]
            hp["muon_lr"] = _log_uniform(cfg["muon_lr_lo"], cfg["muon_lr_hi"], _u53(w[0], w[1]))
        if int(cfg.get("emb_lo", 0) or 0) > 0:
            w = [int(x) for x in philox4x32_10(k, 4, 0, 0, k0, k1)]
            lo, hi, st = int(cfg["emb_lo"]), int(cfg["emb_hi"]), int(cfg["emb_step"])
            hp["d_emb"] = lo + st * int(math.floor(_u53(w[0], w[1]) * ((hi - lo) // st + 1)))
            hp["sigma"] = _log_uniform(cfg["sigma_lo"], cfg["sigma_hi"], _u53(w[2], w[3]))
        out.append(hp)
    return out


def member_hparams(width, dropout, lr, wd, depth=None, muon_lr=None):
    """depth None: the pack's L hidden blocks; muon_lr only for Muon packs."""
    p = float(dropout)
    t = min(int(math.floor(p * 65536.0)), 0xFFFF)
    out = dict(width=int(width), dropout=p, lr=float(lr), wd=float(wd),
               t=t, s=1.0 / (1.0 - p), depth=None if depth is None else int(depth))
    if muon_lr is not None:
        out["muon_lr"] = float(muon_lr)
    return out


def member_depth(cfg, hp):
    """Hidden blocks of a member: its own depth, or the pack's L."""
    d = hp.get("depth") if hp is not None else None
    return int(cfg["L"]) if d is None else int(d)


def layer_shapes(cfg, width, depth=None, d_first=None):
    """[(out, in), ...] for W_1..W_depth and the head W_out of one member;
    d_first: the first layer's input width (d_in * d_emb with embeddings)."""
    L = int(cfg["L"]) if depth is None else int(depth)
    shapes = [(width, cfg["d_in"] if d_first is None else int(d_first))] + [(width, width)] * (L - 1)
    shapes.append((cfg["d_out"], width))
    return shapes


def init_member(cfg, k, width, depth=None, d_first=None):
    """Initial (W, b) pairs of member k, float32 values held in float64 arrays."""
    k0, k1 = stream_key(cfg["seed"], TAG_INIT)
    params = []
    for i, (n_out, n_in) in enumerate(layer_shapes(cfg, width, depth, d_first)):
        bound = 1.0 / math.sqrt(n_in)
        pair = []
        for t, n in ((2 * i, n_out * n_in), (2 * i + 1, n_out)):
            e = np.arange(n, dtype=np.uint64)
            words = philox4x32_10(e >> np.uint64(2) & np.uint64(0xFFFFFFFF),
                                  e >> np.uint64(34), t, k, k0, k1)
            wsel = np.choose((e & np.uint64(3)).astype(np.int64), words)
            u = (wsel >> np.uint32(8)).astype(np.float64) * (2.0 ** -24)
            vals = ((2.0 * u - 1.0) * bound).astype(np.float32).astype(np.float64)
            pair.append(vals)
        params.append((pair[0].reshape(n_out, n_in), pair[1]))
    return params
