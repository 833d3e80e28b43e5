"""Pins of the oracle's Philox block functions and dropout masks (CPU only)."""
import os

import numpy as np
import pytest

from oracle import philox
from oracle.mlp import dropout_mask
from oracle.sampling import TAG_DROPOUT, stream_key

GOLDEN = os.path.join(os.path.dirname(__file__), "golden", "philox_kat.txt")


def _kat():
    rows = []
    for line in open(GOLDEN):
        if line.startswith("#") or not line.strip():
            continue
        f = line.split()
        rows.append((f[0], int(f[1]), [int(x, 16) for x in f[2:6]],
                     [int(x, 16) for x in f[6:8]], [int(x, 16) for x in f[8:12]]))
    return rows


@pytest.mark.parametrize("row", _kat())
def test_known_answer_vectors(row):
    variant, rounds, ctr, key, out = row
    params = philox.PHILOX4x32 if variant == "philox4x32" else philox.PHILOX4x64
    assert philox.philox_scalar(ctr, key, rounds=rounds, **params) == out
    if variant == "philox4x32":
        got = philox.philox4x32_10(*ctr, *key)
        assert [int(x) for x in got] == out


@pytest.mark.parametrize("key,ctr", [((0, 0), (0, 0, 0, 0)), ((12345, 2 ** 63 + 7), (5, 2 ** 64 - 3, 9, 1)),
                                     ((2 ** 64 - 1, 3), (2 ** 64 - 2, 0, 0, 2 ** 40))])
def test_philox4x64_matches_numpy(key, ctr):
    # numpy's Philox is Philox4x64-10 and increments its counter before each block.
    bg = np.random.Philox(key=np.array(key, dtype=np.uint64), counter=np.array(ctr, dtype=np.uint64))
    got = [int(x) for x in bg.random_raw(8)]
    c = list(ctr)
    for blk in range(2):
        c[0] = (c[0] + 1) % 2 ** 64
        if c[0] == 0:
            c[1] = (c[1] + 1) % 2 ** 64
        assert philox.philox_scalar(c, key, **philox.PHILOX4x64) == got[4 * blk:4 * blk + 4]


def test_vectorised_matches_scalar():
    rng = np.random.default_rng(0)
    c = rng.integers(0, 2 ** 32, size=(4, 50), dtype=np.uint64)
    k = [int(x) for x in rng.integers(0, 2 ** 32, size=2)]
    vec = philox.philox4x32_10(c[0], c[1], c[2], c[3], *k)
    for i in range(50):
        ref = philox.philox_scalar([int(x) for x in c[:, i]], k, **philox.PHILOX4x32)
        assert [int(v[i]) for v in vec] == ref


def test_mask_counter_layout_by_hand():
    seed, k, step, layer = 2607053805, 3, 17, 2
    t = 2 ** 15
    m = dropout_mask(seed, k, step, layer, 19, 5, t)
    k0, k1 = stream_key(seed, TAG_DROPOUT)
    for r in range(19):
        for c in range(5):
            w = philox.philox_scalar([r // 8, c, (k << 8) | layer, step], [k0, k1], **philox.PHILOX4x32)
            word = w[(r % 8) // 2]
            half = word % 2 ** 16 if r % 2 == 0 else word // 2 ** 16
            assert m[r, c] == (half >= t)


@pytest.mark.parametrize("p", [0.0, 0.1, 0.25, 0.5, 0.3])
def test_mask_keep_rate(p):
    t = int(np.floor(p * 2 ** 16))
    m = dropout_mask(7, 1, 1, 1, 512, 256, t)
    n = m.size
    keep = 1.0 - t / 2 ** 16
    sigma = np.sqrt(n * keep * (1 - keep)) + 1e-12
    if p == 0.0:
        assert m.all()
    else:
        assert abs(m.sum() - n * keep) < 5 * sigma


def test_thresholds_exact():
    from oracle.sampling import member_hparams
    assert member_hparams(8, 0.0, 1e-3, 1e-3)["t"] == 0
    assert member_hparams(8, 0.25, 1e-3, 1e-3)["t"] == 2 ** 14
    assert member_hparams(8, 0.5, 1e-3, 1e-3)["t"] == 2 ** 15
    assert member_hparams(8, 0.999999, 1e-3, 1e-3)["t"] == 2 ** 16 - 1
    assert member_hparams(8, 0.5, 1e-3, 1e-3)["s"] == 2.0
