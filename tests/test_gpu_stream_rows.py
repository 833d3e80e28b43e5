"""The first layer reading its batch rows straight from a bf16 copy of the
training data (pack_bind_data): every member's base batch is a set of rows of
X chosen by its indices (Section 3.3), so loading them through the indices
inside the first GEMM gives the same bf16 operand as gathering them first.
Steps must be bit-identical to the gathered ones, in every tile set, and
match the oracle like them."""
import numpy as np
import pytest

from oracle.pack import OraclePack
from paper_2607_05380_amd import configs, synth, tabpack
from parity import TOL, check_decisions, check_tensor, compare_member, gpu_hints, make_inputs, oracle_cfg, \
    oracle_hparams, to_dev

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _state(pk, K):
    return [(pk.get_params(k), pk.get_moments(k)) for k in range(K)]


def _assert_same(ref, got, tag):
    for (p1, m1), (p2, m2) in zip(ref, got):
        for (W1, b1), (W2, b2) in zip(p1, p2):
            np.testing.assert_array_equal(W1, W2, err_msg=tag)
            np.testing.assert_array_equal(b1, b2, err_msg=tag)
        for x1, x2 in zip(m1, m2):
            for (W1, b1), (W2, b2) in zip(x1, x2):
                np.testing.assert_array_equal(W1, W2, err_msg=tag)
                np.testing.assert_array_equal(b1, b2, err_msg=tag)


# d_in 900 (the large regression's features, Pin 904: a ragged last depth
# block), d_in 61 (Pin 64, padded columns), ragged B against the 128/256 tiles
CASES = [
    ("regression_large", dict(K=5, B=500), 3000),
    ("binary_wide", dict(K=4, B=260, d_in=61), 2000),
    ("multiclass_lognormal", dict(K=5, B=700), 2500),
]


@pytest.mark.parametrize("tiles", ["small", "tall", "big"])
@pytest.mark.parametrize("name,over,n", CASES)
def test_streamed_rows_bit_identical_to_gathered(monkeypatch, tiles, name, over, n):
    monkeypatch.setenv("TABPACK_GEMM_TILES", tiles)
    cfg = configs.workload(name, **over)
    print(f"[stream_rows] {name} {over} tiles={tiles}", flush=True)
    Xtr, ytr, _, _, orders, _ = make_inputs(cfg, n, 10)
    X, y = to_dev(Xtr, ytr)
    idx = [to_dev(synth.batch_indices(orders, s, cfg["B"]))[0] for s in range(3)]
    runs = []
    for stream in (False, True):
        pk = tabpack.Pack(cfg).bind()
        if stream:
            pk.bind_data(X)
        losses = [pk.train_step(X, y, idx[s], s + 1).cpu().numpy() for s in range(3)]
        runs.append((losses, _state(pk, cfg["K"])))
    for a, b in zip(runs[0][0], runs[1][0]):
        np.testing.assert_array_equal(a, b)
    _assert_same(runs[0][1], runs[1][1], f"{name}.{tiles}")


def test_streamed_rows_parity_with_oracle():
    cfg = configs.workload("regression_large", K=5, B=500)
    Xtr, ytr, _, _, orders, _ = make_inputs(cfg, 3000, 10)
    X, y = to_dev(Xtr, ytr)
    pk = tabpack.Pack(cfg).bind().bind_data(X)
    op = OraclePack(oracle_cfg(cfg), hparams=oracle_hparams(cfg), precision="bf16")
    p0 = [[(W.copy(), b.copy()) for W, b in p] for p in op.params]
    for s in (1, 2):
        idx = synth.batch_indices(orders, s - 1, cfg["B"])
        lg = pk.train_step(X, y, to_dev(idx)[0], s).cpu().numpy()
        hints = {k: gpu_hints(pk, k, cfg, s) for k in range(cfg["K"])}
        lo = op.train_step(Xtr, ytr, idx, s, hints=hints)
        check_tensor(f"stream_rows.loss{s}", lg, lo, TOL["bf16"])
        for k in range(cfg["K"]):
            check_decisions(op, k, f"stream_rows.step{s}.m{k}")
    for k in range(cfg["K"]):
        compare_member(pk, op, k, p0[k], TOL["bf16"], steps=2, prefix="stream_rows.")


def test_streamed_rows_out_of_range_index_reads_row_zero():
    # an index outside [0, N) reads row 0 and raises the status flag, streamed
    # or gathered alike
    cfg = configs.workload("regression_large", K=3, B=300)
    Xtr, ytr, _, _, orders, _ = make_inputs(cfg, 2000, 10)
    X, y = to_dev(Xtr, ytr)
    idx = synth.batch_indices(orders, 0, cfg["B"]).copy()
    idx[1, 17], idx[2, 299] = 2000, -5
    (idx_d,) = to_dev(idx)
    runs = []
    for stream in (False, True):
        pk = tabpack.Pack(cfg).bind()
        if stream:
            pk.bind_data(X)
        loss = pk.train_step(X, y, idx_d, 1).cpu().numpy()
        assert pk.status() == tabpack.STATUS_IDX_RANGE
        runs.append(([loss], _state(pk, cfg["K"])))
    np.testing.assert_array_equal(runs[0][0][0], runs[1][0][0])
    _assert_same(runs[0][1], runs[1][1], "idx_range")


def test_bind_data_rules():
    cfg = configs.workload("regression_large", K=2, B=200)
    Xtr, ytr, _, _, orders, idx = make_inputs(cfg, 1000, 10)
    X, y, idx_d = to_dev(Xtr, ytr, idx)
    pk = tabpack.Pack(cfg).bind().bind_data(X)
    pk.train_step(X, y, idx_d, 1)
    X2 = X.clone()
    with pytest.raises(tabpack.PackError, match="pack_bind_data"):
        pk.train_step(X2, y, idx_d, 2)
    with pytest.raises(tabpack.PackError, match="pack_bind_data"):
        pk.train_step(X[:900], y[:900], idx_d, 2)
    pk.bind_data(None)  # unbound: any X again
    pk.train_step(X2, y, idx_d, 2)
    lib = tabpack.load_library()
    small = torch.empty(100, dtype=torch.bfloat16, device="cuda")
    assert lib.pack_bind_data(pk.h, X.data_ptr(), X.shape[0], small.data_ptr(), 200, None) == -1  # PACK_EINVAL
    assert b"bytes" in lib.pack_last_error()
    for over in (dict(precision="fp32"), dict(emb_lo=8, emb_hi=16, emb_step=4, sigma_lo=0.1, sigma_hi=3.0)):
        c2 = configs.workload("regression_large", K=2, B=200, **over)
        p2 = tabpack.Pack(c2).bind()
        with pytest.raises(tabpack.PackError, match="bf16"):
            p2.bind_data(X)
