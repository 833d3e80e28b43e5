"""Shape, determinism and recipe checks of the synthetic workload generator (CPU)."""
import numpy as np
import pytest

from paper_2607_05380_amd import configs, synth


@pytest.mark.parametrize("name", configs.ORDER)
def test_make_data_shapes_and_determinism(name):
    cfg = configs.workload(name)
    Xtr, ytr, Xva, yva = synth.make_data(cfg, n_train=3000, n_val=500)
    assert Xtr.shape == (3000, cfg["d_in"]) and Xva.shape == (500, cfg["d_in"])
    assert Xtr.dtype == np.float32 and np.isfinite(Xtr).all()
    if cfg["task"] == "multi":
        assert ytr.dtype == np.int32 and ytr.min() >= 0 and ytr.max() < cfg["d_out"]
    else:
        assert ytr.dtype == np.float32
    if cfg["task"] == "bin":
        assert set(np.unique(ytr)) <= {0.0, 1.0}
    if cfg["task"] == "reg":
        assert abs(ytr.mean()) < 1e-5 and abs(ytr.std() - 1) < 1e-4
    again = synth.make_data(cfg, n_train=3000, n_val=500)
    np.testing.assert_array_equal(again[0], Xtr)


def test_recipes():
    X = synth.make_data(configs.workload("regression_large"), 20000, 10)[0]
    c = np.corrcoef(X[:, :60].T)
    assert abs(c[0, 1] - 0.6) < 0.03 and abs(c[0, 35]) < 0.03
    X = synth.make_data(configs.workload("binary_wide"), 5000, 10)[0]
    zero_frac = (X == 0).mean(axis=0)
    assert (zero_frac > 0.4).sum() == round(0.2 * 512)
    X = synth.make_data(configs.workload("regression_onehot"), 1000, 10)[0]
    assert np.all(X[:, 48:].sum(axis=1) == 4)


def test_batch_orders():
    cfg = configs.workload("binary_small")
    o = synth.epoch_orders(cfg, 0, 2048)
    assert o.shape == (4, 2048) and all(np.array_equal(np.sort(r), np.arange(2048)) for r in o)
    idx = synth.batch_indices(o, 3, 256)
    assert idx.dtype == np.int32 and idx.shape == (4, 256)
    np.testing.assert_array_equal(idx[2], o[2, 768:1024])
    assert not np.array_equal(o, synth.epoch_orders(cfg, 1, 2048))
