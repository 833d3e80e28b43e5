"""Host-side checks of the C ABI that need no GPU: the library loads and exports
every declared symbol, pack_init validates its arguments, and the library's own
hyperparameter sampler and initialiser agree with the independent oracle."""
import ctypes
import os
import re

import numpy as np
import pytest

from paper_2607_05380_amd import configs, tabpack
from oracle.sampling import init_member, sample_hparams

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "tabpack.h")


def declared():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^(?:int|const char\*)\s+(pack_\w+)\s*\(", text, flags=re.M)))


def test_library_exports_every_declared_symbol():
    lib = tabpack.load_library()
    names = declared()
    assert len(names) >= 17
    for n in names:
        assert hasattr(lib, n), n
    assert sorted(tabpack.SYMBOLS) == names


def oracle_cfg(cfg):
    out = {k: cfg[k] for k in ("seed", "K", "d_in", "d_out", "L", "width_lo", "width_hi", "dropout_lo",
                               "dropout_hi", "lr_lo", "lr_hi", "wd_lo", "wd_hi")}
    out["depth_lo"], out["depth_hi"] = cfg.get("depth_lo", 0), cfg.get("depth_hi", 0)
    for k, v in (("optimizer", "adamw"), ("muon_lr_lo", 1e-3), ("muon_lr_hi", 1e-1)):
        out[k] = cfg.get(k, v)
    return out


@pytest.mark.parametrize("name", configs.ORDER)
def test_sampled_hparams_match_oracle(name):
    cfg = configs.workload(name)
    pk = tabpack.Pack(cfg)
    got = pk.hparams()
    ref = sample_hparams(oracle_cfg(cfg))
    q = 32
    for g, r in zip(got, ref):
        assert g["width"] == r["width"] and g["t"] == r["t"]
        assert g["padded_width"] == -(-r["width"] // q) * q
        for key in ("dropout", "lr", "wd", "s"):
            assert g[key] == pytest.approx(r[key], rel=4e-16, abs=0), key


@pytest.mark.parametrize("name", ["binary_small", "multiclass_lognormal"])
def test_initial_params_bit_equal_oracle(name):
    cfg = configs.workload(name)
    pk = tabpack.Pack(cfg)
    for k in range(min(cfg["K"], 3)):
        ref = init_member(oracle_cfg(cfg), k, pk.hparams()[k]["width"])
        got = pk.get_params(k)
        for (W, b), (Wr, br) in zip(got, ref):
            np.testing.assert_array_equal(W, Wr.astype(np.float32))
            np.testing.assert_array_equal(b, br.astype(np.float32))


def test_explicit_members_and_roundtrip():
    cfg = configs.workload("binary_small")
    members = [dict(width=w, dropout=p, lr=1e-3, wd=1e-4) for w, p in ((1, 0.0), (31, 0.25), (32, 0.5), (33, 0.1))]
    pk = tabpack.Pack(cfg, members=members)
    hp = pk.hparams()
    assert [h["width"] for h in hp] == [1, 31, 32, 33]
    assert [h["padded_width"] for h in hp] == [32, 32, 32, 64]
    assert hp[1]["t"] == 2 ** 14 and hp[2]["t"] == 2 ** 15 and hp[2]["s"] == 2.0
    p = pk.get_params(3)
    p2 = [(W * 2, b - 1) for W, b in p]
    pk.set_params(3, p2)
    for (W, b), (W2, b2) in zip(pk.get_params(3), p2):
        np.testing.assert_array_equal(W, W2)
        np.testing.assert_array_equal(b, b2)
    n = 33 * 8 + 33 + 33 * 33 + 33 + 33 + 1
    assert pk.param_count(3) == n


@pytest.mark.parametrize("field,value", [("K", 0), ("L", 0), ("L", 9), ("B", 0), ("d_out", 2), ("width_lo", 0),
                                         ("dropout_hi", 1.0), ("lr_lo", 0.0), ("quantum", 12), ("task", "x")])
def test_invalid_configs_rejected(field, value):
    cfg = configs.workload("binary_small")
    cfg[field] = value
    if field == "task":
        with pytest.raises(KeyError):
            tabpack.Pack(cfg)
        return
    with pytest.raises(tabpack.PackError) as e:
        tabpack.Pack(cfg)
    assert "tabpack error -1" in str(e.value)


def test_state_errors_without_bind():
    lib = tabpack.load_library()
    pk = tabpack.Pack(configs.workload("binary_small"))
    rc = lib.pack_train_step(pk.h, 16, 16, 10, 16, 1, 16, None)
    assert rc == -2 and b"pack_bind" in lib.pack_last_error()
    out = np.empty(10, np.float32)
    assert lib.pack_get_grads(pk.h, 0, out.ctypes.data) == -2
    assert lib.pack_get_params(pk.h, 7, out.ctypes.data) == -1
    n = ctypes.c_size_t()
    assert lib.pack_workspace_size(pk.h, ctypes.byref(n)) == 0 and n.value > 0
    assert lib.pack_select_workspace_size(0, 10, ctypes.byref(n)) == -1
    assert lib.pack_init(None, ctypes.byref(ctypes.c_void_p())) == -1


def test_sampled_depths_and_init_match_oracle():
    # App. F samples the number of layers per member: depth ~ UniformInt[lo, hi]
    cfg = configs.workload("regression_onehot", K=40, L=4, depth_lo=1, depth_hi=4)
    pk = tabpack.Pack(cfg)
    got = pk.hparams()
    ref = sample_hparams(oracle_cfg(cfg))
    assert [g["depth"] for g in got] == [r["depth"] for r in ref]
    assert set(g["depth"] for g in got) == {1, 2, 3, 4}
    for k in range(6):
        p = pk.get_params(k)
        r = init_member(oracle_cfg(cfg), k, got[k]["width"], got[k]["depth"])
        assert len(p) == len(r) == got[k]["depth"] + 1
        for (W, b), (Wr, br) in zip(p, r):
            np.testing.assert_array_equal(W, Wr.astype(np.float32))
            np.testing.assert_array_equal(b, br.astype(np.float32))
    # without a range every member has L blocks; explicit depths are taken as given
    assert all(h["depth"] == 4 for h in tabpack.Pack(dict(cfg, depth_lo=0, depth_hi=0)).hparams())
    one = tabpack.Pack(dict(cfg, K=2), members=[dict(width=9, dropout=0.1, lr=1e-3, wd=1e-3, depth=2),
                                                 dict(width=9, dropout=0.1, lr=1e-3, wd=1e-3)])
    assert [h["depth"] for h in one.hparams()] == [2, 4]
    assert one.param_count(0) == 9 * 64 + 9 + 9 * 9 + 9 + 9 + 1


@pytest.mark.parametrize("lo,hi", [(0, 2), (2, 1), (1, 5), (-1, 3)])
def test_invalid_depth_ranges_rejected(lo, hi):
    cfg = configs.workload("regression_onehot", K=2, L=4, depth_lo=lo, depth_hi=hi)
    with pytest.raises(tabpack.PackError, match="depth"):
        tabpack.Pack(cfg)


def test_sampled_muon_lrs_match_oracle():
    cfg = configs.workload("regression_large", K=50, optimizer="muon", muon_lr_lo=1e-3, muon_lr_hi=1e-1)
    got = tabpack.Pack(cfg).hparams()
    ref = sample_hparams(oracle_cfg(cfg))
    for g, r in zip(got, ref):
        assert g["muon_lr"] == pytest.approx(r["muon_lr"], rel=4e-16, abs=0)
        assert g["lr"] == pytest.approx(r["lr"], rel=4e-16, abs=0)
    # the AdamW-only pack draws the same widths, rates and decays
    base = tabpack.Pack(dict(cfg, optimizer="adamw")).hparams()
    assert [(b["width"], b["lr"], b["wd"]) for b in base] == [(g["width"], g["lr"], g["wd"]) for g in got]
    assert all(b["muon_lr"] == 0.0 for b in base)
    with pytest.raises(tabpack.PackError, match="Muon"):
        tabpack.Pack(dict(cfg, muon_lr_lo=0.0))


def test_embedding_hparams_and_init_match_oracle():
    from oracle.embed import init_embedding
    cfg = configs.workload("regression_onehot", K=6, emb_lo=8, emb_hi=32, emb_step=4, sigma_lo=1e-2, sigma_hi=10.0)
    oc = dict(oracle_cfg(cfg), emb_lo=8, emb_hi=32, emb_step=4, sigma_lo=1e-2, sigma_hi=10.0)
    pk = tabpack.Pack(cfg)
    got = pk.hparams()
    ref = sample_hparams(oc)
    for g, r in zip(got, ref):
        assert g["d_emb"] == r["d_emb"] and g["sigma"] == pytest.approx(r["sigma"], rel=4e-16, abs=0)
    for k in range(3):
        params = pk.get_params(k)
        emb, layers = params[0], params[1:]
        ref_emb = init_embedding(oc, k, got[k]["d_emb"], got[k]["sigma"])
        for n in ("w", "b", "alpha", "beta"):
            np.testing.assert_array_equal(emb[n], ref_emb[n].astype(np.float32), err_msg=n)
        ref_layers = init_member(oc, k, got[k]["width"], None, cfg["d_in"] * got[k]["d_emb"])
        assert layers[0][0].shape == (got[k]["width"], cfg["d_in"] * got[k]["d_emb"])
        for (W, b), (Wr, br) in zip(layers, ref_layers):
            np.testing.assert_array_equal(W, Wr.astype(np.float32))
            np.testing.assert_array_equal(b, br.astype(np.float32))
        assert pk.param_count(k) == sum(a.size for a in emb.values()) + sum(W.size + b.size for W, b in layers)


def test_workspace_independent_of_tile_sets(monkeypatch):
    # The GEMM tile sets are chosen per launch (or forced by the environment);
    # the device tile table is sized for the largest choice (small tiles), so
    # the workspace is the same under every setting.  multiclass_lognormal's
    # evaluation launch of all 32 members has 1,280 small tiles: tall by default.
    sizes = {}
    for v in (None, "small", "tall", "big"):
        if v is None:
            monkeypatch.delenv("TABPACK_GEMM_TILES", raising=False)
        else:
            monkeypatch.setenv("TABPACK_GEMM_TILES", v)
        sizes[v] = tabpack.Pack(configs.workload("multiclass_lognormal")).workspace_bytes()
    assert len(set(sizes.values())) == 1, sizes
