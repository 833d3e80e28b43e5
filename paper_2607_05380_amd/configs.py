"""The five synthetic tabular workloads the packed step is tested and measured on.

Each entry holds the pack's hyperparameter ranges (pack_config fields) and the
data recipe consumed by ``synth``.  Shapes follow the paper's datasets: up to
~700K training rows and ~900 features, batch sizes 256-2048, one-hot
categoricals and quantile-normalised skewed columns as in its preprocessing.
Seeds: workload i (1-based) uses S_i = 2607053800 + i; the pack seed is S_i.
"""

_COMMON = dict(lr_lo=1e-4, lr_hi=3e-3, wd_lo=1e-5, wd_hi=1e-2,
               beta1=0.9, beta2=0.999, eps=1e-8, decay_bias=1, quantum=0)

WORKLOADS = {
    "binary_small": dict(
        _COMMON, index=1, n_train=2048, n_val=512, d_in=8, d_out=1, task="bin",
        K=4, L=2, B=256, width_lo=64, width_hi=256, dropout_lo=0.0, dropout_hi=0.3,
        precision="fp32", features="normal", label="sign", score="bce"),
    "regression_onehot": dict(
        _COMMON, index=2, n_train=50_000, n_val=10_000, d_in=64, d_out=1, task="reg",
        K=16, L=3, B=512, width_lo=128, width_hi=512, dropout_lo=0.0, dropout_hi=0.5,
        precision="bf16", features="onehot", label="teacher_noise", score="rmse"),
    "multiclass_lognormal": dict(
        _COMMON, index=3, n_train=200_000, n_val=20_000, d_in=256, d_out=10, task="multi",
        K=32, L=3, B=1024, width_lo=256, width_hi=1024, dropout_lo=0.0, dropout_hi=0.5,
        precision="bf16", features="lognormal_rankgauss", label="argmax", score="ce"),
    "binary_wide": dict(
        _COMMON, index=4, n_train=400_000, n_val=40_000, d_in=512, d_out=1, task="bin",
        K=64, L=4, B=2048, width_lo=64, width_hi=2048, dropout_lo=0.0, dropout_hi=0.5,
        precision="bf16", features="zero_inflated", label="sign", score="bce"),
    "regression_large": dict(
        _COMMON, index=5, n_train=700_000, n_val=70_000, d_in=900, d_out=1, task="reg",
        K=64, L=3, B=1024, width_lo=256, width_hi=1024, dropout_lo=0.0, dropout_hi=0.5,
        precision="bf16", features="block_correlated", label="teacher_t3", score="rmse"),
}

ORDER = ["binary_small", "regression_onehot", "multiclass_lognormal",
         "binary_wide", "regression_large"]

BASE_SEED = 2607053800


def workload(name, **overrides):
    """A copy of workload ``name`` with the pack seed filled in and overrides applied."""
    cfg = dict(WORKLOADS[name])
    cfg["seed"] = BASE_SEED + cfg["index"]
    cfg["name"] = name
    cfg.update(overrides)
    return cfg
