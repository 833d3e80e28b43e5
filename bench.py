"""Throughput of the packed training step (fwd + bwd + AdamW for all K members).

Default workload: the 700K x 900 regression workload with K = 64 members, 3
hidden layers, widths UniformInt[256, 1024], dropout U[0, 0.5], batch 1024,
bf16 MFMA GEMMs with fp32 master weights.  Inputs are synthetic, generated on
the device and resident in HBM before timing.  Prints one JSON line.

  python bench.py [--gpus 1] [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]
"""
import argparse
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "member-samples/sec (fwd+bwd+AdamW) at K=64; % bf16 MFMA peak; % HBM BW"
PEAK = {"mfma_bf16": 2516.6, "mfma_fp32": 157.3, "hbm": 8000.0}  # TFLOP/s, TFLOP/s, GB/s
COPY_BYTES = 256 << 20  # the calibration copy of --copy-calibration


def log(msg):
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def cpu_baseline(cfg, X, y, idx0, budget_s=15.0):
    """The fp64 oracle, timed on the host cores on a bounded sample: members
    0, 1, ... of step 1, then of step 2, ... (each step on the first step's
    batches: the work per member step does not depend on the rows) until the
    time budget is spent."""
    import numpy as np
    from oracle.pack import OraclePack
    keys = ("seed", "K", "d_in", "d_out", "L", "B", "task", "beta1", "beta2", "eps", "decay_bias",
            "width_lo", "width_hi", "dropout_lo", "dropout_hi", "lr_lo", "lr_hi", "wd_lo", "wd_hi")
    op = OraclePack({k: cfg[k] for k in keys})
    try:
        from threadpoolctl import threadpool_info
        threads = max([p.get("num_threads", 1) for p in threadpool_info()] + [1])
    except Exception:
        threads = os.cpu_count()
    B, K = cfg["B"], cfg["K"]
    batches = {}
    done, dt = 0, 0.0
    while dt < budget_s and done < 8 * K:
        k, step = done % K, done // K + 1
        if k not in batches:
            rows = idx0[k].long()  # this member's base batch, copied before timing
            batches[k] = (X[rows].double().cpu().numpy(), y[rows].cpu().numpy())
        Xk, yk = batches[k]
        t0 = time.perf_counter()
        op.member_step(k, Xk, yk, np.arange(B), step)
        dt += time.perf_counter() - t0
        done += 1
    steps, rest = divmod(done, K)
    what = f"{steps} step{'s' if steps != 1 else ''} of members 0..{K - 1}" if steps else ""
    if rest:
        what += (" and " if what else "") + f"members 0..{rest - 1} of step {steps + 1}"
    return {"value": done * B / dt, "unit": "member-samples/s", "cores": int(threads), "kind": "oracle",
            "sample": f"{what} of {cfg['name']} (fp64 numpy, one member at a time, the first step's batches), "
                      f"{dt:.1f} s",
            "cpu_model": cpu_model(), "logical_cpus": os.cpu_count(), "blas": blas_vendor()}


def cpu_model():
    """The host CPU's model name (lscpu, else /proc/cpuinfo)."""
    import subprocess
    try:
        out = subprocess.run(["lscpu"], capture_output=True, text=True, timeout=10).stdout
        for line in out.splitlines():
            if line.startswith("Model name:"):
                return line.split(":", 1)[1].strip()
    except Exception:
        pass
    try:
        for line in open("/proc/cpuinfo"):
            if line.startswith("model name"):
                return line.split(":", 1)[1].strip()
    except OSError:
        pass
    return None


def blas_vendor():
    """The BLAS library numpy calls (threadpoolctl's view; numpy's build config as a fallback)."""
    try:
        from threadpoolctl import threadpool_info
        libs = [f"{p.get('internal_api')} {p.get('version')} ({p.get('threading_layer')}, "
                f"{p.get('num_threads')} threads)" for p in threadpool_info() if p.get("user_api") == "blas"]
        if libs:
            return "; ".join(libs)
    except Exception:
        pass
    try:
        import numpy as np
        cfg = np.show_config(mode="dicts")
        return cfg["Build Dependencies"]["blas"]["name"]
    except Exception:
        return None


def per_epoch(cfg, pk, Xtr, ytr, Xva, yva, step, online_epochs):
    """The per-epoch work around the training steps, timed on the device: the
    validation forward and scores of every member (pack_eval_members), the
    greedy selection over the online pool of the K members plus a previous
    ensemble of 32 (pack_select), the step time with the cheaper half of the
    members removed from the pack (pack_set_active), and whole epochs of the
    online driver (training, validation, selection, snapshots).  Returns
    (results, last step number used)."""
    import torch
    from paper_2607_05380_amd.online import OnlineTrainer

    def timed(fn, reps):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        fn()
        torch.cuda.synchronize()
        e0.record()
        for _ in range(reps):
            r = fn()
        e1.record()
        torch.cuda.synchronize()
        return e0.elapsed_time(e1) / reps, r

    K, L, d_in, d_out = cfg["K"], cfg["L"], cfg["d_in"], cfg["d_out"]
    widths = [h["width"] for h in pk.hparams()]
    Nv = Xva.shape[0]
    res = {}
    ms, (pred, _) = timed(lambda: pk.eval_members(Xva, yva), 3)
    flops = 2.0 * Nv * sum(d_in * w + (L - 1) * w * w + w * d_out for w in widths)
    peak = PEAK["mfma_bf16"] if cfg["precision"] == "bf16" else PEAK["mfma_fp32"]
    res["eval"] = {"ms": round(ms, 3), "rows": Nv, "tflop_per_s": round(flops / ms / 1e9, 1),
                   "frac_mfma_peak": round(flops / ms / 1e9 / peak, 4)}
    g = torch.Generator(device=pred.device)
    g.manual_seed(1)
    prev = pred[:32] + 0.05 * torch.randn(pred[:32].shape, generator=g, device=pred.device)
    cand = torch.cat([pred, prev]).contiguous()
    ms, (picks, _) = timed(lambda: pk.select(cand, yva, 32), 3)
    sweeps = min(len(picks) + 1, 32)
    res["select"] = {"ms": round(ms, 3), "candidates": cand.shape[0], "rows": Nv, "picked": len(picks),
                     "gb_per_s": round(sweeps * cand.numel() * 4 / ms / 1e6, 1)}
    loss = torch.empty(K, dtype=torch.float32, device=Xtr.device)
    cost = sorted(range(K), key=lambda k: widths[k] * (d_in + (L - 1) * widths[k]))
    keep = [False] * K
    for k in cost[K // 2:]:
        keep[k] = True
    idx = synth_idx(cfg, Xtr.shape[0], Xtr.device)

    def one():
        nonlocal step
        step += 1
        pk.train_step(Xtr, ytr, idx, step, loss)

    full_ms, _ = timed(one, 20)
    pk.set_active(keep)
    half_ms, _ = timed(one, 20)
    pk.set_active([True] * K)
    work = [w * (d_in + (L - 1) * w) for w in widths]
    res["removal"] = {"step_ms_all": round(full_ms, 4), "step_ms_costlier_half": round(half_ms, 4),
                      "work_share_kept": round(sum(work[k] for k in range(K) if keep[k]) / sum(work), 4)}
    if online_epochs > 0:
        tr = OnlineTrainer(dict(cfg, keep_grads=0), max_epochs=online_epochs, device=Xtr.device)
        torch.cuda.synchronize()
        t0 = time.perf_counter()
        tr.fit(Xtr, ytr, Xva, yva)
        torch.cuda.synchronize()
        wall = time.perf_counter() - t0
        n = len(tr.history)
        res["online"] = {"epochs": n, "steps_per_epoch": tr.history[0]["steps"], "s_per_epoch": round(wall / n, 4),
                         "ensemble_size": len(tr.ensemble), "ensemble_score": tr.ensemble_score}
        del tr
    return res, step


def variable_depth(cfg, Xtr, ytr, steps=100, warmup=5, stream_rows=True):
    """Step time of the same workload with member depths ~ UniformInt[1, L]
    (App. F samples the number of layers): shallower members leave the deeper
    layers' launches, so the step should scale with the GEMM work."""
    import torch
    from paper_2607_05380_amd import tabpack
    L, d_in = cfg["L"], cfg["d_in"]
    pk = tabpack.Pack(dict(cfg, depth_lo=1, depth_hi=L, keep_grads=0)).bind(Xtr.device)
    if stream_rows and pk.can_bind_data():
        pk.bind_data(Xtr)
    hp = pk.hparams()
    idx = synth_idx(cfg, Xtr.shape[0], Xtr.device)
    loss = torch.empty(cfg["K"], dtype=torch.float32, device=Xtr.device)
    for s in range(warmup):
        pk.train_step(Xtr, ytr, idx, s + 1, loss)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for s in range(steps):
        pk.train_step(Xtr, ytr, idx, warmup + s + 1, loss)
    e1.record()
    torch.cuda.synchronize()
    work = sum(h["width"] * (d_in + (h["depth"] - 1) * h["width"]) for h in hp)
    full = sum(h["width"] * (d_in + (L - 1) * h["width"]) for h in hp)
    return {"depths": [sum(h["depth"] == d for h in hp) for d in range(1, L + 1)],
            "step_ms": round(e0.elapsed_time(e1) / steps, 4), "gemm_work_vs_full_depth": round(work / full, 4)}


MUON_OPTS = dict(optimizer="muon", muon_lr_lo=1e-3, muon_lr_hi=1e-1)
EMB_OPTS = dict(emb_lo=8, emb_hi=32, emb_step=4, sigma_lo=1e-2, sigma_hi=10.0)


def muon_optimizer(cfg, Xtr, ytr, steps=50, warmup=5, stream_rows=True):
    """Step time of the same workload with the paper's default optimizer split:
    Muon for the hidden weights (Newton-Schulz on the grouped GEMMs), AdamW for
    biases and heads; and the Newton-Schulz GEMMs' rate (library events)."""
    import torch
    from paper_2607_05380_amd import tabpack
    pk = tabpack.Pack(dict(cfg, keep_grads=0, **MUON_OPTS)).bind(Xtr.device)
    if stream_rows and pk.can_bind_data():
        pk.bind_data(Xtr)
    idx = synth_idx(cfg, Xtr.shape[0], Xtr.device)
    loss = torch.empty(cfg["K"], dtype=torch.float32, device=Xtr.device)
    for s in range(warmup):
        pk.train_step(Xtr, ytr, idx, s + 1, loss)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for s in range(steps):
        pk.train_step(Xtr, ytr, idx, warmup + s + 1, loss)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    pk.profile(True)
    for s in range(3):
        pk.train_step(Xtr, ytr, idx, warmup + steps + 1 + s, loss)
    stats = pk.profile_read()
    pk.profile(False)
    ns = [x for x in stats if x["name"].endswith("_ns")]
    ns_flops = sum(x["flops"] * x["launches"] for x in ns) / 3
    ns_ms = sum(x["busy_ms"] for x in ns) / 3
    other = sum(x["busy_ms"] for x in stats if x["name"].startswith("muon_")) / 3
    peak = PEAK["mfma_bf16"] if cfg["precision"] == "bf16" else PEAK["mfma_fp32"]
    return {"step_ms": round(ms, 4), "ns_gemm_ms_per_step": round(ns_ms, 4),
            "ns_gemm_gflop_per_step": round(ns_flops / 1e9, 1),
            "ns_gemm_tflop_per_s": round(ns_flops / ns_ms / 1e9, 1) if ns_ms > 0 else None,
            "ns_gemm_frac_mfma_peak": round(ns_flops / ns_ms / 1e9 / peak, 4) if ns_ms > 0 else None,
            "muon_elementwise_ms_per_step": round(other, 4),
            "kernels_ms_per_step": {x["name"]: round(x["busy_ms"] / 3, 4) for x in stats}}


def embeddings(cfg, Xtr, ytr, steps=20, warmup=3):
    """Step time of the same workload with periodic feature embeddings
    (d_emb ~ UniformInt[8, 32] step 4, sigma ~ LogUniform[1e-2, 10]): the first
    layer then reads d_in * d_emb columns per member; per-kernel rates from the
    library's events."""
    import torch
    from paper_2607_05380_amd import tabpack
    pk = tabpack.Pack(dict(cfg, keep_grads=0, **EMB_OPTS)).bind(Xtr.device)
    hp = pk.hparams()
    idx = synth_idx(cfg, Xtr.shape[0], Xtr.device)
    loss = torch.empty(cfg["K"], dtype=torch.float32, device=Xtr.device)
    for s in range(warmup):
        pk.train_step(Xtr, ytr, idx, s + 1, loss)
    torch.cuda.synchronize()
    e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    e0.record()
    for s in range(steps):
        pk.train_step(Xtr, ytr, idx, warmup + s + 1, loss)
    e1.record()
    torch.cuda.synchronize()
    ms = e0.elapsed_time(e1) / steps
    pk.profile(True)
    for s in range(2):
        pk.train_step(Xtr, ytr, idx, warmup + steps + 1 + s, loss)
    stats = pk.profile_read()
    pk.profile(False)
    flops = sum(x["flops"] * x["launches"] for x in stats if x["kind"] == "mfma" or "gemm" in x["name"]) / 2
    out = {"d_emb_mean": round(sum(h["d_emb"] for h in hp) / len(hp), 2), "step_ms": round(ms, 3),
           "workspace_gib": round(pk.workspace_bytes() / 2 ** 30, 2), "gemm_tflop_per_step": round(flops / 1e12, 3),
           "kernels": {x["name"]: {"busy_ms_per_step": round(x["busy_ms"] / 2, 4),
                                   "tflop_per_s": round(x["flops"] * x["launches"] / x["busy_ms"] / 1e9, 1),
                                   "gb_per_s": round(x["bytes"] * x["launches"] / x["busy_ms"] / 1e6, 1)}
                       for x in stats}}
    del pk
    torch.cuda.empty_cache()
    return out


def synth_idx(cfg, n, device):
    from paper_2607_05380_amd import synth
    return synth.epoch_orders_device(cfg, 1, n, device)[:, :cfg["B"]].contiguous()


def measured_traffic(workload, kernel):
    """HBM bytes per launch of `kernel` from the committed profiler counters
    (FETCH_SIZE + WRITE_SIZE, scaled by a plain copy's reading), or None when
    no record exists or the library sources changed since it was taken."""
    from paper_2607_05380_amd.profiles_summary import source_digest
    path = os.path.join(ROOT, "profiles", f"traffic_{workload}.json")
    if not os.path.exists(path):
        return None
    with open(path) as f:
        rec = json.load(f)
    if rec.get("source_sha256") != source_digest():
        return None
    k = rec.get("kernels", {}).get(kernel)
    return None if k is None else round(k["fetch_bytes"] + k["write_bytes"], 1)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=0,
                    help="timed steps (default: one epoch of the workload, n_train // B: 683 for regression_large)")
    ap.add_argument("--warmup", type=int, default=10)
    ap.add_argument("--workload", default="regression_large")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--profile-steps", type=int, default=10)
    ap.add_argument("--copy-calibration", action="store_true",
                    help="accepted for older profiler commands: the 256 MiB copies that scale the hardware byte "
                         "counters run in every invocation (they also time the copy bandwidth)")
    ap.add_argument("--online-epochs", type=int, default=1,
                    help="epochs of the online driver timed after the steps (0: none)")
    ap.add_argument("--no-per-epoch", action="store_true", help="skip the per-epoch measurements")
    ap.add_argument("--keep-grads", action="store_true",
                    help="also write every gradient out (an inspection aid; the optimizer does not need it)")
    ap.add_argument("--members", type=int, default=0,
                    help="pack size K (default: the workload's; other values measure packing efficiency, "
                         "not the metric's configuration)")
    ap.add_argument("--variant", choices=["adamw", "muon", "embeddings"], default="adamw",
                    help="the timed step's options: AdamW for everything (the metric), Muon for the hidden "
                         "weights, or periodic feature embeddings (for profiling those steps on their own)")
    ap.add_argument("--rows", choices=["stream", "gather"], default="stream",
                    help="how the first layer gets its batch rows: read straight from a bf16 copy of X through "
                         "the batch indices (pack_bind_data; bf16 packs without embeddings), or gathered into a "
                         "dense batch before the first GEMM")
    a = ap.parse_args()
    if a.gpus != 1:
        print(f"bench.py measures one GPU: the packed step runs all members on one device and this "
              f"build has no multi-GPU path (asked for --gpus {a.gpus}).", file=sys.stderr)
        sys.exit(2)

    import torch
    from paper_2607_05380_amd import configs, synth, tabpack

    cfg = configs.workload(a.workload, **({"K": a.members} if a.members > 0 else {}))
    dev = torch.device("cuda:0")
    torch.cuda.set_device(dev)
    log(f"generating {cfg['name']} on device: {cfg['n_train']} x {cfg['d_in']}")
    Xtr, ytr, Xva, yva = synth.make_data_device(cfg, dev)
    orders = synth.epoch_orders_device(cfg, 0, cfg["n_train"], dev)
    steps_per_epoch = cfg["n_train"] // cfg["B"]
    if a.steps <= 0:
        a.steps = steps_per_epoch
    total = a.warmup + a.steps + a.profile_steps
    idx_all = torch.stack([orders[:, (s % steps_per_epoch) * cfg["B"]:(s % steps_per_epoch + 1) * cfg["B"]]
                           for s in range(total)]).contiguous()
    # keep_grads=0: hidden-layer weight gradients go straight into the fused
    # AdamW update of the weight-gradient GEMM instead of being stored as well
    variant = {"adamw": {}, "muon": MUON_OPTS, "embeddings": EMB_OPTS}[a.variant]
    pk = tabpack.Pack(dict(cfg, keep_grads=int(a.keep_grads), **variant)).bind(dev)
    log(f"bound: workspace {pk.workspace_bytes() / 2**30:.2f} GiB")
    stream_rows = a.rows == "stream" and pk.can_bind_data()
    if stream_rows:
        pk.bind_data(Xtr)  # one bf16 copy of X, made before any step (like the data upload)
        log(f"first-layer rows streamed from a bf16 copy of X ({pk.xb.numel() * 2 / 2**30:.2f} GiB)")
    loss = torch.empty(cfg["K"], dtype=torch.float32, device=dev)
    step = 0
    for _ in range(a.warmup):
        step += 1
        pk.train_step(Xtr, ytr, idx_all[step - 1], step, loss)
    torch.cuda.synchronize()
    log(f"warmup done, losses[:4] = {loss[:4].tolist()}")
    # streaming copy bandwidth (read + write) with the library's non-temporal
    # copy kernel, the measured reference for the HBM-bound kernels, and
    # torch's copy for comparison; in a profiler run the same copies scale the
    # byte counters (profiles_summary traffic)
    src = torch.ones(COPY_BYTES // 4, dtype=torch.float32, device=dev)
    dst = torch.empty_like(src)

    def copy_rate(fn):
        fn()
        torch.cuda.synchronize()
        c0, c1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        c0.record()
        for _ in range(3):
            fn()
        c1.record()
        torch.cuda.synchronize()
        return 2 * 3 * COPY_BYTES / (c0.elapsed_time(c1) / 1e3) / 1e9

    copy_gbps = copy_rate(lambda: tabpack.stream_copy(src, dst))
    torch_copy_gbps = copy_rate(lambda: dst.copy_(src))
    del src, dst
    log(f"streaming copy: {copy_gbps:.0f} GB/s, torch copy {torch_copy_gbps:.0f} GB/s (read + write)")
    ev0, ev1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev0.record()
    for _ in range(a.steps):
        step += 1
        pk.train_step(Xtr, ytr, idx_all[step - 1], step, loss)
    ev1.record()
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    ms = ev0.elapsed_time(ev1)
    if not torch.isfinite(loss).all():
        raise RuntimeError("non-finite member loss in the timed region")
    ms_per_step = ms / a.steps
    msamples = cfg["K"] * cfg["B"] * a.steps / (ms / 1e3)
    log(f"timed {a.steps} steps: {ms_per_step:.3f} ms/step (wall {wall:.3f} s), {msamples / 1e6:.2f} M member-samples/s")

    # per-kernel durations: HIP events recorded by the library around each launch
    stats = []
    if a.profile_steps > 0:
        pk.profile(True)
        for _ in range(a.profile_steps):
            step += 1
            pk.train_step(Xtr, ytr, idx_all[step - 1], step, loss)
        stats = pk.profile_read()
        pk.profile(False)
    for s in sorted(stats, key=lambda s: -s["busy_ms"]):
        log(f"  {s['name']:26s} launches {s['launches']:4d}  avg {s['avg_ms'] * 1e3:8.1f} us  "
            f"busy/step {s['busy_ms'] / a.profile_steps:6.3f} ms  "
            f"{s['flops'] * s['launches'] / s['busy_ms'] / 1e9:7.1f} TFLOP/s "
            f"{s['bytes'] * s['launches'] / s['busy_ms'] / 1e6:7.1f} GB/s  [{s['kind']}]")
    roofline = None
    if stats:
        # The dominant kernel (largest busy time per step).  achieved = the
        # algorithmic work of one launch / the launch's average duration (HIP
        # events on the stream it runs on; rocprofv3's average duration of the
        # same kernel in profiles/ must agree).  Launches of the concurrent
        # member groups overlap and share the chip, so a launch's duration
        # includes the time other groups' kernels hold CUs; the rate over the
        # kernel's busy time (the union of its launches' intervals) is
        # reported beside it, labelled.
        dom = max(stats, key=lambda s: s["busy_ms"])
        if dom["kind"] == "mfma":
            peak = PEAK["mfma_bf16"] if cfg["precision"] == "bf16" else PEAK["mfma_fp32"]
            work, unit, scale = dom["flops"], "TFLOP/s", 1e12
        else:
            peak, work, unit, scale = PEAK["hbm"], dom["bytes"], "GB/s", 1e9
        achieved = work / (dom["avg_ms"] / 1e3) / scale
        busy_rate = work * dom["launches"] / (dom["busy_ms"] / 1e3) / scale
        roofline = {"bound": dom["kind"], "kernel": dom["name"], "achieved": round(achieved, 2), "peak": peak,
                    "unit": unit, "frac": round(achieved / peak, 4),
                    "traffic": measured_traffic(cfg["name"], dom["name"]),
                    "work_per_launch": work, "flops_per_launch": dom["flops"], "bytes_per_launch": dom["bytes"],
                    "avg_launch_us": round(dom["avg_ms"] * 1e3, 2),
                    "launches_per_step": dom["launches"] / a.profile_steps,
                    "busy_time": {"us_per_step": round(dom["busy_ms"] * 1e3 / a.profile_steps, 2),
                                  "achieved": round(busy_rate, 2), "frac": round(busy_rate / peak, 4)}}
        if dom["kind"] != "mfma":
            roofline["copy_gb_per_s"] = round(copy_gbps, 1)
            roofline["torch_copy_gb_per_s"] = round(torch_copy_gbps, 1)
            roofline["frac_of_copy"] = round(achieved / copy_gbps, 4)
    out = {
        "metric": METRIC, "value": round(msamples, 1), "unit": "member-samples/s", "n_gpus": 1,
        "steps": a.steps, "warmup": a.warmup, "ms_per_step": round(ms_per_step, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": cfg["precision"], "data": "synthetic",
        "config": {"workload": cfg["name"], "K": cfg["K"], "B": cfg["B"], "d_in": cfg["d_in"], "L": cfg["L"],
                   "widths": [cfg["width_lo"], cfg["width_hi"]], "n_train": cfg["n_train"],
                   "task": cfg["task"], "keep_grads": int(a.keep_grads),
                   "first_layer_rows": "streamed" if stream_rows else "gathered",
                   **({} if a.variant == "adamw" else {"variant": a.variant})},
        "roofline": roofline,
        "kernels": [{"name": s["name"], "bound": s["kind"], "avg_us": round(s["avg_ms"] * 1e3, 2),
                     "busy_ms_per_step": round(s["busy_ms"] / a.profile_steps, 4),
                     "launches_per_step": s["launches"] / a.profile_steps, "flops_per_launch": s["flops"],
                     "bytes_per_launch": s["bytes"]}
                    for s in sorted(stats, key=lambda s: -s["busy_ms"])],
    }
    if not a.no_per_epoch:
        log("per-epoch work: validation, selection, member removal, online driver")
        out["per_epoch"], step = per_epoch(cfg, pk, Xtr, ytr, Xva, yva, step, a.online_epochs)
        log(f"  {json.dumps(out['per_epoch'])}")
        out["variable_depth"] = variable_depth(cfg, Xtr, ytr, stream_rows=stream_rows)
        log(f"  variable depth: {json.dumps(out['variable_depth'])}")
        out["muon"] = muon_optimizer(cfg, Xtr, ytr, stream_rows=stream_rows)
        log(f"  Muon optimizer: {json.dumps(out['muon'])}")
        out["embeddings"] = embeddings(cfg, Xtr, ytr)
        log(f"  periodic embeddings: {json.dumps(out['embeddings'])}")
    if not a.no_cpu_baseline and a.variant == "adamw":
        log("timing the fp64 oracle on the host (bounded sample)")
        out["cpu_baseline"] = cpu_baseline(cfg, Xtr, ytr, idx_all[0])
    print(json.dumps(out), flush=True)


if __name__ == "__main__":
    main()
