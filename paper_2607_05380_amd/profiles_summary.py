"""Summaries of rocprofv3 output for the profiles/ folder.

  python -m paper_2607_05380_amd.profiles_summary stats DIR OUT.md --command "..."
      per-kernel launch counts and average durations from a
      `rocprofv3 --kernel-trace --stats --output-format csv` run
  python -m paper_2607_05380_amd.profiles_summary traffic FETCH_DIR WRITE_DIR WORKLOAD OUT_PREFIX --command "..."
      HBM bytes per launch of every library kernel from two `--pmc FETCH_SIZE` /
      `--pmc WRITE_SIZE` runs of `bench.py --copy-calibration`: each counter (KiB per
      dispatch) is scaled by what it reads for the 256 MiB device-to-device copies of
      that run; writes OUT_PREFIX.json (read by bench.py) and OUT_PREFIX.md
  python -m paper_2607_05380_amd.profiles_summary counters WORKLOAD OUT.md PMC_DIR... --command "..."
      per-kernel hardware counters of `--pmc` runs (MFMA busy share, wave
      wait states, L2 hit rate and latency, LDS bank conflicts)
  python -m paper_2607_05380_amd.profiles_summary mfma PMC_DIR BENCH_LOG WORKLOAD OUT.md --command "..."
      executed MFMA work per launch of every GEMM kernel from a `--pmc
      SQ_INSTS_VALU_MFMA_MOPS_BF16` (or _F32) run of `bench.py --profile-steps N`
      (the counter counts in units of 512 flops), against the algorithmic flops
      per launch that the same run's JSON line reports

Kernel names are mapped to the names the library's own profiler uses.
"""
import argparse
import csv
import glob
import hashlib
import json
import os
import re
import statistics
import sys

PKG = os.path.dirname(os.path.abspath(__file__))
COPY_BYTES = 256 << 20
OPS = ["kmaj", "rmaj", "emb"]
EPIS = ["fwd", "fwd_eval", "dx", "dw", "ns", "de"]
SIMPLE = ["dropout_words", "grad_sums", "head_grad_reduce", "head_fwd", "head_bwd", "loss_reduce", "bias_from_partials",
          "gather", "adamw", "to_shadow", "eval_score", "dropout_mask", "select_partial", "select_pick",
          "select_update", "select_init", "select_final", "ensemble_mean", "muon_prep", "muon_norm",
          "muon_convert", "muon_update", "embed_table", "embed_grad", "idx_check", "stream_copy"]


def source_digest():
    """sha256 over the library sources (kernel and host code)."""
    h = hashlib.sha256()
    for f in sorted(glob.glob(os.path.join(PKG, "csrc", "*"))):
        h.update(os.path.basename(f).encode())
        with open(f, "rb") as fh:
            h.update(fh.read())
    return h.hexdigest()


def short_name(kernel):
    """Library profiler name of a rocprofv3 kernel name (mangled, or demangled),
    or None for other kernels.  GEMM kernels are named by their template
    arguments: element type, operand kinds (0 depth-contiguous, 1 row-major, 2 the
    embedded first-layer input produced in the GEMM) and
    epilogue."""
    if "gemm_kernel_emb_wide" in kernel:  # the embedded forward on 8-wave tiles: bf16, E x W_1
        m = re.search(r"gemm_kernel_emb_wide(?:ILi(\d)EE|<(\d)>)", kernel)
        if not m:
            return None
        epi = int(m.group(1) or m.group(2))
        return f"gemm_bf16_{OPS[2]}_{OPS[0]}_{EPIS[epi]}" if epi < len(EPIS) else None
    if "gemm_kernel" in kernel:
        m = re.search(r"gemm_kernel(?:_small|_tall)?I(DF16b|f)?(?:Li(\d)E)(?:Li(\d)E)(?:Li(\d)E)", kernel)
        if m:
            t = "f32" if m.group(1) == "f" else "bf16"
            ak, bk, epi = int(m.group(2)), int(m.group(3)), int(m.group(4))
        else:
            m = re.search(r"gemm_kernel(?:_small|_tall)?<(?:([^,<>]*), )?(\d), (\d), (\d)>", kernel)
            if m:
                t = "f32" if m.group(1) and "float" in m.group(1) else "bf16"
                ak, bk, epi = int(m.group(2)), int(m.group(3)), int(m.group(4))
            else:
                # demangled with the leading arguments lost: the operand kind of A
                # follows from the epilogue (the forward, data-gradient and Newton-
                # Schulz GEMMs read A depth-contiguous, the weight gradient row-major)
                m = re.search(r"gemm_kernel(?:_small|_tall)?<.*, (\d), (\d)>", kernel)
                if not m:
                    return None
                t, bk, epi = "bf16", int(m.group(1)), int(m.group(2))
                ak = 1 if epi == 3 else 0
        if epi >= len(EPIS) or ak >= len(OPS) or bk >= len(OPS):
            return None
        return f"gemm_{t}_{OPS[ak]}_{OPS[bk]}_{EPIS[epi]}"
    for s in sorted(SIMPLE, key=len, reverse=True):
        if s + "_kernel" in kernel:
            return s
    if "select_" in kernel:
        return "select"
    return None


def is_copy(kernel):
    return "copyBuffer" in kernel or "CopyBuffer" in kernel


def busy_ns(intervals):
    """Length of the union of [start, end) intervals."""
    tot, cur_s, cur_e = 0, None, None
    for a, b in sorted(intervals):
        if cur_e is None or a > cur_e:
            if cur_e is not None:
                tot += cur_e - cur_s
            cur_s, cur_e = a, b
        else:
            cur_e = max(cur_e, b)
    if cur_e is not None:
        tot += cur_e - cur_s
    return tot


def trace_busy(d):
    """{kernel: (dispatches, union of its dispatch intervals in ns)} from the
    kernel_trace.csv files of a --kernel-trace run."""
    iv = {}
    for f in glob.glob(os.path.join(d, "**", "*kernel_trace.csv"), recursive=True):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                name = short_name(r["Kernel_Name"])
                if name:
                    iv.setdefault(name, []).append((int(r["Start_Timestamp"]), int(r["End_Timestamp"])))
    return {k: (len(v), busy_ns(v)) for k, v in iv.items()}


def stats(args):
    rows = []
    for f in glob.glob(os.path.join(args.dir, "**", "*kernel_stats.csv"), recursive=True):
        with open(f) as fh:
            rows += list(csv.DictReader(fh))
    if not rows:
        sys.exit(f"no kernel_stats.csv under {args.dir}")
    agg, other = {}, [0, 0.0]
    for r in rows:
        name = short_name(r["Name"])
        a = agg.setdefault(name, [0, 0.0]) if name else other
        a[0] += int(r["Calls"])
        a[1] += float(r["TotalDurationNs"])
    total = sum(v[1] for v in agg.values())
    busy = trace_busy(args.dir)
    lines = [f"# Kernel time summary ({os.path.basename(args.out)[:-3]})", "", "Command:", "", "```",
             args.command, "```", "",
             "Library kernels only; the share is of the library's kernel time.  Other dispatches of the run "
             f"(synthetic data generation in torch): {other[0]} calls, {other[1] / 1e6:.3f} ms.  "
             "Busy ms: the union of the kernel's dispatch intervals in the kernel trace (launches of the "
             "concurrent member-group streams overlap, so it can be less than the total).", "",
             "| kernel | calls | avg us | total ms | busy ms | share |", "|---|---|---|---|---|---|"]
    for name, (calls, ns) in sorted(agg.items(), key=lambda kv: -kv[1][1]):
        b = busy.get(name, (0, 0))[1]
        lines.append(f"| {name} | {calls} | {ns / calls / 1e3:.1f} | {ns / 1e6:.3f} | {b / 1e6:.3f} | "
                     f"{100 * ns / total:.1f}% |")
    with open(args.out, "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def per_dispatch(d, counter):
    """{dispatch id: (kernel name, counter value)} of one --pmc run."""
    out = {}
    for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
        with open(f) as fh:
            for r in csv.DictReader(fh):
                if r["Counter_Name"] != counter:
                    continue
                k = r["Dispatch_Id"]
                name, v = out.get(k, (r["Kernel_Name"], 0.0))
                out[k] = (name, v + float(r["Counter_Value"]))
    if not out:
        sys.exit(f"no {counter} rows under {d}")
    return out


def fmt(x):
    return "n/a" if x is None else f"{x:.3f}"


def traffic(args):
    res = {}
    factors = {}
    torch_factors = {}
    for counter, d in (("FETCH_SIZE", args.fetch), ("WRITE_SIZE", args.write)):
        disp = per_dispatch(d, counter)
        # calibration: the library's non-temporal streaming copy of 256 MiB
        # (the access pattern of the optimizer epilogues); torch's copy kernel
        # is reported beside it
        cal = [v for name, v in disp.values() if short_name(name) == "stream_copy" and v * 1024 >= 0.5 * COPY_BYTES]
        if not cal:
            sys.exit(f"no calibration stream_copy found in the {counter} run")
        factor = statistics.median(cal) * 1024 / COPY_BYTES  # counter bytes per true byte
        factors[counter] = factor
        tc = [v for name, v in disp.values() if is_copy(name) and v * 1024 >= 0.5 * COPY_BYTES]
        torch_factors[counter] = statistics.median(tc) * 1024 / COPY_BYTES if tc else None
        per = {}
        for name, v in disp.values():
            s = short_name(name)
            if s:
                per.setdefault(s, []).append(v * 1024)
        for s, vals in per.items():
            key = "fetch" if counter == "FETCH_SIZE" else "write"
            res.setdefault(s, {})[key + "_bytes"] = statistics.mean(vals) / factor
            res[s][key + "_raw_bytes"] = statistics.mean(vals)
            res[s]["dispatches"] = len(vals)
    rec = {"workload": args.workload, "source_sha256": source_digest(), "command": args.command,
           "copy_factor": {"fetch": factors["FETCH_SIZE"], "write": factors["WRITE_SIZE"]},
           "torch_copy_factor": {"fetch": torch_factors["FETCH_SIZE"], "write": torch_factors["WRITE_SIZE"]},
           "kernels": {k: v for k, v in res.items() if "fetch_bytes" in v and "write_bytes" in v}}
    with open(args.out_prefix + ".json", "w") as f:
        json.dump(rec, f, indent=1)
    lines = [f"# HBM traffic per launch, {args.workload}", "", "Commands (FETCH_SIZE run, then WRITE_SIZE run):",
             "", "```", args.command, "```", "",
             "Calibration: the library's non-temporal streaming copy (`pack_stream_copy`, 256 MiB read and "
             f"256 MiB written) reads FETCH_SIZE x {factors['FETCH_SIZE']:.3f} and WRITE_SIZE x "
             f"{factors['WRITE_SIZE']:.3f} of its true bytes; the scaled figures below are divided by these "
             "factors, the raw ones are the counters as read (KiB x 1024).  torch's device-to-device copy of the "
             f"same size reads FETCH_SIZE x {fmt(torch_factors['FETCH_SIZE'])} and WRITE_SIZE x "
             f"{fmt(torch_factors['WRITE_SIZE'])}.  Bytes served by the 256 MB last-level cache do not reach "
             "HBM and are not counted.", "",
             "| kernel | dispatches | fetch MB | write MB | total MB | raw fetch MB | raw write MB |",
             "|---|---|---|---|---|---|---|"]
    for k, v in sorted(rec["kernels"].items(), key=lambda kv: -(kv[1]["fetch_bytes"] + kv[1]["write_bytes"])):
        lines.append(f"| {k} | {v['dispatches']} | {v['fetch_bytes'] / 1e6:.1f} | {v['write_bytes'] / 1e6:.1f} | "
                     f"{(v['fetch_bytes'] + v['write_bytes']) / 1e6:.1f} | {v['fetch_raw_bytes'] / 1e6:.1f} | "
                     f"{v['write_raw_bytes'] / 1e6:.1f} |")
    with open(args.out_prefix + ".md", "w") as f:
        f.write("\n".join(lines) + "\n")
    print("\n".join(lines))


def mfma(args):
    counter = "SQ_INSTS_VALU_MFMA_MOPS_" + args.dtype.upper()
    disp = per_dispatch(args.dir, counter)
    with open(args.bench_log) as f:
        lines = [ln for ln in f if ln.startswith("{")]
    if not lines:
        sys.exit(f"no JSON line in {args.bench_log}")
    algo = {k["name"]: k["flops_per_launch"] for k in json.loads(lines[-1]).get("kernels", [])}
    per = {}
    for name, v in disp.values():
        s = short_name(name)
        if s and s.startswith("gemm_"):
            per.setdefault(s, []).append(v * 512)
    if not per:
        sys.exit(f"no GEMM dispatches with {counter} under {args.dir}")
    out = ["# Executed MFMA work against algorithmic flops, " + args.workload, "", "Command:", "", "```",
           args.command, "```", "",
           f"`{counter}` x 512 per dispatch (flops the matrix cores executed, padding included), averaged "
           "over the run's dispatches of each kernel, against the algorithmic flops per launch (true member "
           "widths, no padding) that the same run's library events report.  The ratio is the work added by "
           "rounding member widths to tiles and by whole tiles on the diagonal of symmetric products.", "",
           "| kernel | dispatches | executed GFLOP/launch | algorithmic GFLOP/launch | executed / algorithmic |",
           "|---|---|---|---|---|"]
    tot_e = tot_a = 0.0
    for k, vals in sorted(per.items(), key=lambda kv: -sum(kv[1])):
        e = statistics.mean(vals)
        a = algo.get(k)
        if a:
            tot_e += e * len(vals)
            tot_a += a * len(vals)
        out.append(f"| {k} | {len(vals)} | {e / 1e9:.2f} | {a / 1e9 if a else float('nan'):.2f} | "
                   f"{e / a if a else float('nan'):.3f} |")
    out += ["", f"All GEMM launches: executed / algorithmic = {tot_e / tot_a:.3f}."]
    with open(args.out, "w") as f:
        f.write("\n".join(out) + "\n")
    print("\n".join(out))


def counter_means(dirs):
    """{kernel: ({counter: mean per dispatch}, dispatches, mean duration ns)} over
    the counter_collection.csv files of one or more --pmc runs."""
    vals, durs = {}, {}
    for d in dirs:
        for f in glob.glob(os.path.join(d, "**", "*counter_collection.csv"), recursive=True):
            seen = set()
            with open(f) as fh:
                for r in csv.DictReader(fh):
                    s = short_name(r["Kernel_Name"])
                    if not s:
                        continue
                    vals.setdefault(s, {}).setdefault(r["Counter_Name"], []).append(float(r["Counter_Value"]))
                    key = (f, r["Dispatch_Id"])
                    if key not in seen:
                        seen.add(key)
                        durs.setdefault((d, s), []).append(int(r["End_Timestamp"]) - int(r["Start_Timestamp"]))
    out = {}
    for s, cs in vals.items():
        d_all = [x for (dd, ss), v in durs.items() if ss == s for x in v]
        n = max(len(v) for (dd, ss), v in durs.items() if ss == s)
        out[s] = ({c: statistics.mean(v) for c, v in cs.items()}, n, statistics.mean(d_all))
    return out


def counters(args):
    """Where the GEMM kernels' time goes: per-dispatch hardware counters (each
    kernel measured alone: counter collection serialises the dispatches)."""
    res = counter_means(args.dirs)
    cyc = args.clock_ghz * 1e9
    simds = args.cus * 4
    out = ["# Hardware counters of the library kernels, " + args.workload, "", "Commands (one run per counter set):",
           "", "```", args.command, "```", "",
           "Counter collection serialises dispatches, so each kernel runs alone here (in the training step the "
           f"member groups' launches overlap).  Derived per dispatch, at the {args.clock_ghz} GHz shader clock "
           f"measured during the bench (amd-smi) and {args.cus} CUs x 4 SIMDs:", "",
           "* MFMA busy: `SQ_VALU_MFMA_BUSY_CYCLES` / (duration x clock x SIMDs) -- the share of the matrix "
           "cores' cycles spent on MFMA work (one v_mfma_f32_32x32x16_bf16 holds a SIMD for 32 cycles);",
           "* wave states, shares of `SQ_WAVE_CYCLES`: `SQ_WAIT_ANY` (waiting on a counter: memory or LDS "
           "data), `SQ_WAIT_INST_ANY` (ready but not issued), `SQ_ACTIVE_INST_ANY` (issuing);",
           "* L2 hit rate `TCC_HIT` / (`TCC_HIT` + `TCC_MISS`) and mean L2 read latency "
           "`TCP_TCC_READ_REQ_LATENCY` / `TCP_TCC_READ_REQ` (cycles);",
           "* LDS bank conflicts: `SQ_LDS_BANK_CONFLICT` / `SQ_ACTIVE_INST_LDS` (conflict cycles per active LDS "
           "cycle).", "",
           "| kernel | dispatches | avg us | MFMA busy | wait | ready, not issued | issuing | L2 hit | "
           "L2 latency (cyc) | LDS conflict |",
           "|---|---|---|---|---|---|---|---|---|---|"]

    def g(c, k):
        return c.get(k)

    for s, (c, n, dur) in sorted(res.items(), key=lambda kv: -kv[1][2] * kv[1][1]):
        if not s.startswith("gemm_") and s not in args.also:
            continue
        wc = g(c, "SQ_WAVE_CYCLES") or 0.0
        mf = g(c, "SQ_VALU_MFMA_BUSY_CYCLES")
        busy = mf / (dur * 1e-9 * cyc * simds) if mf is not None and dur > 0 else None
        hit, miss = g(c, "TCC_HIT_sum"), g(c, "TCC_MISS_sum")
        lat, req = g(c, "TCP_TCC_READ_REQ_LATENCY_sum"), g(c, "TCP_TCC_READ_REQ_sum")
        lc, la = g(c, "SQ_LDS_BANK_CONFLICT"), g(c, "SQ_ACTIVE_INST_LDS")

        def pct(x):
            return "n/a" if x is None else f"{100 * x:.1f}%"

        def frac(k):
            v = g(c, k)
            return None if v is None or wc <= 0 else v / wc

        out.append(f"| {s} | {n} | {dur / 1e3:.1f} | {pct(busy)} | {pct(frac('SQ_WAIT_ANY'))} | "
                   f"{pct(frac('SQ_WAIT_INST_ANY'))} | {pct(frac('SQ_ACTIVE_INST_ANY'))} | "
                   f"{pct(hit / (hit + miss) if hit is not None and miss is not None and hit + miss > 0 else None)} | "
                   f"{lat / req if lat is not None and req else float('nan'):.0f} | "
                   f"{pct(lc / la if lc is not None and la else None)} |")
    with open(args.out, "w") as f:
        f.write("\n".join(out) + "\n")
    print("\n".join(out))


def main():
    ap = argparse.ArgumentParser()
    sub = ap.add_subparsers(dest="cmd", required=True)
    a = sub.add_parser("stats")
    a.add_argument("dir")
    a.add_argument("out")
    a.add_argument("--command", default="")
    b = sub.add_parser("traffic")
    b.add_argument("fetch")
    b.add_argument("write")
    b.add_argument("workload")
    b.add_argument("out_prefix")
    b.add_argument("--command", default="")
    c = sub.add_parser("mfma")
    c.add_argument("dir")
    c.add_argument("bench_log")
    c.add_argument("workload")
    c.add_argument("out")
    c.add_argument("--dtype", default="bf16")
    c.add_argument("--command", default="")
    e = sub.add_parser("counters")
    e.add_argument("workload")
    e.add_argument("out")
    e.add_argument("dirs", nargs="+")
    e.add_argument("--clock-ghz", type=float, default=2.38)
    e.add_argument("--cus", type=int, default=256)
    e.add_argument("--also", nargs="*", default=[])
    e.add_argument("--command", default="")
    args = ap.parse_args()
    {"stats": stats, "traffic": traffic, "mfma": mfma, "counters": counters}[args.cmd](args)


if __name__ == "__main__":
    main()
