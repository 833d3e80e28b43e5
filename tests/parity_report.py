"""Summary of the parity measurements that a GPU run records (tests/parity.py
writes them to $TABPACK_PARITY_REPORT): per test and kind of tensor, the
worst value of each measure over the tensors of that kind.

  python tests/parity_report.py REPORT.json OUT.md --command "..."
"""
import argparse
import json
from collections import defaultdict

MEASURES = [
    ("strict_frac", "max share of gradient elements outside the strict band"),
    ("strict_misses", "max count of gradient elements outside the strict band in one tensor"),
    ("frob", "max relative Frobenius error"),
    ("tol_ratio", "max |gpu - ref| / (atol + rtol |ref|) (1.0 = the literal bound)"),
    ("exempt_frac", "max share of elements whose gradient sign is undetermined (exempt)"),
    ("flip_frac", "max share of elements whose first update flipped (exempt elements off by more than upd * lr)"),
    ("nonexempt_err_lr", "max update error / lr over the other elements"),
    ("upd_miss_frac", "max share of updates off by more than upd * lr (several steps)"),
    ("max_err_lr", "max update error / lr"),
    ("literal_frac", "max share of elements outside the literal tolerance"),
    ("err_over_omax", "max error / (lr scale max|O|)"),
    ("max_rel", "max relative score difference"),
    ("ens_rel", "max relative ensemble-score difference"),
    ("max_abs", "max absolute difference"),
    ("max_ratio", "ReLU decisions: the furthest disagreement from 0, in rms(Z) of its layer"),
]


def summarize(records):
    groups = defaultdict(list)
    for r in records:
        test = r["test"].split("::", 1)[-1]
        groups[(test, r["kind"])].append(r)
    rows = []
    for (test, kind), rs in sorted(groups.items()):
        vals = {}
        for m, _ in MEASURES:
            xs = [r[m] for r in rs if r.get(m) is not None]
            if xs:
                vals[m] = max(xs)
        rows.append((test, kind, len(rs), vals))
    return rows


def fmt(x):
    if x == 0:
        return "0"
    if x >= 100 or x < 1e-3:
        return f"{x:.2e}"
    return f"{x:.4f}"


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("report")
    ap.add_argument("out")
    ap.add_argument("--command", default="")
    a = ap.parse_args()
    records = json.load(open(a.report))
    rows = summarize(records)
    used = [m for m, _ in MEASURES if any(m in v for _, _, _, v in rows)]
    lines = ["# Parity measurements per test and tensor kind", "", "Command:", "", "```", a.command, "```", "",
             "Worst value over the tensors of each kind (all members) in each test.  Measures:", ""]
    lines += [f"* `{m}`: {d}" for m, d in MEASURES if m in used]
    # the per-test table goes to stdout only; the file keeps the maxima per kind
    per_test = ["| test | kind | tensors | " + " | ".join(used) + " |", "|---|---|---|" + "---|" * len(used)]
    for test, kind, n, vals in rows:
        per_test.append(f"| {test} | {kind} | {n} | " + " | ".join(fmt(vals[m]) if m in vals else "" for m in used)
                        + " |")
    print("\n".join(per_test))
    lines += ["", f"{len(records)} records from {len({r['test'] for r in records})} tests."]
    # overall maxima per kind across tests
    over = defaultdict(dict)
    for _, kind, _, vals in rows:
        for m, v in vals.items():
            over[kind][m] = max(over[kind].get(m, v), v)
    lines += ["", "## Worst per kind over all tests", "", "| kind | " + " | ".join(used) + " |",
              "|---|" + "---|" * len(used)]
    for kind in sorted(over):
        lines.append(f"| {kind} | " + " | ".join(fmt(over[kind][m]) if m in over[kind] else "" for m in used)
                     + " |")
    dec = [r for r in records if r["kind"] == "decisions"]
    if dec:
        tot = {m: sum(r.get(m) or 0 for r in dec) for m in ("decisions", "window", "taken", "outside")}
        lines += ["", "## ReLU decisions (bf16 policy and fp32 comparisons)", "",
                  f"* decisions compared: {tot['decisions']:.0f}",
                  f"* inside the window (|Z| <= window rms(Z)): {tot['window']:.0f}",
                  f"* taken from the GPU there because they differ: {tot['taken']:.0f} "
                  f"({tot['taken'] / max(tot['decisions'], 1):.2e} of all)",
                  f"* differing outside the window: {tot['outside']:.0f}",
                  f"* furthest disagreement: {max(r.get('max_ratio') or 0 for r in dec):.2e} rms(Z)"]
    with open(a.out, "w") as f:
        f.write("\n".join(lines) + "\n")


if __name__ == "__main__":
    main()
