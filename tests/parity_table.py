"""Summarize the parity records a GPU test run appended to the file named by
LIBRA_PARITY_LOG (one JSON object per check) as a Markdown table: per test
and output, the max-abs error, the part of it beyond bf16 storage rounding,
the relative L2 error, max |ref| and the bound.

    python tests/parity_table.py LOG.jsonl "COMMAND" > profiles/parity_errors.md

where LOG.jsonl is the file the run named in LIBRA_PARITY_LOG and COMMAND the
command line of that run (printed in the table's header).
"""
import collections
import json
import sys


def main(path, command):
    rs = [json.loads(l) for l in open(path) if l.strip()]
    print("# Parity errors of the GPU tests against the float64 oracle\n")
    print(f"Command: `{command}`\n")
    print(f"{len(rs)} checks, {sum(not r['ok'] for r in rs)} over their bound.  Bounds: max-abs "
          "2e-2 (bf16 outputs: beyond half a bf16 ulp of the exact value), relative L2 1e-2; "
          "LSE max-abs 1e-3.  Outputs named `fp32` are accumulate-mode dK / dV (no storage "
          "allowance).  Per test, rows that repeat one output over heads keep the worst.\n")
    # worst record per (test, output kind)
    worst = collections.OrderedDict()
    for r in rs:
        name = r["name"]
        kind = name.split(" ")[0] + (" fp32" if "fp32" in name else "")
        if name.startswith(("dK probe", "dV probe", "dK kv", "dV kv", "O head")):
            kind = " ".join(name.split(" ")[:2]) + (" fp32" if "fp32" in name else "")
        key = (r["test"].split("::")[-1], kind)
        m = r["excess"] / r["bound"][0]
        if key not in worst or m > worst[key][0]:
            worst[key] = (m, r)
    print("| test | output | max-abs | beyond storage | rel-L2 | max \\|ref\\| | of bound |")
    print("|---|---|---:|---:|---:|---:|---:|")
    for (test, kind), (m, r) in worst.items():
        print(f"| {test} | {kind} | {r['max_abs']:.3e} | {r['excess']:.3e} | {r['rel_l2']:.2e} | "
              f"{r['ref_max_abs']:.2f} | {m:.2f} |")
    print("\nWorst over all tests, per output:\n")
    per = collections.OrderedDict()
    for (test, kind), (m, r) in worst.items():
        k = kind.split(" ")[0] + (" fp32" if "fp32" in kind else "")
        if k not in per or m > per[k][0]:
            per[k] = (m, test, r)
    print("| output | test | beyond storage | rel-L2 | of bound |")
    print("|---|---|---:|---:|---:|")
    for k, (m, test, r) in per.items():
        print(f"| {k} | {test} | {r['excess']:.3e} | {r['rel_l2']:.2e} | {m:.2f} |")


if __name__ == "__main__":
    main(sys.argv[1], sys.argv[2] if len(sys.argv) > 2 else
         f"LIBRA_PARITY_LOG={sys.argv[1]} python -m pytest tests -m gpu")
