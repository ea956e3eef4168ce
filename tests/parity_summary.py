"""Summarise a parity error log (JSON lines written by the GPU tests when
GPPS_PARITY_LOG is set) as a markdown table: per test label and output, the
error against the oracle, its tolerance and the margin (tolerance / error).

    python tests/parity_summary.py <log.jsonl> [--title TEXT] > out.md
"""
import argparse
import json
import sys


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("log")
    ap.add_argument("--title", default="Parity errors against the fp64 oracle")
    a = ap.parse_args()
    rows = [json.loads(l) for l in open(a.log) if l.strip()]
    print(f"# {a.title}\n")
    print("Relative errors per output (relative Frobenius for whole outputs, over the "
          "sampled entries or rows where marked), from the GPU tests' own comparisons.\n")
    print("| test | case | output | error | tolerance | margin |")
    print("|---|---|---|---|---|---|")
    for r in rows:
        tol = r["tol"]
        marg = f"{tol / r['err']:.0f}x" if tol and r["err"] > 0 else ("exact" if tol else "-")
        t = r["test"].split("::")[-1]
        print(f"| {t} | {r['label']} | {r['what']} | {r['err']:.2e} | "
              f"{'-' if tol is None else f'{tol:.0e}'} | {marg} |")
    worst = max((r for r in rows if r["tol"]), key=lambda r: r["err"] / r["tol"], default=None)
    if worst:
        print(f"\nSmallest margin: {worst['label']} {worst['what']}, {worst['err']:.2e} "
              f"against {worst['tol']:.0e}.")
    return 0


if __name__ == "__main__":
    sys.exit(main())
