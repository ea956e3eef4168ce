"""Summarise a parity error log (JSON lines written by the GPU tests when
GPPS_PARITY_LOG is set) as markdown: the five named workloads by path with the
error of every output, the matrix-core range cases with the route the guard
took, and the smallest margins (tolerance / error) over every comparison.

    GPPS_PARITY_LOG=gpurun_out/parity_errors.jsonl python -m pytest tests -m gpu
    python tests/parity_summary.py gpurun_out/parity_errors.jsonl > profiles/parity_errors.md
"""
import argparse
import json
import sys

OUTPUTS = ["psi0", "Psi1", "Psi2", "dmu", "dS", "dZ", "dsigma_f2", "dl"]
# (label prefix in the tests, name shown)
WORKLOADS = [("tiny/f64/", "tiny fp64"), ("tiny/f32/", "tiny fp32"), ("small/f32/", "small"),
             ("medium/f32/", "medium"), ("large-subset/", "large, 1031-row subset"),
             ("large/", "large, full size (sampled)"), ("stress-subset/", "stress, 1004-row subset"),
             ("stress/", "stress, full size in 8 chunks (sampled)")]


def short(what):
    """Output name of a record ('dZ (2 rows, ...)' -> 'dZ')."""
    return what.split(" (")[0]


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("log")
    a = ap.parse_args()
    rows = [json.loads(l) for l in open(a.log) if l.strip()]
    print("# Parity errors against the fp64 oracle\n")
    print("Relative errors of the GPU outputs against the oracle, as the GPU tests measured them "
          "(relative Frobenius norm per output; over the sampled entries or rows where the "
          "workload runs at full size).  Tolerances: 1e-5 (Psi1), 1e-4 (every other fp32 "
          "output), 1e-10 (fp64).  Produced by\n")
    print("```\nGPPS_PARITY_LOG=gpurun_out/parity_errors.jsonl python -u -m pytest tests -m gpu\n"
          f"python tests/parity_summary.py {a.log} > profiles/parity_errors.md\n```\n")
    print("## The five workloads\n")
    print("| workload | path | " + " | ".join(OUTPUTS) + " |")
    print("|---|---|" + "---|" * len(OUTPUTS))
    for prefix, name in WORKLOADS:
        for path in ("generic", "mfma"):
            sel = [r for r in rows if r["label"].startswith(prefix) and r["label"].endswith(path)
                   and (prefix != "large/" or r["label"] in ("large/generic", "large/mfma"))
                   and (prefix != "stress/" or r["label"] in ("stress/generic", "stress/mfma"))]
            if not sel:
                continue
            cell = {}
            for r in sel:
                cell[short(r["what"])] = r["err"]
            print(f"| {name} | {path} | " + " | ".join(
                f"{cell[o]:.1e}" if o in cell else "-" for o in OUTPUTS) + " |")
    print("\nFull-size rows also carry identity residuals (translation, per-dimension scaling, "
          "sigma_f2 homogeneity) of at most:")
    for lab in ("large/generic", "large/mfma", "stress/generic", "stress/mfma"):
        res = [r for r in rows if r["label"] == lab and "residual" in r["what"]]
        if res:
            print(f"{lab} {max(r['err'] for r in res):.1e};", end=" ")
    print("\n")
    rng = [r for r in rows if r["label"].startswith("range-")]
    if rng:
        print("## Matrix-core range cases (route 0: matrix cores, 1: generic by the guard)\n")
        print("| case | route | " + " | ".join(OUTPUTS) + " |")
        print("|---|---|" + "---|" * len(OUTPUTS))
        labels = sorted({r["label"] for r in rng})
        for lab in labels:
            cell = {short(r["what"]): r["err"] for r in rng if r["label"] == lab}
            route = f"{cell['route']:.0f}" if "route" in cell else "-"
            print(f"| {lab[6:]} | {route} | " + " | ".join(
                f"{cell[o]:.1e}" if o in cell else "-" for o in OUTPUTS) + " |")
        print()
    tol = sorted((r for r in rows if r["tol"] and r["err"] > 0), key=lambda r: -r["err"] / r["tol"])
    print(f"## Smallest margins over all {len(rows)} comparisons\n")
    print("| test | case | output | error | tolerance | margin |")
    print("|---|---|---|---|---|---|")
    for r in tol[:15]:
        print(f"| {r['test'].split('::')[-1]} | {r['label']} | {r['what']} | {r['err']:.2e} | "
              f"{r['tol']:.0e} | {r['tol'] / r['err']:.1f}x |")
    return 0


if __name__ == "__main__":
    sys.exit(main())
