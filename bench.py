"""Benchmark: RBF-ARD psi-statistics + gradients on one MI355X.

One step = gpps_psi_stats (psi0, Psi1, Psi2) + gpps_psi_grads (dmu, dS, dZ,
dsigma_f2, dl) over the whole workload, inputs resident in HBM.  The timed
workload is ``large`` (N=100,000, M=256, Q=20, fp32, synthetic, seed 0).

Timing: the headline runs with the library's per-kernel timing off; every step
is bracketed by one HIP event pair on the library's stream, and ms_per_step is
the median over the steps (the wall clock between the two synchronisations is
reported beside it).  A second pass with per-kernel timing on gives the kernel
table and the roofline.

Metric: N*M^2*Q terms per second (whole step).  Beside it:
  roofline      the dominant kernel's algorithmic fp32 FLOP rate (6 Q flops per
                datapoint and unique pair for the Psi2 gradient) against the fp32
                vector peak of 157.3 TFLOP/s, with what bounds it: its executed
                matrix-core work against the dense f16 peak, and the vector-ALU /
                matrix-core busy shares from the committed SQ counters;
  pct_fp32_peak F_alg = 8 Q N M(M+1)/2 flops over the Psi2 forward and gradient
                kernels with their reductions (and beside it with the per-row
                kernels that feed them);
  exp_per_s     2 N M(M+1)/2 exponentials over the same time, against the
                measured v_exp_f32 rate (gpps_probe_unit_rates);
  cpu_baseline  the fp64 CPU oracle on a bounded row sample of the same
                workload, on this host's cores (a reported baseline only).

Usage: python bench.py [--gpus 1] [--steps 20] [--warmup 3] [--workload large]

--workload tiny|small|medium|stress times the same step on the other seeded
workloads; stress (N = 10^6, M = 512, Q = 30) runs as 8 row chunks of 131,072
per entry point, accumulating psi0, Psi2, dZ, dl and dsigma_f2 on the device.
--dtype f64 times the fp64 (generic) kernels on the same inputs, against the
fp64 vector peak.

--workload gplvm times the next step of the method instead: one evaluation of
the Bayesian GP-LVM bound and all its gradients (gpps_bound) at the shape of
the paper's experiment (section 4: Q = 1, M = 100, D = 3, here N = 64,000,
fp64), in evaluations per second, with the fp64 oracle timed on one full
evaluation beside it.

--workload known times the known-input (S = 0) path at the large workload's
shape and distributions (N=100,000, M=256, Q=20, the S array dropped):
gpps_psi_stats + gpps_psi_grads with S = NULL, where Psi2 = Kfu^T Kfu and
dL/dKfu = G1 + 2 Kfu G2s run on the matrix cores.  Same metric and unit;
--dtype f64 runs it in double precision.

--copy-probe-mib X runs a plain device copy (torch.neg into a second buffer) of
X MiB three times before the timed steps: under a rocprofv3 --pmc run its
FETCH_SIZE / WRITE_SIZE calibrate the counters against a known byte count.
"""
from __future__ import annotations

import argparse
import ctypes
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_FP32 = 157.3e12          # MI355X FP32 vector peak (packed FMA), FLOP/s
PEAK_FP64 = 78.6e12           # MI355X FP64 vector peak, FLOP/s
PEAK_F16_MFMA = 2.5e15        # MI355X dense fp16 / bf16 matrix-core peak, FLOP/s
PEAK_HBM = 8.0e12             # B/s
# vector issue peak: 256 CUs x 4 SIMDs x 16 lanes per cycle at 2.4 GHz (a wave64
# instruction takes four cycles of a SIMD; 2 flops per lane for an FMA gives the
# unpacked fp32 rate, half of the packed 157.3 TFLOP/s)
PEAK_VALU_LANE_OPS = 256 * 4 * 16 * 2.4e9
METRIC = "N·M²·Q psi-stat+grad terms/sec (fp32) and % of FP32 VALU peak, 1 MI355X"


def algorithmic(kernel: str, N: int, M: int, Q: int):
    """(bound, flops or bytes per launch, unit) of each kernel's algorithmic work.

    Per unique pair (m <= m') and datapoint, the Psi2 forward needs one FMA per
    latent dimension (the Gram term) and the Psi2 gradient three (Gram
    recompute plus W*d on both sides of the pair): 2 and 6 flops per
    (n, pair, q).  Psi1 kernels are counted by their compulsory HBM bytes."""
    P = M * (M + 1) // 2
    fwd, grad = 2.0 * Q * N * P, 6.0 * Q * N * P
    table = {
        "generic_psi2_partial": ("alu", fwd, "flop"),
        "generic_grad_rows": ("alu", 4.0 * Q * N * P, "flop"),
        "generic_grad_cols": ("alu", 2.0 * Q * N * P, "flop"),
        "generic_grad_pairs": ("alu", grad, "flop"),
        "generic_grad_wide": ("alu", grad, "flop"),
        # the matrix-core Psi2 kernels are bound by instruction issue on the SIMD,
        # mostly vector ALU (exp2, weighting, operand splits); their algorithmic
        # flops are priced against the fp32 vector peak
        "mfma_psi2_fwd": ("alu", fwd, "flop"),
        "mfma_psi2_grad": ("alu", grad, "flop"),
        "generic_psi1": ("hbm", 4.0 * (N * M + 2 * N * Q), "byte"),
        "mfma_psi1_fwd": ("hbm", 4.0 * (N * M + 2 * N * Q), "byte"),
        "mfma_psi1_grad": ("hbm", 4.0 * (N * M + 4 * N * Q), "byte"),
        # known inputs (S = 0): the rank-k update over the unique pairs, the
        # gradient GEMM over all M x M, Kfu, and the chain rule per (n, m, q):
        # rows a difference and an FMA, columns a difference, a product, a sum
        # and an FMA (8 flops)
        "known_syrk": ("mfma", 2.0 * N * P, "flop"),
        "known_dkfu": ("mfma", 2.0 * N * M * M, "flop"),
        "known_kfu": ("alu", 3.0 * N * M * Q, "flop"),
        "known_chain": ("alu", 8.0 * N * M * Q, "flop"),
    }
    return table.get(kernel)


def traffic_for(kernel: str, workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, if it
    was taken on the current source of the kernel; else None."""
    f = os.path.join(ROOT, "profiles", f"traffic_{kernel}_{workload}.json")
    if not os.path.exists(f):
        return None
    rec = json.load(open(f))
    src = os.path.join(ROOT, rec["source"])
    if not os.path.exists(src):
        return None
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec["source_sha256"]:
        return None
    return rec["bytes_per_launch"]


def counters_for(kernel: str, workload: str):
    """The committed rocprofv3 SQ counter summary of a kernel (per dispatch), if
    it was taken on the current source of the kernel; else None."""
    f = os.path.join(ROOT, "profiles", f"counters_{kernel}_{workload}.json")
    if not os.path.exists(f):
        return None
    rec = json.load(open(f))
    src = os.path.join(ROOT, rec["source"])
    if not os.path.exists(src):
        return None
    if hashlib.sha256(open(src, "rb").read()).hexdigest() != rec["source_sha256"]:
        return None
    return rec


def time_steps(step, steps: int, stream):
    """Headline timing with the library's per-kernel timing off: one event pair
    per step on the library's stream.  Returns (median ms, wall-clock ms per
    step between the two synchronisations, every step's ms)."""
    import torch
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(steps)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    for a, b in ev:
        a.record(stream)
        step()
        b.record(stream)
    torch.cuda.synchronize()
    wall = (time.perf_counter() - t0) * 1e3 / steps
    per = [a.elapsed_time(b) for a, b in ev]
    return float(sorted(per)[len(per) // 2]), wall, per


def kernel_pass(step, steps: int):
    """Per-kernel timing (HIP events around every library launch on its stream)
    over a separate set of steps."""
    import torch

    import paper_1410_4984_amd as gpps
    L = gpps.lib()
    torch.cuda.synchronize()
    L.gpps_timing_enable(1)
    for _ in range(steps):
        step()
    torch.cuda.synchronize()
    L.gpps_timing_enable(0)
    return timed_kernels(L)


def cpu_baseline(inp, target_s: float):
    """Time the fp64 oracle (forward + gradients) on a row sample of the workload."""
    import numpy as np

    import oracle

    oracle.build(force=False)
    N, Q = inp["mu"].shape
    M = inp["Z"].shape[0]

    def run(rows):
        sub = {k: inp[k][rows] for k in ("mu", "S", "dL_dPsi1")}
        t0 = time.perf_counter()
        oracle.psi_stats(sub["mu"], sub["S"], inp["Z"], inp["sigma_f2"], inp["l"])
        oracle.psi_grads(sub["mu"], sub["S"], inp["Z"], inp["sigma_f2"], inp["l"],
                         inp["dL_dpsi0"], sub["dL_dPsi1"], inp["dL_dPsi2"])
        return time.perf_counter() - t0

    threads = oracle.num_threads()
    # two calibration runs (the first one pays thread start-up), then the sample
    n = max(threads, 16)
    for aim in (1.0, target_s):
        t = run(np.linspace(0, N - 1, n).astype(np.int64))
        n = int(min(N, max(threads, n * aim / max(t, 1e-6))))
    rows = np.linspace(0, N - 1, n).astype(np.int64)
    t = run(rows)
    return {"value": n * M * M * Q / t, "unit": "terms/s", "cores": threads, "kind": "oracle",
            "sample": f"{n} of {N} rows (evenly spaced) of the same workload, fp64 oracle, "
                      f"forward + gradients, {t:.1f} s wall"}


def timed_kernels(L):
    cap = 64
    names = (ctypes.c_char_p * cap)()
    tot = (ctypes.c_double * cap)()
    cnt = (ctypes.c_int64 * cap)()
    n = L.gpps_timing_collect(cap, names, tot, cnt)
    if n < 0:
        raise RuntimeError("kernel timing failed")
    return {names[i].decode(): {"avg_ms": tot[i] / cnt[i], "launches": int(cnt[i])}
            for i in range(n)}


def bench_gplvm(args):
    """One step = gpps_bound (L and every gradient) at the paper's experiment shape."""
    import numpy as np
    import torch

    import paper_1410_4984_amd as gpps
    from paper_1410_4984_amd import gplvm

    N, M, Q, D = 64_000, 100, 1, 3
    Y, _ = gplvm.paper_data(N, D=D, seed=0)
    Y = Y - Y.mean(0)
    mu, S, Z, sf2, l, beta = gplvm.init_params(Y, Q, M, seed=0)
    # A well-conditioned point of this shape (the work does not depend on it):
    # evenly spaced inducing inputs and a lengthscale below their spacing give
    # cond(Kmm) ~ 1e2 and cond(Kmm + beta Psi2) ~ 1e4.  At the data-driven start
    # (inducing inputs among the means, unit lengthscale) cond(Kmm + beta Psi2)
    # is ~1e14 and the bound itself is undetermined to ~1e-2 in fp64.
    Z = np.linspace(mu.min(), mu.max(), M)[:, None]
    l = np.array([0.03])
    jitter = 1e-6
    dev, dt = "cuda:0", torch.float64
    t = {k: torch.tensor(v, dtype=dt, device=dev) for k, v in (("mu", mu), ("S", S), ("Z", Z),
                                                                ("Y", Y))}
    ws = torch.empty(gpps.bound_workspace_bytes(dt, N, M, Q, D), dtype=torch.uint8, device=dev)
    out = None

    def step():
        nonlocal out
        out = gpps.bound(t["mu"], t["S"], t["Z"], t["Y"], sf2, l, beta, jitter, out=out,
                         workspace=ws)

    for _ in range(args.warmup):
        step()
    stream = torch.cuda.current_stream()
    ms, wall, _ = time_steps(step, args.steps, stream)
    kernels = kernel_pass(step, args.kernel_steps)
    dom = max(kernels, key=lambda k: kernels[k]["avg_ms"] * kernels[k]["launches"])
    alg = algorithmic(dom, N, M, Q)
    roofline = None
    if alg:
        bound, work, unit = alg
        avg_s = kernels[dom]["avg_ms"] * 1e-3
        if unit == "flop":
            ach, peak, u = work / avg_s / 1e12, PEAK_FP64 / 1e12, "TFLOP/s"
        else:
            ach, peak, u = work / avg_s / 1e9, PEAK_HBM / 1e9, "GB/s"
        roofline = {"kernel": dom, "bound": bound, "achieved": round(ach, 4), "peak": peak,
                    "unit": u, "frac": round(ach / peak, 5), "traffic": None,
                    "algorithmic_per_launch": work}
    # at Q = 1 the statistic kernels are bound by fp64 exponentials, one per
    # datapoint and unique pair in both (the gradient's symmetric form, which
    # runs whenever one workgroup holds all of M)
    P = M * (M + 1) // 2
    exps = {"generic_psi2_partial": N * P, "generic_grad_pairs": N * P}
    exp_rate = {k: round(v / (kernels[k]["avg_ms"] * 1e-3), 1) for k, v in exps.items() if k in kernels}
    rec = {
        "metric": "Bayesian GP-LVM bound + gradient evaluations/sec (fp64), 1 MI355X",
        "value": 1e3 / ms, "unit": "evals/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "ms_per_step_wall_mean": round(wall, 4), "higher_is_better": True,
        "scaling": "weak", "vs_baseline": None, "dtype": "f64", "data": "synthetic",
        "config": {"workload": f"gplvm-paper (N={N}, M={M}, Q={Q}, D={D}, seed 0)", "N": N,
                   "M": M, "Q": Q, "D": D, "L": float(out["L"].item())},
        "roofline": roofline,
        "exp_per_s": exp_rate,
        "kernels": {k: {"avg_ms": round(v["avg_ms"], 4), "launches": v["launches"]}
                    for k, v in sorted(kernels.items())},
    }
    if not args.no_cpu_baseline:
        import oracle
        from oracle import bound as ob
        oracle.build(force=False)
        t0 = time.perf_counter()
        ref = ob.grads(mu, S, Z, Y, sf2, l, beta, jitter)
        tc = time.perf_counter() - t0
        rec["cpu_baseline"] = {"value": 1.0 / tc, "unit": "evals/s",
                               "cores": oracle.num_threads(), "kind": "oracle",
                               "sample": f"one full evaluation (all {N} rows), fp64 oracle, "
                                         f"{tc:.2f} s wall, L = {ref['L']:.6f}"}
        rec["config"]["L_rel_diff_oracle"] = abs(rec["config"]["L"] - ref["L"]) / abs(ref["L"])
    print(json.dumps(rec), flush=True)


def copy_probe(args, dev):
    """A plain device copy of args.copy_probe_mib MiB, three times (counter calibration)."""
    import torch
    if args.copy_probe_mib <= 0:
        return
    n_el = args.copy_probe_mib * (1 << 20) // 4
    src = torch.ones(n_el, device=dev)
    dst = torch.empty_like(src)
    for _ in range(3):
        torch.neg(src, out=dst)
    torch.cuda.synchronize()
    del src, dst


def bench_known(args):
    """One step = gpps_psi_stats + gpps_psi_grads with S = NULL (known inputs) at
    the large workload's shape."""
    import numpy as np
    import torch

    import paper_1410_4984_amd as gpps
    from paper_1410_4984_amd import synth

    w = synth.WORKLOADS["large"]
    N, M, Q = w.N, w.M, w.Q
    f64 = args.dtype == "f64"
    dt = torch.float64 if f64 else torch.float32
    inp = synth.make_workload("large")
    inp["S"] = None
    if not f64:
        inp = synth.to_f32(inp)
    dev = "cuda:0"
    t = {k: torch.tensor(v, dtype=dt, device=dev) for k, v in inp.items()
         if isinstance(v, np.ndarray)}
    psi0 = torch.zeros(1, dtype=dt, device=dev)
    P1 = torch.empty((N, M), dtype=dt, device=dev)
    P2 = torch.empty((M, M), dtype=dt, device=dev)
    g = {"dmu": torch.empty((N, Q), dtype=dt, device=dev), "dS": None,
         "dZ": torch.empty((M, Q), dtype=dt, device=dev),
         "dsigma_f2": torch.empty(1, dtype=dt, device=dev),
         "dl": torch.empty(Q, dtype=dt, device=dev)}
    ws = torch.empty(gpps.workspace_bytes(dt, N, M, Q), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        gpps.psi_stats(t["mu"], None, t["Z"], inp["sigma_f2"], inp["l"], out=(psi0, P1, P2),
                       workspace=ws, stream=stream)
        gpps.psi_grads(t["mu"], None, t["Z"], inp["sigma_f2"], inp["l"], inp["dL_dpsi0"],
                       t["dL_dPsi1"], t["dL_dPsi2"], out=g, workspace=ws, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    copy_probe(args, dev)
    ms, wall, _ = time_steps(step, args.steps, stream)
    kernels = kernel_pass(step, args.kernel_steps)
    dom = max(kernels, key=lambda k: kernels[k]["avg_ms"] * kernels[k]["launches"])
    peak_f = PEAK_FP64 if f64 else PEAK_FP32
    roofline = None
    alg = algorithmic(dom, N, M, Q)
    if alg:
        bound, work, unit = alg
        ach = work / (kernels[dom]["avg_ms"] * 1e-3) / 1e12
        roofline = {"kernel": dom, "bound": bound, "achieved": round(ach, 3),
                    "peak": peak_f / 1e12, "unit": "TFLOP/s", "frac": round(ach * 1e12 / peak_f, 4),
                    "traffic": None if f64 else traffic_for(dom, "large_known"),
                    "algorithmic_per_launch": work}
    mm = {}
    for k in ("known_syrk", "known_dkfu"):
        if k in kernels:
            a = algorithmic(k, N, M, Q)[1] / (kernels[k]["avg_ms"] * 1e-3)
            mm[k] = {"tflops": round(a / 1e12, 2), "frac": round(a / peak_f, 4)}
    rec = {
        "metric": METRIC.replace("(fp32)", "(fp64)") if f64 else METRIC,
        "value": float(N) * M * M * Q / (ms * 1e-3), "unit": "terms/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "ms_per_step_wall_mean": round(wall, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64" if f64 else "f32", "data": "synthetic",
        "config": {"workload": f"large-known (N={N}, M={M}, Q={Q}, S = 0: known inputs, seed 0)",
                   "N": N, "M": M, "Q": Q},
        "matrix_core": mm,
        "roofline": roofline,
        "kernels": {k: {"avg_ms": round(v["avg_ms"], 4), "launches": v["launches"]}
                    for k, v in sorted(kernels.items())},
    }
    if not args.no_cpu_baseline:
        base = dict(inp, S=np.zeros_like(inp["mu"]))
        rec["cpu_baseline"] = cpu_baseline(base, args.cpu_seconds)
        rec["cpu_baseline"]["sample"] += " (S = 0)"
    print(json.dumps(rec), flush=True)


def bench_views(args):
    """One step = gpps_psi_stats_views + gpps_psi_grads_views over three views
    sharing q(X) (section 1, MRD): N = 100,000, Q = 20, M = 256, 192, 128."""
    import numpy as np
    import torch

    import paper_1410_4984_amd as gpps
    from paper_1410_4984_amd import synth

    name = "views-large"
    N, Ms, Q = synth.VIEW_WORKLOADS[name]
    w = synth.views_to_f32(synth.make_views_workload(name))
    dev, dt = "cuda:0", torch.float32
    t = lambda a: torch.tensor(a, dtype=dt, device=dev)  # noqa: E731
    mu, S = t(w["mu"]), t(w["S"])
    V = w["views"]
    Zs = [t(v["Z"]) for v in V]
    sf, ls = [v["sigma_f2"] for v in V], [v["l"] for v in V]
    d0 = [v["dL_dpsi0"] for v in V]
    G1, G2 = [t(v["dL_dPsi1"]) for v in V], [t(v["dL_dPsi2"]) for v in V]
    ws = torch.empty(gpps.views_workspace_bytes(dt, N, list(Ms), Q), dtype=torch.uint8, device=dev)
    st_out = [(torch.zeros(1, device=dev), torch.empty((N, M), device=dev),
               torch.empty((M, M), device=dev)) for M in Ms]
    g_out = {"dmu": torch.empty((N, Q), device=dev), "dS": torch.empty((N, Q), device=dev),
             "dZ": [torch.empty((M, Q), device=dev) for M in Ms],
             "dsigma_f2": [torch.empty(1, device=dev) for _ in Ms],
             "dl": [torch.empty(Q, device=dev) for _ in Ms]}
    stream = torch.cuda.current_stream()

    def step():
        gpps.psi_stats_views(mu, S, Zs, sf, ls, out=st_out, workspace=ws, stream=stream)
        gpps.psi_grads_views(mu, S, Zs, sf, ls, d0, G1, G2, out=g_out, workspace=ws,
                             stream=stream)

    for _ in range(args.warmup):
        step()
    ms, wall, per = time_steps(step, args.steps, stream)
    kernels = kernel_pass(step, args.kernel_steps)
    terms = float(N) * Q * sum(M * M for M in Ms)
    rec = {
        "metric": "sum over views of N·M_v²·Q psi-stat+grad terms/sec (fp32), 1 MI355X",
        "value": terms / (ms * 1e-3), "unit": "terms/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(ms, 4), "ms_per_step_wall_mean": round(wall, 4),
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "f32",
        "data": "synthetic",
        "config": {"workload": f"{name} (three views sharing q(X): N={N}, Q={Q}, M={list(Ms)}, "
                               f"seed 0)", "N": N, "M": list(Ms), "Q": Q},
        "kernels": {k: {"avg_ms": round(v["avg_ms"], 4), "launches": v["launches"]}
                    for k, v in sorted(kernels.items())},
    }
    if not args.no_cpu_baseline:
        import oracle
        oracle.build(force=False)
        rows = np.linspace(0, N - 1, 400).astype(np.int64)
        t0 = time.perf_counter()
        for v in V:
            oracle.psi_stats(w["mu"][rows], w["S"][rows], v["Z"], v["sigma_f2"], v["l"])
            oracle.psi_grads(w["mu"][rows], w["S"][rows], v["Z"], v["sigma_f2"], v["l"],
                             v["dL_dpsi0"], v["dL_dPsi1"][rows], v["dL_dPsi2"])
        tc = time.perf_counter() - t0
        rec["cpu_baseline"] = {"value": len(rows) * Q * sum(M * M for M in Ms) / tc,
                               "unit": "terms/s", "cores": oracle.num_threads(), "kind": "oracle",
                               "sample": f"{len(rows)} of {N} rows (evenly spaced), every view, "
                                         f"fp64 oracle, forward + gradients, {tc:.1f} s wall"}
    print(json.dumps(rec), flush=True)


def main():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=3)
    ap.add_argument("--kernel-steps", type=int, default=5,
                    help="steps of the second pass with per-kernel timing on")
    ap.add_argument("--workload", default="large")
    ap.add_argument("--path", default="auto", choices=["auto", "generic", "mfma"])
    ap.add_argument("--cpu-seconds", type=float, default=20.0)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-probe-mib", type=int, default=0)
    ap.add_argument("--dtype", default="f32", choices=["f32", "f64"],
                    help="element type (f64: the generic fp64 kernels; not for gplvm, which "
                         "is fp64, or views)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the multi-GPU path (row sharding with an "
              "all-reduce of Psi2 and the global gradients) is a design, not built here.",
              file=sys.stderr)
        sys.exit(2)

    if args.workload == "gplvm":
        bench_gplvm(args)
        return
    if args.workload == "known":
        bench_known(args)
        return
    if args.workload == "views":
        bench_views(args)
        return

    import numpy as np
    import torch

    import paper_1410_4984_amd as gpps
    from paper_1410_4984_amd import synth

    w = synth.WORKLOADS[args.workload]
    N, M, Q = w.N, w.M, w.Q
    f64 = args.dtype == "f64"
    npdt = np.float64 if f64 else np.float32
    inp = synth.make_workload(args.workload)
    if not f64:
        inp = synth.to_f32(inp)
    C = w.chunk_rows or N
    chunks = [(r0, min(N, r0 + C)) for r0 in range(0, N, C)]
    if w.chunk_rows:
        # row chunks accumulating on the device, each chunk's dL/dPsi1 from its own seed
        inp["dL_dPsi1"] = np.concatenate([
            synth.stress_dL_dPsi1_chunk(0, c, r1 - r0, M).astype(npdt)
            for c, (r0, r1) in enumerate(chunks)])
    dev = "cuda:0"
    dt = torch.float64 if f64 else torch.float32
    t = {k: torch.tensor(v, dtype=dt, device=dev) for k, v in inp.items()
         if isinstance(v, np.ndarray)}
    gpps.set_path(args.path)
    psi0 = torch.zeros(1, dtype=dt, device=dev)
    P1 = torch.empty((N, M), dtype=dt, device=dev)
    P2 = torch.empty((M, M), dtype=dt, device=dev)
    g = {k: torch.empty(shape, dtype=dt, device=dev)
         for k, shape in (("dmu", (N, Q)), ("dS", (N, Q)), ("dZ", (M, Q)), ("dsigma_f2", (1,)),
                          ("dl", (Q,)))}
    ws = torch.empty(gpps.workspace_bytes(dt, C, M, Q), dtype=torch.uint8, device=dev)
    stream = torch.cuda.current_stream()

    def step():
        for c, (r0, r1) in enumerate(chunks):
            gpps.psi_stats(t["mu"][r0:r1], t["S"][r0:r1], t["Z"], inp["sigma_f2"], inp["l"],
                           accumulate=c > 0, out=(psi0, P1[r0:r1], P2), workspace=ws,
                           stream=stream)
        for c, (r0, r1) in enumerate(chunks):
            sub = dict(g, dmu=g["dmu"][r0:r1], dS=g["dS"][r0:r1])
            gpps.psi_grads(t["mu"][r0:r1], t["S"][r0:r1], t["Z"], inp["sigma_f2"], inp["l"],
                           inp["dL_dpsi0"], t["dL_dPsi1"][r0:r1], t["dL_dPsi2"],
                           accumulate=c > 0, out=sub, workspace=ws, stream=stream)

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    copy_probe(args, dev)
    ms, wall, per = time_steps(step, args.steps, stream)
    kernels = kernel_pass(step, args.kernel_steps)
    rates = gpps.unit_rates(dev)
    terms = float(N) * M * M * Q
    P = M * (M + 1) // 2

    # which kernels computed the step: the matrix-core ones unless the range guard
    # sent the call to the generic kernels (the route word; fp64 is always generic)
    on_mfma = any(k.startswith("mfma_psi2") for k in kernels) and \
        gpps.route_taken(ws, dt, C, M, Q) == 0
    PEAK_VALU = PEAK_FP64 if f64 else PEAK_FP32
    # dominant kernel and its roofline (a chunked workload launches each kernel
    # once per chunk: the mean launch covers N / chunks rows)
    dom = max(kernels, key=lambda k: kernels[k]["avg_ms"] * kernels[k]["launches"])
    alg = algorithmic(dom, N / len(chunks), M, Q)
    roofline = None
    if alg:
        bound, work, unit = alg
        avg_s = kernels[dom]["avg_ms"] * 1e-3
        if unit == "flop":
            ach, peak, u = work / avg_s / 1e12, PEAK_VALU / 1e12, "TFLOP/s"
        else:
            ach, peak, u = work / avg_s / 1e9, PEAK_HBM / 1e9, "GB/s"
        roofline = {"kernel": dom, "bound": bound, "achieved": round(ach, 3), "peak": peak,
                    "unit": u, "frac": round(ach / peak, 4),
                    "traffic": traffic_for(dom, args.workload),
                    "algorithmic_per_launch": work}
        if unit == "flop" and on_mfma:
            roofline["note"] = (
                "algorithmic fp32 flops (each unordered pair once) against the fp32 vector peak; "
                "the Q-long contractions run on the matrix cores, so the fraction can pass 1; "
                "'issue' gives what each unit executed")
        cnt = counters_for(dom, args.workload) if on_mfma else None
        if cnt is not None and unit == "flop":
            c = cnt["per_dispatch"]
            mfma_flops = c["SQ_INSTS_MFMA"] * cnt["flops_per_mfma"]
            roofline["limiter"] = (
                "SIMD instruction issue: vector ALU and matrix cores share each wave's issue; "
                "busy shares per SIMD from the committed SQ counters")
            roofline["issue"] = {
                "valu_busy": cnt["derived"]["valu_busy"],
                "mfma_busy": cnt["derived"]["mfma_busy"],
                "both_busy": cnt["derived"]["both_busy"],
                "mfma_executed_flops_per_launch": mfma_flops,
                "mfma_executed_tflops": round(mfma_flops / avg_s / 1e12, 2),
                "mfma_peak_f16_tflops": PEAK_F16_MFMA / 1e12,
                "mfma_frac_f16_peak": round(mfma_flops / avg_s / PEAK_F16_MFMA, 4),
                "mfma_frac_f16_measured": round(mfma_flops / avg_s / rates["mfma_f16_flops"], 4),
                "valu_insts_per_launch": c["SQ_INSTS_VALU"],
                "valu_lane_ops_per_s": float(f"{c['SQ_INSTS_VALU'] * 64 / avg_s:.4g}"),
                "valu_frac_lane_issue_peak": round(c["SQ_INSTS_VALU"] * 64 / avg_s
                                                   / PEAK_VALU_LANE_OPS, 4),
                "exp_executed_per_launch": c["SQ_INSTS_VALU_TRANS_F32"] * 64,
                "exp_unique_pairs_per_launch": float(N) / len(chunks) * P,
                "counters": f"profiles/counters_{dom}_{args.workload}.md"}
    # Psi2 forward + gradient kernels with their reductions (F_alg's kernels), and
    # beside them with the per-row kernels that feed them
    core = ("psi2_partial", "psi2_fwd", "psi2_grad", "grad_rows", "grad_cols", "grad_pairs",
            "grad_wide",
            "psi2_reduce", "psi2_finalize", "grad_reduce")
    feed = ("mfma_rows", "mfma_rowterm", "mfma_centre", "mfma_guard", "mfma_sym",
            "mfma_absmax", "generic_rows_pre", "generic_sym", "generic_circ", "generic_psi1")
    per_step = {k: v["avg_ms"] * v["launches"] / args.kernel_steps for k, v in kernels.items()}
    t_psi2 = sum(v for k, v in per_step.items() if any(c in k for c in core)) * 1e-3
    t_feed = sum(v for k, v in per_step.items() if any(c in k for c in feed)) * 1e-3
    F_alg = 8.0 * Q * N * P
    rec = {
        "metric": METRIC, "value": terms / (ms * 1e-3), "unit": "terms/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": round(ms, 4),
        "ms_per_step_wall_mean": round(wall, 4),
        "ms_per_step_min_max": [round(min(per), 4), round(max(per), 4)],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None,
        "dtype": "f64" if f64 else "f32", "data": "synthetic",
        "config": {"workload": (f"{args.workload} (N={N}, M={M}, Q={Q}, seed 0"
                                + (f", {len(chunks)} row chunks of {C} accumulating on the device)"
                                   if len(chunks) > 1 else ")")),
                   "N": N, "M": M, "Q": Q, "path": args.path,
                   "arithmetic": (("matrix-core path: Gram and W [Z | 1] products on "
                                   "v_mfma_f32_32x32x16_f16 with two-part fp16 operands (22 "
                                   "significant bits, three cross products) accumulated in fp32; "
                                   "exponentials, weighting and epilogues in fp32 on the vector "
                                   "ALU") if on_mfma else
                                  f"generic path: {'fp64' if f64 else 'fp32'} on the vector ALU")},
        f"pct_{'fp64' if f64 else 'fp32'}_peak": (round(100.0 * F_alg / t_psi2 / PEAK_VALU, 2)
                                                  if t_psi2 > 0 else None),
        f"pct_{'fp64' if f64 else 'fp32'}_peak_with_row_kernels": (
            round(100.0 * F_alg / (t_psi2 + t_feed) / PEAK_VALU, 2) if t_psi2 > 0 else None),
        "exp_per_s": 2.0 * N * P / t_psi2 if t_psi2 > 0 else None,
        "exp_frac_measured_rate": (round(2.0 * N * P / t_psi2 / rates["exp"], 4)
                                   if t_psi2 > 0 and not f64 else None),
        "unit_rates_measured": {k: float(f"{v:.4g}") for k, v in rates.items()},
        "roofline": roofline,
        "kernels": {k: {"avg_ms": round(v["avg_ms"], 4), "launches": v["launches"]}
                    for k, v in sorted(kernels.items())},
    }
    if not args.no_cpu_baseline:
        rec["cpu_baseline"] = cpu_baseline(inp, args.cpu_seconds)
    print(json.dumps(rec), flush=True)


if __name__ == "__main__":
    main()
