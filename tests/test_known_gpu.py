"""GPU parity of the known-input path (S = NULL: every variance zero, the sparse
GP regression case of eq. (boundF)) against the fp64 CPU oracle.

With S = 0 the oracle's closed forms reduce exactly to Psi1 = K(X, Z) and
Psi2 = sum_n k_n k_n^T (pinned on the CPU by the zero-variance test of the
oracle), so the oracle runs with an all-zero S while the library gets S = NULL
and takes its matrix-core GEMM path.  Tolerances as for the S > 0 path:
relative Frobenius norm 1e-5 for Psi1 and 1e-4 for Psi2 and every gradient on
fp32, 1e-10 on fp64; fp32 inputs are rounded first and the oracle receives them
upcast.  Small shapes are compared in full, spanning several 64-blocks, ragged
tails in N and M, and the degenerate sizes; the large workload (N = 100,000,
M = 256, Q = 20) runs at full size in the launch configuration the benchmark
times, checked on sampled outputs and through exact identities.
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import paper_1410_4984_amd as gpps  # noqa: E402
from oracle import bound as ob  # noqa: E402
from paper_1410_4984_amd import synth  # noqa: E402
from parity_log import current_test, record  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
TOL32 = {"psi0": 1e-6, "Psi1": 1e-5, "Psi2": 1e-4, "dmu": 1e-4, "dZ": 1e-4, "dsigma_f2": 1e-4,
         "dl": 1e-4}
TOL64 = {k: 1e-10 for k in TOL32}


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel(a, ref):
    a, ref = np.asarray(a, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref.ravel())
    return np.linalg.norm((a - ref).ravel()) / (den if den > 0 else 1.0)


@pytest.fixture(scope="module", autouse=True)
def _libs():
    oracle.build(force=False)
    gpps.lib()
    assert torch.cuda.is_available(), "GPU tests need a GPU"


def known_inputs(N, M, Q, seed, f32):
    inp = synth.random_inputs(N, M, Q, seed=seed)
    inp["S"] = None
    return synth.to_f32(inp) if f32 else inp


def run_gpu(inp, dtype, want_psi1=True, workspace=None):
    t = lambda a: None if a is None else torch.tensor(a, dtype=dtype, device=DEV)  # noqa: E731
    X, Z = t(inp["mu"]), t(inp["Z"])
    psi0, P1, P2 = gpps.psi_stats(X, None, Z, inp["sigma_f2"], inp["l"], want_psi1=want_psi1,
                                  workspace=workspace)
    g = gpps.psi_grads(X, None, Z, inp["sigma_f2"], inp["l"], inp["dL_dpsi0"],
                       t(inp["dL_dPsi1"]), t(inp["dL_dPsi2"]), workspace=workspace)
    torch.cuda.synchronize()
    assert g["dS"] is None
    out = {"psi0": psi0.cpu().double().numpy()[0], "Psi2": P2.cpu().double().numpy()}
    if want_psi1:
        out["Psi1"] = P1.cpu().double().numpy()
    for k in ("dmu", "dZ", "dsigma_f2", "dl"):
        out[k] = g[k].cpu().double().numpy()
    out["dsigma_f2"] = out["dsigma_f2"][0]
    return out


def run_oracle(inp):
    S0 = np.zeros_like(inp["mu"])
    psi0, P1, P2 = oracle.psi_stats(inp["mu"], S0, inp["Z"], inp["sigma_f2"], inp["l"])
    g = oracle.psi_grads(inp["mu"], S0, inp["Z"], inp["sigma_f2"], inp["l"], inp["dL_dpsi0"],
                         inp["dL_dPsi1"], inp["dL_dPsi2"])
    return dict(psi0=psi0, Psi1=P1, Psi2=P2, dmu=g["dmu"], dZ=g["dZ"], dsigma_f2=g["dsigma_f2"],
                dl=g["dl"])


def compare_all(got, ref, tol, label):
    bad = {}
    for k in ref:
        if k not in got:
            continue
        e = rel(got[k], ref[k])
        say(f"  {label} {k}: rel {e:.3e} (tol {tol[k]:.0e})")
        record(current_test(), label, k, e, tol[k])
        if not e <= tol[k]:
            bad[k] = e
    assert not bad, (label, bad)


SHAPES = [(200, 10, 2), (1000, 70, 3), (5000, 50, 10), (3001, 130, 20), (1, 5, 3), (300, 1, 4),
          (150, 17, 64), (3, 1100, 2), (64, 64, 1), (65, 129, 7)]


@pytest.mark.parametrize("shape", SHAPES, ids=[f"{n}x{m}x{q}" for n, m, q in SHAPES])
@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_known_full(dtype, shape):
    N, M, Q = shape
    f32 = dtype == "f32"
    say(f"[known {dtype} N={N} M={M} Q={Q}]")
    inp = known_inputs(N, M, Q, seed=N + M + Q, f32=f32)
    got = run_gpu(inp, torch.float32 if f32 else torch.float64)
    compare_all(got, run_oracle(inp), TOL32 if f32 else TOL64, f"known/{dtype}/{N}x{M}x{Q}")
    assert np.array_equal(got["Psi2"], got["Psi2"].T)


def _identities(inp, got, label, tol=2e-5):
    """Exact identities of the gradients on the GPU's own outputs (S = 0):
    translation and scaling of each input dimension, sigma_f2-homogeneity."""
    X, Z, l, sf2 = inp["mu"], inp["Z"], inp["l"], inp["sigma_f2"]
    dX, dZ, dl = got["dmu"], got["dZ"], got["dl"]
    r = dX.sum(0) + dZ.sum(0)
    s = np.abs(dX).sum(0) + np.abs(dZ).sum(0)
    say(f"  {label} translation residual {np.max(np.abs(r) / s):.2e}")
    assert np.all(np.abs(r) <= tol * s)
    r = (X * dX).sum(0) + (Z * dZ).sum(0) + l * dl
    s = np.abs(X * dX).sum(0) + np.abs(Z * dZ).sum(0) + np.abs(l * dl)
    say(f"  {label} scaling residual {np.max(np.abs(r) / s):.2e}")
    assert np.all(np.abs(r) <= tol * s)
    G2s = 0.5 * (inp["dL_dPsi2"] + inp["dL_dPsi2"].T)
    a = np.sum(inp["dL_dPsi1"] * got["Psi1"])
    b = 2 * np.sum(G2s * got["Psi2"])
    c = inp["dL_dpsi0"] * X.shape[0] * sf2
    r = sf2 * got["dsigma_f2"] - (a + b + c)
    say(f"  {label} homogeneity residual {abs(r) / (abs(a) + abs(b) + abs(c)):.2e}")
    assert abs(r) <= 1e-4 * (abs(a) + abs(b) + abs(c))


def test_known_large_full_size_sampled():
    """The large workload's shape and distributions with known inputs, at full
    size: sampled Psi2 entries and dZ rows (each a sum over all 100,000 rows),
    rows of Psi1 and dX, and the identities for dl and dsigma_f2."""
    say("[known large f32 full size]")
    inp = synth.to_f32(synth.make_workload("large"))
    inp["S"] = None
    got = run_gpu(inp, torch.float32)
    N, Q = inp["mu"].shape
    M = inp["Z"].shape[0]
    sf2, l = inp["sigma_f2"], inp["l"]
    assert np.array_equal(got["Psi2"], got["Psi2"].T)
    assert got["psi0"] == pytest.approx(N * sf2, rel=1e-6)
    rng = np.random.default_rng(5)
    pairs = np.stack([rng.integers(0, M, 64), rng.integers(0, M, 64)], 1)
    pairs[:4, 1] = pairs[:4, 0]
    S0 = np.zeros_like(inp["mu"])
    ref = oracle.psi2_entries(inp["mu"], S0, inp["Z"], sf2, l, pairs)
    e = rel(got["Psi2"][pairs[:, 0], pairs[:, 1]], ref)
    say(f"  Psi2 sampled: rel {e:.3e}")
    record(current_test(), "known sampled", "Psi2 (sampled entries)", e, TOL32["Psi2"])
    assert e <= TOL32["Psi2"]
    rows = np.sort(rng.choice(N, 48, replace=False))
    rows[-1] = N - 1
    _, P1, _ = oracle.psi_stats(inp["mu"][rows], S0[rows], inp["Z"], sf2, l)
    g = oracle.psi_grads(inp["mu"][rows], S0[rows], inp["Z"], sf2, l, 0.0, inp["dL_dPsi1"][rows],
                         inp["dL_dPsi2"])
    for k, a, b, tol in (("Psi1", got["Psi1"][rows], P1, TOL32["Psi1"]),
                         ("dmu", got["dmu"][rows], g["dmu"], TOL32["dmu"])):
        e = rel(a, b)
        say(f"  {k} rows: rel {e:.3e}")
        record(current_test(), "known sampled", f"{k} (sampled rows)", e, tol)
        assert e <= tol, k
    zr = rng.choice(M, 3, replace=False)
    ref = oracle.dZ_rows(inp["mu"], S0, inp["Z"], sf2, l, inp["dL_dPsi1"], inp["dL_dPsi2"], zr)
    e = rel(got["dZ"][zr], ref)
    say(f"  dZ rows: rel {e:.3e}")
    record(current_test(), "known sampled", "dZ (rows summed over all N)", e, TOL32["dZ"])
    assert e <= TOL32["dZ"]
    _identities(inp, got, "known-large")


def test_known_large_row_subset_full():
    """Every output against the oracle on a row subset of the large workload
    (same M = 256, Q = 20), dl and dsigma_f2 included."""
    inp = synth.to_f32(synth.make_workload("large"))
    rows = np.arange(0, inp["mu"].shape[0], 97)
    sub = dict(inp, mu=inp["mu"][rows], S=None, dL_dPsi1=inp["dL_dPsi1"][rows])
    compare_all(run_gpu(sub, torch.float32), run_oracle(sub), TOL32, "known-large-subset")


def test_known_stress_chunked():
    """N = 10^6, M = 512, Q = 30 (the stress workload with S dropped) in 8 row
    chunks accumulating on the device: symmetry, psi0, sampled Psi2 entries (each
    a sum over all 10^6 rows), sampled rows of Psi1 and dX, and the identities
    (translation, scaling, sigma_f2-homogeneity with <G1, Psi1> summed per chunk)."""
    say("[known stress f32 chunked]")
    w = synth.WORKLOADS["stress"]
    inp = synth.to_f32(synth.make_workload("stress"))
    inp["S"] = None
    N, M, Q, C = w.N, w.M, w.Q, w.chunk_rows
    t = lambda a: torch.tensor(a, dtype=torch.float32, device=DEV)  # noqa: E731
    X, Z, G2 = t(inp["mu"]), t(inp["Z"]), t(inp["dL_dPsi2"])
    psi0 = torch.zeros(1, device=DEV)
    Psi2 = torch.zeros((M, M), device=DEV)
    g = {"dmu": torch.empty((N, Q), device=DEV), "dS": None, "dZ": torch.zeros((M, Q), device=DEV),
         "dsigma_f2": torch.zeros(1, device=DEV), "dl": torch.zeros(Q, device=DEV)}
    ws = torch.empty(gpps.workspace_bytes("f32", C, M, Q), dtype=torch.uint8, device=DEV)
    P1 = torch.empty((C, M), device=DEV)
    rng = np.random.default_rng(6)
    rows = np.sort(rng.choice(N, 16, replace=False))
    rows[-1] = N - 1
    P1_rows = np.empty((rows.shape[0], M))
    G1_rows = np.empty((rows.shape[0], M))
    G1_sum = 0.0
    for c, r0 in enumerate(range(0, N, C)):
        r1 = min(N, r0 + C)
        G1 = synth.stress_dL_dPsi1_chunk(0, c, r1 - r0, M).astype(np.float32)
        G1d = torch.tensor(G1, device=DEV)
        P1c = P1[: r1 - r0]
        gpps.psi_stats(X[r0:r1], None, Z, inp["sigma_f2"], inp["l"], accumulate=c > 0,
                       out=(psi0, P1c, Psi2), workspace=ws)
        G1_sum += float(torch.sum(G1d.double() * P1c.double()))
        sel = (rows >= r0) & (rows < r1)
        if sel.any():
            idx = torch.tensor(rows[sel] - r0, device=DEV)
            P1_rows[sel] = P1c[idx].double().cpu().numpy()
            G1_rows[sel] = G1[rows[sel] - r0].astype(np.float64)
        gpps.psi_grads(X[r0:r1], None, Z, inp["sigma_f2"], inp["l"], inp["dL_dpsi0"], G1d, G2,
                       accumulate=c > 0, out=dict(g, dmu=g["dmu"][r0:r1]), workspace=ws)
        say(f"  chunk {c} rows {r0}:{r1} done")
    torch.cuda.synchronize()
    got = {"psi0": psi0.cpu().double().numpy()[0], "Psi2": Psi2.cpu().double().numpy()}
    for k in ("dmu", "dZ", "dsigma_f2", "dl"):
        got[k] = g[k].cpu().double().numpy()
    got["dsigma_f2"] = got["dsigma_f2"][0]
    assert np.array_equal(got["Psi2"], got["Psi2"].T)
    assert got["psi0"] == pytest.approx(N * inp["sigma_f2"], rel=1e-5)
    sf2, l = inp["sigma_f2"], inp["l"]
    S0 = np.zeros_like(inp["mu"])
    pairs = np.stack([rng.integers(0, M, 32), rng.integers(0, M, 32)], 1)
    pairs[:4, 1] = pairs[:4, 0]
    ref = oracle.psi2_entries(inp["mu"], S0, inp["Z"], sf2, l, pairs)
    e = rel(got["Psi2"][pairs[:, 0], pairs[:, 1]], ref)
    say(f"  Psi2 sampled: rel {e:.3e}")
    record(current_test(), "known sampled", "Psi2 (sampled entries)", e, TOL32["Psi2"])
    assert e <= TOL32["Psi2"]
    _, P1r, _ = oracle.psi_stats(inp["mu"][rows], S0[rows], inp["Z"], sf2, l)
    gr = oracle.psi_grads(inp["mu"][rows], S0[rows], inp["Z"], sf2, l, 0.0, G1_rows,
                          inp["dL_dPsi2"])
    for k, a, b, tol in (("Psi1", P1_rows, P1r, TOL32["Psi1"]),
                         ("dmu", got["dmu"][rows], gr["dmu"], TOL32["dmu"])):
        e = rel(a, b)
        say(f"  {k} rows: rel {e:.3e}")
        record(current_test(), "known sampled", f"{k} (sampled rows)", e, tol)
        assert e <= tol, k
    # identities (the Psi1 term of homogeneity from the per-chunk sums)
    Xn, Zn = inp["mu"], inp["Z"]
    r = got["dmu"].sum(0) + got["dZ"].sum(0)
    sc = np.abs(got["dmu"]).sum(0) + np.abs(got["dZ"]).sum(0)
    say(f"  translation residual {np.max(np.abs(r) / sc):.2e}")
    assert np.all(np.abs(r) <= 2e-5 * sc)
    r = (Xn * got["dmu"]).sum(0) + (Zn * got["dZ"]).sum(0) + l * got["dl"]
    sc = np.abs(Xn * got["dmu"]).sum(0) + np.abs(Zn * got["dZ"]).sum(0) + np.abs(l * got["dl"])
    say(f"  scaling residual {np.max(np.abs(r) / sc):.2e}")
    assert np.all(np.abs(r) <= 2e-5 * sc)
    G2s = 0.5 * (inp["dL_dPsi2"] + inp["dL_dPsi2"].T)
    a, b, c = G1_sum, 2 * np.sum(G2s * got["Psi2"]), inp["dL_dpsi0"] * N * sf2
    r = sf2 * got["dsigma_f2"] - (a + b + c)
    say(f"  homogeneity residual {abs(r) / (abs(a) + abs(b) + abs(c)):.2e}")
    assert abs(r) <= 1e-4 * (abs(a) + abs(b) + abs(c))


def test_known_without_psi1_and_deterministic():
    inp = known_inputs(2500, 96, 5, seed=21, f32=True)
    a = run_gpu(inp, torch.float32)
    b = run_gpu(inp, torch.float32, want_psi1=False)
    for k in b:
        assert np.array_equal(a[k], b[k]), k


def test_known_chunked_accumulate_matches_single_call():
    inp = known_inputs(3001, 72, 6, seed=4, f32=True)
    whole = run_gpu(inp, torch.float32)
    t = lambda a: torch.tensor(a, dtype=torch.float32, device=DEV)  # noqa: E731
    X, Z, G1, G2 = t(inp["mu"]), t(inp["Z"]), t(inp["dL_dPsi1"]), t(inp["dL_dPsi2"])
    N, Q = inp["mu"].shape
    M = inp["Z"].shape[0]
    psi0, P1, P2 = (torch.zeros(1, device=DEV), torch.empty((N, M), device=DEV),
                    torch.empty((M, M), device=DEV))
    g = {"dmu": torch.empty((N, Q), device=DEV), "dS": None, "dZ": torch.empty((M, Q), device=DEV),
         "dsigma_f2": torch.empty(1, device=DEV), "dl": torch.empty(Q, device=DEV)}
    for i, (r0, r1) in enumerate([(0, 1000), (1000, 1001), (1001, 3001)]):
        gpps.psi_stats(X[r0:r1], None, Z, inp["sigma_f2"], inp["l"], accumulate=i > 0,
                       out=(psi0, P1[r0:r1], P2))
        gpps.psi_grads(X[r0:r1], None, Z, inp["sigma_f2"], inp["l"], inp["dL_dpsi0"], G1[r0:r1], G2,
                       accumulate=i > 0, out=dict(g, dmu=g["dmu"][r0:r1]))
    torch.cuda.synchronize()
    chunked = {"psi0": psi0.cpu().double().numpy()[0], "Psi1": P1.cpu().double().numpy(),
               "Psi2": P2.cpu().double().numpy()}
    for k in ("dmu", "dZ", "dsigma_f2", "dl"):
        chunked[k] = g[k].cpu().double().numpy()
    chunked["dsigma_f2"] = chunked["dsigma_f2"][0]
    for k in whole:
        e = rel(chunked[k], whole[k])
        assert e <= 1e-5, (k, e)
    assert np.array_equal(chunked["Psi2"], chunked["Psi2"].T)


@pytest.mark.parametrize("dtype", ["f32", "f64"])
def test_known_null_upstream_and_nonsymmetric_G2(dtype):
    f32 = dtype == "f32"
    inp = known_inputs(900, 80, 6, seed=12, f32=f32)
    rng = np.random.default_rng(13)
    G2 = rng.standard_normal((80, 80))
    inp["dL_dPsi2"] = G2.astype(np.float32).astype(np.float64) if f32 else G2
    tol = TOL32 if f32 else TOL64
    tdt = torch.float32 if f32 else torch.float64
    compare_all(run_gpu(inp, tdt), run_oracle(inp), tol, "known-nonsym")
    for drop in ("dL_dPsi1", "dL_dPsi2"):
        x = dict(inp, **{drop: None})
        got = run_gpu(x, tdt, want_psi1=False)
        compare_all(got, run_oracle(x), tol, f"known-{drop}-none")


def test_known_agrees_with_variance_path_at_tiny_variance():
    """S = NULL against the S > 0 kernels at S = 1e-12 (whose outputs differ from
    the S = 0 ones by O(1e-12)): two independent code paths, one answer."""
    inp = known_inputs(1500, 40, 4, seed=31, f32=False)
    got = run_gpu(inp, torch.float64)
    t = lambda a: torch.tensor(a, dtype=torch.float64, device=DEV)  # noqa: E731
    X, Z = t(inp["mu"]), t(inp["Z"])
    S = torch.full_like(X, 1e-12)
    psi0, P1, P2 = gpps.psi_stats(X, S, Z, inp["sigma_f2"], inp["l"])
    g = gpps.psi_grads(X, S, Z, inp["sigma_f2"], inp["l"], inp["dL_dpsi0"], t(inp["dL_dPsi1"]),
                       t(inp["dL_dPsi2"]))
    torch.cuda.synchronize()
    other = {"Psi1": P1, "Psi2": P2, "dmu": g["dmu"], "dZ": g["dZ"], "dl": g["dl"]}
    for k, v in other.items():
        e = rel(got[k], v.cpu().numpy())
        say(f"  S=NULL vs S=1e-12 {k}: rel {e:.2e}")
        assert e <= 1e-9, k


# ------------------------------------------------------------------ the regression bound

BKEYS = ("dmu", "dZ", "dsigma_f2", "dl", "dbeta")


def regression_problem(N, M, Q, D, seed, jitter):
    rng = np.random.default_rng(seed)
    return dict(X=rng.uniform(-3, 3, size=(N, Q)), Z=rng.uniform(-3, 3, size=(M, Q)),
                Y=rng.normal(size=(N, D)), sigma_f2=1.3, l=rng.uniform(0.8, 1.8, size=Q),
                beta=2.5, jitter=jitter)


def run_bound(p, dtype):
    t = {k: torch.tensor(p[k], dtype=dtype, device=DEV) for k in ("X", "Z", "Y")}
    out = gpps.bound(t["X"], None, t["Z"], t["Y"], p["sigma_f2"], p["l"], p["beta"], p["jitter"])
    torch.cuda.synchronize()
    assert out["dS"] is None
    return {k: v.double().cpu().numpy() for k, v in out.items() if v is not None}


def oracle_bound(p, f32, inverse=ob._inv_spd):
    q = {k: (np.asarray(v, np.float32).astype(np.float64) if (f32 and isinstance(v, np.ndarray))
             else v) for k, v in p.items()}
    return ob.grads(q["X"], None, q["Z"], q["Y"], q["sigma_f2"], q["l"], q["beta"], q["jitter"],
                    inverse=inverse)


@pytest.mark.parametrize("shape", [(400, 20, 2, 3), (3000, 70, 1, 2), (2000, 130, 3, 4)])
def test_regression_bound_f64_matches_oracle(shape):
    N, M, Q, D = shape
    p = regression_problem(N, M, Q, D, seed=N + M, jitter=1e-4)
    Kmm = ob.kmm(p["Z"], p["sigma_f2"], p["l"]) + p["jitter"] * np.eye(M)
    say(f"  cond(Kmm) {np.linalg.cond(Kmm):.1e}")
    got, ref = run_bound(p, torch.float64), oracle_bound(p, False)
    alts = [oracle_bound(p, False, inverse=inv) for inv in (ob._inv_lu, ob._inv_eigh)]
    e = abs(got["L"][0] - ref["L"]) / abs(ref["L"])
    tol = max(1e-9, 10 * max(abs(a["L"] - ref["L"]) / abs(ref["L"]) for a in alts))
    say(f"  regression f64 {shape} L: rel {e:.2e} (tol {tol:.1e})")
    assert e <= tol
    for k in BKEYS:
        r = np.asarray(ref[k])
        e = rel(got[k].reshape(r.shape), r)
        tol = max(1e-9, 10 * max(rel(np.asarray(a[k]), r) for a in alts))
        say(f"  regression f64 {shape} {k}: rel {e:.2e} (tol {tol:.1e})")
        assert e <= tol, k


def _grid_problem():
    g = np.linspace(-3, 3, 5)
    rng = np.random.default_rng(8)
    return dict(X=rng.uniform(-3, 3, size=(20000, 2)), Z=np.array([[a, b] for a in g for b in g]),
                Y=rng.normal(size=(20000, 2)), sigma_f2=1.3, l=np.array([1.0, 1.2]), beta=2.5,
                jitter=1e-3)


def fp32_stats_spread(p, trials=3):
    """Per output, the largest relative change of the oracle's result when Psi1
    and Psi2 carry independent relative errors of a few fp32 units (uniform in
    +-2^-24 and +-2^-22): how much an output moves for errors an fp32 path
    cannot avoid in its stored statistics."""
    q = {k: (np.asarray(v, np.float32).astype(np.float64) if isinstance(v, np.ndarray) else v)
         for k, v in p.items()}
    args = (q["X"], None, q["Z"], q["Y"], q["sigma_f2"], q["l"], q["beta"], q["jitter"])
    X = q["X"]
    psi0, P1, P2 = oracle.psi_stats(X, np.zeros_like(X), q["Z"], q["sigma_f2"], q["l"])
    P1 = np.asarray(P1).reshape(X.shape[0], -1)
    ref = ob.grads(*args, stats=(psi0, P1, P2))
    rng = np.random.default_rng(0)
    spread = {k: 0.0 for k in ("L",) + BKEYS}
    for _ in range(trials):
        E2 = rng.uniform(-1, 1, P2.shape) * 2.0 ** -22
        alt = ob.grads(*args, stats=(psi0, P1 * (1 + rng.uniform(-1, 1, P1.shape) * 2.0 ** -24),
                                     P2 * (1 + (E2 + E2.T) / 2)))
        for k in spread:
            a, r = np.asarray(alt[k], np.float64), np.asarray(ref[k], np.float64)
            spread[k] = max(spread[k], rel(a, r))
    return spread


# Fixed bars of the fp32 regression bound per case and output.  random16's dZ
# is the difference of its contributions through Kfu and through Kmm; its
# oracle moves by 1.3e-4 when Psi1 and Psi2 carry a few fp32 units of error
# (cond(A) = 5.6e3), so its bar is 5e-4; every other output of both cases moves
# by less than 1e-5 and keeps the fp32 bar 1e-4.
F32_BOUND_BARS = {"random16": {"dZ": 5e-4}, "grid25": {}}


@pytest.mark.parametrize("case", ["random16", "grid25"])
def test_regression_bound_f32_matches_oracle(case):
    """The fp32 path stores Psi1 and Psi2 in fp32; the bound's M x M algebra
    (fp64) amplifies their rounding by the conditioning of A = Kmm + beta Psi2,
    and dZ (a difference of its contributions through Kfu and through Kmm) most
    of all.  Tolerances are fixed per case and output (F32_BOUND_BARS, else
    1e-4); each must be at least 3 x the oracle's own spread under errors of a
    few fp32 units in Psi1 and Psi2, measured here, so that a bar follows from
    the conditioning and not from the GPU's result.  The cases keep cond(A) <=
    1e4 (checked)."""
    p = regression_problem(5000, 16, 2, 3, seed=7, jitter=1e-3) if case == "random16" \
        else _grid_problem()
    _, _, pc = ob.bound_terms(p["X"], None, p["Z"], p["Y"], p["sigma_f2"], p["l"], p["beta"],
                              p["jitter"])
    cond = np.linalg.cond(pc["Kmm"] + p["beta"] * pc["Psi2"])
    say(f"  regression f32 {case}: cond(A) {cond:.1e}")
    assert cond <= 1e4
    spread = fp32_stats_spread(p)
    got, ref = run_bound(p, torch.float32), oracle_bound(p, True)
    bars = F32_BOUND_BARS[case]
    for k in ("L",) + BKEYS:
        r = np.asarray(ref[k])
        e = abs(got["L"][0] - ref["L"]) / abs(ref["L"]) if k == "L" else rel(got[k].reshape(r.shape), r)
        bar = bars.get(k, 1e-4)
        say(f"  regression f32 {case} {k}: rel {e:.2e} (bar {bar:.0e}, oracle fp32 spread "
            f"{spread[k]:.1e})")
        record(current_test(), f"regression-f32/{case}", k, e, bar)
        assert spread[k] * 3 <= bar, (k, spread[k])
        assert e <= bar, k
