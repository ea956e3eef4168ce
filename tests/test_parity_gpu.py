"""GPU parity: the HIP library (through its C ABI) against the fp64 CPU oracle.

Tolerances are relative Frobenius norms per output, ||gpu - ref|| / ||ref||:
fp32 path 1e-5 for Psi1 and 1e-4 for Psi2 and every gradient; fp64 path 1e-10.
The oracle receives the fp32-rounded inputs upcast to fp64, so the comparison
measures the kernels' arithmetic, not input rounding.

Small workloads are compared element by element in full.  The large and stress
workloads run at full size in the launch configuration the benchmark times;
there the oracle computes sampled outputs one by one (Psi2 entries, rows of
Psi1 / dmu / dS, rows of dZ, each summed over every datapoint), and the
outputs it cannot afford (dl, dsigma_f2, dZ at stress) are checked through
identities that hold at any size: translation and per-dimension scaling of the
latent space, and sigma_f2-homogeneity.
"""
import os
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import paper_1410_4984_amd as gpps  # noqa: E402
from paper_1410_4984_amd import synth  # noqa: E402
from parity_log import current_test, record  # noqa: E402

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL32 = {"psi0": 1e-6, "Psi1": 1e-5, "Psi2": 1e-4, "dmu": 1e-4, "dS": 1e-4, "dZ": 1e-4,
         "dsigma_f2": 1e-4, "dl": 1e-4}
TOL64 = {k: 1e-10 for k in TOL32}
PATHS = ["generic", "mfma"]


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel(a, ref):
    a, ref = np.asarray(a, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref.ravel())
    return np.linalg.norm((a - ref).ravel()) / (den if den > 0 else 1.0)


@pytest.fixture(autouse=True)
def _restore_path():
    yield
    gpps.set_path("auto")


def use_path(path, dtype):
    if path == "mfma":
        if dtype != torch.float32:
            pytest.skip("the matrix-core path is F32 only")
    gpps.set_path(path)


def dev(inp, dtype):
    t = lambda a: None if a is None else torch.tensor(a, dtype=dtype, device=DEV)  # noqa: E731
    return {k: (t(v) if isinstance(v, np.ndarray) else v) for k, v in inp.items()}


def routes(ws, dtype, N, M, Q):
    """Route word of the last call on ws (0 matrix cores, 1 generic by the range
    guard), or None where the call could not have taken the matrix-core path."""
    if dtype != torch.float32 or gpps.get_path() == "generic":
        return None
    return gpps.route_taken(ws, dtype, N, M, Q)


def run_gpu(inp, dtype, want_psi1=True, expect_route=None):
    """Both entry points on the GPU.  Where the call takes the matrix-core path
    (forced, or expect_route given) the route word of each call must equal
    expect_route (default 0: the matrix cores computed it)."""
    d = dev(inp, dtype)
    N, Q = inp["mu"].shape
    M = inp["Z"].shape[0]
    ws = torch.full((gpps.workspace_bytes(dtype, N, M, Q),), 0x7F, dtype=torch.uint8, device=DEV)
    mfma = dtype == torch.float32 and (gpps.get_path() == "mfma" or
                                       (gpps.get_path() == "auto" and expect_route is not None))
    if expect_route is None:
        expect_route = 0
    try:
        psi0, P1, P2 = gpps.psi_stats(d["mu"], d["S"], d["Z"], inp["sigma_f2"], inp["l"],
                                      want_psi1=want_psi1, workspace=ws)
        if mfma:
            assert routes(ws, dtype, N, M, Q) == expect_route, "psi_stats route"
        g = gpps.psi_grads(d["mu"], d["S"], d["Z"], inp["sigma_f2"], inp["l"], inp["dL_dpsi0"],
                           d["dL_dPsi1"], d["dL_dPsi2"], workspace=ws)
        if mfma:
            assert routes(ws, dtype, N, M, Q) == expect_route, "psi_grads route"
    except gpps.GppsError as e:
        if e.status == 8:
            pytest.skip("path does not support this shape")
        raise
    torch.cuda.synchronize()
    out = {"psi0": psi0.cpu().double().numpy()[0], "Psi2": P2.cpu().double().numpy()}
    if want_psi1:
        out["Psi1"] = P1.cpu().double().numpy()
    for k, v in g.items():
        out[k] = v.cpu().double().numpy()
    out["dsigma_f2"] = out["dsigma_f2"][0]
    return out


def run_oracle(inp):
    psi0, P1, P2 = oracle.psi_stats(inp["mu"], inp["S"], inp["Z"], inp["sigma_f2"], inp["l"])
    g = oracle.psi_grads(inp["mu"], inp["S"], inp["Z"], inp["sigma_f2"], inp["l"],
                         inp["dL_dpsi0"], inp["dL_dPsi1"], inp["dL_dPsi2"])
    return dict(psi0=psi0, Psi1=P1, Psi2=P2, **g)


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


_ORACLE_CACHE = {}


def oracle_for(name, f32):
    key = (name, f32)
    if key not in _ORACLE_CACHE:
        inp = synth.make_workload(name)
        if f32:
            inp = synth.to_f32(inp)
        _ORACLE_CACHE[key] = (inp, run_oracle(inp))
    return _ORACLE_CACHE[key]


@pytest.fixture(scope="module", autouse=True)
def _libs():
    oracle.build(force=False)
    gpps.lib()
    assert torch.cuda.is_available(), "GPU tests need a GPU"


# ------------------------------------------------------------------ full comparisons

@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("dtype", ["f64", "f32"])
def test_tiny_full(dtype, path):
    tdt = torch.float64 if dtype == "f64" else torch.float32
    use_path(path, tdt)
    say(f"[tiny {dtype} {path}]")
    inp, ref = oracle_for("tiny", dtype == "f32")
    got = run_gpu(inp, tdt)
    compare_all(got, ref, TOL64 if dtype == "f64" else TOL32, f"tiny/{dtype}/{path}")
    assert np.array_equal(got["Psi2"], got["Psi2"].T)


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("name", ["small", "medium"])
def test_full_f32(name, path):
    use_path(path, torch.float32)
    say(f"[{name} f32 {path}]")
    inp, ref = oracle_for(name, True)
    got = run_gpu(inp, torch.float32)
    compare_all(got, ref, TOL32, f"{name}/f32/{path}")
    assert np.array_equal(got["Psi2"], got["Psi2"].T)


def test_small_f64_generic():
    use_path("generic", torch.float64)
    inp, ref = oracle_for("small", False)
    got = run_gpu(inp, torch.float64)
    compare_all(got, ref, TOL64, "small/f64")


# ------------------------------------------------------------------ full size, sampled

def _sampled_checks(inp, got, rng, label, n_rows=48, n_pairs=64, dz_rows=3, G1_rows=None,
                    dz_ref=None):
    """Compare sampled outputs against the oracle and check the identities.
    dz_ref(rows) gives the oracle's dZ rows where dL/dPsi1 is not held whole."""
    N, Q = inp["mu"].shape
    M = inp["Z"].shape[0]
    sf2, l = inp["sigma_f2"], inp["l"]
    # Psi2 entries (each a sum over all N datapoints), incl. the diagonal
    pairs = np.stack([rng.integers(0, M, n_pairs), rng.integers(0, M, n_pairs)], 1)
    pairs[:4, 1] = pairs[:4, 0]
    ref = oracle.psi2_entries(inp["mu"], inp["S"], inp["Z"], sf2, l, pairs)
    e = rel(got["Psi2"][pairs[:, 0], pairs[:, 1]], ref)
    say(f"  {label} Psi2 sampled: rel {e:.3e}")
    record(current_test(), label, f"Psi2 ({n_pairs} sampled entries)", e, TOL32["Psi2"])
    assert e <= TOL32["Psi2"]
    # rows of Psi1, dmu, dS: per-row outputs depend on their own row only
    rows = np.sort(rng.choice(N, n_rows, replace=False))
    rows[-1] = N - 1
    G1 = inp["dL_dPsi1"] if G1_rows is None else G1_rows(rows)
    G1r = G1[rows] if G1_rows is None else G1
    _, P1, _ = oracle.psi_stats(inp["mu"][rows], inp["S"][rows], inp["Z"], sf2, l)
    g = oracle.psi_grads(inp["mu"][rows], inp["S"][rows], inp["Z"], sf2, l, 0.0, G1r,
                         inp["dL_dPsi2"])
    for k, got_k, ref_k, tol in (("Psi1", got.get("Psi1"), P1, TOL32["Psi1"]),
                                 ("dmu", got["dmu"], g["dmu"], TOL32["dmu"]),
                                 ("dS", got["dS"], g["dS"], TOL32["dS"])):
        if got_k is None:
            continue
        e = rel(got_k[rows], ref_k)
        say(f"  {label} {k} rows: rel {e:.3e}")
        record(current_test(), label, f"{k} ({n_rows} sampled rows)", e, tol)
        assert e <= tol, (k, e)
    # rows of dZ (sums over every datapoint)
    if dz_rows:
        zr = rng.choice(M, dz_rows, replace=False)
        if dz_ref is None:
            ref = oracle.dZ_rows(inp["mu"], inp["S"], inp["Z"], sf2, l, inp["dL_dPsi1"],
                                 inp["dL_dPsi2"], zr)
        else:
            ref = dz_ref(zr)
        e = rel(got["dZ"][zr], ref)
        say(f"  {label} dZ rows: rel {e:.3e}")
        record(current_test(), label, f"dZ ({dz_rows} rows, each summed over all N)", e,
               TOL32["dZ"])
        assert e <= TOL32["dZ"]
    _identities(inp, got, label)


def _identities(inp, got, label, tol=2e-5):
    """Exact identities of the gradients, evaluated on the GPU's own outputs.
    Each residual is compared with the sum of the magnitudes of its terms."""
    mu, S, Z, l, sf2 = inp["mu"], inp["S"], inp["Z"], inp["l"], inp["sigma_f2"]
    dmu, dS, dZ, dl = got["dmu"], got["dS"], got["dZ"], got["dl"]
    # translation of latent dimension q
    r = dmu.sum(0) + dZ.sum(0)
    s = np.abs(dmu).sum(0) + np.abs(dZ).sum(0)
    say(f"  {label} translation residual {np.max(np.abs(r) / s):.2e}")
    record(current_test(), label, "translation identity residual", np.max(np.abs(r) / s), tol)
    assert np.all(np.abs(r) <= tol * s)
    # scaling of latent dimension q (mu, z, l scaled by c, S by c^2)
    terms = [(mu * dmu).sum(0), (Z * dZ).sum(0), l * dl, 2 * (S * dS).sum(0)]
    r = sum(terms)
    s = (np.abs(mu * dmu).sum(0) + np.abs(Z * dZ).sum(0) + np.abs(l * dl)
         + 2 * np.abs(S * dS).sum(0))
    say(f"  {label} scaling residual {np.max(np.abs(r) / s):.2e}")
    record(current_test(), label, "scaling identity residual", np.max(np.abs(r) / s), tol)
    assert np.all(np.abs(r) <= tol * s)
    # sf2 homogeneity: sf2 dL/dsf2 = <G1, Psi1> + 2 <G2s, Psi2> + dL_dpsi0 N sf2
    if "Psi1" in got and inp.get("dL_dPsi1") is not None:
        G2s = 0.5 * (inp["dL_dPsi2"] + inp["dL_dPsi2"].T)
        a = np.sum(inp["dL_dPsi1"] * got["Psi1"])
        b = 2 * np.sum(G2s * got["Psi2"])
        c = inp["dL_dpsi0"] * mu.shape[0] * sf2
        r = sf2 * got["dsigma_f2"] - (a + b + c)
        s = abs(a) + abs(b) + abs(c)
        say(f"  {label} homogeneity residual {abs(r) / s:.2e}")
        record(current_test(), label, "sigma_f2 homogeneity residual", abs(r) / s, 1e-4)
        assert abs(r) <= 1e-4 * s


@pytest.mark.parametrize("path", PATHS)
def test_large_full_size_sampled(path):
    use_path(path, torch.float32)
    say(f"[large f32 {path} full size]")
    inp = synth.to_f32(synth.make_workload("large"))
    got = run_gpu(inp, torch.float32)
    assert np.array_equal(got["Psi2"], got["Psi2"].T)
    assert got["psi0"] == pytest.approx(inp["mu"].shape[0] * inp["sigma_f2"], rel=1e-6)
    _sampled_checks(inp, got, np.random.default_rng(1), f"large/{path}")


@pytest.mark.parametrize("path", PATHS)
def test_large_row_subset_full(path):
    """Every output, dl and dsigma_f2 included, against the oracle on a row subset
    of the large workload (same M = 256, Q = 20)."""
    use_path(path, torch.float32)
    inp = synth.to_f32(synth.make_workload("large"))
    rows = np.arange(0, inp["mu"].shape[0], 97)  # 1031 rows
    sub = dict(inp, mu=inp["mu"][rows], S=inp["S"][rows], dL_dPsi1=inp["dL_dPsi1"][rows])
    got = run_gpu(sub, torch.float32)
    compare_all(got, run_oracle(sub), TOL32, f"large-subset/{path}")


@pytest.mark.parametrize("path", PATHS)
def test_stress_chunked(path):
    """N = 10^6, M = 512, Q = 30 in 8 row chunks, accumulating on the device."""
    use_path(path, torch.float32)
    say(f"[stress f32 {path} chunked]")
    w = synth.WORKLOADS["stress"]
    inp = synth.to_f32(synth.make_workload("stress"))
    N, M, Q, C = w.N, w.M, w.Q, w.chunk_rows
    d = dev({k: v for k, v in inp.items() if k != "dL_dPsi1"}, torch.float32)
    psi0 = torch.zeros(1, dtype=torch.float32, device=DEV)
    Psi2 = torch.zeros((M, M), dtype=torch.float32, device=DEV)
    gout = {"dmu": torch.empty((N, Q), device=DEV), "dS": torch.empty((N, Q), device=DEV),
            "dZ": torch.zeros((M, Q), device=DEV), "dsigma_f2": torch.zeros(1, device=DEV),
            "dl": torch.zeros(Q, device=DEV)}
    ws = torch.empty(gpps.workspace_bytes("f32", C, M, Q), dtype=torch.uint8, device=DEV)
    G1_sum = 0.0
    try:
        for c, r0 in enumerate(range(0, N, C)):
            r1 = min(N, r0 + C)
            G1 = synth.stress_dL_dPsi1_chunk(0, c, r1 - r0, M).astype(np.float32)
            G1d = torch.tensor(G1, device=DEV)
            _, P1, _ = gpps.psi_stats(d["mu"][r0:r1], d["S"][r0:r1], d["Z"], inp["sigma_f2"],
                                      inp["l"], accumulate=c > 0,
                                      out=(psi0, torch.empty((r1 - r0, M), device=DEV), Psi2),
                                      workspace=ws)
            G1_sum += float(torch.sum(G1d.double() * P1.double()))
            sub = {k: gout[k] for k in gout}
            sub["dmu"], sub["dS"] = gout["dmu"][r0:r1], gout["dS"][r0:r1]
            gpps.psi_grads(d["mu"][r0:r1], d["S"][r0:r1], d["Z"], inp["sigma_f2"], inp["l"],
                           inp["dL_dpsi0"], G1d, d["dL_dPsi2"], accumulate=c > 0, out=sub,
                           workspace=ws)
            say(f"  chunk {c} rows {r0}:{r1} enqueued")
    except gpps.GppsError as e:
        if e.status == 8:
            pytest.skip("path does not support this shape")
        raise
    torch.cuda.synchronize()
    got = {"psi0": psi0.cpu().double().numpy()[0], "Psi2": Psi2.cpu().double().numpy()}
    for k, v in gout.items():
        got[k] = v.cpu().double().numpy()
    got["dsigma_f2"] = got["dsigma_f2"][0]
    assert np.array_equal(got["Psi2"], got["Psi2"].T)
    assert got["psi0"] == pytest.approx(N * inp["sigma_f2"], rel=1e-5)

    def g1_rows(rows):
        out = np.empty((rows.shape[0], M))
        for i, r in enumerate(rows):
            c = r // C
            out[i] = synth.stress_dL_dPsi1_chunk(0, c, min(N, (c + 1) * C) - c * C, M)[r - c * C]
        return out.astype(np.float32).astype(np.float64)

    def g1_columns(cols):
        """dL/dPsi1[:, cols] over all N rows, chunk by chunk."""
        out = np.empty((N, len(cols)))
        for c, r0 in enumerate(range(0, N, C)):
            r1 = min(N, r0 + C)
            out[r0:r1] = synth.stress_dL_dPsi1_chunk(0, c, r1 - r0, M)[:, cols]
        return out.astype(np.float32).astype(np.float64)

    def dz_ref(zr):
        """dZ rows summed over all N: the Psi2 part (oracle.dZ_rows without dL/dPsi1)
        plus the Psi1 part of each z_m, which involves only column m of dL/dPsi1
        (oracle.psi_grads on that single inducing input)."""
        ref = oracle.dZ_rows(inp["mu"], inp["S"], inp["Z"], inp["sigma_f2"], inp["l"], None,
                             inp["dL_dPsi2"], zr)
        G1c = g1_columns(zr)
        for k, m in enumerate(zr):
            g = oracle.psi_grads(inp["mu"], inp["S"], inp["Z"][[m]], inp["sigma_f2"], inp["l"],
                                 0.0, np.ascontiguousarray(G1c[:, [k]]), None)
            ref[k] += g["dZ"][0]
        return ref

    _sampled_checks(inp, got, np.random.default_rng(2), f"stress/{path}", n_rows=16,
                    n_pairs=32, dz_rows=2, G1_rows=g1_rows, dz_ref=dz_ref)
    # sf2 homogeneity with <G1, Psi1> accumulated per chunk above
    G2s = 0.5 * (inp["dL_dPsi2"] + inp["dL_dPsi2"].T)
    a, b, c = G1_sum, 2 * np.sum(G2s * got["Psi2"]), inp["dL_dpsi0"] * N * inp["sigma_f2"]
    r = inp["sigma_f2"] * got["dsigma_f2"] - (a + b + c)
    assert abs(r) <= 1e-4 * (abs(a) + abs(b) + abs(c))


@pytest.mark.parametrize("path", PATHS)
def test_stress_row_subset_full(path):
    """Every output, dl and dsigma_f2 included, against the oracle on an evenly
    spaced row subset of the stress workload (same M = 512, Q = 30, l ~ U(0.5, 4)),
    its dL/dPsi1 rows taken from their chunks."""
    use_path(path, torch.float32)
    w = synth.WORKLOADS["stress"]
    inp = synth.to_f32(synth.make_workload("stress"))
    N, M, C = w.N, w.M, w.chunk_rows
    rows = np.arange(0, N, 997)          # 1004 rows, spread over all 8 chunks
    G1 = np.empty((rows.shape[0], M))
    for c in range(0, (N + C - 1) // C):
        sel = (rows >= c * C) & (rows < (c + 1) * C)
        if sel.any():
            G1[sel] = synth.stress_dL_dPsi1_chunk(0, c, min(N, (c + 1) * C) - c * C, M)[rows[sel] - c * C]
    sub = dict(inp, mu=inp["mu"][rows], S=inp["S"][rows],
               dL_dPsi1=G1.astype(np.float32).astype(np.float64))
    say(f"[stress subset {rows.shape[0]} rows {path}]")
    got = run_gpu(sub, torch.float32)
    compare_all(got, run_oracle(sub), TOL32, f"stress-subset/{path}")


# ------------------------------------------------------------------ determinism, chunking

@pytest.mark.parametrize("workload", ["medium", "large"])
@pytest.mark.parametrize("path", PATHS)
def test_bitwise_deterministic(path, workload):
    """Two calls give identical bits.  At large the matrix-core gradient runs
    every exchange round of its workgroups (eight blocks) over 196-row chunks."""
    use_path(path, torch.float32)
    inp = synth.to_f32(synth.make_workload(workload))
    a = run_gpu(inp, torch.float32)
    b = run_gpu(inp, torch.float32)
    for k in a:
        assert np.array_equal(a[k], b[k]), k


@pytest.mark.parametrize("path", PATHS)
def test_chunked_accumulate_matches_single_call(path):
    use_path(path, torch.float32)
    inp = synth.to_f32(synth.random_inputs(3001, 40, 7, seed=4))
    whole = run_gpu(inp, torch.float32)
    d = dev(inp, torch.float32)
    N, Q = inp["mu"].shape
    M = inp["Z"].shape[0]
    psi0 = torch.zeros(1, device=DEV)
    P1 = torch.empty((N, M), device=DEV)
    P2 = torch.empty((M, M), device=DEV)
    g = {"dmu": torch.empty((N, Q), device=DEV), "dS": torch.empty((N, Q), device=DEV),
         "dZ": torch.empty((M, Q), device=DEV), "dsigma_f2": torch.empty(1, device=DEV),
         "dl": torch.empty(Q, device=DEV)}
    for i, (r0, r1) in enumerate([(0, 1000), (1000, 1001), (1001, 3001)]):
        gpps.psi_stats(d["mu"][r0:r1], d["S"][r0:r1], d["Z"], inp["sigma_f2"], inp["l"],
                       accumulate=i > 0, out=(psi0, P1[r0:r1], P2))
        sub = dict(g, dmu=g["dmu"][r0:r1], dS=g["dS"][r0:r1])
        gpps.psi_grads(d["mu"][r0:r1], d["S"][r0:r1], d["Z"], inp["sigma_f2"], inp["l"],
                       inp["dL_dpsi0"], d["dL_dPsi1"][r0:r1],
                       d["dL_dPsi2"], accumulate=i > 0, out=sub)
    torch.cuda.synchronize()
    chunked = {"psi0": psi0.cpu().double().numpy()[0], "Psi1": P1.cpu().double().numpy(),
               "Psi2": P2.cpu().double().numpy()}
    for k, v in g.items():
        chunked[k] = v.cpu().double().numpy()
    chunked["dsigma_f2"] = chunked["dsigma_f2"][0]
    for k in whole:
        e = rel(chunked[k], whole[k])
        assert e <= 1e-5, (k, e)
    assert np.array_equal(chunked["Psi2"], chunked["Psi2"].T)


# ------------------------------------------------------------------ edge cases

EDGE = [
    ("N1", dict(N=1, M=5, Q=3)),
    ("M1", dict(N=300, M=1, Q=4)),
    ("Q1", dict(N=500, M=33, Q=1)),
    ("ragged", dict(N=777, M=65, Q=13)),
    ("Qmax", dict(N=150, M=17, Q=64)),
    ("Mbig", dict(N=3, M=1100, Q=2)),
]


@pytest.mark.parametrize("path", PATHS)
@pytest.mark.parametrize("case", EDGE, ids=[c[0] for c in EDGE])
def test_edge_shapes(case, path):
    name, kw = case
    use_path(path, torch.float32)
    say(f"[edge {name} {kw} {path}]")
    inp = synth.to_f32(synth.random_inputs(kw["N"], kw["M"], kw["Q"], seed=9))
    got = run_gpu(inp, torch.float32)
    compare_all(got, run_oracle(inp), TOL32, f"edge-{name}/{path}")


@pytest.mark.parametrize("path", PATHS)
def test_edge_shapes_f64(path):
    use_path(path, torch.float64)
    for N, M, Q in [(1, 1, 1), (37, 19, 5), (64, 16, 64)]:
        inp = synth.random_inputs(N, M, Q, seed=10)
        got = run_gpu(inp, torch.float64)
        compare_all(got, run_oracle(inp), TOL64, f"f64-{N}x{M}x{Q}")


@pytest.mark.parametrize("path", PATHS)
def test_null_upstream_gradients_and_nonsymmetric_G2(path):
    use_path(path, torch.float32)
    inp = synth.to_f32(synth.random_inputs(900, 24, 6, seed=12))
    rng = np.random.default_rng(13)
    inp["dL_dPsi2"] = rng.standard_normal((24, 24)).astype(np.float32).astype(np.float64)
    compare_all(run_gpu(inp, torch.float32), run_oracle(inp), TOL32, "nonsym")
    for drop in ("dL_dPsi1", "dL_dPsi2"):
        x = dict(inp, **{drop: None})
        compare_all(run_gpu(x, torch.float32, want_psi1=False), run_oracle(x), TOL32, drop)


@pytest.mark.parametrize("path", PATHS)
def test_zero_variance_limit(path):
    """S = 0: Psi1 is the plain kernel matrix K(mu, Z) and Psi2 = K^T K."""
    use_path(path, torch.float32)
    inp = synth.to_f32(synth.random_inputs(400, 20, 5, seed=14))
    inp["S"] = np.zeros_like(inp["S"])
    got = run_gpu(inp, torch.float32)
    r2 = (((inp["mu"][:, None, :] - inp["Z"][None]) / inp["l"]) ** 2).sum(-1)
    K = inp["sigma_f2"] * np.exp(-0.5 * r2)
    assert rel(got["Psi1"], K) <= 1e-5
    assert rel(got["Psi2"], K.T @ K) <= 1e-4


@pytest.mark.parametrize("path", PATHS)
def test_far_inducing_points_underflow_cleanly(path):
    """Inducing inputs far from every datapoint: the exponentials underflow to 0
    and nothing turns into NaN or Inf."""
    use_path(path, torch.float32)
    inp = synth.to_f32(synth.random_inputs(200, 12, 3, seed=15))
    inp["Z"][6:] += 60.0
    got = run_gpu(inp, torch.float32)
    for k, v in got.items():
        assert np.all(np.isfinite(v)), k
    compare_all(got, run_oracle(inp), TOL32, "far")


# Dimensions at both ends of every instruction count of the matrix-core Gram
# product: the three fp16 cross products of each dimension share one packed K
# range (Q <= 4, 8, 14, 20, 30, 40, 52, 62 take 1, 2, 3, 4, 6, 8, 10, 12
# instructions), so a slot misplaced in the layout shows up at one of these.
GRAM_Q = [4, 5, 8, 9, 14, 15, 20, 21, 30, 31, 32, 40, 41, 52, 53, 62]


@pytest.mark.parametrize("Q", GRAM_Q)
def test_mfma_gram_layout_dimensions(Q):
    use_path("mfma", torch.float32)
    say(f"[gram layout Q={Q}]")
    inp = synth.to_f32(synth.random_inputs(300, 70, Q, seed=100 + Q))
    got = run_gpu(inp, torch.float32)
    compare_all(got, run_oracle(inp), TOL32, f"gram-Q{Q}")


# Block counts of the symmetric gradient kernel (one workgroup of nb waves covers
# every block pair; odd nb has (nb - 1) / 2 exchange rounds and no shared tile,
# even nb one shared tile): nb = 5, 7 (two and three rounds), 7 at Q = 30
# (its tables fill 159.9 of the 160 KB of LDS), 8 with a partial last block, 6;
# N leaves partial batches of rows at the ends of the row chunks.  Batches are
# eight rows at nb >= 5 where the tables fit (150 x 9, 150 x 30, 200 x 20,
# 180 x 14, and nb = 8 at Q = 10 and Q = 4), four otherwise.
@pytest.mark.parametrize("N,M,Q", [(301, 150, 9), (333, 150, 30), (299, 200, 20),
                                   (257, 200, 30), (311, 250, 20), (205, 180, 14),
                                   (263, 256, 10), (250, 240, 4)])
def test_mfma_symmetric_block_counts(N, M, Q):
    use_path("mfma", torch.float32)
    say(f"[symmetric gradient N={N} M={M} Q={Q}]")
    inp = synth.to_f32(synth.random_inputs(N, M, Q, seed=300 + M + Q))
    got = run_gpu(inp, torch.float32)
    compare_all(got, run_oracle(inp), TOL32, f"sym-{M}x{Q}")


# Block counts of the symmetric forward past eight blocks: from nb = 10 each wave's
# tiles are split into two ranges of k with workgroups of their own, and each
# workgroup stages a window of eight blocks taken mod nb.  nb = 9 (one range, a
# window smaller than nb), 10 and 12 (column groups that straddle nb / 2, where
# the waves' tile counts differ), 11 and 13 (odd), 15 and 16 (the largest
# windows), at Q from 3 to 30 (one to six Gram instructions).
@pytest.mark.parametrize("N,M,Q", [(150, 270, 20), (160, 310, 12), (140, 350, 30),
                                   (130, 384, 6), (150, 410, 20), (120, 449, 25),
                                   (129, 512, 30), (100, 500, 3)])
def test_mfma_symmetric_forward_ranges(N, M, Q):
    use_path("mfma", torch.float32)
    say(f"[symmetric forward ranges N={N} M={M} Q={Q}]")
    inp = synth.to_f32(synth.random_inputs(N, M, Q, seed=400 + M + Q))
    got = run_gpu(inp, torch.float32)
    compare_all(got, run_oracle(inp), TOL32, f"fsym-{M}x{Q}")


# The gradient for 13 <= nb <= 16 (where the halves' tables fit): the symmetric
# kernel on blocks 0 .. 7 and on 8 .. nb - 1, the tile kernel on the tiles
# between them; nb = 13 (a half of five blocks), 14, 15 (odd half) and 16, with
# eight-row batches (Q <= 14) and four (Q = 20), ragged M and partial batches.
@pytest.mark.parametrize("N,M,Q", [(150, 410, 20), (170, 448, 20), (201, 480, 14),
                                   (140, 512, 10), (100, 500, 3)])
def test_mfma_split_gradient(N, M, Q):
    use_path("mfma", torch.float32)
    say(f"[split gradient N={N} M={M} Q={Q}]")
    inp = synth.to_f32(synth.random_inputs(N, M, Q, seed=500 + M + Q))
    got = run_gpu(inp, torch.float32)
    compare_all(got, run_oracle(inp), TOL32, f"split-{M}x{Q}")


# Ragged ranges of row blocks on the matrix-core path: M = 257 (9 blocks of 32,
# three ranges of four, the last with one real block) at Q = 20, and M = 300 at
# Q = 31 (eight Gram instructions, the widest single [Z | 1] column block).
@pytest.mark.parametrize("N,M,Q", [(400, 257, 20), (300, 300, 31)])
def test_mfma_ragged_block_ranges(N, M, Q):
    use_path("mfma", torch.float32)
    say(f"[ragged ranges N={N} M={M} Q={Q}]")
    inp = synth.to_f32(synth.random_inputs(N, M, Q, seed=200 + M))
    got = run_gpu(inp, torch.float32)
    compare_all(got, run_oracle(inp), TOL32, f"ragged-{M}x{Q}")


# ------------------------------------------------------------------ fp16 range of the matrix cores
# The matrix-core path carries its Gram operands and the column bias as two-part
# fp16 values, scaled per dimension and with the n-independent pair factor taken
# out of the sum over datapoints.  A device guard routes a call to the generic
# kernels when an operand bound leaves the fp16 range, or when the inducing
# inputs spread over more than 64 lengthscales (the gradient's accuracy limit).
# Each case is compared with the oracle element by element, with the route the
# guard must take (0 matrix cores, 1 generic).
def _scaled(c):
    """Psi1 and Psi2 are invariant under mu, Z, l -> c mu, c Z, c l, S -> c^2 S."""
    inp = synth.random_inputs(2000, 70, 8, seed=36)
    return dict(inp, mu=c * inp["mu"], Z=c * inp["Z"], l=c * inp["l"], S=c * c * inp["S"]), 0


def _range_case(name):
    if name.startswith("scaled"):
        inp, route = _scaled({"scaled-1e-3": 1e-3, "scaled-1e3": 1e3}[name])
        return synth.to_f32(inp), route
    rng = np.random.default_rng({"l002-zspread": 31, "q1-l0008": 32, "tiny-l-trip": 33,
                                 "far-mu-trip": 34, "wide-s": 35, "spread-at-limit": 37}[name])
    if name == "l002-zspread":       # Q = 10, l = 0.02, mu ~ N(0, 0.3^2), Z ~ N(0, 2.5^2)
        N, M, Q = 400, 40, 10
        mu = 0.3 * rng.standard_normal((N, Q))
        S = rng.uniform(0.01, 0.5, (N, Q))
        Z = 2.5 * rng.standard_normal((M, Q))
        l = np.full(Q, 0.02)
        route = 1                    # R / l ~ 330
    elif name == "q1-l0008":         # a 1-D latent over [-3.5, 3.5], l = 0.008
        N, M, Q = 2000, 100, 1
        mu = rng.uniform(-3.5, 3.5, (N, Q))
        S = rng.uniform(0.01, 0.5, (N, Q))
        Z = np.linspace(-3.5, 3.5, M)[:, None]
        l = np.array([0.008])
        route = 1                    # R / l ~ 440
    elif name == "spread-at-limit":  # the first case with l raised to R / 60
        N, M, Q = 400, 40, 10
        mu = 0.3 * rng.standard_normal((N, Q))
        S = rng.uniform(0.01, 0.5, (N, Q))
        Z = 2.5 * rng.standard_normal((M, Q))
        l = np.abs(Z - Z.mean(0)).max(0) / 60.0
        route = 0
    elif name == "wide-s":           # S >> l^2 in every dimension, Z spread past mu
        N, M, Q = 600, 64, 6
        mu = rng.standard_normal((N, Q))
        S = rng.uniform(1.0, 4.0, (N, Q))
        Z = 3.0 * rng.standard_normal((M, Q))
        l = rng.uniform(0.3, 0.6, Q)
        route = 0
    elif name == "tiny-l-trip":      # l ~ 1e-3, S ~ 1e-7: R / l ~ 2000
        N, M, Q = 300, 20, 2
        mu = rng.standard_normal((N, Q))
        S = rng.uniform(1e-8, 1e-7, (N, Q))
        Z = mu[:M] + 1e-4 * rng.standard_normal((M, Q))
        l = np.array([1e-3, 2e-3])
        route = 1
    else:                            # "far-mu-trip": half the data 300 lengthscales away:
        N, M, Q = 300, 24, 3         # the column bias and Gram operands leave the fp16 range
        mu = rng.standard_normal((N, Q))
        mu[: N // 2] += 300.0
        S = rng.uniform(0.01, 0.5, (N, Q))
        Z = rng.standard_normal((M, Q))
        l = rng.uniform(0.8, 1.2, Q)
        route = 1
    dL_dpsi0 = float(rng.standard_normal())
    G1 = rng.standard_normal((N, M))
    A = rng.standard_normal((M, M))
    inp = {"mu": mu, "S": S, "Z": Z, "sigma_f2": 1.0, "l": l, "dL_dpsi0": dL_dpsi0,
           "dL_dPsi1": G1, "dL_dPsi2": 0.5 * (A + A.T)}
    return synth.to_f32(inp), route


RANGE = ["l002-zspread", "q1-l0008", "spread-at-limit", "wide-s", "scaled-1e-3", "scaled-1e3",
         "tiny-l-trip", "far-mu-trip"]


@pytest.mark.parametrize("path", ["auto", "mfma"])
@pytest.mark.parametrize("name", RANGE)
def test_matrix_core_operand_range(name, path):
    gpps.set_path(path)
    inp, route = _range_case(name)
    say(f"[range {name} {path}: expect route {route}]")
    got = run_gpu(inp, torch.float32, expect_route=route)
    record(current_test(), f"range-{name}/{path}", "route", route, None)
    for k, v in got.items():
        assert np.all(np.isfinite(v)), k
    compare_all(got, run_oracle(inp), TOL32, f"range-{name}/{path}")
