"""GPU parity of the Bayesian GP-LVM bound (gpps_bound, through the C ABI) against
the fp64 oracle in oracle/bound.py, and the optimiser loop built on it.

fp64 calls run the generic psi-statistic path and the fp64 M x M algebra.  The
library and the oracle factorise Kmm and A by different (blocked vs. LAPACK)
Cholesky codes, so on an ill-conditioned problem an output can differ by as much
as two backward-stable fp64 evaluations of the same definition do.  The test
measures that spread on the oracle itself (Cholesky-based inverses against
LU-based and eigendecomposition-based ones; one pair alone under-samples it: the
LU spread of dsigma_f2 at the paper's shape measured 1.3e-10 on one host and
4.4e-10 on another, the eigendecomposition's 1.1e-9) and allows, per output,
max(1e-9, 10 x the largest spread).  At the
paper's shape (Q = 1, M = 100) cond(A) reaches ~1e7 and dZ is the difference of
two nearly equal contributions (through the psi-statistics and through Kmm), so
its spread is ~1e-6; every other case and output is held to 1e-9.  The parity
cases also keep cond(Kmm) <= 1e4 (checked) by spreading the inducing inputs or,
at the paper's shape, with jitter 1e-2.  fp32 calls run the
matrix-core psi-statistics: their errors (~1e-6 relative in Psi2) are amplified
in the bound by the conditioning of Kmm and A = Kmm + beta Psi2, so the fp32
cases use well-conditioned problems (spread inducing inputs, jitter 1e-4) and a
tolerance of 1e-4 on L and every gradient.
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_1410_4984_amd as gpps  # noqa: E402
from oracle import bound as ob  # noqa: E402
import oracle  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
KEYS = ("dmu", "dS", "dZ", "dsigma_f2", "dl", "dbeta")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def rel(a, ref):
    a, ref = np.asarray(a, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref.ravel())
    return np.linalg.norm((a - ref).ravel()) / (den if den > 0 else 1.0)


def problem(N, M, Q, D, seed, jitter=1e-6, spread=1.0):
    rng = np.random.default_rng(seed)
    mu = rng.normal(size=(N, Q))
    S = rng.uniform(0.05, 0.5, size=(N, Q))
    Z = rng.normal(scale=spread, size=(M, Q))
    Y = rng.normal(size=(N, D))
    l = rng.uniform(0.7, 1.8, size=Q)
    return dict(mu=mu, S=S, Z=Z, Y=Y, sigma_f2=1.3, l=l, beta=2.5, jitter=jitter)


def run_gpu(p, dtype):
    t = {k: torch.tensor(p[k], dtype=dtype, device=DEV) for k in ("mu", "S", "Z", "Y")}
    out = gpps.bound(t["mu"], t["S"], t["Z"], t["Y"], p["sigma_f2"], p["l"], p["beta"], p["jitter"])
    torch.cuda.synchronize()
    return {k: v.double().cpu().numpy() for k, v in out.items()}


def run_oracle(p, f32, inverse=None):
    q = dict(p)
    if f32:
        q = {k: (np.asarray(v, np.float32).astype(np.float64) if isinstance(v, np.ndarray) else v)
             for k, v in p.items()}
    oracle.build(force=False)
    args = (q["mu"], q["S"], q["Z"], q["Y"], q["sigma_f2"], q["l"], q["beta"], q["jitter"])
    return ob.grads(*args) if inverse is None else ob.grads(*args, inverse=inverse)


def spread_tol(p, ref):
    """max(1e-9, 10 x the largest relative spread between the Cholesky-based oracle
    run and the LU- and eigendecomposition-based ones)."""
    tol = {k: 0.0 for k in ("L",) + KEYS}
    for inv in (ob._inv_lu, ob._inv_eigh):
        alt = run_oracle(p, False, inverse=inv)
        tol["L"] = max(tol["L"], abs(alt["L"] - ref["L"]) / abs(ref["L"]))
        for k in KEYS:
            tol[k] = max(tol[k], rel(np.asarray(alt[k]), np.asarray(ref[k])))
    return {k: max(1e-9, 10.0 * v) for k, v in tol.items()}


@pytest.fixture(autouse=True)
def _auto_path():
    gpps.set_path("auto")
    yield
    gpps.set_path("auto")


def kmm_cond(p):
    M = p["Z"].shape[0]
    return np.linalg.cond(ob.kmm(p["Z"], p["sigma_f2"], p["l"]) + p["jitter"] * np.eye(M))


@pytest.mark.parametrize("shape,spread,jitter", [((300, 20, 3, 4), 1.0, 1e-6),
                                                 ((777, 45, 2, 1), 3.0, 1e-6),
                                                 ((64, 33, 5, 7), 1.0, 1e-6),
                                                 ((1000, 100, 1, 3), 2.0, 1e-2),
                                                 ((1500, 150, 3, 3), 3.0, 1e-6)])
def test_bound_f64_matches_oracle(shape, spread, jitter):
    N, M, Q, D = shape
    p = problem(N, M, Q, D, seed=N + M, spread=spread, jitter=jitter)
    cond = kmm_cond(p)
    assert cond <= 1e4
    got, ref = run_gpu(p, torch.float64), run_oracle(p, False)
    tol = spread_tol(p, ref)
    e = abs(got["L"][0] - ref["L"]) / abs(ref["L"])
    say(f"  f64 {shape} L: rel {e:.2e} (tol {tol['L']:.1e}, cond(Kmm) {cond:.1e})")
    assert e <= tol["L"]
    for k in KEYS:
        e = rel(got[k].reshape(np.shape(ref[k])), ref[k])
        say(f"  f64 {shape} {k}: rel {e:.2e} (tol {tol[k]:.1e})")
        assert e <= tol[k], k


@pytest.mark.parametrize("shape", [(2000, 32, 4, 3), (5000, 64, 10, 5)])
def test_bound_f32_matches_oracle(shape):
    N, M, Q, D = shape
    p = problem(N, M, Q, D, seed=N, jitter=1e-4, spread=1.5)
    assert kmm_cond(p) <= 1e4
    got, ref = run_gpu(p, torch.float32), run_oracle(p, True)
    e = abs(got["L"][0] - ref["L"]) / abs(ref["L"])
    say(f"  f32 {shape} L: rel {e:.2e} (path {gpps.get_path()})")
    assert e <= 1e-4
    for k in KEYS:
        e = rel(got[k].reshape(np.shape(ref[k])), ref[k])
        say(f"  f32 {shape} {k}: rel {e:.2e}")
        assert e <= 1e-4, k


def test_bound_is_deterministic():
    p = problem(500, 40, 3, 2, seed=3)
    a, b = run_gpu(p, torch.float64), run_gpu(p, torch.float64)
    for k in ("L",) + KEYS:
        assert np.array_equal(a[k], b[k]), k


def test_bound_not_positive_definite_gives_nan():
    # two coincident inducing inputs and no jitter: Kmm is singular
    p = problem(100, 6, 2, 2, seed=4, jitter=0.0)
    p["Z"][1] = p["Z"][0]
    got = run_gpu(p, torch.float64)
    assert np.isnan(got["L"][0]) and np.isnan(got["dbeta"][0])
