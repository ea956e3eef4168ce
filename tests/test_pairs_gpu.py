"""GPU parity of the generic path's pair kernels against the fp64 oracle.

The gradient's pairs kernel has three forms.  The symmetric ones (each
unordered pair (m, m') evaluated once by thread m for m' = m + k mod M,
k <= M/2, and exchanged through LDS bands) run whenever one workgroup holds all
of M (M <= 256): with several rows per workgroup where its LDS fits (every
case here up to M = 256 except fp64 at Q = 4 for M = 100, 255, 256), else one
row at a time (those three).  The ordered form runs beyond.  The symmetric schedule
depends on the parity of M and on the band edges, so M runs over 1, 2, 3, small
odd and even values, the paper's 100, the largest symmetric sizes 255 and 256,
and the ordered 257 and 300.  The forward Psi2 kernel puts one thread on each unique pair, in the
row-major order of the upper triangle, for the same sizes.  Every output is
compared element by element (relative Frobenius norm, 1e-10 fp64, fp32 as in
the main parity tests).
"""
import sys

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import oracle  # noqa: E402
import paper_1410_4984_amd as gpps  # noqa: E402
from paper_1410_4984_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu

DEV = "cuda:0"
TOL32 = {"psi0": 1e-6, "Psi1": 1e-5, "Psi2": 1e-4, "dmu": 1e-4, "dS": 1e-4, "dZ": 1e-4,
         "dsigma_f2": 1e-4, "dl": 1e-4}
TOL64 = {k: 1e-10 for k in TOL32}


def rel(a, ref):
    a, ref = np.asarray(a, dtype=np.float64), np.asarray(ref, dtype=np.float64)
    den = np.linalg.norm(ref.ravel())
    return np.linalg.norm((a - ref).ravel()) / (den if den > 0 else 1.0)


@pytest.fixture(scope="module", autouse=True)
def _setup():
    oracle.build(force=False)
    gpps.lib()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    gpps.set_path("generic")
    yield
    gpps.set_path("auto")


def check(N, M, Q, dtype, seed):
    print(f"[pairs N={N} M={M} Q={Q} {dtype}]", flush=True)
    inp = synth.random_inputs(N, M, Q, seed=seed)
    tol = TOL64
    if dtype == torch.float32:
        inp, tol = synth.to_f32(inp), TOL32
    t = lambda a: torch.tensor(a, dtype=dtype, device=DEV)  # noqa: E731
    mu, S, Z = t(inp["mu"]), t(inp["S"]), t(inp["Z"])
    psi0, P1, P2 = gpps.psi_stats(mu, S, Z, inp["sigma_f2"], inp["l"])
    g = gpps.psi_grads(mu, S, Z, inp["sigma_f2"], inp["l"], inp["dL_dpsi0"],
                       t(inp["dL_dPsi1"]), t(inp["dL_dPsi2"]))
    torch.cuda.synchronize()
    got = {"psi0": psi0.cpu().double().numpy()[0], "Psi1": P1.cpu().double().numpy(),
           "Psi2": P2.cpu().double().numpy(), **{k: v.cpu().double().numpy() for k, v in g.items()}}
    got["dsigma_f2"] = got["dsigma_f2"][0]
    r0, R1, R2 = oracle.psi_stats(inp["mu"], inp["S"], inp["Z"], inp["sigma_f2"], inp["l"])
    ref = dict(psi0=r0, Psi1=R1, Psi2=R2,
               **oracle.psi_grads(inp["mu"], inp["S"], inp["Z"], inp["sigma_f2"], inp["l"],
                                  inp["dL_dpsi0"], inp["dL_dPsi1"], inp["dL_dPsi2"]))
    bad = {}
    for k, v in ref.items():
        e = rel(got[k], v)
        print(f"  {k}: rel {e:.3e}", flush=True)
        if not e <= tol[k]:
            bad[k] = e
    assert not bad, (N, M, Q, bad)
    assert np.array_equal(got["Psi2"], got["Psi2"].T)
    sys.stdout.flush()


@pytest.mark.parametrize("M", [1, 2, 3, 8, 9, 100, 255, 256, 257, 300])
@pytest.mark.parametrize("Q", [1, 2, 4])
def test_pairs_f64(M, Q):
    check(N=53, M=M, Q=Q, dtype=torch.float64, seed=11 + M + Q)


@pytest.mark.parametrize("M", [3, 100, 256, 257])
def test_pairs_f32(M):
    check(N=41, M=M, Q=7, dtype=torch.float32, seed=5 + M)
