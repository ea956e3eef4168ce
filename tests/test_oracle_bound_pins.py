"""Pins of the fp64 Bayesian GP-LVM bound oracle (CPU only).

Each check ties oracle/bound.py to something other than itself:
  * central finite differences of L for every parameter (mu, S, Z, sigma_f2, l,
    beta): the closed-form gradients (dL/dPsi assembly, the chain rule through
    Kmm and the psi-statistics, the KL term) must match;
  * S = 0, Z = X, no jitter: the collapsed bound is then exact, equal to the GP
    log marginal likelihood log N(Y | 0, Knn + I / beta) (written out here
    with numpy's slogdet and solve);
  * the KL term of q(x) = N(mu, S) against N(0, 1) by 1-D quadrature;
  * rotating the output columns (Y -> Y R, R orthogonal) leaves L unchanged;
  * the bound of D columns is the sum of the D single-column bounds (the
    factor D on the log-determinant and trace terms).
"""
from __future__ import annotations

import numpy as np
import pytest

import oracle
from oracle import bound as ob


def _problem(N=12, M=5, Q=2, D=3, seed=3):
    rng = np.random.default_rng(seed)
    mu = rng.normal(size=(N, Q))
    S = rng.uniform(0.05, 0.5, size=(N, Q))
    Z = rng.normal(size=(M, Q))
    Y = rng.normal(size=(N, D))
    l = rng.uniform(0.7, 1.8, size=Q)
    return dict(mu=mu, S=S, Z=Z, Y=Y, sigma_f2=1.3, l=l, beta=2.5, jitter=1e-6)


def _L(p):
    return ob.bound(p["mu"], p["S"], p["Z"], p["Y"], p["sigma_f2"], p["l"], p["beta"],
                    p["jitter"])


@pytest.fixture(scope="module", autouse=True)
def _built():
    oracle.build(force=False)


def test_gradients_match_finite_differences():
    p = _problem()
    g = ob.grads(p["mu"], p["S"], p["Z"], p["Y"], p["sigma_f2"], p["l"], p["beta"], p["jitter"])
    assert abs(g["L"] - _L(p)) <= 1e-12 * abs(g["L"])

    def fd(key, idx=None):
        q = {k: (np.array(v, dtype=np.float64, copy=True) if isinstance(v, np.ndarray) else v)
             for k, v in p.items()}
        x0 = q[key][idx] if idx is not None else q[key]
        h = 1e-6 * max(1.0, abs(x0))
        vals = []
        for s in (+1, -1):
            if idx is not None:
                q[key][idx] = x0 + s * h
            else:
                q[key] = x0 + s * h
            vals.append(_L(q))
        return (vals[0] - vals[1]) / (2 * h)

    for key, gk in (("mu", "dmu"), ("S", "dS"), ("Z", "dZ"), ("l", "dl")):
        num = np.array([fd(key, idx) for idx in np.ndindex(p[key].shape)]).reshape(p[key].shape)
        ana = np.asarray(g[gk])
        err = np.linalg.norm(num - ana) / np.linalg.norm(ana)
        assert err <= 1e-7, (key, err)
    for key, gk in (("sigma_f2", "dsigma_f2"), ("beta", "dbeta")):
        num = fd(key)
        assert abs(num - g[gk]) <= 1e-7 * max(1.0, abs(g[gk])), (key, num, g[gk])


def test_exact_gp_marginal_likelihood_when_inducing_inputs_are_the_data():
    rng = np.random.default_rng(7)
    N, Q, D = 7, 2, 3
    mu = rng.uniform(-3, 3, size=(N, Q))
    Y = rng.normal(size=(N, D))
    l = np.array([1.1, 0.8])
    sf2, beta = 1.7, 3.0
    S = np.zeros((N, Q))
    F, _, _ = ob.bound_terms(mu, S, mu, Y, sf2, l, beta, 0.0)
    K = ob.kmm(mu, sf2, l)
    Cov = K + np.eye(N) / beta
    sign, logdet = np.linalg.slogdet(Cov)
    assert sign > 0
    lml = (-0.5 * float(np.sum(Y * np.linalg.solve(Cov, Y))) - 0.5 * D * logdet
           - 0.5 * N * D * np.log(2 * np.pi))
    assert abs(F - lml) <= 1e-9 * abs(lml), (F, lml)


def test_kl_matches_quadrature():
    from scipy import integrate
    for m, s in ((0.0, 1.0), (0.7, 0.2), (-1.3, 2.5), (0.1, 0.01)):
        def integrand(x):
            lq = -0.5 * np.log(2 * np.pi * s) - 0.5 * (x - m) ** 2 / s
            lp = -0.5 * np.log(2 * np.pi) - 0.5 * x * x
            return np.exp(lq) * (lq - lp)
        w = 12 * np.sqrt(s)
        val, _ = integrate.quad(integrand, m - w, m + w, epsabs=0, epsrel=1e-12, limit=200)
        assert abs(ob.kl(np.array([[m]]), np.array([[s]])) - val) <= 1e-10 * max(1.0, abs(val))


def test_output_rotation_invariance():
    p = _problem(seed=5)
    rng = np.random.default_rng(11)
    R, _ = np.linalg.qr(rng.normal(size=(3, 3)))
    q = dict(p, Y=p["Y"] @ R)
    g1 = ob.grads(p["mu"], p["S"], p["Z"], p["Y"], p["sigma_f2"], p["l"], p["beta"], p["jitter"])
    g2 = ob.grads(q["mu"], q["S"], q["Z"], q["Y"], q["sigma_f2"], q["l"], q["beta"], q["jitter"])
    assert abs(g1["L"] - g2["L"]) <= 1e-12 * abs(g1["L"])
    for k in ("dmu", "dS", "dZ", "dl"):
        assert np.allclose(g1[k], g2[k], rtol=1e-10, atol=1e-12), k
    assert abs(g1["dbeta"] - g2["dbeta"]) <= 1e-10 * abs(g1["dbeta"])


def test_bound_is_the_sum_of_single_column_bounds():
    p = _problem(seed=9)
    F, K, _ = ob.bound_terms(p["mu"], p["S"], p["Z"], p["Y"], p["sigma_f2"], p["l"], p["beta"],
                             p["jitter"])
    parts = [ob.bound_terms(p["mu"], p["S"], p["Z"], p["Y"][:, [d]], p["sigma_f2"], p["l"],
                            p["beta"], p["jitter"])[0] for d in range(p["Y"].shape[1])]
    assert abs(F - sum(parts)) <= 1e-11 * abs(F)
    assert K == ob.kl(p["mu"], p["S"])


# ---------------------------------------------------------------- known inputs (S = None)
# The sparse GP regression bound of eq. (boundF) itself, written out densely the
# way the variational sparse GP literature states it:
#     F = log N(Y | 0, Qff + I / beta) - (beta D / 2) tr(Kff - Qff),
#     Qff = Kfu Kuu^-1 Kuf,  Kuu = k(Z, Z) + jitter I,
# with an N x N covariance (numpy slogdet and solve), i.e. without the matrix
# inversion lemma and the M x M algebra the oracle uses.

def _regression_problem(seed=13, N=12, M=5, Q=2, D=3):
    rng = np.random.default_rng(seed)
    return dict(X=rng.uniform(-2.5, 2.5, size=(N, Q)), Z=rng.normal(size=(M, Q)),
                Y=rng.normal(size=(N, D)), sigma_f2=1.4, l=rng.uniform(0.6, 1.7, size=Q),
                beta=4.0, jitter=1e-6)


def _dense_titsias(X, Z, Y, sf2, l, beta, jitter):
    def k(A, B):
        d = (A[:, None, :] - B[None, :, :]) / l
        return sf2 * np.exp(-0.5 * np.sum(d * d, axis=-1))
    N, D = Y.shape
    Kfu = k(X, Z)
    Kuu = k(Z, Z) + jitter * np.eye(Z.shape[0])
    Qff = Kfu @ np.linalg.solve(Kuu, Kfu.T)
    Cov = Qff + np.eye(N) / beta
    sign, logdet = np.linalg.slogdet(Cov)
    assert sign > 0
    lml = (-0.5 * float(np.sum(Y * np.linalg.solve(Cov, Y))) - 0.5 * D * logdet
           - 0.5 * N * D * np.log(2 * np.pi))
    return lml - 0.5 * beta * D * float(np.trace(k(X, X)) - np.trace(Qff))


@pytest.mark.parametrize("jitter", [1e-6, 1e-2])
def test_regression_bound_matches_dense_form(jitter):
    p = _regression_problem()
    F, kl_term, _ = ob.bound_terms(p["X"], None, p["Z"], p["Y"], p["sigma_f2"], p["l"], p["beta"],
                                   jitter)
    ref = _dense_titsias(p["X"], p["Z"], p["Y"], p["sigma_f2"], p["l"], p["beta"], jitter)
    assert kl_term == 0.0
    assert abs(F - ref) <= 1e-10 * abs(ref), (F, ref)
    g = ob.grads(p["X"], None, p["Z"], p["Y"], p["sigma_f2"], p["l"], p["beta"], jitter)
    assert g["dS"] is None and g["L"] == F


def test_regression_gradients_match_finite_differences():
    p = _regression_problem(seed=17)
    g = ob.grads(p["X"], None, p["Z"], p["Y"], p["sigma_f2"], p["l"], p["beta"], p["jitter"])

    def L(q):
        return _dense_titsias(q["X"], q["Z"], q["Y"], q["sigma_f2"], q["l"], q["beta"], q["jitter"])

    def fd(key, idx=None):
        q = {k: (np.array(v, dtype=np.float64, copy=True) if isinstance(v, np.ndarray) else v)
             for k, v in p.items()}
        x0 = q[key][idx] if idx is not None else q[key]
        h = 1e-6 * max(1.0, abs(x0))
        vals = []
        for s in (+1, -1):
            if idx is not None:
                q[key][idx] = x0 + s * h
            else:
                q[key] = x0 + s * h
            vals.append(L(q))
        return (vals[0] - vals[1]) / (2 * h)

    # differences of the dense form, so the gradient pin does not lean on the
    # oracle's own bound either
    for key, gk in (("X", "dmu"), ("Z", "dZ"), ("l", "dl")):
        num = np.array([fd(key, idx) for idx in np.ndindex(p[key].shape)]).reshape(p[key].shape)
        ana = np.asarray(g[gk])
        err = np.linalg.norm(num - ana) / np.linalg.norm(ana)
        assert err <= 1e-6, (key, err)
    for key, gk in (("sigma_f2", "dsigma_f2"), ("beta", "dbeta")):
        num = fd(key)
        assert abs(num - g[gk]) <= 1e-6 * max(1.0, abs(g[gk])), (key, num, g[gk])
