"""Bayesian GP-LVM fitting with the bound evaluated on the GPU.

Section 2 (end): the parameters are the variational means and variances
(mu, S) of q(X), the inducing inputs Z, the kernel parameters (sigma_f2, l) and
the noise precision beta; the gradients of every parameter are collected on one
node and passed to an existing optimiser (L-BFGS-B in SciPy).  Here the bound
and all its gradients come from ``gpps_bound`` (one call per evaluation, all on
the device); only the optimiser's vector arithmetic runs on the host.

Positive parameters are optimised through their logarithms (S, sigma_f2, l,
beta); the chain rule d/dlog x = x d/dx is applied to the gradients the library
returns.  A step whose parameters overflow is reported as infeasible (the line
search backs off); the regression fit also bounds its log parameters (L-BFGS-B's
box constraints), which its first line-search step needs.

    fit(Y, Q, M, iters=...) -> FitResult
    fit_staged(Y, Q, M) -> (FitResult, FitResult, rows)   large N with many inducing inputs
    fit_regression(X, Y, M, iters=...) -> RegressionResult
    paper_data(N, D=3, seed=0) -> (Y, x_true)   the synthetic data of section 4

fit_regression is the sparse GP regression model of eq. (boundF) itself: the
inputs X are observed (``gpps_bound`` with S = NULL, no q(X) and no KL term) and
the optimiser adjusts the inducing inputs Z and the kernel and noise
parameters only.
"""
from __future__ import annotations

import dataclasses
import time

import numpy as np

from . import bound


def paper_data(N: int, D: int = 3, seed: int = 0, noise: float = 0.05, lengthscale: float = 1.0):
    """Synthetic data in the manner of section 4: a one-dimensional latent
    variable mapped to D dimensions by functions drawn from an RBF-kernel GP,
    plus Gaussian noise.

    x_n ~ U(-3, 3).  Each output function is drawn exactly at 512 grid points of
    [-3.5, 3.5] (Cholesky of the kernel matrix plus 1e-10 jitter) and linearly
    interpolated at the x_n, which keeps the draw O(N) for large N.  Returns
    (Y [N x D], x [N])."""
    rng = np.random.default_rng(seed)
    x = rng.uniform(-3.0, 3.0, size=N)
    g = np.linspace(-3.5, 3.5, 512)
    K = np.exp(-0.5 * (g[:, None] - g[None, :]) ** 2 / lengthscale ** 2)
    L = np.linalg.cholesky(K + 1e-10 * np.eye(g.size))
    F = L @ rng.normal(size=(g.size, D))
    Y = np.stack([np.interp(x, g, F[:, d]) for d in range(D)], axis=1)
    Y = Y + noise * rng.normal(size=Y.shape)
    return Y, x


@dataclasses.dataclass
class FitResult:
    mu: np.ndarray
    S: np.ndarray
    Z: np.ndarray
    sigma_f2: float
    l: np.ndarray
    beta: float
    bound_trace: list        # L after every evaluation
    evals: int
    iterations: int
    seconds: float           # wall time of the optimisation
    gpu_seconds: float       # wall time inside the bound evaluations (device synchronised)
    message: str


def _pack(mu, S, Z, sf2, l, beta):
    return np.concatenate([mu.ravel(), np.log(S).ravel(), Z.ravel(), [np.log(sf2)], np.log(l),
                           [np.log(beta)]])


def _unpack(x, N, M, Q):
    o = 0
    mu = x[o:o + N * Q].reshape(N, Q); o += N * Q
    S = np.exp(x[o:o + N * Q]).reshape(N, Q); o += N * Q
    Z = x[o:o + M * Q].reshape(M, Q); o += M * Q
    sf2 = float(np.exp(x[o])); o += 1
    l = np.exp(x[o:o + Q]); o += Q
    beta = float(np.exp(x[o]))
    return mu, S, Z, sf2, l, beta


def init_params(Y: np.ndarray, Q: int, M: int, seed: int = 0, spread: bool = False):
    """PCA means (scaled to unit variance), sigma_f2 = var(Y), beta = 100 / var(Y), and

    spread=False: S = 0.5, Z a random subset of the means, unit lengthscales;
    spread=True (Q = 1): Z evenly spaced over the range of the means, S = 0.05 and
      a lengthscale of 0.1 (below the spacing of the data's features, about the
      size of a few inducing-input spacings at M = 100).  With many inducing
      inputs among the means and a unit lengthscale the start has
      cond(Kmm + beta Psi2) ~ 1e14 (the bound is then undetermined to ~1e-2 in
      fp64); the spread start is well conditioned."""
    rng = np.random.default_rng(seed)
    Yc = Y - Y.mean(0)
    _, _, Vt = np.linalg.svd(Yc, full_matrices=False)
    mu = Yc @ Vt[:Q].T
    mu = mu / mu.std(0)
    var = float(Yc.var())
    if spread:
        if Q != 1:
            raise ValueError("the spread start is defined for a one-dimensional latent space")
        Z = np.linspace(mu.min(), mu.max(), M)[:, None]
        return mu, np.full_like(mu, 0.05), Z, var, np.array([0.1]), 100.0 / var
    S = np.full_like(mu, 0.5)
    Z = mu[rng.choice(mu.shape[0], size=M, replace=False)].copy()
    return mu, S, Z, var, np.ones(Q), 100.0 / var


def fit(Y: np.ndarray, Q: int, M: int, *, iters: int = 200, dtype=None, jitter: float = 1e-6,
        seed: int = 0, init=None, device: str = "cuda:0", tol: float = 1e-9) -> FitResult:
    """Maximise the bound over (mu, S, Z, sigma_f2, l, beta) with L-BFGS-B.

    Y is centred internally.  Every objective evaluation is one ``gpps_bound``
    call on ``device`` (dtype float64 unless given)."""
    import scipy.optimize
    import torch

    dtype = torch.float64 if dtype is None else dtype
    Y = np.asarray(Y, np.float64)
    Y = Y - Y.mean(0)
    N, D = Y.shape
    mu0, S0, Z0, sf20, l0, beta0 = init if init is not None else init_params(Y, Q, M, seed)
    x0 = _pack(mu0, S0, Z0, sf20, l0, beta0)
    Yt = torch.tensor(Y, dtype=dtype, device=device)
    trace = []
    gpu_s = [0.0]
    ws = torch.empty(max(1, _ws_bytes(dtype, N, M, Q, D)), dtype=torch.uint8, device=device)
    out = None

    def objective(x):
        nonlocal out
        mu, S, Z, sf2, l, beta = _unpack(x, N, M, Q)
        if not _feasible(S, sf2, l, beta):
            return 1e300, np.zeros_like(x)
        t = {k: torch.tensor(v, dtype=dtype, device=device) for k, v in (("mu", mu), ("S", S),
                                                                           ("Z", Z))}
        t0 = time.perf_counter()
        out = bound(t["mu"], t["S"], t["Z"], Yt, sf2, l, beta, jitter, out=out, workspace=ws)
        torch.cuda.synchronize()
        gpu_s[0] += time.perf_counter() - t0
        g = {k: v.double().cpu().numpy() for k, v in out.items()}
        L = float(g["L"][0])
        if not np.isfinite(L):
            # an infeasible step (a matrix lost positive definiteness): tell the
            # line search to back off
            return 1e300, np.zeros_like(x)
        trace.append(L)
        grad = np.concatenate([g["dmu"].ravel(), (g["dS"] * S).ravel(), g["dZ"].ravel(),
                               [float(g["dsigma_f2"][0]) * sf2], g["dl"] * l,
                               [float(g["dbeta"][0]) * beta]])
        return -L, -grad

    t0 = time.perf_counter()
    res = scipy.optimize.minimize(objective, x0, jac=True, method="L-BFGS-B",
                                  options={"maxiter": iters, "ftol": tol, "gtol": 1e-8})
    secs = time.perf_counter() - t0
    mu, S, Z, sf2, l, beta = _unpack(res.x, N, M, Q)
    return FitResult(mu, S, Z, sf2, l, beta, trace, int(res.nfev), int(res.nit), secs, gpu_s[0],
                     str(res.message))


def fit_staged(Y: np.ndarray, Q: int, M: int, *, every: int = 16, iters: int = 300,
               jitter: float = 1e-4, dtype=None, device: str = "cuda:0", tol: float = 1e-12):
    """Two-stage fit for large N with many inducing inputs (the section 4 shape:
    Q = 1, M = 100, N up to 64,000).

    Stage 1 fits every ``every``-th row from the spread start (init_params with
    spread=True).  Stage 2 fits all rows, starting from stage 1's Z and kernel
    and noise parameters, each row's (mu, S) taken from its nearest stage-1 row in
    data space (a k-d tree on Y: the PCA coordinate of a folded 1-D curve is not
    monotone in the latent).  From a cold start at full N, with 100 inducing
    inputs spaced far below the lengthscale, the line search keeps stepping into
    parameters where A = Kmm + beta Psi2 is not positive definite in fp64 and the
    optimiser stops early.  Returns (stage-1 result, stage-2 result, rows of
    stage 1)."""
    from scipy.spatial import cKDTree

    Y = np.asarray(Y, np.float64)
    Yc = Y - Y.mean(0)
    mu, S, Z, var, l, beta = init_params(Yc, Q, M, spread=True)
    sub = np.arange(0, Y.shape[0], every)
    r1 = fit(Y[sub], Q, M, iters=iters, init=(mu[sub], S[sub], Z, var, l, beta), jitter=jitter,
             dtype=dtype, device=device, tol=tol)
    _, nn = cKDTree(Yc[sub]).query(Yc)
    r2 = fit(Y, Q, M, iters=iters, init=(r1.mu[nn], r1.S[nn], r1.Z, r1.sigma_f2, r1.l, r1.beta),
             jitter=jitter, dtype=dtype, device=device, tol=tol)
    return r1, r2, sub


_LOG_BOUND = 30.0


def _feasible(S, sf2, l, beta) -> bool:
    """A line-search step can overflow exp() of a log parameter: such a point is
    infeasible (the library would reject it), so the objective reports a huge
    value and the line search backs off."""
    vals = [sf2, beta, *np.ravel(l)] + ([] if S is None else [float(np.min(S)), float(np.max(S))])
    return all(np.isfinite(v) and v > 0 for v in vals)


def _ws_bytes(dtype, N, M, Q, D):
    from . import bound_workspace_bytes
    return bound_workspace_bytes(dtype, N, M, Q, D)


@dataclasses.dataclass
class RegressionResult:
    Z: np.ndarray
    sigma_f2: float
    l: np.ndarray
    beta: float
    bound_trace: list        # L after every evaluation
    evals: int
    iterations: int
    seconds: float
    message: str


def fit_regression(X: np.ndarray, Y: np.ndarray, M: int, *, iters: int = 200, dtype=None,
                   jitter: float = 1e-6, seed: int = 0, device: str = "cuda:0",
                   tol: float = 1e-9) -> RegressionResult:
    """Maximise the regression bound of eq. (boundF) over (Z, log sigma_f2, log l,
    log beta) with L-BFGS-B, X fixed.  Y is centred internally.  Start: Z a random
    subset of X, sigma_f2 = var(Y), l = the spread of each input dimension,
    beta = 100 / var(Y).  Every objective evaluation is one ``gpps_bound`` call
    with S = None on ``device`` (dtype float64 unless given)."""
    import scipy.optimize
    import torch

    dtype = torch.float64 if dtype is None else dtype
    X = np.asarray(X, np.float64)
    Y = np.asarray(Y, np.float64)
    Y = Y - Y.mean(0)
    N, Q = X.shape
    D = Y.shape[1]
    rng = np.random.default_rng(seed)
    Z0 = X[rng.choice(N, size=M, replace=False)].copy()
    var = float(Y.var())
    x0 = np.concatenate([Z0.ravel(), [np.log(var)], np.log(X.std(0) + 1e-12), [np.log(100.0 / var)]])
    Xt = torch.tensor(X, dtype=dtype, device=device)
    Yt = torch.tensor(Y, dtype=dtype, device=device)
    ws = torch.empty(max(1, _ws_bytes(dtype, N, M, Q, D)), dtype=torch.uint8, device=device)
    trace = []
    out = None

    def unpack(x):
        Z = x[:M * Q].reshape(M, Q)
        return Z, float(np.exp(x[M * Q])), np.exp(x[M * Q + 1:M * Q + 1 + Q]), float(np.exp(x[-1]))

    def objective(x):
        nonlocal out
        Z, sf2, l, beta = unpack(x)
        if not _feasible(None, sf2, l, beta):
            return 1e300, np.zeros_like(x)
        Zt = torch.tensor(Z, dtype=dtype, device=device)
        out = bound(Xt, None, Zt, Yt, sf2, l, beta, jitter, out=out, workspace=ws)
        torch.cuda.synchronize()
        g = {k: v.double().cpu().numpy() for k, v in out.items() if v is not None}
        L = float(g["L"][0])
        if not np.isfinite(L):
            return 1e300, np.zeros_like(x)
        trace.append(L)
        grad = np.concatenate([g["dZ"].ravel(), [float(g["dsigma_f2"][0]) * sf2], g["dl"] * l,
                               [float(g["dbeta"][0]) * beta]])
        return -L, -grad

    # the log parameters are bounded to +-30 (e^30 ~ 1e13): from this start the
    # first line-search step is long enough to overflow exp() otherwise
    bounds = [(None, None)] * (M * Q) + [(-_LOG_BOUND, _LOG_BOUND)] * (Q + 2)
    t0 = time.perf_counter()
    res = scipy.optimize.minimize(objective, x0, jac=True, method="L-BFGS-B", bounds=bounds,
                                  options={"maxiter": iters, "ftol": tol, "gtol": 1e-8})
    secs = time.perf_counter() - t0
    Z, sf2, l, beta = unpack(res.x)
    return RegressionResult(Z, sf2, l, beta, trace, int(res.nfev), int(res.nit), secs,
                            str(res.message))
