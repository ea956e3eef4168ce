"""Bayesian GP-LVM fitting with the bound evaluated on the GPU.

Section 2 (end): the parameters are the variational means and variances
(mu, S) of q(X), the inducing inputs Z, the kernel parameters (sigma_f2, l) and
the noise precision beta; the gradients of every parameter are collected on one
node and passed to an existing optimiser (L-BFGS-B in SciPy).  Here the bound
and all its gradients come from ``gpps_bound`` (one call per evaluation, all on
the device); only the optimiser's vector arithmetic runs on the host.

Positive parameters are optimised through their logarithms (S, sigma_f2, l,
beta); the chain rule d/dlog x = x d/dx is applied to the gradients the library
returns.

    fit(Y, Q, M, iters=...) -> FitResult
    paper_data(N, D=3, seed=0) -> (Y, x_true)   the synthetic data of section 4
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


def init_params(Y: np.ndarray, Q: int, M: int, seed: int = 0):
    """PCA means (scaled to unit variance), S = 0.5, Z a random subset of the
    means, unit lengthscales, sigma_f2 = var(Y), beta = 100 / var(Y)."""
    rng = np.random.default_rng(seed)
    Yc = Y - Y.mean(0)
    _, _, Vt = np.linalg.svd(Yc, full_matrices=False)
    mu = Yc @ Vt[:Q].T
    mu = mu / mu.std(0)
    S = np.full_like(mu, 0.5)
    Z = mu[rng.choice(mu.shape[0], size=M, replace=False)].copy()
    var = float(Yc.var())
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


def _ws_bytes(dtype, N, M, Q, D):
    from . import bound_workspace_bytes
    return bound_workspace_bytes(dtype, N, M, Q, D)
