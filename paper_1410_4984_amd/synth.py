"""Seeded synthetic workloads for the psi-statistics path.

This module only draws random inputs (numpy ``default_rng``); it contains none
of the psi-statistic arithmetic, so both the HIP path and the CPU oracle can
consume what it produces.  Every array is drawn in float64; ``to_f32`` rounds
a workload to float32 for the fp32 path (the oracle then receives the rounded
values upcast back to float64).

The five named workloads follow the shapes of the paper's setting (section 4:
Bayesian GP-LVM with a latent space of dimension Q and M inducing inputs,
time dominated by the O(N M^2 Q) statistic) scaled to one modern GPU:

  tiny    N=200,       M=10,  Q=2   parity case, fp64 and fp32
  small   N=5,000,     M=50,  Q=10
  medium  N=50,000,    M=100, Q=10  clustered latents, inducing inputs picked from them
  large   N=100,000,   M=256, Q=20  the timed workload
  stress  N=1,000,000, M=512, Q=30  processed in row chunks of 131,072

Draw order for every workload: mu, S, Z, l, dL_dpsi0, dL_dPsi1, A; then
dL_dPsi2 = (A + A^T) / 2.  For ``stress`` dL_dPsi1 is drawn per row chunk from
``default_rng([seed, chunk])`` so that it never has to exist whole on the host.
"""
from __future__ import annotations

from dataclasses import dataclass

import numpy as np


@dataclass(frozen=True)
class Workload:
    name: str
    N: int
    M: int
    Q: int
    description: str
    chunk_rows: int = 0  # > 0: rows are processed in chunks of this size


WORKLOADS = {
    "tiny": Workload("tiny", 200, 10, 2, "mu~N(0,1), S~U(0.01,0.5), Z = subset of mu + N(0,0.1^2), "
                     "sigma_f2=1.3, l~U(0.5,2)"),
    "small": Workload("small", 5_000, 50, 10, "mu~N(0,1), S~U(0.05,1), Z~N(0,1), sigma_f2=1, "
                      "l~U(0.3,3)"),
    "medium": Workload("medium", 50_000, 100, 10, "mu from a 3-component Gaussian mixture "
                       "(centres ~N(0,9 I), unit covariance), S~logU(1e-3,1), Z = k-means++ "
                       "D^2-seeded picks of mu, sigma_f2=1, l~U(0.5,2)"),
    "large": Workload("large", 100_000, 256, 20, "mu~N(0,1), S~U(0.01,0.5), Z~N(0,1), "
                      "sigma_f2=1, l~U(0.5,2)"),
    "stress": Workload("stress", 1_000_000, 512, 30, "mu~N(0,1), S~U(0.01,0.5), Z~N(0,1), "
                       "sigma_f2=1, l~U(0.5,4)", chunk_rows=131_072),
}


def _kmeanspp_picks(rng, X, M):
    """Indices of M rows of X chosen by k-means++ D^2 seeding (no Lloyd steps)."""
    N = X.shape[0]
    idx = [int(rng.integers(N))]
    d2 = np.sum((X - X[idx[0]]) ** 2, axis=1)
    for _ in range(1, M):
        p = d2 / d2.sum()
        i = int(rng.choice(N, p=p))
        idx.append(i)
        d2 = np.minimum(d2, np.sum((X - X[i]) ** 2, axis=1))
    return np.array(idx)


def _gradients(rng, N, M, with_G1=True):
    dL_dpsi0 = float(rng.standard_normal())
    G1 = rng.standard_normal((N, M)) if with_G1 else None
    A = rng.standard_normal((M, M))
    return dL_dpsi0, G1, 0.5 * (A + A.T)


def make_workload(name: str, seed: int = 0) -> dict:
    """Inputs of a named workload (float64).  For ``stress`` dL_dPsi1 is None: use
    :func:`stress_dL_dPsi1_chunk`."""
    w = WORKLOADS[name]
    rng = np.random.default_rng(seed)
    N, M, Q = w.N, w.M, w.Q
    if name == "tiny":
        mu = rng.standard_normal((N, Q))
        S = rng.uniform(0.01, 0.5, (N, Q))
        Z = mu[rng.choice(N, M, replace=False)] + 0.1 * rng.standard_normal((M, Q))
        sf2 = 1.3
        l = rng.uniform(0.5, 2.0, Q)
    elif name == "small":
        mu = rng.standard_normal((N, Q))
        S = rng.uniform(0.05, 1.0, (N, Q))
        Z = rng.standard_normal((M, Q))
        sf2 = 1.0
        l = rng.uniform(0.3, 3.0, Q)
    elif name == "medium":
        centres = 3.0 * rng.standard_normal((3, Q))
        comp = rng.integers(0, 3, N)
        mu = centres[comp] + rng.standard_normal((N, Q))
        S = np.exp(rng.uniform(np.log(1e-3), np.log(1.0), (N, Q)))
        Z = mu[_kmeanspp_picks(rng, mu, M)].copy()
        sf2 = 1.0
        l = rng.uniform(0.5, 2.0, Q)
    elif name == "large":
        mu = rng.standard_normal((N, Q))
        S = rng.uniform(0.01, 0.5, (N, Q))
        Z = rng.standard_normal((M, Q))
        sf2 = 1.0
        l = rng.uniform(0.5, 2.0, Q)
    elif name == "stress":
        mu = rng.standard_normal((N, Q))
        S = rng.uniform(0.01, 0.5, (N, Q))
        Z = rng.standard_normal((M, Q))
        sf2 = 1.0
        l = rng.uniform(0.5, 4.0, Q)
    else:  # pragma: no cover
        raise KeyError(name)
    dL_dpsi0, G1, G2 = _gradients(rng, N, M, with_G1=(name != "stress"))
    return {"mu": mu, "S": S, "Z": Z, "sigma_f2": sf2, "l": l, "dL_dpsi0": dL_dpsi0,
            "dL_dPsi1": G1, "dL_dPsi2": G2}


def stress_dL_dPsi1_chunk(seed: int, chunk: int, rows: int, M: int) -> np.ndarray:
    """dL/dPsi1 rows of one chunk of the ``stress`` workload."""
    return np.random.default_rng([seed, chunk]).standard_normal((rows, M))


def random_inputs(N: int, M: int, Q: int, seed: int = 0, s_range=(0.01, 0.5),
                  l_range=(0.5, 2.0), sigma_f2: float = 1.0, z_scale: float = 1.0) -> dict:
    """Generic seeded inputs of any shape (same distributions as ``large``)."""
    rng = np.random.default_rng(seed)
    mu = rng.standard_normal((N, Q))
    S = rng.uniform(s_range[0], s_range[1], (N, Q))
    Z = z_scale * rng.standard_normal((M, Q))
    l = rng.uniform(l_range[0], l_range[1], Q)
    dL_dpsi0, G1, G2 = _gradients(rng, N, M)
    return {"mu": mu, "S": S, "Z": Z, "sigma_f2": float(sigma_f2), "l": l,
            "dL_dpsi0": dL_dpsi0, "dL_dPsi1": G1, "dL_dPsi2": G2}


def to_f32(inputs: dict) -> dict:
    """Round every array (and the scalar hypers) to float32; values stay float64 arrays
    holding exactly representable float32 numbers."""
    out = {}
    for k, v in inputs.items():
        if isinstance(v, np.ndarray):
            out[k] = v.astype(np.float32).astype(np.float64)
        elif isinstance(v, float):
            out[k] = float(np.float32(v))
        else:
            out[k] = v
    return out


# Several views sharing one q(X) (section 1: MRD): shared mu, S drawn as in
# ``large``; per view, inducing inputs Z_v ~ N(0, 1), sigma_f2_v ~ U(0.5, 2),
# l_v ~ U(0.5, 2) per dimension, and Gaussian dL/dPsi of the view's shape.
# Draw order: mu, S, then per view Z, sigma_f2, l, dL_dpsi0, dL_dPsi1, A.
VIEW_WORKLOADS = {
    "views-tiny": (300, (10, 7, 12), 3),
    "views-small": (5_000, (50, 30, 20), 10),
    "views-large": (100_000, (256, 192, 128), 20),
}


def make_views_workload(name: str, seed: int = 0) -> dict:
    N, Ms, Q = VIEW_WORKLOADS[name]
    rng = np.random.default_rng(seed)
    mu = rng.standard_normal((N, Q))
    S = rng.uniform(0.01, 0.5, (N, Q))
    views = []
    for M in Ms:
        Z = rng.standard_normal((M, Q))
        sf2 = float(rng.uniform(0.5, 2.0))
        l = rng.uniform(0.5, 2.0, Q)
        d0 = float(rng.standard_normal())
        G1 = rng.standard_normal((N, M))
        A = rng.standard_normal((M, M))
        views.append({"Z": Z, "sigma_f2": sf2, "l": l, "dL_dpsi0": d0, "dL_dPsi1": G1,
                      "dL_dPsi2": 0.5 * (A + A.T)})
    return {"mu": mu, "S": S, "views": views}


def views_to_f32(w: dict) -> dict:
    f = lambda a: a.astype(np.float32).astype(np.float64)  # noqa: E731
    return {"mu": f(w["mu"]), "S": f(w["S"]),
            "views": [{k: (f(v) if isinstance(v, np.ndarray) else float(np.float32(v)))
                       for k, v in vw.items()} for vw in w["views"]]}
