"""Plain fp64 oracle for the Bayesian GP-LVM variational bound and its gradients.

TEST INFRASTRUCTURE ONLY, like the rest of ``oracle/``: only ``tests/``,
``__graft_entry__.smoke()`` and the CPU-baseline leg of ``bench.py`` may use it.

What it computes (section 2): the collapsed sparse-GP bound of eq. (boundF) for
all D output columns, with the kernel statistics replaced by their expectations
under q(X) (phi -> psi0, Phi -> Psi2, Psi = Psi1^T Y), minus the KL term of
eq. (boundBGPLVM) against the standard normal prior p(x_n) = N(0, I):

    F = -(N D / 2) log(2 pi) + (N D / 2) log beta + (D / 2) log|Kmm| - (D / 2) log|A|
        - (beta / 2) tr(Y^T Y) + (beta^2 / 2) tr(Psi^T A^-1 Psi)
        - (beta D / 2) psi0 + (beta D / 2) tr(Kmm^-1 Psi2),
    A = Kmm + beta Psi2,        Kmm = k(Z, Z) + jitter I,
    KL = 1/2 sum_nq (mu^2 + S - log S - 1),          L = F - KL.

Readings taken where the printed equation is garbled: the data term is the
scalar tr(Y^T Y); the Psi-term carries a trace; the log-determinant terms of the
per-column bound are multiplied by D; jitter is an absolute value added to the
diagonal of Kmm.  The psi-statistics and their chain rule come from the C
oracle (``oracle.psi_stats`` / ``oracle.psi_grads``); the M x M algebra here uses
numpy's Cholesky and triangular solves, the library primitives the definition
is written with.

Gradients (all matrices symmetric, C = A^-1 Psi, P = C C^T):
    dL/dpsi0 = -beta D / 2
    dL/dPsi1 = beta^2 Y C^T
    dL/dPsi2 = -(beta D / 2) A^-1 - (beta^3 / 2) P + (beta D / 2) Kmm^-1
    dL/dKmm  = (D / 2) Kmm^-1 - (D / 2) A^-1 - (beta^2 / 2) P - (beta D / 2) Kmm^-1 Psi2 Kmm^-1
    dL/dbeta = N D / (2 beta) - tr(Y^T Y) / 2 - (D / 2) tr(A^-1 Psi2) + beta tr(Psi^T C)
               - (beta^2 / 2) tr(P Psi2) - (D / 2) psi0 + (D / 2) tr(Kmm^-1 Psi2)
then through Kmm to (Z, sigma_f^2, l), through the psi-statistics to
(mu, S, Z, sigma_f^2, l), and the KL adds dmu -= mu, dS -= (1 - 1/S) / 2.

S = None is the sparse GP regression case of eq. (boundF) itself: the inputs are
known (mu holds X, every variance is zero), so the statistics are the plain
kernel quantities (psi0 = tr Kff, Psi1 = Kfu, Psi2 = Kfu^T Kfu), there is no
q(X) and no KL term, L = F, and the gradient w.r.t. the inputs is dL/dX (no dS).
"""
from __future__ import annotations

import numpy as np

from . import psi_grads, psi_stats


def kmm(Z, sigma_f2, l):
    """ARD RBF kernel matrix of the inducing inputs (no jitter)."""
    Z = np.asarray(Z, np.float64)
    l = np.asarray(l, np.float64)
    d = (Z[:, None, :] - Z[None, :, :]) / l
    return sigma_f2 * np.exp(-0.5 * np.sum(d * d, axis=-1))


def _chol(A):
    return np.linalg.cholesky(A)


def _inv_spd(L):
    """A^-1 from its lower Cholesky factor."""
    M = L.shape[0]
    Li = np.linalg.solve(L, np.eye(M))
    return Li.T @ Li


def _inv_lu(L):
    """A^-1 of A = L L^T by LU with partial pivoting (numpy's inv): a second
    backward-stable evaluation, used to measure how much an output of an
    ill-conditioned problem moves between two correct fp64 evaluations."""
    return np.linalg.inv(L @ L.T)


def _inv_eigh(L):
    """A^-1 of A = L L^T through its eigendecomposition (numpy's eigh): a third
    backward-stable evaluation for the same purpose as _inv_lu."""
    w, V = np.linalg.eigh(L @ L.T)
    return (V / w) @ V.T


def kl(mu, S):
    """KL(q(X) || N(0, I)) summed over datapoints and dimensions."""
    mu = np.asarray(mu, np.float64)
    S = np.asarray(S, np.float64)
    with np.errstate(divide="ignore"):
        return 0.5 * float(np.sum(mu * mu + S - np.log(S) - 1.0))


def bound_terms(mu, S, Z, Y, sigma_f2, l, beta, jitter, inverse=_inv_spd, stats=None):
    """(F, KL, pieces): the collapsed bound F and the KL term, plus the
    intermediate matrices the gradient needs.  ``inverse`` maps a Cholesky
    factor to the inverse of its matrix (default: triangular solves).  S = None:
    known inputs (zero variances), KL = 0.  ``stats`` = (psi0, Psi1, Psi2) uses
    the given statistics instead of computing them (to measure how sensitive
    the bound is to errors in them)."""
    mu = np.asarray(mu, np.float64)
    Y = np.asarray(Y, np.float64)
    N, D = Y.shape
    if stats is None:
        psi0, Psi1, Psi2 = psi_stats(mu, np.zeros_like(mu) if S is None else S, Z, sigma_f2, l)
    else:
        psi0, Psi1, Psi2 = stats
    Psi1 = np.asarray(Psi1).reshape(N, -1)
    Psi2 = np.asarray(Psi2)
    M = Psi2.shape[0]
    K0 = kmm(Z, sigma_f2, l)
    Kmm = K0 + jitter * np.eye(M)
    A = Kmm + beta * Psi2
    Lk, La = _chol(Kmm), _chol(A)
    Kinv, Ainv = inverse(Lk), inverse(La)
    Psi = Psi1.T @ Y
    C = Ainv @ Psi
    yy = float(np.sum(Y * Y))
    logdet_k = 2.0 * float(np.sum(np.log(np.diag(Lk))))
    logdet_a = 2.0 * float(np.sum(np.log(np.diag(La))))
    F = (-0.5 * N * D * np.log(2.0 * np.pi) + 0.5 * N * D * np.log(beta)
         + 0.5 * D * logdet_k - 0.5 * D * logdet_a - 0.5 * beta * yy
         + 0.5 * beta * beta * float(np.sum(Psi * C))
         - 0.5 * beta * D * float(psi0) + 0.5 * beta * D * float(np.sum(Kinv * Psi2)))
    pieces = dict(N=N, D=D, M=M, psi0=float(psi0), Psi1=Psi1, Psi2=Psi2, K0=K0, Kmm=Kmm,
                  Kinv=Kinv, Ainv=Ainv, Psi=Psi, C=C, yy=yy)
    return F, (0.0 if S is None else kl(mu, S)), pieces


def bound(mu, S, Z, Y, sigma_f2, l, beta, jitter):
    """L = F - KL."""
    F, K, _ = bound_terms(mu, S, Z, Y, sigma_f2, l, beta, jitter)
    return F - K


def upstream(mu, S, Z, Y, sigma_f2, l, beta, jitter, inverse=_inv_spd, stats=None):
    """(L, dL/dpsi0, dL/dPsi1, dL/dPsi2, dL/dKmm, dL/dbeta, pieces)."""
    F, K, p = bound_terms(mu, S, Z, Y, sigma_f2, l, beta, jitter, inverse, stats)
    D = p["D"]
    Kinv, Ainv, C, Psi2, Psi = p["Kinv"], p["Ainv"], p["C"], p["Psi2"], p["Psi"]
    P = C @ C.T
    d_psi0 = -0.5 * beta * D
    d_Psi1 = beta * beta * (np.asarray(Y, np.float64) @ C.T)
    d_Psi2 = -0.5 * beta * D * Ainv - 0.5 * beta ** 3 * P + 0.5 * beta * D * Kinv
    d_Kmm = 0.5 * D * Kinv - 0.5 * D * Ainv - 0.5 * beta * beta * P \
        - 0.5 * beta * D * (Kinv @ Psi2 @ Kinv)
    d_beta = (0.5 * p["N"] * D / beta - 0.5 * p["yy"] - 0.5 * D * float(np.sum(Ainv * Psi2))
              + beta * float(np.sum(Psi * C)) - 0.5 * beta * beta * float(np.sum(P * Psi2))
              - 0.5 * D * p["psi0"] + 0.5 * D * float(np.sum(Kinv * Psi2)))
    return F - K, d_psi0, d_Psi1, d_Psi2, d_Kmm, d_beta, p


def kmm_grads(Z, sigma_f2, l, G):
    """Chain rule through Kmm = k(Z, Z) + jitter I for an upstream dL/dKmm = G
    (any square matrix; only its symmetric part matters): (dZ, dsigma_f2, dl)."""
    Z = np.asarray(Z, np.float64)
    l = np.asarray(l, np.float64)
    Gs = 0.5 * (G + G.T)
    K0 = kmm(Z, sigma_f2, l)
    W = Gs * K0
    diff = Z[:, None, :] - Z[None, :, :]                       # [m, m', q]
    dZ = -2.0 * np.einsum("ab,abq->aq", W, diff) / (l * l)
    dl = np.einsum("ab,abq->q", W, diff * diff) / (l ** 3)
    dsf2 = float(np.sum(W)) / sigma_f2
    return dZ, dsf2, dl


def grads(mu, S, Z, Y, sigma_f2, l, beta, jitter, inverse=_inv_spd, stats=None):
    """L and its gradient w.r.t. every parameter:
    dict(L, dmu, dS, dZ, dsigma_f2, dl, dbeta).  S = None (known inputs): dmu is
    dL/dX and dS is None.  ``stats`` as for bound_terms (the chain rule through
    the statistics is still taken at mu, S, Z)."""
    L, d_psi0, d_Psi1, d_Psi2, d_Kmm, d_beta, p = upstream(mu, S, Z, Y, sigma_f2, l, beta,
                                                            jitter, inverse, stats)
    mu = np.asarray(mu, np.float64)
    known = S is None
    S = np.zeros_like(mu) if known else np.asarray(S, np.float64)
    g = psi_grads(mu, S, Z, sigma_f2, l, d_psi0, d_Psi1, d_Psi2)
    kz, ks, kl_ = kmm_grads(Z, sigma_f2, l, d_Kmm)
    return dict(L=L,
                dmu=np.asarray(g["dmu"]) - (0.0 if known else mu),
                dS=None if known else np.asarray(g["dS"]) - 0.5 * (1.0 - 1.0 / S),
                dZ=np.asarray(g["dZ"]) + kz,
                dsigma_f2=float(np.asarray(g["dsigma_f2"]).ravel()[0]) + ks,
                dl=np.asarray(g["dl"]) + kl_,
                dbeta=d_beta)
