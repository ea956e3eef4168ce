"""Plain fp64 CPU oracle for the RBF-ARD psi-statistics and their gradients.

TEST INFRASTRUCTURE ONLY: only ``tests/``, ``__graft_entry__.smoke()`` and the
CPU-baseline leg of ``bench.py`` may import this package.  The product path
(the HIP library and its Python binding) never imports, links or calls it,
and the two share no code.

The psi-statistic arithmetic lives in ``psi_oracle.c`` (plain loops, fp64,
libm); this module only compiles it with gcc and marshals numpy arrays through
ctypes.  ``bound.py`` adds the Bayesian GP-LVM bound and its gradients on top
(fp64 numpy).  What each
function computes, and the passage of the paper it follows, is stated in the C
source.  Every function here takes float64 arrays; callers that compare against
the fp32 GPU path first round their inputs to float32 and pass them upcast, so
that a comparison measures compute error, not input rounding.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "psi_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None

_ERRORS = {1: "bad size", 2: "null pointer", 3: "bad hyper-parameter", 4: "out of memory"}


def build(force: bool = True) -> str:
    """Compile the oracle into ``oracle/liboracle.so`` (gcc, -O2, OpenMP, no fast-math)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp"
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-fopenmp", "-fno-fast-math",
             "-Wall", "-Wextra", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        i64, dp, d = ctypes.c_int64, ctypes.c_void_p, ctypes.c_double
        lib.oracle_psi_stats.argtypes = [i64, i64, i64, dp, dp, dp, d, dp, dp, dp, dp]
        lib.oracle_psi_grads.argtypes = [i64, i64, i64, dp, dp, dp, d, dp, d, dp, dp,
                                         dp, dp, dp, dp, dp]
        lib.oracle_psi2_entries.argtypes = [i64, i64, i64, dp, dp, dp, d, dp, i64, dp, dp]
        lib.oracle_dZ_rows.argtypes = [i64, i64, i64, dp, dp, dp, d, dp, dp, dp, i64, dp, dp]
        for f in (lib.oracle_psi_stats, lib.oracle_psi_grads, lib.oracle_psi2_entries,
                  lib.oracle_dZ_rows):
            f.restype = ctypes.c_int
        lib.oracle_num_threads.restype = ctypes.c_int
        _lib = lib
    return _lib


def _f64(a):
    return None if a is None else np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a):
    return None if a is None else a.ctypes.data


def _check(rc):
    if rc != 0:
        raise ValueError(f"oracle: {_ERRORS.get(rc, rc)}")


def _common(mu, S, Z, l):
    mu, S, Z, l = _f64(mu), _f64(S), _f64(Z), _f64(l)
    N, Q = mu.shape
    M = Z.shape[0]
    assert S.shape == (N, Q) and Z.shape == (M, Q) and l.shape == (Q,)
    return mu, S, Z, l, N, M, Q


def num_threads() -> int:
    return int(_load().oracle_num_threads())


def psi_stats(mu, S, Z, sigma_f2, l, want_psi1=True):
    """Return (psi0, Psi1 [N x M] or None, Psi2 [M x M]) in float64."""
    mu, S, Z, l, N, M, Q = _common(mu, S, Z, l)
    psi0 = np.zeros(1)
    Psi1 = np.empty((N, M)) if want_psi1 else None
    Psi2 = np.empty((M, M))
    _check(_load().oracle_psi_stats(N, M, Q, _ptr(mu), _ptr(S), _ptr(Z), float(sigma_f2),
                                    _ptr(l), _ptr(psi0), _ptr(Psi1), _ptr(Psi2)))
    return float(psi0[0]), Psi1, Psi2


def psi_grads(mu, S, Z, sigma_f2, l, dL_dpsi0, dL_dPsi1, dL_dPsi2):
    """Return dict with dmu, dS [N x Q], dZ [M x Q], dsigma_f2 (float), dl [Q]."""
    mu, S, Z, l, N, M, Q = _common(mu, S, Z, l)
    G1, G2 = _f64(dL_dPsi1), _f64(dL_dPsi2)
    if G1 is not None:
        assert G1.shape == (N, M)
    if G2 is not None:
        assert G2.shape == (M, M)
    dmu, dS = np.empty((N, Q)), np.empty((N, Q))
    dZ, dl, dsf2 = np.empty((M, Q)), np.empty(Q), np.zeros(1)
    _check(_load().oracle_psi_grads(N, M, Q, _ptr(mu), _ptr(S), _ptr(Z), float(sigma_f2),
                                    _ptr(l), float(dL_dpsi0), _ptr(G1), _ptr(G2), _ptr(dmu),
                                    _ptr(dS), _ptr(dZ), _ptr(dsf2), _ptr(dl)))
    return {"dmu": dmu, "dS": dS, "dZ": dZ, "dsigma_f2": float(dsf2[0]), "dl": dl}


def psi2_entries(mu, S, Z, sigma_f2, l, pairs):
    """Psi2[m, m'] for each (m, m') row of ``pairs`` (int array k x 2), summed over all N."""
    mu, S, Z, l, N, M, Q = _common(mu, S, Z, l)
    pairs = np.ascontiguousarray(pairs, dtype=np.int64).reshape(-1, 2)
    out = np.empty(pairs.shape[0])
    _check(_load().oracle_psi2_entries(N, M, Q, _ptr(mu), _ptr(S), _ptr(Z), float(sigma_f2),
                                       _ptr(l), pairs.shape[0], _ptr(pairs), _ptr(out)))
    return out


def dZ_rows(mu, S, Z, sigma_f2, l, dL_dPsi1, dL_dPsi2, rows):
    """dL/dZ[m, :] for each m in ``rows``, summed over all N (k x Q)."""
    mu, S, Z, l, N, M, Q = _common(mu, S, Z, l)
    G1, G2 = _f64(dL_dPsi1), _f64(dL_dPsi2)
    rows = np.ascontiguousarray(rows, dtype=np.int64).reshape(-1)
    out = np.empty((rows.shape[0], Q))
    _check(_load().oracle_dZ_rows(N, M, Q, _ptr(mu), _ptr(S), _ptr(Z), float(sigma_f2),
                                  _ptr(l), _ptr(G1), _ptr(G2), rows.shape[0], _ptr(rows),
                                  _ptr(out)))
    return out
