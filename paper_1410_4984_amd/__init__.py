"""RBF-ARD psi-statistics and their gradients on AMD Instinct MI355X (HIP, gfx950).

Thin binding over the C ABI of ``libgpps.so`` (declared in ``include/gpps.h``):
it checks torch tensors (device, dtype, contiguity, shape), allocates outputs
and workspace with torch, and passes raw pointers plus the current HIP stream.
Every step of the computation runs in the library's HIP kernels; there is no
fallback of any kind: if the library is missing or cannot run, calls raise.

    psi_stats(mu, S, Z, sigma_f2, l)   -> (psi0, Psi1, Psi2)
    psi_grads(mu, S, Z, sigma_f2, l, dL_dpsi0, dL_dPsi1, dL_dPsi2)
                                       -> dict(dmu, dS, dZ, dsigma_f2, dl)
    bound(mu, S, Z, Y, sigma_f2, l, beta, jitter)
                                       -> dict(L, dmu, dS, dZ, dsigma_f2, dl, dbeta)

Notation follows the paper (section 2, Alg. 1-2): mu, S (variances) are N x Q,
Z is M x Q, sigma_f2 the kernel variance, l the Q ARD lengthscales.  S = None
means known inputs (every variance zero: the sparse GP regression case of
eq. (boundF), with mu holding the inputs X); the library then computes
Psi1 = Kfu and Psi2 = Kfu^T Kfu on its matrix-core GEMM path, and dS is None.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libgpps.so")

F32, F64 = 0, 1
ACCUMULATE = 1
PATHS = {"auto": 0, "generic": 2, "mfma": 4}   # path flags of the C ABI
MAX_Q = 64
MAX_M = 4096

_lib = None
_default_path = "auto"


class GppsError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"gpps status {status}: {msg}")
        self.status = status


def lib():
    """The loaded ``libgpps.so`` (ctypes handle with argument types set)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise RuntimeError(f"{LIB_PATH} is not built; run `python -m paper_1410_4984_amd.build` "
                           "(or __graft_entry__.build())")
    import torch  # noqa: F401  -- load torch's HIP runtime first so the library shares it
    L = ctypes.CDLL(LIB_PATH)
    i64, vp, d, sz, i32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_double, ctypes.c_size_t, ctypes.c_int
    L.gpps_workspace_bytes.argtypes = [i32, i64, i64, i64]
    L.gpps_workspace_bytes.restype = sz
    L.gpps_route_word_offset.argtypes = [i32, i64, i64, i64]
    L.gpps_route_word_offset.restype = sz
    L.gpps_psi_stats.argtypes = [i32, i64, i64, i64, vp, vp, vp, d, vp, vp, vp, vp, i32, vp, sz, vp]
    L.gpps_psi_stats.restype = i32
    L.gpps_psi_grads.argtypes = [i32, i64, i64, i64, vp, vp, vp, d, vp, d, vp, vp, vp, vp, vp, vp,
                                 vp, i32, vp, sz, vp]
    L.gpps_psi_grads.restype = i32
    L.gpps_bound_workspace_bytes.argtypes = [i32, i64, i64, i64, i64]
    L.gpps_bound_workspace_bytes.restype = sz
    L.gpps_bound.argtypes = [i32, i64, i64, i64, i64, vp, vp, vp, vp, d, vp, d, d, vp, vp, vp, vp,
                             vp, vp, vp, i32, vp, sz, vp]
    L.gpps_bound.restype = i32
    L.gpps_views_workspace_bytes.argtypes = [i32, i64, i64, vp, i64]
    L.gpps_views_workspace_bytes.restype = sz
    L.gpps_psi_stats_views.argtypes = [i32, i64, i64, vp, i64, vp, vp, vp, vp, vp, vp, vp, vp, i32,
                                       vp, sz, vp]
    L.gpps_psi_stats_views.restype = i32
    L.gpps_psi_grads_views.argtypes = [i32, i64, i64, vp, i64, vp, vp, vp, vp, vp, vp, vp, vp, vp,
                                       vp, vp, vp, vp, i32, vp, sz, vp]
    L.gpps_psi_grads_views.restype = i32
    L.gpps_probe_sink_bytes.restype = sz
    L.gpps_probe_unit_rates.argtypes = [vp, sz, vp, vp]
    L.gpps_probe_unit_rates.restype = i32
    L.gpps_timing_enable.argtypes = [i32]
    L.gpps_timing_enable.restype = i32
    L.gpps_timing_collect.argtypes = [i32, vp, vp, vp]
    L.gpps_timing_collect.restype = i32
    L.gpps_status_string.argtypes = [i32]
    L.gpps_status_string.restype = ctypes.c_char_p
    L.gpps_version.restype = i32
    _lib = L
    return L


def _check(status: int):
    if status != 0:
        raise GppsError(status, lib().gpps_status_string(status).decode())


def status_string(status: int) -> str:
    return lib().gpps_status_string(status).decode()


def set_path(path: str) -> None:
    """Default kernel path of this module's calls that pass no ``path``:
    'auto', 'generic' or 'mfma'.  The C library itself keeps no path setting;
    every call hands its choice over as a flag."""
    global _default_path
    if path not in PATHS:
        raise ValueError(f"unknown path {path!r}")
    _default_path = path


def get_path() -> str:
    return _default_path


def _flags(path, accumulate=False) -> int:
    path = _default_path if path is None else path
    if path not in PATHS:
        raise ValueError(f"unknown path {path!r}")
    return PATHS[path] | (ACCUMULATE if accumulate else 0)


def route_word_offset(dtype, N: int, M: int, Q: int) -> int:
    return int(lib().gpps_route_word_offset(_dt(dtype), N, M, Q))


def route_taken(workspace, dtype, N: int, M: int, Q: int) -> int:
    """The route word a matrix-core call left in ``workspace`` (synchronises):
    0 = computed on the matrix cores, 1 = the range guard sent it to the
    generic kernels."""
    import torch
    off = route_word_offset(dtype, N, M, Q)
    torch.cuda.synchronize(workspace.device)
    return int(workspace[off:off + 4].cpu().view(torch.int32).item())


def unit_rates(device="cuda:0") -> dict:
    """Measured sustained rates of the device's units (see gpps_probe_unit_rates):
    fp32 vector FMA flops/s, v_exp_f32 results/s, f16 matrix-core flops/s."""
    import torch
    n = int(lib().gpps_probe_sink_bytes())
    sink = torch.empty(n, dtype=torch.uint8, device=device)
    rates = (ctypes.c_double * 3)()
    _check(lib().gpps_probe_unit_rates(sink.data_ptr(), n, ctypes.addressof(rates),
                                       _stream(None)))
    return {"fp32_fma_flops": rates[0], "exp": rates[1], "mfma_f16_flops": rates[2]}


def workspace_bytes(dtype, N: int, M: int, Q: int) -> int:
    return int(lib().gpps_workspace_bytes(_dt(dtype), N, M, Q))


def _dt(dtype) -> int:
    import torch
    if dtype in (torch.float32, "f32", "float32", F32):
        return F32
    if dtype in (torch.float64, "f64", "float64", F64):
        return F64
    raise TypeError(f"unsupported dtype {dtype}")


def _dev_tensor(x, name, dtype, shape, device):
    import torch
    if not isinstance(x, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if x.device.type != "cuda":
        raise ValueError(f"{name} must be a GPU tensor (got {x.device})")
    if x.device != device or x.dtype != dtype:
        raise ValueError(f"{name}: expected {dtype} on {device}, got {x.dtype} on {x.device}")
    if tuple(x.shape) != tuple(shape):
        raise ValueError(f"{name}: expected shape {tuple(shape)}, got {tuple(x.shape)}")
    if not x.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return x


def _host_l(l, Q):
    import numpy as np
    import torch
    if isinstance(l, torch.Tensor):
        l = l.detach().cpu().double().numpy()
    arr = np.ascontiguousarray(np.asarray(l, dtype=np.float64).reshape(-1))
    if arr.shape[0] != Q:
        raise ValueError(f"l: expected {Q} lengthscales, got {arr.shape[0]}")
    return arr


def _workspace(dtype, N, M, Q, device, workspace):
    import torch
    need = workspace_bytes(dtype, N, M, Q)
    if need == 0:
        raise GppsError(2, status_string(2))
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=device)
    elif workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace too small: need {need} bytes")
    return workspace, workspace.numel() * workspace.element_size()


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return ctypes.c_void_p(s.cuda_stream)


def psi_stats(mu, S, Z, sigma_f2, l, *, want_psi1=True, accumulate=False, out=None,
              workspace=None, stream=None, path=None):
    """Forward statistics (section 2, eq. (4); Alg. 1).

    Returns (psi0 [1], Psi1 [N x M] or None, Psi2 [M x M]).  With
    ``accumulate=True`` and ``out=(psi0, Psi1, Psi2)`` the N-summed outputs are
    added to the given tensors (row chunking); Psi1 rows are always written.
    ``path``: 'auto', 'generic' or 'mfma' (default: the module default).
    """
    import torch
    dtype, device = mu.dtype, mu.device
    N, Q = mu.shape
    M = Z.shape[0]
    _dev_tensor(mu, "mu", dtype, (N, Q), device)
    if S is not None:
        _dev_tensor(S, "S", dtype, (N, Q), device)
    _dev_tensor(Z, "Z", dtype, (M, Q), device)
    lh = _host_l(l, Q)
    if out is None:
        psi0 = torch.zeros(1, dtype=dtype, device=device)
        Psi1 = torch.empty((N, M), dtype=dtype, device=device) if want_psi1 else None
        Psi2 = torch.empty((M, M), dtype=dtype, device=device)
    else:
        psi0, Psi1, Psi2 = out
        _dev_tensor(psi0, "psi0", dtype, (1,), device)
        if Psi1 is not None:
            _dev_tensor(Psi1, "Psi1", dtype, (N, M), device)
        _dev_tensor(Psi2, "Psi2", dtype, (M, M), device)
    ws, ws_bytes = _workspace(dtype, N, M, Q, device, workspace)
    _check(lib().gpps_psi_stats(
        _dt(dtype), N, M, Q, mu.data_ptr(), None if S is None else S.data_ptr(), Z.data_ptr(),
        float(sigma_f2), lh.ctypes.data, psi0.data_ptr(), None if Psi1 is None else Psi1.data_ptr(),
        Psi2.data_ptr(), _flags(path, accumulate), ws.data_ptr(), ws_bytes, _stream(stream)))
    return psi0, Psi1, Psi2


def psi_grads(mu, S, Z, sigma_f2, l, dL_dpsi0, dL_dPsi1, dL_dPsi2, *, accumulate=False,
              out=None, workspace=None, stream=None, path=None):
    """Gradients of L = dL_dpsi0 psi0 + <dL_dPsi1, Psi1> + <dL_dPsi2, Psi2> (Alg. 2).

    ``dL_dPsi1`` / ``dL_dPsi2`` may be None (zero).  Returns a dict with dmu, dS
    (N x Q; None when S is None), dZ (M x Q), dsigma_f2 (1), dl (Q).  With
    ``accumulate=True`` and ``out`` (a dict of the same tensors) dZ, dsigma_f2
    and dl are added to.
    """
    import torch
    dtype, device = mu.dtype, mu.device
    N, Q = mu.shape
    M = Z.shape[0]
    _dev_tensor(mu, "mu", dtype, (N, Q), device)
    if S is not None:
        _dev_tensor(S, "S", dtype, (N, Q), device)
    _dev_tensor(Z, "Z", dtype, (M, Q), device)
    if dL_dPsi1 is not None:
        _dev_tensor(dL_dPsi1, "dL_dPsi1", dtype, (N, M), device)
    if dL_dPsi2 is not None:
        _dev_tensor(dL_dPsi2, "dL_dPsi2", dtype, (M, M), device)
    lh = _host_l(l, Q)
    if out is None:
        out = {"dmu": torch.empty((N, Q), dtype=dtype, device=device),
               "dS": None if S is None else torch.empty((N, Q), dtype=dtype, device=device),
               "dZ": torch.zeros((M, Q), dtype=dtype, device=device),
               "dsigma_f2": torch.zeros(1, dtype=dtype, device=device),
               "dl": torch.zeros(Q, dtype=dtype, device=device)}
    else:
        for k, shp in (("dmu", (N, Q)), ("dS", (N, Q)), ("dZ", (M, Q)), ("dsigma_f2", (1,)),
                       ("dl", (Q,))):
            if k == "dS" and S is None:
                continue
            _dev_tensor(out[k], k, dtype, shp, device)
    ws, ws_bytes = _workspace(dtype, N, M, Q, device, workspace)
    ptr = lambda t: None if t is None else t.data_ptr()  # noqa: E731
    _check(lib().gpps_psi_grads(
        _dt(dtype), N, M, Q, mu.data_ptr(), ptr(S), Z.data_ptr(), float(sigma_f2),
        lh.ctypes.data, float(dL_dpsi0), ptr(dL_dPsi1), ptr(dL_dPsi2), out["dmu"].data_ptr(),
        ptr(None if S is None else out["dS"]), out["dZ"].data_ptr(), out["dsigma_f2"].data_ptr(),
        out["dl"].data_ptr(), _flags(path, accumulate), ws.data_ptr(), ws_bytes,
        _stream(stream)))
    return out


def bound_workspace_bytes(dtype, N: int, M: int, Q: int, D: int) -> int:
    return int(lib().gpps_bound_workspace_bytes(_dt(dtype), N, M, Q, D))


def bound(mu, S, Z, Y, sigma_f2, l, beta, jitter=0.0, *, out=None, workspace=None, stream=None,
          path=None):
    """The Bayesian GP-LVM bound L = <F>_q(X) - KL and its gradients (section 2,
    eq. (boundF) with the psi-statistics as expectations, eq. (boundBGPLVM)).

    Y is N x D.  Returns a dict with L (1), dmu, dS (N x Q), dZ (M x Q),
    dsigma_f2 (1), dl (Q) and dbeta (1), all tensors of mu's dtype on its device.
    S = None: known inputs mu = X, the sparse GP regression bound of eq. (boundF)
    itself (no KL term), dmu = dL/dX and dS is None.
    """
    import torch
    dtype, device = mu.dtype, mu.device
    N, Q = mu.shape
    M = Z.shape[0]
    D = Y.shape[1] if Y.dim() == 2 else -1
    _dev_tensor(mu, "mu", dtype, (N, Q), device)
    if S is not None:
        _dev_tensor(S, "S", dtype, (N, Q), device)
    _dev_tensor(Z, "Z", dtype, (M, Q), device)
    _dev_tensor(Y, "Y", dtype, (N, D), device)
    lh = _host_l(l, Q)
    shapes = (("L", (1,)), ("dmu", (N, Q)), ("dS", (N, Q)), ("dZ", (M, Q)), ("dsigma_f2", (1,)),
              ("dl", (Q,)), ("dbeta", (1,)))
    if S is None:
        shapes = tuple(kv for kv in shapes if kv[0] != "dS")
    if out is None:
        out = {k: torch.empty(shp, dtype=dtype, device=device) for k, shp in shapes}
        if S is None:
            out["dS"] = None
    else:
        for k, shp in shapes:
            _dev_tensor(out[k], k, dtype, shp, device)
    need = bound_workspace_bytes(dtype, N, M, Q, D)
    if need == 0:
        raise GppsError(2, status_string(2))
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=device)
    elif workspace.numel() * workspace.element_size() < need:
        raise ValueError(f"workspace too small: need {need} bytes")
    _check(lib().gpps_bound(
        _dt(dtype), N, M, Q, D, mu.data_ptr(), None if S is None else S.data_ptr(), Z.data_ptr(),
        Y.data_ptr(), float(sigma_f2), lh.ctypes.data, float(beta), float(jitter),
        out["L"].data_ptr(), out["dmu"].data_ptr(),
        None if S is None else out["dS"].data_ptr(), out["dZ"].data_ptr(),
        out["dsigma_f2"].data_ptr(), out["dl"].data_ptr(), out["dbeta"].data_ptr(),
        _flags(path), workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream(stream)))
    return out


# ---------------------------------------------------------------- several views (MRD)

def _ptrs(ts):
    arr = (ctypes.c_void_p * len(ts))()
    for i, t in enumerate(ts):
        arr[i] = None if t is None else t.data_ptr()
    return arr


def views_workspace_bytes(dtype, N: int, Ms, Q: int) -> int:
    Ma = (ctypes.c_int64 * len(Ms))(*Ms)
    return int(lib().gpps_views_workspace_bytes(_dt(dtype), len(Ms), N, Ma, Q))


def _views_common(mu, S, Zs, sigma_f2s, ls):
    dtype, device = mu.dtype, mu.device
    N, Q = mu.shape
    V = len(Zs)
    if not (len(sigma_f2s) == len(ls) == V):
        raise ValueError("one Z, sigma_f2 and l per view")
    _dev_tensor(mu, "mu", dtype, (N, Q), device)
    if S is not None:
        _dev_tensor(S, "S", dtype, (N, Q), device)
    Ms = []
    for v, Z in enumerate(Zs):
        _dev_tensor(Z, f"Z[{v}]", dtype, (Z.shape[0], Q), device)
        Ms.append(int(Z.shape[0]))
    lh = np.ascontiguousarray(np.concatenate([_host_l(l, Q) for l in ls]))
    sf = np.ascontiguousarray(np.asarray(sigma_f2s, dtype=np.float64).reshape(V))
    return dtype, device, N, Q, V, Ms, lh, sf


def psi_stats_views(mu, S, Zs, sigma_f2s, ls, *, want_psi1=True, accumulate=False, out=None,
                    workspace=None, stream=None, path=None):
    """Statistics of V views sharing q(X) (section 1, MRD): one (psi0, Psi1, Psi2)
    per view, each as psi_stats would give it.  Returns a list of triples."""
    import torch
    dtype, device, N, Q, V, Ms, lh, sf = _views_common(mu, S, Zs, sigma_f2s, ls)
    if out is None:
        out = [(torch.zeros(1, dtype=dtype, device=device),
                torch.empty((N, M), dtype=dtype, device=device) if want_psi1 else None,
                torch.empty((M, M), dtype=dtype, device=device)) for M in Ms]
    need = views_workspace_bytes(dtype, N, Ms, Q)
    if need == 0:
        raise GppsError(2, status_string(2))
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=device)
    Ma = (ctypes.c_int64 * V)(*Ms)
    _check(lib().gpps_psi_stats_views(
        _dt(dtype), V, N, Ma, Q, mu.data_ptr(), None if S is None else S.data_ptr(),
        _ptrs(Zs), sf.ctypes.data, lh.ctypes.data, _ptrs([o[0] for o in out]),
        _ptrs([o[1] for o in out]), _ptrs([o[2] for o in out]), _flags(path, accumulate),
        workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream(stream)))
    return out


def psi_grads_views(mu, S, Zs, sigma_f2s, ls, dL_dpsi0s, dL_dPsi1s, dL_dPsi2s, *,
                    accumulate=False, out=None, workspace=None, stream=None, path=None):
    """Gradients of L = sum_v L_v over V views sharing q(X): dmu, dS summed over the
    views, and per view dZ, dsigma_f2, dl.  Returns a dict with dmu, dS and lists
    dZ, dsigma_f2, dl."""
    import torch
    dtype, device, N, Q, V, Ms, lh, sf = _views_common(mu, S, Zs, sigma_f2s, ls)
    G1 = list(dL_dPsi1s) if dL_dPsi1s is not None else [None] * V
    G2 = list(dL_dPsi2s) if dL_dPsi2s is not None else [None] * V
    for v in range(V):
        if G1[v] is not None:
            _dev_tensor(G1[v], f"dL_dPsi1[{v}]", dtype, (N, Ms[v]), device)
        if G2[v] is not None:
            _dev_tensor(G2[v], f"dL_dPsi2[{v}]", dtype, (Ms[v], Ms[v]), device)
    if out is None:
        out = {"dmu": torch.empty((N, Q), dtype=dtype, device=device),
               "dS": None if S is None else torch.empty((N, Q), dtype=dtype, device=device),
               "dZ": [torch.zeros((M, Q), dtype=dtype, device=device) for M in Ms],
               "dsigma_f2": [torch.zeros(1, dtype=dtype, device=device) for _ in Ms],
               "dl": [torch.zeros(Q, dtype=dtype, device=device) for _ in Ms]}
    need = views_workspace_bytes(dtype, N, Ms, Q)
    if need == 0:
        raise GppsError(2, status_string(2))
    if workspace is None:
        workspace = torch.empty(need, dtype=torch.uint8, device=device)
    Ma = (ctypes.c_int64 * V)(*Ms)
    d0 = np.ascontiguousarray(np.asarray(dL_dpsi0s, dtype=np.float64).reshape(V))
    _check(lib().gpps_psi_grads_views(
        _dt(dtype), V, N, Ma, Q, mu.data_ptr(), None if S is None else S.data_ptr(), _ptrs(Zs),
        sf.ctypes.data, lh.ctypes.data, d0.ctypes.data, _ptrs(G1), _ptrs(G2),
        out["dmu"].data_ptr(), None if out["dS"] is None else out["dS"].data_ptr(),
        _ptrs(out["dZ"]), _ptrs(out["dsigma_f2"]), _ptrs(out["dl"]), _flags(path, accumulate),
        workspace.data_ptr(), workspace.numel() * workspace.element_size(), _stream(stream)))
    return out
