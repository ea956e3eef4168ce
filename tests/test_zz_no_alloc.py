"""The allocation-free entry point (gpps_psi_stats_noalloc, static device
scratch) against gpps_psi_stats with a caller workspace, through the C ABI:
two calls in a row, the second with a smaller input, each bitwise equal to the
workspace entry point (same kernels and launch shapes), plus an oversized call
that is refused before any launch."""
import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_1410_4984_amd as gpps  # noqa: E402
from paper_1410_4984_amd import synth  # noqa: E402

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
SCRATCH_BYTES = 64 << 20


def _lib():
    L = gpps.lib()
    i64, vp, d, i32 = ctypes.c_int64, ctypes.c_void_p, ctypes.c_double, ctypes.c_int
    L.gpps_psi_stats_noalloc.argtypes = [i32, i64, i64, i64, vp, vp, vp, d, vp, vp, vp, vp, i32, vp]
    L.gpps_psi_stats_noalloc.restype = i32
    return L


def _call(fn_noalloc, inp, dtype, flags=0):
    t = {k: torch.tensor(v, dtype=dtype, device=DEV) for k, v in inp.items()
         if isinstance(v, np.ndarray) and k in ("mu", "S", "Z")}
    N, Q = inp["mu"].shape
    M = inp["Z"].shape[0]
    psi0 = torch.full((1,), 7.0, dtype=dtype, device=DEV)
    P1 = torch.full((N, M), 7.0, dtype=dtype, device=DEV)
    P2 = torch.full((M, M), 7.0, dtype=dtype, device=DEV)
    l = np.ascontiguousarray(inp["l"], dtype=np.float64)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    dt = 0 if dtype == torch.float32 else 1
    L = _lib()
    if fn_noalloc:
        st = L.gpps_psi_stats_noalloc(dt, N, M, Q, t["mu"].data_ptr(), t["S"].data_ptr(),
                                      t["Z"].data_ptr(), float(inp["sigma_f2"]), l.ctypes.data,
                                      psi0.data_ptr(), P1.data_ptr(), P2.data_ptr(), flags, stream)
    else:
        need = L.gpps_workspace_bytes(dt, N, M, Q)
        ws = torch.empty(need, dtype=torch.uint8, device=DEV)
        st = L.gpps_psi_stats(dt, N, M, Q, t["mu"].data_ptr(), t["S"].data_ptr(),
                              t["Z"].data_ptr(), float(inp["sigma_f2"]), l.ctypes.data,
                              psi0.data_ptr(), P1.data_ptr(), P2.data_ptr(), flags,
                              ws.data_ptr(), need, stream)
    assert st == 0, gpps.status_string(st)
    torch.cuda.synchronize()
    return psi0.cpu().numpy(), P1.cpu().numpy(), P2.cpu().numpy()


@pytest.mark.parametrize("dtype", [torch.float32, torch.float64])
def test_noalloc_matches_workspace_entry_point_twice(dtype):
    # first a larger call, then a smaller one on the same (shared) scratch
    for N, M, Q, seed in ((3000, 70, 8, 51), (700, 33, 5, 52)):
        inp = synth.random_inputs(N, M, Q, seed=seed)
        if dtype == torch.float32:
            inp = synth.to_f32(inp)
        assert gpps.workspace_bytes(dtype, N, M, Q) <= SCRATCH_BYTES
        a = _call(True, inp, dtype)
        b = _call(False, inp, dtype)
        for x, y, name in zip(a, b, ("psi0", "Psi1", "Psi2")):
            assert np.array_equal(x, y), (N, M, Q, name)
        assert np.array_equal(a[2], a[2].T)


def test_noalloc_accumulates_row_chunks():
    """Row chunks through the static scratch with GPPS_ACCUMULATE add up to the
    whole call (within fp32 rounding of the different summation order)."""
    inp = synth.to_f32(synth.random_inputs(2000, 50, 6, seed=53))
    whole = _call(False, inp, torch.float32)
    L = _lib()
    t = {k: torch.tensor(inp[k], dtype=torch.float32, device=DEV) for k in ("mu", "S", "Z")}
    psi0 = torch.zeros(1, device=DEV)
    P1 = torch.empty((2000, 50), device=DEV)
    P2 = torch.zeros((50, 50), device=DEV)
    l = np.ascontiguousarray(inp["l"], dtype=np.float64)
    stream = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    for i, (r0, r1) in enumerate(((0, 1200), (1200, 2000))):
        st = L.gpps_psi_stats_noalloc(0, r1 - r0, 50, 6, t["mu"][r0:r1].data_ptr(),
                                      t["S"][r0:r1].data_ptr(), t["Z"].data_ptr(),
                                      float(inp["sigma_f2"]), l.ctypes.data, psi0.data_ptr(),
                                      P1[r0:r1].data_ptr(), P2.data_ptr(), 1 if i else 0, stream)
        assert st == 0
    torch.cuda.synchronize()
    assert np.array_equal(P1.cpu().numpy(), whole[1])
    d = np.linalg.norm(P2.cpu().numpy() - whole[2]) / np.linalg.norm(whole[2])
    assert d <= 1e-6, d


def test_noalloc_refuses_oversized_calls():
    L = _lib()
    N, M, Q = 1_000_000, 512, 30
    assert gpps.workspace_bytes("f32", N, M, Q) > SCRATCH_BYTES
    fake = 0x7F0000000000   # never dereferenced: the size check stops the call first
    l = (ctypes.c_double * Q)(*([1.0] * Q))
    st = L.gpps_psi_stats_noalloc(0, N, M, Q, fake, fake, fake, 1.0, l, fake, fake, fake, 0, None)
    assert st == 5   # GPPS_ERR_WORKSPACE
