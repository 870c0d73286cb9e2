"""The gather-rate probe bench.py uses to measure the memory system's own rate
for a pass's row reads (a measurement helper, not part of the follow path).

Host: the probe library is built and exports its entry point, and rejects bad
arguments without touching the GPU.  GPU: the probe really reads the rows it
is timed on -- its per-chunk sums equal the sums of the indexed rows (integer
values, so float addition is exact in any order).
"""
import ctypes
import os

import numpy as np
import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROBE = os.path.join(ROOT, "paper_2002_06115_amd", "_lib", "libkbprobe.so")


def _lib():
    lib = ctypes.CDLL(PROBE)
    lib.kbp_gather_time.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                    ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                    ctypes.c_int32, ctypes.c_void_p,
                                    ctypes.POINTER(ctypes.c_float)]
    return lib


def test_probe_library_exports_entry_points():
    assert os.path.exists(PROBE), "run __graft_entry__.build() first"
    lib = ctypes.CDLL(PROBE)
    assert hasattr(lib, "kbp_gather_time")
    assert hasattr(lib, "kbp_stream_read_time")
    assert hasattr(lib, "kbp_stream_copy_time")
    assert hasattr(lib, "kbp_stream_write_time")


def _copy_lib():
    lib = ctypes.CDLL(PROBE)
    lib.kbp_stream_copy_time.argtypes = [ctypes.c_void_p, ctypes.c_void_p, ctypes.c_int64,
                                         ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p,
                                         ctypes.POINTER(ctypes.c_float)]
    return lib


@pytest.mark.parametrize("n4,blocks,reps", [(0, 4, 1), (16, 0, 1), (16, 4, 0)])
def test_stream_copy_rejects_bad_arguments(n4, blocks, reps):
    dummy = ctypes.c_void_p(16)  # never dereferenced: arguments are checked first
    ms = ctypes.c_float()
    assert _copy_lib().kbp_stream_copy_time(dummy, dummy, n4, blocks, reps, None,
                                            ctypes.byref(ms)) == -1


def _write_lib():
    lib = ctypes.CDLL(PROBE)
    lib.kbp_stream_write_time.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                          ctypes.c_int32, ctypes.c_void_p,
                                          ctypes.POINTER(ctypes.c_float)]
    return lib


@pytest.mark.parametrize("n4,blocks,reps", [(0, 4, 1), (16, 0, 1), (16, 4, 0)])
def test_stream_write_rejects_bad_arguments(n4, blocks, reps):
    dummy = ctypes.c_void_p(16)  # never dereferenced: arguments are checked first
    ms = ctypes.c_float()
    assert _write_lib().kbp_stream_write_time(dummy, n4, blocks, reps, None,
                                              ctypes.byref(ms)) == -1


@pytest.mark.parametrize("n4,blocks,reps", [(0, 4, 1), (16, 0, 1), (16, 4, 0)])
def test_stream_read_rejects_bad_arguments(n4, blocks, reps):
    lib = ctypes.CDLL(PROBE)
    lib.kbp_stream_read_time.argtypes = [ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32,
                                         ctypes.c_void_p, ctypes.c_int32, ctypes.c_void_p,
                                         ctypes.POINTER(ctypes.c_float)]
    dummy = ctypes.c_void_p(16)  # never dereferenced: arguments are checked first
    ms = ctypes.c_float()
    assert lib.kbp_stream_read_time(dummy, n4, blocks, dummy, reps, None, ctypes.byref(ms)) == -1


@pytest.mark.parametrize("n,chunk,b,reps", [(0, 256, 32, 1), (10, 0, 32, 1), (10, 256, 30, 1),
                                            (10, 256, 260, 1), (10, 256, 32, 0)])
def test_probe_rejects_bad_arguments(n, chunk, b, reps):
    lib = _lib()
    dummy = ctypes.c_void_p(16)  # never dereferenced: arguments are checked first
    ms = ctypes.c_float()
    assert lib.kbp_gather_time(dummy, n, chunk, dummy, b, dummy, reps, None,
                               ctypes.byref(ms)) == -1


@pytest.mark.gpu
@pytest.mark.parametrize("b,n,chunk", [(32, 5000, 256), (8, 777, 64), (256, 3001, 128),
                                       (4, 1, 256)])
def test_probe_sums_the_indexed_rows(b, n, chunk):
    import torch
    rows = 1000
    rng = np.random.default_rng(7)
    X = rng.integers(-8, 9, size=(rows, b)).astype(np.float32)
    idx = rng.integers(0, rows, size=n).astype(np.int32)
    n_chunks = -(-n // chunk)
    Xd = torch.from_numpy(X).cuda()
    idxd = torch.from_numpy(idx).cuda()
    out = torch.full((n_chunks * b,), float("nan"), device="cuda")
    ms = ctypes.c_float()
    rc = _lib().kbp_gather_time(idxd.data_ptr(), n, chunk, Xd.data_ptr(), b, out.data_ptr(), 2,
                                None, ctypes.byref(ms))
    assert rc == 0
    assert ms.value > 0
    want = np.stack([X[idx[g * chunk:(g + 1) * chunk]].sum(axis=0) for g in range(n_chunks)])
    np.testing.assert_array_equal(out.cpu().numpy().reshape(n_chunks, b), want)


@pytest.mark.gpu
def test_stream_copy_copies():
    import torch
    src = torch.arange(4 * 5000, dtype=torch.float32, device="cuda")
    dst = torch.full_like(src, float("nan"))
    ms = ctypes.c_float()
    assert _copy_lib().kbp_stream_copy_time(src.data_ptr(), dst.data_ptr(), 5000, 7, 2, None,
                                            ctypes.byref(ms)) == 0
    assert torch.equal(src, dst) and ms.value > 0


@pytest.mark.gpu
def test_stream_write_zero_fills():
    import torch
    dst = torch.full((4 * 5003,), float("nan"), device="cuda")
    guard = torch.full((64,), 7.0, device="cuda")
    ms = ctypes.c_float()
    assert _write_lib().kbp_stream_write_time(dst.data_ptr(), 5000, 7, 2, None,
                                              ctypes.byref(ms)) == 0
    torch.cuda.synchronize()
    assert torch.equal(dst[:20000], torch.zeros(20000, device="cuda")) and ms.value > 0
    assert torch.isnan(dst[20000:]).all()  # only n_float4 float4s written
    assert torch.equal(guard, torch.full((64,), 7.0, device="cuda"))
