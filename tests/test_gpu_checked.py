"""The checked build (KBFOLLOW_CHECKED): every row, slot and combine index the
kernels use is validated against its table.  On every plan shape -- small and
large chunks, split hub rows over several combine levels, empty rows, soft
weights, the residual hop -- the checked library must count no violation and
produce bitwise the results of the normal library (the checks never change a
valid index).
"""
import ctypes

import numpy as np
import pytest

import kbgen
from gpu_util import to_em

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def libs():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2002_06115_amd as kbf
    from paper_2002_06115_amd import build as kbuild
    lib = ctypes.CDLL(kbuild.CHECKED_LIB)
    P, I64, I32, SZ = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int32, ctypes.c_size_t
    lib.kb_create.argtypes = [I64, I64, I64, P, P, P, P, P, ctypes.POINTER(P)]
    lib.kb_destroy.argtypes = [P]
    lib.kb_workspace_size.argtypes = [P, I32]
    lib.kb_workspace_size.restype = SZ
    lib.kb_follow_residual.argtypes = [P, I32, P, P, ctypes.c_float, P, P, SZ, P]
    lib.kb_follow_backward_residual.argtypes = [P, I32, P, P, P, ctypes.c_float, P, P, P, SZ, P]
    lib.kb_checked_violations.argtypes = [ctypes.POINTER(ctypes.c_uint64), I32]
    return kbf, lib


def run_checked(lib, kb, w, X, R, dY, weight, gamma):
    """Forward and backward through the checked library (residual hop with
    gamma; gamma = 0 is the plain follow)."""
    import torch
    ptr = lambda a: a.ctypes.data_as(ctypes.c_void_p)
    h = ctypes.c_void_p()
    arr = [np.ascontiguousarray(a, np.int32) for a in (kb.subj, kb.rel, kb.obj)]
    wt = None if weight is None else np.ascontiguousarray(weight, np.float32)
    assert lib.kb_create(w.n_entities, w.n_relations, kb.n_triples, *map(ptr, arr),
                         None if wt is None else ptr(wt), None, ctypes.byref(h)) == 0
    b = X.shape[1]
    n_ws = lib.kb_workspace_size(h, b)
    ws = torch.empty(max(1, n_ws), dtype=torch.uint8, device="cuda")
    Y, dX, dR = torch.empty_like(X), torch.empty_like(X), torch.empty_like(R)
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    s = ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)
    assert lib.kb_follow_residual(h, b, p(X), p(R), gamma, p(Y), p(ws), n_ws, s) == 0
    assert lib.kb_follow_backward_residual(h, b, p(X), p(R), p(dY), gamma, p(dX), p(dR), p(ws),
                                           n_ws, s) == 0
    torch.cuda.synchronize()
    lib.kb_destroy(h)
    return Y, dX, dR


CASES = {
    "tiny": (kbgen.TINY, None, None),
    "metaqa_s": (kbgen.METAQA.scaled(20_000, 150_000, batch=32, tag=5), None, None),
    "large_s chunk 16": (kbgen.LARGE.scaled(200_000, 1_000_000, tag=1), "16", None),
    "train_s weighted": (kbgen.TRAIN.scaled(50_000, 400_000, batch=64, n_relations=50, tag=2),
                         None, 0.5),
}


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("gamma", [0.0, 1.0])
def test_checked_build_counts_nothing_and_matches(libs, name, gamma, monkeypatch):
    import torch
    kbf, lib = libs
    w, chunk, weight_scale = CASES[name]
    if chunk:
        monkeypatch.setenv("KBFOLLOW_CHUNK", chunk)
        monkeypatch.setenv("KBFOLLOW_REL_CHUNK", chunk)
    kb = kbgen.make_kb(w)
    weight = None
    if weight_scale is not None:
        weight = np.random.default_rng(9).uniform(0.1, 2.0, kb.n_triples).astype(np.float32)
    X, R, dY = to_em(kbgen.make_x(w)), to_em(kbgen.make_r(w)), to_em(kbgen.make_dy(w))
    count = ctypes.c_uint64(1)
    assert lib.kb_checked_violations(ctypes.byref(count), 1) == 0
    got = run_checked(lib, kb, w, X, R, dY, weight, gamma)
    assert lib.kb_checked_violations(ctypes.byref(count), 1) == 0
    assert count.value == 0, f"{count.value} index violations"
    gkb = kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations, weight=weight)
    want_y = gkb.follow(X, R, residual=gamma)
    want_dx, want_dr = gkb.follow_backward(X, R, dY, residual=gamma)
    torch.cuda.synchronize()
    bits = lambda t: t.view(torch.int32)
    for n, g, e in zip(("Y", "dX", "dR"), got, (want_y, want_dx, want_dr)):
        assert torch.equal(bits(g), bits(e)), f"{name}: checked {n} differs"
    gkb.close()
