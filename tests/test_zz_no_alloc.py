"""kb_follow_noalloc: the forward pass with the library's fixed per-GPU
scratch instead of a caller workspace, for callers that cannot allocate.

Called through the C ABI (ctypes on libkbfollow.so) and compared bit for bit
with kb_follow's output on the same inputs -- two calls in a row on one GPU,
the second on a smaller KB and batch, so the scratch still holds the first
call's partials -- and with the oracle (bit-exact on integer inputs, rtol
1e-5 / atol 1e-7 otherwise).  A KB whose workspace exceeds the scratch is
refused before anything is enqueued.
"""
import ctypes

import numpy as np
import pytest

import kbgen
import oracle
from gpu_util import assert_bitexact, assert_close, to_em, from_em

pytestmark = pytest.mark.gpu

SCRATCH_BYTES = 64 << 20  # KB_NOALLOC_SCRATCH_BYTES


@pytest.fixture(scope="module")
def kbf():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2002_06115_amd as kbf
    return kbf


def _stream():
    import torch
    return ctypes.c_void_p(torch.cuda.current_stream().cuda_stream)


def noalloc(kbf, gkb, X, R, Y):
    """Y = follow(X, R) through kb_follow_noalloc; returns the status."""
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    return kbf._lib.kb_follow_noalloc(gkb._handle, X.shape[1], p(X), p(R), p(Y), _stream())


def with_workspace(kbf, gkb, X, R, Y):
    """Y = follow(X, R) through kb_follow with a workspace of its own."""
    import torch
    b = X.shape[1]
    n = gkb.workspace_size(b)
    ws = torch.empty(max(n, 1), dtype=torch.uint8, device="cuda")
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    st = kbf._lib.kb_follow(gkb._handle, b, p(X), p(R), p(Y), p(ws) if n else None, n, _stream())
    torch.cuda.synchronize()
    return st


def check_case(kbf, w, integer):
    import torch
    kb = kbgen.make_kb(w)
    if integer:
        X, R, _ = kbgen.make_integer_inputs(w)
    else:
        X, R = kbgen.make_x(w), kbgen.make_r(w)
    print(f"[noalloc] {w.label} integer={integer}", flush=True)
    gkb = kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations)
    need = gkb.workspace_size(w.batch)
    assert need <= SCRATCH_BYTES
    Xe, Re = to_em(X), to_em(R)
    Y = torch.full_like(Xe, float("nan"))
    assert noalloc(kbf, gkb, Xe, Re, Y) == kbf.KB_OK, kbf._lib.kb_last_error()
    Yref = torch.full_like(Xe, float("nan"))
    assert with_workspace(kbf, gkb, Xe, Re, Yref) == kbf.KB_OK
    torch.cuda.synchronize()
    assert torch.equal(Y.view(torch.int32), Yref.view(torch.int32)), "differs from kb_follow"
    want = oracle.follow(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations, X, R)
    (assert_bitexact if integer else assert_close)(from_em(Y), want, f"{w.name} noalloc Y")
    info = gkb.info()
    gkb.close()
    return need, info


def test_two_calls_second_smaller(kbf):
    """A KB with split rows (hub objects), then a smaller KB and batch whose
    partials land in scratch that still holds the first call's."""
    need1, info1 = check_case(kbf, kbgen.METAQA, integer=False)
    assert info1["n_slots"][0] > 0 and need1 > 0, "the first KB must use the scratch"
    w2 = kbgen.TINY
    need2, info2 = check_case(kbf, w2, integer=True)
    assert 0 < need2 < need1 and info2["n_slots"][0] > 0
    # And once more on the first KB, after the second.
    check_case(kbf, kbgen.METAQA, integer=False)


def test_kb_without_partials(kbf):
    """No row crosses a chunk: no scratch is needed and none is addressed."""
    import torch
    s = np.array([0, 1, 2], np.int32)
    r = np.array([0, 1, 0], np.int32)
    o = np.array([1, 2, 0], np.int32)
    gkb = kbf.KB(s, r, o, 3, 2)
    assert gkb.workspace_size(4) == 0
    X = torch.arange(12, dtype=torch.float32, device="cuda").reshape(3, 4).contiguous()
    R = torch.tensor([[1.0, 2.0, 3.0, 4.0], [0.5, 0.5, 0.5, 0.5]], device="cuda")
    Y = torch.full_like(X, float("nan"))
    assert noalloc(kbf, gkb, X, R, Y) == kbf.KB_OK
    torch.cuda.synchronize()
    want = oracle.follow(s, r, o, 3, 2, X.t().contiguous().cpu().numpy(),
                         R.t().contiguous().cpu().numpy())
    assert_bitexact(from_em(Y), want, "three-triple KB")
    gkb.close()


def test_refuses_a_kb_larger_than_the_scratch(kbf, monkeypatch):
    """A KB whose partials exceed the scratch: KB_EINVAL before any launch,
    the output untouched."""
    import torch
    monkeypatch.setenv("KBFOLLOW_CHUNK", "16")
    g = np.random.default_rng(5)
    n_t = 300_000
    s = g.integers(0, 1000, n_t).astype(np.int32)
    o = g.integers(0, 100, n_t).astype(np.int32)   # 100 hub rows
    r = g.integers(0, 4, n_t).astype(np.int32)
    gkb = kbf.KB(s, r, o, 1000, 4)
    b = 512
    assert gkb.workspace_size(b) > SCRATCH_BYTES
    X = torch.ones((1000, b), device="cuda")
    R = torch.ones((4, b), device="cuda")
    Y = torch.full_like(X, 7.0)
    st = noalloc(kbf, gkb, X, R, Y)
    assert st == kbf.KB_EINVAL
    assert b"fixed scratch" in kbf._lib.kb_last_error()
    torch.cuda.synchronize()
    assert bool((Y == 7.0).all())
    # The same KB at a batch that fits runs and matches kb_follow.
    b = 8
    assert gkb.workspace_size(b) <= SCRATCH_BYTES
    X, R = X[:, :b].contiguous(), R[:, :b].contiguous()
    Y = torch.full_like(X, float("nan"))
    assert noalloc(kbf, gkb, X, R, Y) == kbf.KB_OK
    Yref = torch.empty_like(X)
    assert with_workspace(kbf, gkb, X, R, Yref) == kbf.KB_OK
    assert torch.equal(Y.view(torch.int32), Yref.view(torch.int32))
    gkb.close()
