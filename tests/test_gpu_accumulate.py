"""The accumulating follow, Y = follow(X, R) + gamma * Z (kb_follow_accumulate),
against the oracle: an independent Z and Z = Y in place, on KBs with hubs
split over many chunks (the combine adds gamma * Z), empty rows (the fill
writes gamma * Z), soft weights and odd batch widths; bit for bit on integer
inputs; Z = X reproduces the residual hop bit for bit; bad overlaps are
refused."""
import ctypes

import numpy as np
import pytest

import oracle
from gpu_util import assert_bitexact, assert_close, from_em, to_em

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kbf():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2002_06115_amd as kbf
    return kbf


def hub_kb(seed, n_e=3000, n_r=9, n_t=40_000):
    g = np.random.default_rng(seed)
    # hubs on both sides and a block of entities no triple reaches
    s = np.where(g.random(n_t) < 0.3, g.integers(0, 3, n_t), g.integers(0, n_e - 500, n_t))
    o = np.where(g.random(n_t) < 0.3, g.integers(0, 3, n_t), g.integers(0, n_e - 500, n_t))
    r = g.integers(0, n_r, n_t)
    return s.astype(np.int32), r.astype(np.int32), o.astype(np.int32), n_e, n_r


@pytest.mark.parametrize("b", [4, 5, 32, 260])
@pytest.mark.parametrize("gamma", [1.0, -0.5])
@pytest.mark.parametrize("weighted", [False, True])
def test_accumulate_matches_oracle(kbf, b, gamma, weighted, monkeypatch):
    monkeypatch.setenv("KBFOLLOW_CHUNK", "32")  # hub rows over many chunks
    s, r, o, n_e, n_r = hub_kb(b + 3 * weighted)
    g = np.random.default_rng(b)
    w = g.uniform(0.1, 2.0, len(s)).astype(np.float32) if weighted else None
    X = g.standard_normal((b, n_e)).astype(np.float32)
    R = g.standard_normal((b, n_r)).astype(np.float32)
    Z = g.standard_normal((b, n_e)).astype(np.float32)
    kb = kbf.KB(s, r, o, n_e, n_r, weight=w)
    want = oracle.follow_accumulate(s, r, o, n_e, n_r, X, R, Z, gamma, weight=w)
    got = from_em(kb.follow_accumulate(to_em(X), to_em(R), to_em(Z), gamma))
    assert_close(got, want, f"b={b} gamma={gamma} weighted={weighted}")
    # In place: Z is the output.
    Yz = to_em(Z)
    kb.follow_accumulate(to_em(X), to_em(R), Yz, gamma, out=Yz)
    assert_close(from_em(Yz), want, "in place")
    kb.close()


def test_accumulate_integer_exact_in_place(kbf):
    import torch
    s, r, o, n_e, n_r = hub_kb(11)
    b = 8
    g = np.random.default_rng(11)
    X = g.integers(0, 3, (b, n_e)).astype(np.float32)
    R = g.integers(0, 2, (b, n_r)).astype(np.float32)
    Z = g.integers(-4, 5, (b, n_e)).astype(np.float32)
    kb = kbf.KB(s, r, o, n_e, n_r)
    want = oracle.follow_accumulate(s, r, o, n_e, n_r, X, R, Z, 2.0)
    Y = to_em(Z)
    kb.follow_accumulate(to_em(X), to_em(R), Y, 2.0, out=Y)
    assert_bitexact(from_em(Y), want, "integer in place")
    # Twice in place adds the hop twice: Z + 2 (f + f) = oracle with Z' = Y.
    kb.follow_accumulate(to_em(X), to_em(R), Y, 1.0, out=Y)
    want2 = oracle.follow_accumulate(s, r, o, n_e, n_r, X, R, want, 1.0)
    assert_bitexact(from_em(Y), want2, "second accumulation")
    torch.cuda.synchronize()
    kb.close()


def test_z_equal_x_is_the_residual_hop(kbf):
    import torch
    s, r, o, n_e, n_r = hub_kb(12)
    b = 32
    g = np.random.default_rng(12)
    X = to_em(g.standard_normal((b, n_e)).astype(np.float32))
    R = to_em(g.standard_normal((b, n_r)).astype(np.float32))
    kb = kbf.KB(s, r, o, n_e, n_r)
    a = kb.follow_accumulate(X, R, X, 0.75)
    c = kb.follow(X, R, residual=0.75)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), c.view(torch.int32))
    kb.close()


def test_accumulate_is_deterministic(kbf):
    import torch
    s, r, o, n_e, n_r = hub_kb(13)
    b = 32
    g = np.random.default_rng(13)
    X, R, Z = (to_em(g.standard_normal((b, n)).astype(np.float32)) for n in (n_e, n_r, n_e))
    kb = kbf.KB(s, r, o, n_e, n_r)
    a = kb.follow_accumulate(X, R, Z, -1.5)
    c = kb.follow_accumulate(X, R, Z, -1.5)
    torch.cuda.synchronize()
    assert torch.equal(a.view(torch.int32), c.view(torch.int32))
    kb.close()


def test_accumulate_refuses_partial_overlap(kbf):
    import torch
    s, r, o, n_e, n_r = hub_kb(14)
    b = 4
    kb = kbf.KB(s, r, o, n_e, n_r)
    X = torch.rand(n_e, b, device="cuda")
    R = torch.rand(n_r, b, device="cuda")
    big = torch.zeros(n_e + 8, b, device="cuda")
    Y, Zshift = big[:n_e], big[4:]          # Z starts 4 rows into Y
    lib = ctypes.CDLL(kbf.LIB_PATH)
    P = ctypes.c_void_p
    lib.kb_follow_accumulate.argtypes = [P, ctypes.c_int32, P, P, P, ctypes.c_float, P, P,
                                         ctypes.c_size_t, P]
    ws = kb.workspace(b)
    nws = 0 if ws is None else ws.numel()
    p = lambda t: P(t.data_ptr())
    wsp = None if ws is None else p(ws)
    rc = lib.kb_follow_accumulate(kb._handle, b, p(X), p(R), p(Zshift), 1.0, p(Y), wsp, nws, None)
    assert rc == kbf.KB_EINVAL
    rc = lib.kb_follow_accumulate(kb._handle, b, p(X), p(R), None, 1.0, p(Y), wsp, nws, None)
    assert rc == kbf.KB_EINVAL
    assert torch.count_nonzero(big) == 0  # nothing was launched
    kb.close()
