"""GPU edge cases against the oracle: empty KB, odd batch sizes, one-hub KBs,
a single relation, a single entity with duplicate self-loops, empty rows next
to 2^20-triple rows, and argument errors."""
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


def both(kbf, s, r, o, n_e, n_r, X, R, dY, exact, label, weight=None):
    print(f"[edge] {label} NE={n_e} NR={n_r} NT={len(s)} b={X.shape[0]}", flush=True)
    kb = kbf.KB(s, r, o, n_e, n_r, weight=weight)
    Y = from_em(kb.follow(to_em(X), to_em(R)))
    dX, dR = kb.follow_backward(to_em(X), to_em(R), to_em(dY))
    got = (Y, from_em(dX), from_em(dR))
    Yo = oracle.follow(s, r, o, n_e, n_r, X, R, weight=weight)
    dXo, dRo = oracle.follow_backward(s, r, o, n_e, n_r, X, R, dY, weight=weight)
    for name, g, e in zip(("Y", "dX", "dR"), got, (Yo, dXo, dRo)):
        (assert_bitexact if exact else assert_close)(g, e, f"{label} {name}")
    return kb


def rand_kb(seed, n_e, n_r, n_t):
    g = np.random.default_rng(seed)
    return (g.integers(0, n_e, n_t).astype(np.int32), g.integers(0, n_r, n_t).astype(np.int32),
            g.integers(0, n_e, n_t).astype(np.int32))


def rand_io(seed, b, n_e, n_r):
    g = np.random.default_rng(seed)
    return (g.standard_normal((b, n_e)).astype(np.float32), g.standard_normal((b, n_r)).astype(np.float32),
            g.standard_normal((b, n_e)).astype(np.float32))


@pytest.mark.parametrize("b", [1, 2, 3, 4, 5, 8, 12, 33, 64, 100, 260, 300, 513, 4095, 4096])
def test_batch_sizes(kbf, b):
    # Rows are gathered as records of a structured buffer whose stride is the
    # row's bytes, at most 16383: b = 4095 is the widest row read that way,
    # b = 4096 takes plain loads.
    n_e, n_r = 700, 6
    s, r, o = rand_kb(b, n_e, n_r, 6000)
    X, R, dY = rand_io(b, b, n_e, n_r)
    both(kbf, s, r, o, n_e, n_r, X, R, dY, False, f"b={b}")


def test_empty_kb(kbf):
    e = np.zeros(0, np.int32)
    X, R, dY = rand_io(1, 4, 50, 3)
    both(kbf, e, e, e, 50, 3, X, R, dY, True, "empty")


def test_one_hub_holds_every_triple(kbf):
    n_e, n_r, n_t = 20_000, 4, 300_000
    g = np.random.default_rng(2)
    s = np.full(n_t, 17, np.int32)
    r = g.integers(0, n_r, n_t).astype(np.int32)
    o = g.integers(0, n_e, n_t).astype(np.int32)
    X, R, dY = rand_io(2, 32, n_e, n_r)
    both(kbf, s, r, o, n_e, n_r, X, R, dY, False, "subject hub")
    both(kbf, o, r, s, n_e, n_r, X, R, dY, False, "object hub")


def test_single_relation(kbf):
    s, r, o = rand_kb(3, 5000, 1, 40_000)
    X, R, dY = rand_io(3, 16, 5000, 1)
    both(kbf, s, r, o, 5000, 1, X, R, dY, False, "N_R=1")


def test_single_entity_duplicate_self_loops(kbf):
    n_t = 5000
    s = np.zeros(n_t, np.int32)
    r = (np.arange(n_t) % 3).astype(np.int32)
    X = np.full((8, 1), 1.0, np.float32)
    R = np.ones((8, 3), np.float32)
    dY = np.ones((8, 1), np.float32)
    both(kbf, s, r, s, 1, 3, X, R, dY, True, "N_E=1 duplicates")


def test_empty_rows_beside_huge_rows(kbf):
    # Two rows of 2^20 triples (several combine levels), the rest mostly empty.
    n_e, n_r = 50_000, 5
    g = np.random.default_rng(4)
    big = 1 << 20
    s = np.concatenate([np.full(big, 11), np.full(big, 40_000), g.integers(0, 100, 5000)]).astype(np.int32)
    o = np.concatenate([g.integers(0, 30, big), g.integers(0, n_e, big), np.full(5000, 7)]).astype(np.int32)
    r = g.integers(0, n_r, len(s)).astype(np.int32)
    Xi = (g.random((4, n_e)) < 0.3).astype(np.float32)
    Ri = np.zeros((4, n_r), np.float32)
    Ri[np.arange(4), g.integers(0, n_r, 4)] = 1.0
    both(kbf, s, r, o, n_e, n_r, Xi, Ri, np.ones((4, n_e), np.float32), True, "hubs+empty int")
    X, R, dY = rand_io(4, 32, n_e, n_r)
    kb = both(kbf, s, r, o, n_e, n_r, X, R, dY, False, "hubs+empty real")
    info = kb.info()
    assert max(info["n_levels"]) >= 2 and info["n_empty_rows"][1] > 0


def test_argument_errors(kbf):
    import torch
    s, r, o = rand_kb(5, 100, 3, 2000)
    kb = kbf.KB(s, r, o, 100, 3)
    X = torch.zeros((100, 8), device="cuda")
    R = torch.zeros((3, 8), device="cuda")
    lib = kbf._lib
    h = kb._handle
    p = lambda t: ctypes.c_void_p(t.data_ptr())
    ws = kb.workspace(8)
    nws = 0 if ws is None else ws.numel()
    wsp = None if ws is None else p(ws)
    assert lib.kb_follow(h, 0, p(X), p(R), p(X), wsp, nws, None) == kbf.KB_EINVAL       # b < 1
    assert lib.kb_follow(h, 8, p(X), p(R), p(X), wsp, nws, None) == kbf.KB_EINVAL       # Y aliases X
    assert lib.kb_follow(h, 8, None, p(R), p(X), wsp, nws, None) == kbf.KB_EINVAL       # NULL X
    Xo = torch.zeros(100 * 8 + 1, device="cuda")[1:].view(100, 8)
    Y = torch.zeros((100, 8), device="cuda")
    assert lib.kb_follow(h, 8, p(Xo), p(R), p(Y), wsp, nws, None) == kbf.KB_EINVAL      # misaligned
    need = lib.kb_workspace_size(h, 8)
    assert need > 0  # rows of this small KB cross its 16-entry chunks
    # A workspace overlapping an input or an output is refused before any launch.
    big = torch.zeros(need // 4 + 2 * 100 * 8, device="cuda")
    inside = big[: 100 * 8].view(100, 8)
    dX = torch.zeros((100, 8), device="cuda")
    dR = torch.zeros((3, 8), device="cuda")
    assert lib.kb_follow(h, 8, p(inside), p(R), p(Y), p(big), need, None) == kbf.KB_EINVAL
    assert lib.kb_follow(h, 8, p(X), p(R), p(inside), p(big), need, None) == kbf.KB_EINVAL
    assert lib.kb_follow_backward(h, 8, p(X), p(R), p(Y), p(inside), p(dR), p(big), need,
                                  None) == kbf.KB_EINVAL
    assert b"overlaps" in lib.kb_last_error()
    assert lib.kb_follow_backward(h, 8, p(X), p(R), p(Y), p(dX), p(dR), wsp, nws,
                                  None) == kbf.KB_OK
    torch.cuda.synchronize()
    with pytest.raises(ValueError):
        kb.follow(X, torch.zeros((3, 7), device="cuda"))


@pytest.mark.parametrize("chunk,fan_in", [(2, 2), (8, 32), (16, 3), (24, 2), (40, 4), (64, 2), (4096, 32)])
def test_chunk_and_combine_plans(kbf, chunk, fan_in, monkeypatch):
    # Tiny chunks put a marker every few entries: runs cut by chunk ends,
    # no-op markers, rows split into many slots, deep combine trees.  Chunks
    # of an odd number of 8-entry steps end on a lone step of the paired
    # entry fetch (8-lane groups: b = 7 and 32, and dR at b = 256).
    monkeypatch.setenv("KBFOLLOW_CHUNK", str(chunk))
    monkeypatch.setenv("KBFOLLOW_REL_CHUNK", str(chunk))
    monkeypatch.setenv("KBFOLLOW_FAN_IN", str(fan_in))
    n_e, n_r = 300, 4
    g = np.random.default_rng(chunk * 100 + fan_in)
    s = np.concatenate([g.integers(0, n_e, 3000), np.full(700, 5)]).astype(np.int32)
    r = g.integers(0, n_r, len(s)).astype(np.int32)
    o = np.concatenate([g.integers(0, n_e, 3000), g.integers(0, 3, 700)]).astype(np.int32)
    for b, exact in ((4, True), (12, False), (7, False), (32, True), (256, False)):
        if exact:
            X = (g.random((b, n_e)) < 0.2).astype(np.float32)
            R = np.zeros((b, n_r), np.float32)
            R[np.arange(b), g.integers(0, n_r, b)] = 1.0
            dY = np.ones((b, n_e), np.float32)
        else:
            X, R, dY = rand_io(b + chunk, b, n_e, n_r)
        kb = both(kbf, s, r, o, n_e, n_r, X, R, dY, exact, f"chunk={chunk} fan_in={fan_in} b={b}")
    info = kb.info()
    rounded = max(8, (chunk + 7) // 8 * 8)      # chunks are whole 8-entry steps
    assert info["chunk_len"] == [rounded] * 3


@pytest.mark.parametrize("b", [4, 32, 33, 256])
def test_plain_load_path(kbf, b, monkeypatch):
    # Tables of 4 GB or more are read with plain loads instead of raw buffer
    # loads; force that path at a small size.
    monkeypatch.setenv("KBFOLLOW_PLAIN_LOADS", "1")
    n_e, n_r = 2000, 7
    s, r, o = rand_kb(50 + b, n_e, n_r, 20_000)
    s[:3000] = 9                       # a hub, split across chunks
    X, R, dY = rand_io(50 + b, b, n_e, n_r)
    both(kbf, s, r, o, n_e, n_r, X, R, dY, False, f"plain loads b={b}")
    wt = np.random.default_rng(b).uniform(0.5, 1.5, len(s)).astype(np.float32)
    both(kbf, s, r, o, n_e, n_r, X, R, dY, False, f"plain loads weighted b={b}", weight=wt)


@pytest.mark.parametrize("b", [1, 7, 32, 36, 256])
def test_empty_rows_into_nan_outputs(kbf, b):
    """Rows no triple reaches, in runs of one to three rows and one long run,
    written into outputs prefilled with NaN (a row left unwritten stays NaN):
    zeros from the plain passes, gamma * Z from the residual and
    accumulating ones."""
    import torch
    n_e, n_r = 3000, 5
    g = np.random.default_rng(700 + b)
    ids = np.array([i for i in range(2000) if i % 7 in (0, 3, 4)], np.int32)
    n_t = 12_000
    s = g.choice(ids, n_t).astype(np.int32)
    o = g.choice(ids, n_t).astype(np.int32)
    r = g.integers(0, n_r, n_t).astype(np.int32)
    s[:800] = ids[5]   # a hub row, split over chunks
    o[800:1600] = ids[9]
    X, R, dY = rand_io(b + 11, b, n_e, n_r)
    Z = np.random.default_rng(b).standard_normal((b, n_e)).astype(np.float32)
    kb = kbf.KB(s, r, o, n_e, n_r)
    tX, tR, tdY, tZ = to_em(X), to_em(R), to_em(dY), to_em(Z)
    nan = lambda t: torch.full_like(t, float("nan"))
    Y = nan(tX)
    kb.follow(tX, tR, out=Y)
    Yr = nan(tX)
    kb.follow(tX, tR, out=Yr, residual=0.5)
    Ya = nan(tX)
    kb.follow_accumulate(tX, tR, tZ, 0.25, out=Ya)
    dX, dR = nan(tX), nan(tR)
    kb.follow_backward(tX, tR, tdY, dX=dX, dR=dR)
    torch.cuda.synchronize()
    label = f"empty rows b={b}"
    for name, t in (("Y", Y), ("residual", Yr), ("accumulate", Ya), ("dX", dX), ("dR", dR)):
        assert not torch.isnan(t).any(), f"{label}: {name} has unwritten rows"
    assert_close(from_em(Y), oracle.follow(s, r, o, n_e, n_r, X, R), label + " Y")
    assert_close(from_em(Yr), oracle.follow_residual(s, r, o, n_e, n_r, X, R, gamma=0.5),
                 label + " residual")
    assert_close(from_em(Ya), oracle.follow_accumulate(s, r, o, n_e, n_r, X, R, Z, gamma=0.25),
                 label + " accumulate")
    wdX, wdR = oracle.follow_backward(s, r, o, n_e, n_r, X, R, dY)
    assert_close(from_em(dX), wdX, label + " dX")
    assert_close(from_em(dR), wdR, label + " dR")
    kb.close()
