"""The stream kernel's two ways of reading the B operand: the whole column
slice of B staged in LDS (up to 80 KB with two workgroups per CU, up to 160 KB
with one for the hard KB, rows cut into 32-column slices where that makes B
fit; used when the LDS variant keeps at least as many waves on a CU as the
register variant), or one B row per run loaded into registers.  Both do the
same FMAs in the same order, so their outputs must agree bit for bit, and
both must match the oracle.  The KBs sit on either side of the 80 KB and
160 KB limits (R with 640 / 641 and 1280 / 1281 rows at b = 32), need the
32-column slices (b = 128 with 161 relations, b = 256 with 1000, b = 260 with
700: nine slices, the last four columns wide), include relation hubs split
over many chunks, and cover the dR pass of a small-entity KB whose B table
(X) fits LDS too."""
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


def kb_arrays(seed, n_e, n_r, n_t):
    g = np.random.default_rng(seed)
    s = np.where(g.random(n_t) < 0.2, g.integers(0, 4, n_t), g.integers(0, n_e, n_t))
    o = np.where(g.random(n_t) < 0.2, g.integers(0, 4, n_t), g.integers(0, n_e, n_t))
    # a Zipf-like relation mix: a few relations with long runs, many short ones
    r = np.minimum(g.zipf(1.3, n_t) - 1, n_r - 1)
    return s.astype(np.int32), r.astype(np.int32), o.astype(np.int32)


def run(kbf, monkeypatch, lds, s, r, o, n_e, n_r, X, R, dY, weight=None, gamma=None):
    monkeypatch.setenv("KBFOLLOW_B_IN_LDS", "1" if lds else "0")
    kb = kbf.KB(s, r, o, n_e, n_r, weight=weight)
    Y = from_em(kb.follow(to_em(X), to_em(R), residual=gamma))
    dX, dR = kb.follow_backward(to_em(X), to_em(R), to_em(dY), residual=gamma)
    out = Y, from_em(dX), from_em(dR)
    kb.close()
    return out


@pytest.mark.parametrize("b,n_r", [(32, 640), (32, 641), (32, 1280), (32, 1281), (128, 160),
                                   (128, 161), (5, 300), (1, 2000), (256, 80), (256, 1000),
                                   (260, 40), (260, 700)])
def test_lds_and_register_paths_agree(kbf, monkeypatch, b, n_r):
    monkeypatch.setenv("KBFOLLOW_CHUNK", "32")
    n_e, n_t = 5000, 60_000
    s, r, o = kb_arrays(b * 1000 + n_r, n_e, n_r, n_t)
    g = np.random.default_rng(b + n_r)
    X = g.standard_normal((b, n_e)).astype(np.float32)
    R = g.standard_normal((b, n_r)).astype(np.float32)
    dY = g.standard_normal((b, n_e)).astype(np.float32)
    with_lds = run(kbf, monkeypatch, True, s, r, o, n_e, n_r, X, R, dY)
    in_regs = run(kbf, monkeypatch, False, s, r, o, n_e, n_r, X, R, dY)
    for name, a, c in zip(("Y", "dX", "dR"), with_lds, in_regs):
        assert_bitexact(a, c, f"b={b} n_r={n_r} {name}: LDS vs registers")
    wantY = oracle.follow(s, r, o, n_e, n_r, X, R)
    wantdX, wantdR = oracle.follow_backward(s, r, o, n_e, n_r, X, R, dY)
    for name, a, want in zip(("Y", "dX", "dR"), with_lds, (wantY, wantdX, wantdR)):
        assert_close(a, want, f"b={b} n_r={n_r} {name}")


@pytest.mark.parametrize("weighted,gamma", [(True, None), (False, 0.5), (True, -1.0)])
@pytest.mark.parametrize("b", [32, 64])
def test_soft_and_residual_variants_agree(kbf, monkeypatch, b, weighted, gamma):
    monkeypatch.setenv("KBFOLLOW_CHUNK", "32")
    n_e, n_r, n_t = 4000, 200, 50_000
    s, r, o = kb_arrays(7 * b + weighted, n_e, n_r, n_t)
    g = np.random.default_rng(b)
    w = g.uniform(0.1, 2.0, n_t).astype(np.float32) if weighted else None
    X = g.standard_normal((b, n_e)).astype(np.float32)
    R = g.standard_normal((b, n_r)).astype(np.float32)
    dY = g.standard_normal((b, n_e)).astype(np.float32)
    a = run(kbf, monkeypatch, True, s, r, o, n_e, n_r, X, R, dY, weight=w, gamma=gamma)
    c = run(kbf, monkeypatch, False, s, r, o, n_e, n_r, X, R, dY, weight=w, gamma=gamma)
    for name, x, y in zip(("Y", "dX", "dR"), a, c):
        assert_bitexact(x, y, f"b={b} weighted={weighted} gamma={gamma} {name}")


def test_integer_inputs_exact_on_the_lds_path(kbf, monkeypatch):
    """k-hot X and one-hot R: every sum is an integer, so the result is the
    oracle's bit for bit (R with 600 rows at b = 32 sits in LDS)."""
    monkeypatch.setenv("KBFOLLOW_B_IN_LDS", "1")
    n_e, n_r, n_t, b = 20_000, 600, 200_000, 32
    s, r, o = kb_arrays(99, n_e, n_r, n_t)
    g = np.random.default_rng(99)
    X = np.zeros((b, n_e), np.float32)
    for beta in range(b):
        X[beta, g.choice(n_e, 5, replace=False)] = 1.0
    X[:, :4] = 1.0  # the hub subjects too
    R = np.zeros((b, n_r), np.float32)
    R[np.arange(b), g.integers(0, 8, b)] = 1.0
    dY = np.ones((b, n_e), np.float32)
    kb = kbf.KB(s, r, o, n_e, n_r)
    Y = from_em(kb.follow(to_em(X), to_em(R)))
    dX, dR = kb.follow_backward(to_em(X), to_em(R), to_em(dY))
    assert_bitexact(Y, oracle.follow(s, r, o, n_e, n_r, X, R), "Y")
    wdX, wdR = oracle.follow_backward(s, r, o, n_e, n_r, X, R, dY)
    assert_bitexact(from_em(dX), wdX, "dX")
    assert_bitexact(from_em(dR), wdR, "dR")
    kb.close()
