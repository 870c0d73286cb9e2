"""Every kernel variant against the oracle.

The stream kernel is instantiated per lane layout (4 floats per lane when
b % 4 == 0, else 1; lane groups of 1..32 lanes; column slices beyond 128
columns), per load path (raw buffer loads with the B table staged in LDS or
with B rows held in registers, or plain loads as for tables of 4 GB or more),
per hard or soft KB (App. A weights) and per plain or residual
hop (Sec. 3.2, App. E).  Each combination runs forward and backward on a KB
with 16-entry chunks (rows split over many chunks, deep combine trees, runs
cut by chunk ends) and is compared elementwise with the oracle.
"""
import itertools

import numpy as np
import pytest

import oracle
from gpu_util import assert_close, from_em, to_em

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kbf():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2002_06115_amd as kbf
    return kbf


def small_kb(seed, n_e=300, n_r=7, n_t=6000):
    g = np.random.default_rng(seed)
    # A few hub subjects and objects beside uniform ones.
    s = np.where(g.random(n_t) < 0.3, g.integers(0, 3, n_t), g.integers(0, n_e, n_t))
    o = np.where(g.random(n_t) < 0.3, g.integers(0, 3, n_t), g.integers(0, n_e, n_t))
    r = g.integers(0, n_r, n_t)
    return s.astype(np.int32), r.astype(np.int32), o.astype(np.int32), n_e, n_r


COMBOS = list(itertools.product([1, 4, 5, 36, 260], [False, True], [None, 0.5],
                                ["lds", "regs", "plain"]))


@pytest.mark.parametrize("b,weighted,gamma,path", COMBOS)
def test_variant(kbf, b, weighted, gamma, path, monkeypatch):
    monkeypatch.setenv("KBFOLLOW_CHUNK", "16")
    monkeypatch.setenv("KBFOLLOW_REL_CHUNK", "16")
    monkeypatch.setenv("KBFOLLOW_FAN_IN", "3")
    if path == "plain":
        monkeypatch.setenv("KBFOLLOW_PLAIN_LOADS", "1")
    if path == "regs":
        monkeypatch.setenv("KBFOLLOW_B_IN_LDS", "0")
    s, r, o, n_e, n_r = small_kb(b * 7 + weighted)
    g = np.random.default_rng(b)
    w = g.uniform(0.1, 2.0, len(s)).astype(np.float32) if weighted else None
    X = g.standard_normal((b, n_e)).astype(np.float32)
    R = g.standard_normal((b, n_r)).astype(np.float32)
    dY = g.standard_normal((b, n_e)).astype(np.float32)
    kb = kbf.KB(s, r, o, n_e, n_r, weight=w)
    Y = from_em(kb.follow(to_em(X), to_em(R), residual=gamma))
    dX, dR = kb.follow_backward(to_em(X), to_em(R), to_em(dY), residual=gamma)
    if gamma is None:
        wantY = oracle.follow(s, r, o, n_e, n_r, X, R, weight=w)
        wantdX, wantdR = oracle.follow_backward(s, r, o, n_e, n_r, X, R, dY, weight=w)
    else:
        wantY = oracle.follow_residual(s, r, o, n_e, n_r, X, R, gamma=gamma, weight=w)
        wantdX, wantdR = oracle.follow_backward_residual(s, r, o, n_e, n_r, X, R, dY,
                                                         gamma=gamma, weight=w)
    label = f"b={b} weighted={weighted} gamma={gamma} path={path}"
    assert_close(Y, wantY, label + " Y")
    assert_close(from_em(dX), wantdX, label + " dX")
    assert_close(from_em(dR), wantdR, label + " dR")
    kb.close()


@pytest.mark.parametrize("class_b,blocks,objects", itertools.product(
    ["0", "1", None], ["0", "5", "64"], ["hubs", "uniform"]))
def test_dr_layout_choices(kbf, class_b, blocks, objects, monkeypatch):
    """dR's chunk lists classed by object or by subject (forced, or picked by
    the object skew when None), its hub segments led by 0, 5 or 64 blocks of
    the object id: every choice is a reordering of the same sums, checked
    against the oracle on a KB with hub objects and on one with uniform
    objects (the two sides of the skew rule)."""
    if class_b is not None:
        monkeypatch.setenv("KBFOLLOW_DR_CLASS_B", class_b)
    monkeypatch.setenv("KBFOLLOW_DR_BLOCKS", blocks)
    monkeypatch.setenv("KBFOLLOW_REL_CHUNK", "16")
    monkeypatch.setenv("KBFOLLOW_HUB_MIN", "32")
    if objects == "hubs":
        s, r, o, n_e, n_r = small_kb(91)
    else:
        g = np.random.default_rng(92)
        n_e, n_r, n_t = 400, 5, 8000
        s = g.integers(0, n_e, n_t).astype(np.int32)
        r = g.integers(0, n_r, n_t).astype(np.int32)
        o = g.integers(0, n_e, n_t).astype(np.int32)
    g = np.random.default_rng(93)
    b = 32
    X = g.standard_normal((b, n_e)).astype(np.float32)
    R = g.standard_normal((b, n_r)).astype(np.float32)
    dY = g.standard_normal((b, n_e)).astype(np.float32)
    kb = kbf.KB(s, r, o, n_e, n_r)
    dX, dR = kb.follow_backward(to_em(X), to_em(R), to_em(dY))
    wantdX, wantdR = oracle.follow_backward(s, r, o, n_e, n_r, X, R, dY)
    label = f"class_b={class_b} blocks={blocks} objects={objects}"
    assert_close(from_em(dX), wantdX, label + " dX")
    assert_close(from_em(dR), wantdR, label + " dR")
    kb.close()
