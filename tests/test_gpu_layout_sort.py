"""The two ways the KB build sorts the triples -- radix sorts of one packed
64-bit key per triple, or chained counting sorts (KBFOLLOW_LAYOUT_SORT=counting)
-- give the same stable orders, so every pass must give bitwise the same
results whichever built the layouts: hard and soft KBs, hubs and empty rows,
a sparse id space, and the residual hop."""
import numpy as np
import pytest

import kbgen
from gpu_util import to_em

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def kbf():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2002_06115_amd as kbf
    return kbf


def hub_kb(seed, n_e=5000, n_r=40, n_t=60_000):
    g = np.random.default_rng(seed)
    s = np.where(g.random(n_t) < 0.2, g.integers(0, 4, n_t), g.integers(0, n_e, n_t))
    o = np.where(g.random(n_t) < 0.2, g.integers(0, 4, n_t), g.integers(0, n_e // 2, n_t))
    r = g.integers(0, n_r, n_t)
    return s.astype(np.int32), r.astype(np.int32), o.astype(np.int32), n_e, n_r


def sparse_kb(seed, n_e=1 << 26, n_r=50, n_t=20_000):
    g = np.random.default_rng(seed)
    s = np.where(g.random(n_t) < 0.5, g.integers(n_e - 100, n_e, n_t), g.integers(0, n_e, n_t))
    o = g.integers(0, 1000, n_t)
    r = g.integers(0, n_r, n_t)
    return s.astype(np.int32), r.astype(np.int32), o.astype(np.int32), n_e, n_r


CASES = {
    "tiny": lambda: (lambda kb: (kb.subj, kb.rel, kb.obj, kbgen.TINY.n_entities,
                                 kbgen.TINY.n_relations))(kbgen.make_kb(kbgen.TINY)),
    "hubs": lambda: hub_kb(1),
    "sparse ids": lambda: sparse_kb(2),
}


@pytest.mark.parametrize("name", list(CASES))
@pytest.mark.parametrize("weighted", [False, True])
@pytest.mark.parametrize("gamma", [None, 0.5])
def test_radix_and_counting_layouts_agree(kbf, name, weighted, gamma, monkeypatch):
    import torch
    s, r, o, n_e, n_r = CASES[name]()
    g = np.random.default_rng(len(s))
    w = g.uniform(0.1, 2.0, len(s)).astype(np.float32) if weighted else None
    b = 8
    X = torch.from_numpy(g.standard_normal((n_e, b)).astype(np.float32)).cuda() \
        if n_e <= 1 << 20 else torch.randn(n_e, b, device="cuda")
    R = to_em(g.standard_normal((b, n_r)).astype(np.float32))
    dY = torch.randn_like(X)
    outs = []
    for how in ("auto", "counting"):
        if how == "counting":
            monkeypatch.setenv("KBFOLLOW_LAYOUT_SORT", "counting")
        else:
            monkeypatch.delenv("KBFOLLOW_LAYOUT_SORT", raising=False)
        kb = kbf.KB(s, r, o, n_e, n_r, weight=w)
        Y = kb.follow(X, R, residual=gamma)
        dX, dR = kb.follow_backward(X, R, dY, residual=gamma)
        torch.cuda.synchronize()
        outs.append((kb.info(), Y, dX, dR))
        kb.close()
    (ia, *a), (ib, *c) = outs
    assert ia == ib, f"{name}: plans differ"
    for label, x, y in zip(("Y", "dX", "dR"), a, c):
        assert torch.equal(x.view(torch.int32), y.view(torch.int32)), f"{name}: {label} differs"
