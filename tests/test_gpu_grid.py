"""The n x n grid KB of the scalability experiment (Sec. 3.1) on the GPU:
closed-form one- and two-hop answers, and parity with the oracle across the
relation sweep (edges renamed into m relations, weights 1 + U(0, 0.001))."""
import numpy as np
import pytest

import kbgen
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


def test_grid_closed_form(kbf):
    n = 64
    s, r, o = kbgen.grid_kb(n)
    kb = kbf.KB(s, r, o, n * n, 4)
    g = np.random.default_rng(0)
    b = 128
    cells = g.integers(0, n * n, b)
    dirs = g.integers(0, 4, b)
    X = np.zeros((b, n * n), np.float32)
    X[np.arange(b), cells] = 1.0
    R = np.zeros((b, 4), np.float32)
    R[np.arange(b), dirs] = 1.0
    Y1 = kb.follow(to_em(X), to_em(R))
    Y2 = from_em(kb.follow(Y1, to_em(R)))
    Y1 = from_em(Y1)
    moves = [(-1, 0), (1, 0), (0, 1), (0, -1)]
    for q in range(b):
        a, c = divmod(int(cells[q]), n)
        da, dc = moves[dirs[q]]
        for hops, Y in ((1, Y1), (2, Y2)):
            want = np.zeros(n * n, np.float32)
            a2, c2 = a + hops * da, c + hops * dc
            if 0 <= a2 < n and 0 <= c2 < n:
                want[a2 * n + c2] = 1.0
            assert np.array_equal(Y[q], want), (q, hops)


@pytest.mark.parametrize("m", [4, 20, 1000])
def test_grid_relation_sweep_two_hops(kbf, m):
    n = 100
    s, r, o = kbgen.grid_kb(n, m)
    X, R = kbgen.grid_inputs(n, m, 128)
    kb = kbf.KB(s, r, o, n * n, m)
    Y1 = kb.follow(to_em(X), to_em(R))
    Y2 = kb.follow(Y1, to_em(R))
    Y1o = oracle.follow(s, r, o, n * n, m, X, R)
    assert_close(from_em(Y1), Y1o, f"grid m={m} hop 1")
    assert_close(from_em(Y2), oracle.follow(s, r, o, n * n, m, from_em(Y1), R), f"grid m={m} hop 2")
    # Integer version: one-hot relation sets are exact.
    Ri = np.zeros_like(R)
    Ri[np.arange(128), np.arange(128) % m] = 1.0
    assert_bitexact(from_em(kb.follow(to_em(X), to_em(Ri))), oracle.follow(s, r, o, n * n, m, X, Ri),
                    f"grid m={m} one-hot")
