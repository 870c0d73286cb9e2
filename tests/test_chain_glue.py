"""The multi-hop chain glue (include/kbchain.h): column-wise softmax, L1
normalisation and softmax cross-entropy, and their backwards.

Host: libkbchain.so exports every entry point the header declares and
rejects bad arguments before launching anything.  GPU: every operation
against a float64 numpy evaluation of its formula (the softmax of the chain
oracle, oracle/chain.py, for the forward softmax), on column counts that are
and are not multiples of the 16-column tile and on row counts from 1 up, and
bitwise reproducibility.
"""
import ctypes
import os
import re

import numpy as np
import pytest

from gpu_util import assert_close

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "kbchain.h")
LIB = os.path.join(ROOT, "paper_2002_06115_amd", "_lib", "libkbchain.so")


def declared():
    text = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    return sorted(set(re.findall(r"\b(kbc_[a-z0-9_]+)\s*\(", text)))


def test_library_exports_every_declared_symbol():
    names = declared()
    assert set(names) >= {"kbc_softmax", "kbc_softmax_backward", "kbc_l1_normalize",
                          "kbc_l1_normalize_backward", "kbc_softmax_xent"}
    lib = ctypes.CDLL(LIB)
    for n in names:
        assert hasattr(lib, n), n


def test_bad_arguments_are_refused_before_any_launch():
    lib = ctypes.CDLL(LIB)
    P = ctypes.c_void_p
    d = P(16)  # never dereferenced: arguments are checked first
    lib.kbc_softmax.argtypes = [ctypes.c_int64, ctypes.c_int32, P, P, P]
    lib.kbc_softmax_xent.argtypes = [ctypes.c_int64, ctypes.c_int32, P, P, P, P, P, P]
    assert lib.kbc_softmax(0, 4, d, d, None) == 1
    assert lib.kbc_softmax(4, 0, d, d, None) == 1
    assert lib.kbc_softmax(4, 4, None, d, None) == 1
    assert lib.kbc_softmax_xent(4, 4, d, d, d, None, d, None) == 1


SHAPES = [(1, 1), (7, 15), (18, 16), (1000, 17), (300, 64), (1000, 256), (43, 130), (3, 1100),
          (50_000, 3)]


@pytest.fixture(scope="module")
def chain():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2002_06115_amd import chain
    return chain


def cuda(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, np.float32)).cuda()


def host(t):
    return t.cpu().numpy()


@pytest.mark.gpu
@pytest.mark.parametrize("n,b", SHAPES)
def test_softmax_and_backward(chain, n, b):
    from oracle.chain import softmax as oracle_softmax
    g = np.random.default_rng(n * 131 + b)
    z = (3 * g.standard_normal((n, b))).astype(np.float32)
    dp = g.standard_normal((n, b)).astype(np.float32)
    p = chain.softmax(cuda(z))
    want = oracle_softmax(z.T.astype(np.float64)).T      # the oracle works in [b][n]
    assert_close(host(p), want, "softmax")
    pg = host(p).astype(np.float64)
    want_dz = pg * (dp - (dp * pg).sum(axis=0, keepdims=True))
    assert_close(host(chain.softmax_backward(p, cuda(dp))), want_dz, "softmax backward")


@pytest.mark.gpu
@pytest.mark.parametrize("n,b", SHAPES)
def test_l1_normalize_and_backward(chain, n, b):
    g = np.random.default_rng(n * 17 + b)
    u = g.random((n, b)).astype(np.float32) + 0.01
    dx = g.standard_normal((n, b)).astype(np.float32)
    x, sums = chain.l1_normalize(cuda(u))
    s = u.astype(np.float64).sum(axis=0)
    np.testing.assert_allclose(host(sums), s, rtol=1e-13)
    assert_close(host(x), u / s, "l1 normalize")
    xg = host(x).astype(np.float64)
    want = (dx - (dx * xg).sum(axis=0, keepdims=True)) / s
    assert_close(host(chain.l1_normalize_backward(x, sums, cuda(dx))), want, "l1 backward")


@pytest.mark.gpu
@pytest.mark.parametrize("n,b", SHAPES)
def test_softmax_xent(chain, n, b):
    g = np.random.default_rng(n * 7 + b)
    z = g.standard_normal((n, b)).astype(np.float32)
    t = np.zeros((n, b), np.float32)
    for c in range(b):   # a uniform distribution over 1..5 answers per example
        k = min(n, int(g.integers(1, 6)))
        t[g.choice(n, k, replace=False), c] = 1.0 / k
    loss, col, dz = chain.softmax_xent(cuda(z), cuda(t))
    z64 = z.astype(np.float64)
    m = z64.max(axis=0, keepdims=True)
    logp = z64 - m - np.log(np.exp(z64 - m).sum(axis=0, keepdims=True))
    col_want = -(t * logp).sum(axis=0)
    np.testing.assert_allclose(host(col), col_want, rtol=1e-12, atol=1e-15)
    assert abs(float(loss) - col_want.sum() / b) <= 1e-12 * max(1.0, abs(col_want.sum() / b))
    p = np.exp(logp)
    assert_close(host(dz), (p * t.sum(axis=0, keepdims=True) - t) / b, "xent dz")


@pytest.mark.gpu
def test_non_normalised_targets_gradient(chain):
    """dz is the gradient of the loss also when a column's targets do not sum
    to one: central differences of the float64 loss formula."""
    g = np.random.default_rng(3)
    n, b = 6, 2
    z = g.standard_normal((n, b)).astype(np.float32)
    t = g.random((n, b)).astype(np.float32) * 2
    _, _, dz = chain.softmax_xent(cuda(z), cuda(t))

    def loss(zz):
        m = zz.max(axis=0, keepdims=True)
        lp = zz - m - np.log(np.exp(zz - m).sum(axis=0, keepdims=True))
        return -(t * lp).sum() / b

    z64, h = z.astype(np.float64), 1e-6
    fd = np.zeros_like(z64)
    for i in range(n):
        for c in range(b):
            e = np.zeros_like(z64)
            e[i, c] = h
            fd[i, c] = (loss(z64 + e) - loss(z64 - e)) / (2 * h)
    np.testing.assert_allclose(host(dz), fd, rtol=1e-5, atol=1e-7)


@pytest.mark.gpu
def test_glue_is_deterministic(chain):
    import torch
    g = np.random.default_rng(5)
    z = cuda(g.standard_normal((20_000, 96)))
    u = cuda(g.random((20_000, 96)) + 0.1)
    a = [chain.softmax(z), chain.l1_normalize(u)[0], chain.softmax_xent(z, u)[2]]
    c = [chain.softmax(z), chain.l1_normalize(u)[0], chain.softmax_xent(z, u)[2]]
    for x, y in zip(a, c):
        assert torch.equal(x.view(torch.int32), y.view(torch.int32))
