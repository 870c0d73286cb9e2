"""GPU parity: the HIP path (through the C ABI) against the CPU oracle.

Integer-valued inputs (k-hot X, one-hot R, dY = 1) must match bit for bit;
real-valued inputs within |gpu - oracle| <= 1e-7 + 1e-5 |oracle| elementwise.
Sizes: the tiny and MetaQA-shaped workloads at full size, the large and
training-shaped workloads scaled down so the whole oracle runs in seconds
(still thousands of chunks, split hub rows and ragged tails); the full-size
large and training workloads are in test_gpu_fullsize.py.
"""
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


def run_gpu(kbf, kb_arrays, n_e, n_r, X, R, dY, weight=None, kb=None):
    s, r, o = kb_arrays
    if kb is None:
        kb = kbf.KB(s, r, o, n_e, n_r, weight=weight)
    Xe, Re, dYe = to_em(X), to_em(R), to_em(dY)
    Y = kb.follow(Xe, Re)
    dX, dR = kb.follow_backward(Xe, Re, dYe)
    return from_em(Y), from_em(dX), from_em(dR), kb


def run_oracle(kb_arrays, n_e, n_r, X, R, dY, weight=None):
    s, r, o = kb_arrays
    Y = oracle.follow(s, r, o, n_e, n_r, X, R, weight=weight)
    dX, dR = oracle.follow_backward(s, r, o, n_e, n_r, X, R, dY, weight=weight)
    return Y, dX, dR


def check(kbf, w, kb, X, R, dY, exact, label, weight=None):
    arrays = (kb.subj, kb.rel, kb.obj)
    print(f"[parity] {label} {w.label} exact={exact}", flush=True)
    got = run_gpu(kbf, arrays, w.n_entities, w.n_relations, X, R, dY, weight)[:3]
    want = run_oracle(arrays, w.n_entities, w.n_relations, X, R, dY, weight)
    for name, g, e in zip(("Y", "dX", "dR"), got, want):
        if exact:
            assert_bitexact(g, e, f"{label} {name}")
        else:
            assert_close(g, e, f"{label} {name}")


SCALED = {
    "tiny": kbgen.TINY,
    "metaqa": kbgen.METAQA,
    "large_s": kbgen.LARGE.scaled(200_000, 1_000_000, tag=1),
    "train_s": kbgen.TRAIN.scaled(100_000, 1_000_000, batch=64, n_relations=200, tag=1),
}


@pytest.mark.parametrize("name", list(SCALED))
def test_integer_inputs_bitexact(kbf, name):
    w = SCALED[name]
    kb = kbgen.make_kb(w)
    X, R, dY = kbgen.make_integer_inputs(w)
    check(kbf, w, kb, X, R, dY, True, name + "/int")


@pytest.mark.parametrize("name", ["metaqa", "large_s", "train_s"])
def test_real_inputs_within_tolerance(kbf, name):
    w = SCALED[name]
    kb = kbgen.make_kb(w)
    check(kbf, w, kb, kbgen.make_x(w), kbgen.make_r(w), kbgen.make_dy(w), False, name)


def test_tiny_workload_as_specified(kbf):
    w = kbgen.TINY
    kb = kbgen.make_kb(w)
    check(kbf, w, kb, kbgen.make_x(w), kbgen.make_r(w), kbgen.make_dy(w), True, "tiny")


def test_weighted_kb(kbf):
    w = kbgen.METAQA.scaled(5_000, 40_000, batch=36, tag=3)
    kb = kbgen.make_kb(w)
    wt = np.random.default_rng(3).uniform(0.1, 2.0, kb.n_triples).astype(np.float32)
    check(kbf, w, kb, kbgen.make_x(w), kbgen.make_r(w), kbgen.make_dy(w), False, "weighted", weight=wt)


@pytest.mark.parametrize("name", list(SCALED))
def test_deterministic(kbf, name):
    """Two calls on the same inputs give bitwise-equal Y, dX and dR: no
    atomics, every sum in a fixed order (also with a freshly built KB)."""
    w = SCALED[name]
    kb = kbgen.make_kb(w)
    X, R, dY = kbgen.make_x(w), kbgen.make_r(w), kbgen.make_dy(w)
    arrays = (kb.subj, kb.rel, kb.obj)
    a = run_gpu(kbf, arrays, w.n_entities, w.n_relations, X, R, dY)
    c = run_gpu(kbf, arrays, w.n_entities, w.n_relations, X, R, dY, kb=a[3])
    d = run_gpu(kbf, arrays, w.n_entities, w.n_relations, X, R, dY)
    for g1, g2, g3 in zip(a[:3], c[:3], d[:3]):
        assert np.array_equal(g1.view(np.uint32), g2.view(np.uint32))
        assert np.array_equal(g1.view(np.uint32), g3.view(np.uint32))


def chain_gpu(kbf, kb, x0, rho, target):
    """The three-hop chain entirely in this project's kernels: follow and its
    backward (libkbfollow), the softmax over relations, the per-example L1
    normalisation and the softmax cross-entropy with their backwards
    (libkbchain).  No torch arithmetic."""
    from paper_2002_06115_amd import chain
    hops = len(rho)
    xs = [to_em(x0)]
    rs, sums = [], []
    for t in range(hops):
        r = chain.softmax(to_em(rho[t]))
        rs.append(r)
        x, s = chain.l1_normalize(kb.follow(xs[-1], r))
        sums.append(s)
        xs.append(x)
    loss, _, dx = chain.softmax_xent(xs[-1], to_em(target))
    drho = [None] * hops
    for t in range(hops, 0, -1):
        du = chain.l1_normalize_backward(xs[t], sums[t - 1], dx)
        dx, dr = kb.follow_backward(xs[t - 1], rs[t - 1], du)
        drho[t - 1] = from_em(chain.softmax_backward(rs[t - 1], dr))
    return float(loss), from_em(dx), drho


def test_three_hop_chain(kbf):
    from oracle import chain
    w = kbgen.CHAIN3
    kb = kbgen.make_kb(w)
    x0, rho, tgt = kbgen.make_chain_inputs(w, kb)
    arrays = (kb.subj, kb.rel, kb.obj)
    loss_o, dx0_o, drho_o = chain.chain_grad(arrays, w.n_entities, w.n_relations, x0, rho, tgt)
    gkb = kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations)
    loss_g, dx0_g, drho_g = chain_gpu(kbf, gkb, x0, rho, tgt)
    assert abs(loss_g - loss_o) <= 1e-7 + 1e-5 * abs(loss_o)
    assert_close(dx0_g, dx0_o, "chain dx0")
    for t in range(3):
        assert_close(drho_g[t], drho_o[t], f"chain drho{t + 1}")
    # The whole three-hop chain is bitwise reproducible.
    loss_2, dx0_2, drho_2 = chain_gpu(kbf, gkb, x0, rho, tgt)
    assert loss_2 == loss_g
    assert np.array_equal(dx0_2, dx0_g)
    for t in range(3):
        assert np.array_equal(drho_2[t], drho_g[t])


def test_autograd_function(kbf):
    import torch
    w = kbgen.METAQA.scaled(3_000, 20_000, batch=8, tag=4)
    kb = kbgen.make_kb(w)
    X, R, dY = kbgen.make_x(w), kbgen.make_r(w), kbgen.make_dy(w)
    gkb = kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations)
    Xe = to_em(X).requires_grad_(True)
    Re = to_em(R).requires_grad_(True)
    Y = kbf.follow(gkb, Xe, Re)
    Y.backward(to_em(dY))
    Yo, dXo, dRo = run_oracle((kb.subj, kb.rel, kb.obj), w.n_entities, w.n_relations, X, R, dY)
    assert_close(from_em(Y.detach()), Yo, "autograd Y")
    assert_close(from_em(Xe.grad), dXo, "autograd dX")
    assert_close(from_em(Re.grad), dRo, "autograd dR")
