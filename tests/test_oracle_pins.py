"""Pins of the CPU oracle against what the paper and the mathematics fix.

None of these checks re-types the oracle's loop: they compare it with dense
matrix evaluations of Eq. 1-4, brute-force neighbour sets (Claim 1), the grid
KB's closed form (Sec. 3.1), linearity, the adjoint identity, finite
differences, the triple-shard identity (App. D) and triple-order invariance.
"""
import itertools

import numpy as np
import pytest

import oracle
from oracle import chain
import dense_ref


def tiny_kb(seed, n_e=37, n_r=5, n_t=300, dup=False, weighted=False):
    g = np.random.default_rng(seed)
    s = g.integers(0, n_e, n_t).astype(np.int32)
    r = g.integers(0, n_r, n_t).astype(np.int32)
    o = g.integers(0, n_e, n_t).astype(np.int32)
    if not dup:
        key = (s.astype(np.int64) * n_r + r) * n_e + o
        _, first = np.unique(key, return_index=True)
        first.sort()
        s, r, o = s[first], r[first], o[first]
    w = g.uniform(0.25, 2.0, len(s)).astype(np.float32) if weighted else None
    return s, r, o, w


def rand_inputs(seed, b, n_e, n_r, signed=False):
    g = np.random.default_rng(seed + 1000)
    lo = -1.0 if signed else 0.0
    X = g.uniform(lo, 1.0, (b, n_e)).astype(np.float32)
    R = g.uniform(lo, 1.0, (b, n_r)).astype(np.float32)
    dY = g.standard_normal((b, n_e)).astype(np.float32)
    return X, R, dY


def assert_rounded_once(got32, exact64):
    """got32 is exact64 rounded to float32 (ties aside): within half an ulp."""
    exact64 = np.asarray(exact64, np.float64)
    err = np.abs(got32.astype(np.float64) - exact64)
    bound = np.spacing(np.abs(exact64).astype(np.float32)).astype(np.float64) * 0.5 + 1e-300
    assert np.all(err <= bound * (1 + 1e-6) + 1e-12 * np.abs(exact64).max(initial=0)), \
        float((err / bound).max())


# ---------------------------------------------------------------------------
# O1: dense Eq. 4 == naive mixing (Eq. 1-2) == late mixing (Eq. 3) == oracle
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("seed,weighted,dup,signed",
                         [(1, False, False, False), (2, True, False, False),
                          (3, False, True, True), (4, True, True, True)])
def test_dense_formulations_agree_with_oracle(seed, weighted, dup, signed):
    n_e, n_r, b = 37, 5, 6
    s, r, o, w = tiny_kb(seed, n_e, n_r, 300, dup=dup, weighted=weighted)
    X, R, _ = rand_inputs(seed, b, n_e, n_r, signed)
    ref = dense_ref.reified(s, r, o, n_e, n_r, X, R, w)
    np.testing.assert_allclose(dense_ref.naive(s, r, o, n_e, n_r, X, R, w), ref, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dense_ref.late(s, r, o, n_e, n_r, X, R, w), ref, rtol=1e-12, atol=1e-13)
    Y = oracle.follow(s, r, o, n_e, n_r, X, R, weight=w)
    assert_rounded_once(Y, ref)
    Y64 = oracle.follow_f64(s, r, o, n_e, n_r, X, R, weight=w)
    np.testing.assert_allclose(Y64, ref, rtol=1e-12, atol=1e-13)


def test_dense_integer_inputs_exact():
    n_e, n_r, b = 50, 4, 5
    s, r, o, _ = tiny_kb(7, n_e, n_r, 600, dup=True)
    g = np.random.default_rng(7)
    X = g.integers(0, 4, (b, n_e)).astype(np.float32)
    R = g.integers(0, 3, (b, n_r)).astype(np.float32)
    Y = oracle.follow(s, r, o, n_e, n_r, X, R)
    assert np.array_equal(Y, dense_ref.reified(s, r, o, n_e, n_r, X, R).astype(np.float32))
    assert np.array_equal(Y, dense_ref.late(s, r, o, n_e, n_r, X, R).astype(np.float32))


# ---------------------------------------------------------------------------
# O2: brute-force neighbour counts and Claim 1 (support == R-neighbours)
# ---------------------------------------------------------------------------

def test_claim1_support_and_counts():
    n_e, n_r, b = 60, 6, 12
    s, r, o, _ = tiny_kb(11, n_e, n_r, 400)
    facts = set(zip(s.tolist(), r.tolist(), o.tolist()))
    g = np.random.default_rng(11)
    X = np.zeros((b, n_e), np.float32)
    R = np.zeros((b, n_r), np.float32)
    sets = []
    for beta in range(b):
        S = set(g.choice(n_e, size=int(g.integers(1, 6)), replace=False).tolist())
        Rs = set(g.choice(n_r, size=int(g.integers(1, 3)), replace=False).tolist())
        X[beta, list(S)] = 1.0
        R[beta, list(Rs)] = 1.0
        sets.append((S, Rs))
    Y = oracle.follow(s, r, o, n_e, n_r, X, R)
    for beta, (S, Rs) in enumerate(sets):
        # R-neighbors(X) = {x_j : exists r in R, x_i in X, (x_i, x_j) in r} (Sec. 2.2)
        neigh = {j for (i, k, j) in facts if i in S and k in Rs}
        assert set(np.nonzero(Y[beta])[0].tolist()) == neigh
        for j in range(n_e):
            count = sum(1 for i in S for k in Rs if (i, k, j) in facts)
            assert Y[beta, j] == count


def test_claim1_nonnegative_weighted_support():
    # Claim 1 holds for any non-negative weights: the support only depends on
    # which entries are non-zero (App. B).
    n_e, n_r, b = 40, 4, 8
    s, r, o, _ = tiny_kb(12, n_e, n_r, 250)
    g = np.random.default_rng(12)
    X = (g.random((b, n_e)) < 0.1) * g.uniform(0.5, 2.0, (b, n_e))
    R = (g.random((b, n_r)) < 0.5) * g.uniform(0.5, 2.0, (b, n_r))
    Y = oracle.follow(s, r, o, n_e, n_r, X.astype(np.float32), R.astype(np.float32))
    for beta in range(b):
        S = set(np.nonzero(X[beta])[0].tolist())
        Rs = set(np.nonzero(R[beta])[0].tolist())
        neigh = {int(oo) for ss, rr, oo in zip(s, r, o) if ss in S and rr in Rs}
        assert set(np.nonzero(Y[beta])[0].tolist()) == neigh


# ---------------------------------------------------------------------------
# O9: grid KB closed form (Sec. 3.1, App. E grid experiments)
# ---------------------------------------------------------------------------

def grid_kb(n):
    """n x n grid; relations 0..3 = north, south, east, west; cell (a, c) -> a * n + c."""
    s, r, o = [], [], []
    moves = [(-1, 0), (1, 0), (0, 1), (0, -1)]
    for a in range(n):
        for c in range(n):
            for k, (da, dc) in enumerate(moves):
                a2, c2 = a + da, c + dc
                if 0 <= a2 < n and 0 <= c2 < n:
                    s.append(a * n + c)
                    r.append(k)
                    o.append(a2 * n + c2)
    return (np.array(s, np.int32), np.array(r, np.int32), np.array(o, np.int32))


def test_grid_one_and_two_hops_closed_form():
    n = 9
    s, r, o = grid_kb(n)
    n_e, n_r = n * n, 4
    moves = [(-1, 0), (1, 0), (0, 1), (0, -1)]
    cells = [(a, c) for a in range(n) for c in range(n)]
    b = len(cells) * 4
    X = np.zeros((b, n_e), np.float32)
    R = np.zeros((b, n_r), np.float32)
    for q, ((a, c), k) in enumerate(itertools.product(cells, range(4))):
        X[q, a * n + c] = 1.0
        R[q, k] = 1.0
    Y1 = oracle.follow(s, r, o, n_e, n_r, X, R)
    Y2 = oracle.follow(s, r, o, n_e, n_r, Y1, R)
    for q, ((a, c), k) in enumerate(itertools.product(cells, range(4))):
        da, dc = moves[k]
        want1 = np.zeros(n_e, np.float32)
        if 0 <= a + da < n and 0 <= c + dc < n:
            want1[(a + da) * n + c + dc] = 1.0
        want2 = np.zeros(n_e, np.float32)
        if 0 <= a + 2 * da < n and 0 <= c + 2 * dc < n:
            want2[(a + 2 * da) * n + c + 2 * dc] = 1.0
        assert np.array_equal(Y1[q], want1)
        assert np.array_equal(Y2[q], want2)


def test_grid_all_directions_counts_neighbours():
    # With every relation weighted 1, one hop from a cell reaches its 2-4 grid
    # neighbours; two hops reach cell (a', c') with the number of 2-step paths.
    n = 7
    s, r, o = grid_kb(n)
    n_e = n * n
    X = np.eye(n_e, dtype=np.float32)
    R = np.ones((n_e, 4), np.float32)
    Y2 = oracle.follow(s, r, o, n_e, 4, oracle.follow(s, r, o, n_e, 4, X, R), R)
    for a, c in itertools.product(range(n), range(n)):
        for a2, c2 in itertools.product(range(n), range(n)):
            paths = 0
            for (d1a, d1c), (d2a, d2c) in itertools.product([(-1, 0), (1, 0), (0, 1), (0, -1)], repeat=2):
                ma, mc = a + d1a, c + d1c
                if 0 <= ma < n and 0 <= mc < n and (ma + d2a, mc + d2c) == (a2, c2):
                    paths += 1
            assert Y2[a * n + c, a2 * n + c2] == paths


# ---------------------------------------------------------------------------
# O3 linearity, O5 adjoint identity, O4 finite differences, dense gradients
# ---------------------------------------------------------------------------

def test_linearity_in_x_and_r():
    n_e, n_r, b = 41, 6, 4
    s, r, o, w = tiny_kb(21, n_e, n_r, 350, weighted=True)
    g = np.random.default_rng(21)
    X1, X2 = g.standard_normal((2, b, n_e))
    R1, R2 = g.standard_normal((2, b, n_r))
    a, c = 0.7, -1.3
    f = lambda X, R: oracle.follow_f64(s, r, o, n_e, n_r, X, R, weight=w)
    np.testing.assert_allclose(f(a * X1 + c * X2, R1), a * f(X1, R1) + c * f(X2, R1), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(f(X1, a * R1 + c * R2), a * f(X1, R1) + c * f(X1, R2), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("weighted", [False, True])
def test_backward_against_dense_adjoint(weighted):
    n_e, n_r, b = 33, 7, 5
    s, r, o, w = tiny_kb(31, n_e, n_r, 280, dup=True, weighted=weighted)
    X, R, dY = rand_inputs(31, b, n_e, n_r, signed=True)
    dX_ref, dR_ref = dense_ref.reified_grads(s, r, o, n_e, n_r, X, R, dY, w)
    dX, dR = oracle.follow_backward(s, r, o, n_e, n_r, X, R, dY, weight=w)
    assert_rounded_once(dX, dX_ref)
    assert_rounded_once(dR, dR_ref)
    dX64, dR64 = oracle.follow_backward_f64(s, r, o, n_e, n_r, X, R, dY, weight=w)
    np.testing.assert_allclose(dX64, dX_ref, rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(dR64, dR_ref, rtol=1e-12, atol=1e-13)


def test_backward_finite_differences_of_dense_forward():
    # L(X, R) = <dY, follow(X, R)> is linear in X and in R, so a central
    # difference along any direction V is exact up to rounding.
    n_e, n_r, b = 29, 5, 3
    s, r, o, w = tiny_kb(41, n_e, n_r, 200, weighted=True)
    X, R, dY = rand_inputs(41, b, n_e, n_r, signed=True)
    g = np.random.default_rng(41)
    V, U = g.standard_normal((b, n_e)), g.standard_normal((b, n_r))
    L = lambda X_, R_: float((dY * dense_ref.reified(s, r, o, n_e, n_r, X_, R_, w)).sum())
    dX, dR = oracle.follow_backward_f64(s, r, o, n_e, n_r, X, R, dY, weight=w)
    h = 1e-3
    fd_x = (L(X + h * V, R) - L(X - h * V, R)) / (2 * h)
    fd_r = (L(X, R + h * U) - L(X, R - h * U)) / (2 * h)
    assert abs(fd_x - (dX * V).sum()) <= 1e-9 * max(1.0, abs(fd_x))
    assert abs(fd_r - (dR * U).sum()) <= 1e-9 * max(1.0, abs(fd_r))


def test_adjoint_identity():
    n_e, n_r, b = 45, 6, 4
    s, r, o, w = tiny_kb(51, n_e, n_r, 400, weighted=True)
    X, R, dY = rand_inputs(51, b, n_e, n_r, signed=True)
    Y = oracle.follow_f64(s, r, o, n_e, n_r, X, R, weight=w)
    dX, dR = oracle.follow_backward_f64(s, r, o, n_e, n_r, X, R, dY, weight=w)
    brute = sum(float(w[l]) * float(X[beta, s[l]]) * float(R[beta, r[l]]) * float(dY[beta, o[l]])
                for beta in range(b) for l in range(len(s)))
    for v in ((dY * Y).sum(), (dX * X).sum(), (dR * R).sum()):
        assert abs(v - brute) <= 1e-12 * max(1.0, abs(brute))


def test_dx_is_forward_on_inverse_kb():
    n_e, n_r, b = 38, 5, 4
    s, r, o, w = tiny_kb(61, n_e, n_r, 300, weighted=True)
    X, R, dY = rand_inputs(61, b, n_e, n_r, signed=True)
    dX, _ = oracle.follow_backward(s, r, o, n_e, n_r, X, R, dY, weight=w)
    # KB' = {(o, r, s)}: the gradient w.r.t. X is following dY backwards.
    assert np.array_equal(dX, oracle.follow(o, r, s, n_e, n_r, dY, R, weight=w))


# ---------------------------------------------------------------------------
# O7 shard identity (App. D), O8 triple-order invariance
# ---------------------------------------------------------------------------

def test_triple_shards_sum_to_whole():
    n_e, n_r, b = 64, 8, 6
    s, r, o, _ = tiny_kb(71, n_e, n_r, 900)
    g = np.random.default_rng(71)
    X = g.integers(0, 3, (b, n_e)).astype(np.float32)
    R = g.integers(0, 2, (b, n_r)).astype(np.float32)
    whole = oracle.follow(s, r, o, n_e, n_r, X, R)
    shard = g.integers(0, 3, len(s))
    parts = [oracle.follow(s[shard == i], r[shard == i], o[shard == i], n_e, n_r, X, R) for i in range(3)]
    assert np.array_equal(parts[0] + parts[1] + parts[2], whole)


def test_triple_order_invariance():
    n_e, n_r, b = 52, 6, 5
    s, r, o, w = tiny_kb(81, n_e, n_r, 500, weighted=True)
    X, R, dY = rand_inputs(81, b, n_e, n_r, signed=True)
    p = np.random.default_rng(81).permutation(len(s))
    Y1 = oracle.follow_f64(s, r, o, n_e, n_r, X, R, weight=w)
    Y2 = oracle.follow_f64(s[p], r[p], o[p], n_e, n_r, X, R, weight=w[p])
    np.testing.assert_allclose(Y1, Y2, rtol=1e-12, atol=1e-13)
    Xi = np.random.default_rng(82).integers(0, 3, (b, n_e)).astype(np.float32)
    Ri = np.random.default_rng(83).integers(0, 3, (b, n_r)).astype(np.float32)
    a1 = oracle.follow_backward(s, r, o, n_e, n_r, Xi, Ri, np.ones((b, n_e), np.float32))
    a2 = oracle.follow_backward(s[p], r[p], o[p], n_e, n_r, Xi, Ri, np.ones((b, n_e), np.float32))
    assert np.array_equal(a1[0], a2[0]) and np.array_equal(a1[1], a2[1])


# ---------------------------------------------------------------------------
# sampled outputs == the matching columns of the full evaluation
# ---------------------------------------------------------------------------

def test_sampled_matches_full():
    n_e, n_r, b = 70, 9, 5
    s, r, o, w = tiny_kb(91, n_e, n_r, 700, weighted=True)
    X, R, dY = rand_inputs(91, b, n_e, n_r, signed=True)
    Y = oracle.follow(s, r, o, n_e, n_r, X, R, weight=w)
    dX, dR = oracle.follow_backward(s, r, o, n_e, n_r, X, R, dY, weight=w)
    ids = np.array([0, 5, 17, 69, 33], np.int32)
    rids = np.array([8, 0, 3], np.int32)
    assert np.array_equal(oracle.sampled(0, s, r, o, n_e, n_r, ids, X=X, R=R, weight=w), Y[:, ids])
    assert np.array_equal(oracle.sampled(1, s, r, o, n_e, n_r, ids, R=R, dY=dY, weight=w), dX[:, ids])
    assert np.array_equal(oracle.sampled(2, s, r, o, n_e, n_r, rids, X=X, dY=dY, weight=w), dR[:, rids])


def test_thread_count_does_not_change_result():
    n_e, n_r, b = 80, 7, 9
    s, r, o, w = tiny_kb(92, n_e, n_r, 800, weighted=True)
    X, R, dY = rand_inputs(92, b, n_e, n_r, signed=True)
    a = oracle.follow_backward(s, r, o, n_e, n_r, X, R, dY, weight=w, nthreads=1)
    c = oracle.follow_backward(s, r, o, n_e, n_r, X, R, dY, weight=w, nthreads=4)
    assert np.array_equal(a[0], c[0]) and np.array_equal(a[1], c[1])


# ---------------------------------------------------------------------------
# edge cases and argument validation
# ---------------------------------------------------------------------------

def test_empty_kb_and_zero_rows():
    X = np.ones((3, 10), np.float32)
    R = np.ones((3, 2), np.float32)
    e = np.zeros(0, np.int32)
    assert not oracle.follow(e, e, e, 10, 2, X, R).any()
    dX, dR = oracle.follow_backward(e, e, e, 10, 2, X, R, X)
    assert not dX.any() and not dR.any()


def test_rejects_out_of_range_ids():
    s = np.array([0, 5], np.int32)
    r = np.array([0, 0], np.int32)
    o = np.array([1, 1], np.int32)
    with pytest.raises(ValueError):
        oracle.follow(s, r, o, 5, 1, np.ones((1, 5), np.float32), np.ones((1, 1), np.float32))
    with pytest.raises(ValueError):
        oracle.follow(o, np.array([0, 1], np.int32), o, 5, 1, np.ones((1, 5), np.float32),
                      np.ones((1, 1), np.float32))


# ---------------------------------------------------------------------------
# planted mistakes: each plausible slip fails one of the pins above
# ---------------------------------------------------------------------------

def test_pins_detect_planted_mistakes():
    n_e, n_r, b = 37, 5, 6
    s, r, o, w = tiny_kb(101, n_e, n_r, 300, weighted=True)
    X, R, dY = rand_inputs(101, b, n_e, n_r)
    ref = dense_ref.reified(s, r, o, n_e, n_r, X, R, w)
    close = lambda Y: np.allclose(Y, ref, rtol=1e-5, atol=1e-7)
    assert close(oracle.follow(s, r, o, n_e, n_r, X, R, weight=w))
    assert not close(oracle.follow(o, r, s, n_e, n_r, X, R, weight=w))            # subject/object swapped
    assert not close(oracle.follow(s, r, o, n_e, n_r, X, R))                      # weight dropped
    assert not close(oracle.follow(s, (r + 1) % n_r, o, n_e, n_r, X, R, weight=w))  # wrong relation index
    assert not close(oracle.follow(s, r, o, n_e, n_r, X, -R, weight=w))           # sign
    assert not close(oracle.follow(s[1:], r[1:], o[1:], n_e, n_r, X, R, weight=w[1:]))  # dropped term
    dX_ref, dR_ref = dense_ref.reified_grads(s, r, o, n_e, n_r, X, R, dY, w)
    dX, dR = oracle.follow_backward(o, r, s, n_e, n_r, X, R, dY, weight=w)
    assert not np.allclose(dX, dX_ref, rtol=1e-5, atol=1e-7)
    assert not np.allclose(dR, dR_ref, rtol=1e-5, atol=1e-7)


# ---------------------------------------------------------------------------
# O10: the three-hop chain's gradients against central differences
# ---------------------------------------------------------------------------

def test_chain_gradients_finite_differences():
    n_e, n_r, b = 30, 4, 3
    s, r, o, _ = tiny_kb(111, n_e, n_r, 260)
    kb = (s, r, o)
    adj = {}
    for ss, oo in zip(s.tolist(), o.tolist()):
        adj.setdefault(ss, set()).add(oo)
    g = np.random.default_rng(111)
    x0 = np.zeros((b, n_e))
    for beta in range(b):
        while True:
            e = int(g.integers(0, n_e))
            f1 = adj.get(e, set())
            f2 = set().union(*[adj.get(v, set()) for v in f1]) if f1 else set()
            f3 = set().union(*[adj.get(v, set()) for v in f2]) if f2 else set()
            if f3:
                break
        x0[beta, e] = 1.0
    x0 = x0 + 0.05 * g.random((b, n_e))          # a dense, positive start for the X gradient
    rho = g.standard_normal((3, b, n_r))
    tgt = np.zeros((b, n_e))
    for beta in range(b):
        tgt[beta, g.choice(n_e, 2, replace=False)] = 0.5
    loss, dx0, drho = chain.chain_grad(kb, n_e, n_r, x0, rho, tgt)
    h = 1e-6
    V = g.standard_normal((b, n_e))
    fd = (chain.chain_loss(kb, n_e, n_r, x0 + h * V, rho, tgt)
          - chain.chain_loss(kb, n_e, n_r, x0 - h * V, rho, tgt)) / (2 * h)
    assert abs(fd - (dx0 * V).sum()) <= 1e-6 * max(1e-3, abs(fd))
    for t in range(3):
        U = np.zeros_like(rho)
        U[t] = g.standard_normal((b, n_r))
        fd = (chain.chain_loss(kb, n_e, n_r, x0, rho + h * U, tgt)
              - chain.chain_loss(kb, n_e, n_r, x0, rho - h * U, tgt)) / (2 * h)
        assert abs(fd - (drho[t] * U[t]).sum()) <= 1e-6 * max(1e-3, abs(fd))


# ---------------------------------------------------------------------------
# Residual hop and residual chains (Sec. 3.2 KB completion, App. E)
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("gamma", [0.0, 1.0, -0.75])
def test_residual_hop_against_dense(gamma):
    n_e, n_r, b = 36, 5, 6
    s, r, o, w = tiny_kb(121, n_e, n_r, 280, weighted=True)
    X, R, dY = rand_inputs(121, b, n_e, n_r, signed=True)
    Y = oracle.follow_residual(s, r, o, n_e, n_r, X, R, gamma, weight=w)
    assert_rounded_once(Y, dense_ref.reified(s, r, o, n_e, n_r, X, R, w) + gamma * X.astype(np.float64))
    dX, dR = oracle.follow_backward_residual(s, r, o, n_e, n_r, X, R, dY, gamma, weight=w)
    dX_ref, dR_ref = dense_ref.reified_grads(s, r, o, n_e, n_r, X, R, dY, w)
    assert_rounded_once(dX, dX_ref + gamma * dY.astype(np.float64))
    assert_rounded_once(dR, dR_ref)
    if gamma == 0.0:
        assert np.array_equal(Y, oracle.follow(s, r, o, n_e, n_r, X, R, weight=w))


@pytest.mark.parametrize("gamma", [0.0, 1.0, -0.75])
def test_accumulate_against_dense(gamma):
    """follow(X, R) + gamma * Z for an independent Z: the dense Eq. 4 plus
    gamma * Z, rounded once; Z = X is the residual hop, gamma = 0 is follow."""
    n_e, n_r, b = 36, 5, 6
    s, r, o, w = tiny_kb(131, n_e, n_r, 280, weighted=True)
    X, R, Z = rand_inputs(131, b, n_e, n_r, signed=True)
    Y = oracle.follow_accumulate(s, r, o, n_e, n_r, X, R, Z, gamma, weight=w)
    assert_rounded_once(Y, dense_ref.reified(s, r, o, n_e, n_r, X, R, w) + gamma * Z.astype(np.float64))
    assert np.array_equal(oracle.follow_accumulate(s, r, o, n_e, n_r, X, R, X, gamma, weight=w),
                          oracle.follow_residual(s, r, o, n_e, n_r, X, R, gamma, weight=w))
    if gamma == 0.0:
        assert np.array_equal(Y, oracle.follow(s, r, o, n_e, n_r, X, R, weight=w))


def test_accumulate_integer_inputs_exact():
    """On integer inputs every sum is exact: Y = counts + gamma * Z exactly."""
    n_e, n_r, b = 40, 4, 5
    s, r, o, _ = tiny_kb(7, n_e, n_r, 300)
    g = np.random.default_rng(7)
    X = g.integers(0, 3, (b, n_e)).astype(np.float32)
    R = g.integers(0, 2, (b, n_r)).astype(np.float32)
    Z = g.integers(-5, 6, (b, n_e)).astype(np.float32)
    Y = oracle.follow_accumulate(s, r, o, n_e, n_r, X, R, Z, 2.0)
    want = dense_ref.reified(s, r, o, n_e, n_r, X, R, None) + 2.0 * Z
    assert np.array_equal(Y, want.astype(np.float32))


def test_residual_chain_is_the_path_expansion():
    # App. E: with x^t = f^t(x^{t-1}) + x^{t-1}, x^T expands by linearity into
    # the sum, over every subset S of {1..T}, of the hops in S applied in order.
    n_e, n_r, b, T = 30, 4, 3, 3
    s, r, o, w = tiny_kb(131, n_e, n_r, 220, weighted=True)
    g = np.random.default_rng(131)
    x0 = g.random((b, n_e))
    rs = [g.random((b, n_r)) for _ in range(T)]
    xs = chain.residual_chain((s, r, o), n_e, n_r, x0, rs, weight=w)
    total = np.zeros((b, n_e))
    for mask in range(1 << T):
        x = x0
        for t in range(T):
            if mask >> t & 1:
                x = dense_ref.reified(s, r, o, n_e, n_r, x, rs[t], w)
        total += x
    np.testing.assert_allclose(xs[-1], total, rtol=1e-12, atol=1e-12)


def test_residual_chain_gradients_finite_differences():
    n_e, n_r, b, T = 25, 4, 2, 3
    s, r, o, w = tiny_kb(141, n_e, n_r, 200, weighted=True)
    g = np.random.default_rng(141)
    x0 = g.standard_normal((b, n_e))
    rs = [g.standard_normal((b, n_r)) for _ in range(T)]
    G = g.standard_normal((b, n_e))
    L = lambda x, rr: float((G * chain.residual_chain((s, r, o), n_e, n_r, x, rr, weight=w)[-1]).sum())
    dx0, drs = chain.residual_chain_grad((s, r, o), n_e, n_r, x0, rs, G, weight=w)
    h = 1e-3
    V = g.standard_normal((b, n_e))
    fd = (L(x0 + h * V, rs) - L(x0 - h * V, rs)) / (2 * h)   # exact: L is linear in x0
    assert abs(fd - (dx0 * V).sum()) <= 1e-9 * max(1.0, abs(fd))
    for t in range(T):
        U = g.standard_normal((b, n_r))
        plus = [rr + h * U if i == t else rr for i, rr in enumerate(rs)]
        minus = [rr - h * U if i == t else rr for i, rr in enumerate(rs)]
        fd = (L(x0, plus) - L(x0, minus)) / (2 * h)           # exact: L is linear in each r^t
        assert abs(fd - (drs[t] * U).sum()) <= 1e-9 * max(1.0, abs(fd))
