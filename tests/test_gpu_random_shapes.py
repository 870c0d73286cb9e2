"""Seeded random shapes against the oracle.

Each case draws a KB shape (entities, relations, triples; uniform or
Zipf-skewed ids), a batch width, a plan (chunk length, combine fan-in), a
load path (B in LDS allowed or not, raw buffer or plain loads) and an
operation (plain follow, soft KB, residual hop, accumulating follow), and
compares forward and backward with the oracle: within rtol 1e-5 / atol 1e-7
on real-valued inputs, bit for bit on integer-valued ones.  Relation counts
and batch widths are drawn so that B tables fall on both sides of the LDS
limits and rows are cut into column slices.
"""
import numpy as np
import pytest

import oracle
from gpu_util import assert_bitexact, assert_close, from_em, to_em

pytestmark = pytest.mark.gpu

N_CASES = 120


@pytest.fixture(scope="module")
def kbf():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2002_06115_amd as kbf
    return kbf


def draw(seed):
    g = np.random.default_rng([2002, 6115, seed])
    n_e = int(g.choice([1, 7, 300, 2000, 5000]))
    n_r = int(g.choice([1, 3, 18, 160, 161, 640, 641, 1000, 1281]))
    n_t = int(g.choice([0, 1, 500, 20_000, 60_000]))
    b = int(g.choice([1, 3, 4, 16, 32, 36, 64, 128, 200, 256, 260]))
    skew = bool(g.random() < 0.5)

    def ids(n):
        if skew:
            return np.minimum(g.zipf(1.2, n_t) - 1, n - 1)
        return g.integers(0, n, n_t)

    s, r, o = ids(n_e), ids(n_r), ids(n_e)
    case = {
        "n_e": n_e, "n_r": n_r, "b": b, "skew": skew,
        "s": s.astype(np.int32), "r": r.astype(np.int32), "o": o.astype(np.int32),
        "chunk": int(g.choice([16, 32, 64, 256])),
        "fan_in": int(g.choice([2, 3, 32])),
        "lds": bool(g.random() < 0.7),
        "plain": bool(g.random() < 0.15),
        "op": str(g.choice(["follow", "follow", "soft", "residual", "accumulate"])),
        "integer": bool(g.random() < 0.3),
    }
    if case["integer"]:
        case["X"] = g.integers(0, 3, (b, n_e)).astype(np.float32)
        case["R"] = g.integers(0, 2, (b, n_r)).astype(np.float32)
        case["dY"] = g.integers(-2, 3, (b, n_e)).astype(np.float32)
        case["Z"] = g.integers(-3, 4, (b, n_e)).astype(np.float32)
        case["w"] = g.integers(1, 4, n_t).astype(np.float32)
        case["gamma"] = 2.0
    else:
        case["X"] = g.standard_normal((b, n_e)).astype(np.float32)
        case["R"] = g.standard_normal((b, n_r)).astype(np.float32)
        case["dY"] = g.standard_normal((b, n_e)).astype(np.float32)
        case["Z"] = g.standard_normal((b, n_e)).astype(np.float32)
        case["w"] = g.uniform(0.1, 2.0, n_t).astype(np.float32)
        case["gamma"] = float(g.uniform(-1.5, 1.5))
    return case


@pytest.mark.parametrize("seed", range(N_CASES))
def test_random_shape(kbf, seed, monkeypatch):
    c = draw(seed)
    label = (f"seed={seed} NE={c['n_e']} NR={c['n_r']} NT={len(c['s'])} b={c['b']} "
             f"skew={c['skew']} chunk={c['chunk']} fan_in={c['fan_in']} lds={c['lds']} "
             f"plain={c['plain']} op={c['op']} integer={c['integer']}")
    print(f"[random] {label}", flush=True)
    monkeypatch.setenv("KBFOLLOW_CHUNK", str(c["chunk"]))
    monkeypatch.setenv("KBFOLLOW_REL_CHUNK", str(c["chunk"]))
    monkeypatch.setenv("KBFOLLOW_FAN_IN", str(c["fan_in"]))
    monkeypatch.setenv("KBFOLLOW_B_IN_LDS", "1" if c["lds"] else "0")
    monkeypatch.setenv("KBFOLLOW_PLAIN_LOADS", "1" if c["plain"] else "0")
    s, r, o, n_e, n_r = c["s"], c["r"], c["o"], c["n_e"], c["n_r"]
    X, R, dY, Z, gamma = c["X"], c["R"], c["dY"], c["Z"], c["gamma"]
    w = c["w"] if c["op"] == "soft" else None
    kb = kbf.KB(s, r, o, n_e, n_r, weight=w)
    res = gamma if c["op"] == "residual" else None
    if c["op"] == "accumulate":
        Y = from_em(kb.follow_accumulate(to_em(X), to_em(R), to_em(Z), gamma))
        wantY = oracle.follow_accumulate(s, r, o, n_e, n_r, X, R, Z, gamma)
    elif res is not None:
        Y = from_em(kb.follow(to_em(X), to_em(R), residual=res))
        wantY = oracle.follow_residual(s, r, o, n_e, n_r, X, R, gamma=res)
    else:
        Y = from_em(kb.follow(to_em(X), to_em(R)))
        wantY = oracle.follow(s, r, o, n_e, n_r, X, R, weight=w)
    dX, dR = kb.follow_backward(to_em(X), to_em(R), to_em(dY), residual=res)
    if res is not None:
        wantdX, wantdR = oracle.follow_backward_residual(s, r, o, n_e, n_r, X, R, dY, gamma=res)
    else:
        wantdX, wantdR = oracle.follow_backward(s, r, o, n_e, n_r, X, R, dY, weight=w)
    check = assert_bitexact if c["integer"] else assert_close
    check(Y, wantY, label + " Y")
    check(from_em(dX), wantdX, label + " dX")
    check(from_em(dR), wantdR, label + " dR")
    kb.close()
