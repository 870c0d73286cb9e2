"""HIP graph capture of the library's calls.

Every call only enqueues kernels on the caller's stream (no allocation, no
synchronisation, no memset), so a caller can capture whole passes -- or a
multi-hop chain -- into one graph and replay it without host launches.  Each
test replays the graph several times, with eager work and synchronisation in
between, and checks every replay bit for bit against the eager result.
"""
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


def bits(t):
    import torch
    return t.view(torch.int32)


def capture(fn):
    """torch CUDA graph of fn(), after one warm-up call on the capture stream."""
    import torch
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        fn()
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        fn()
    return g


def test_forward_and_backward_replay(kbf):
    import torch
    # Small chunks: rows split into many slots, several combine levels, and
    # empty rows, so every kernel of a pass is in the graph.
    w = kbgen.METAQA.scaled(20_000, 150_000, batch=32, tag=5)
    kb = kbgen.make_kb(w)
    gkb = kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations)
    X, R, dY = to_em(kbgen.make_x(w)), to_em(kbgen.make_r(w)), to_em(kbgen.make_dy(w))
    Y0 = gkb.follow(X, R)
    dX0, dR0 = gkb.follow_backward(X, R, dY)
    torch.cuda.synchronize()
    info = gkb.info()
    assert max(info["n_levels"]) >= 1 and info["n_empty_rows"][0] > 0

    Y, dX, dR = torch.empty_like(Y0), torch.empty_like(dX0), torch.empty_like(dR0)

    def step():
        gkb.follow(X, R, out=Y)
        gkb.follow_backward(X, R, dY, dX=dX, dR=dR)

    g = capture(step)
    for i in range(4):
        for t in (Y, dX, dR):
            t.fill_(float("nan"))
        # Eager work between replays: the same passes into other buffers.
        Ye = gkb.follow(X, R)
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(bits(Y), bits(Y0)), f"replay {i}: Y"
        assert torch.equal(bits(dX), bits(dX0)), f"replay {i}: dX"
        assert torch.equal(bits(dR), bits(dR0)), f"replay {i}: dR"
        assert torch.equal(bits(Ye), bits(Y0))


def test_residual_chain_replay(kbf):
    """Three residual hops x^t = follow(x^{t-1}, r^t) + x^{t-1} (Sec. 3.2,
    App. E) captured as one graph: no host launch between hops."""
    import torch
    w = kbgen.METAQA.scaled(8_000, 60_000, batch=16, tag=6)
    kb = kbgen.make_kb(w)
    gkb = kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations)
    rng = np.random.default_rng(6)
    x0 = to_em(rng.random((w.batch, w.n_entities), dtype=np.float32))
    rs = [to_em(rng.random((w.batch, w.n_relations), dtype=np.float32)) for _ in range(3)]
    xs = [x0] + [torch.empty_like(x0) for _ in range(3)]

    def chain():
        for t in range(3):
            gkb.follow(xs[t], rs[t], out=xs[t + 1], residual=1.0)

    chain()
    torch.cuda.synchronize()
    want = xs[3].clone()
    g = capture(chain)
    for i in range(3):
        for t in xs[1:]:
            t.zero_()
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(bits(xs[3]), bits(want)), f"replay {i}"


def test_first_launch_under_capture(kbf):
    """The launcher's first call for a kernel and LDS size queries the
    occupancy calculator and sets the kernel's LDS limit; when that first call
    is being captured, the graph must still replay correctly.  (37 relations
    at b = 32 give an LDS size no other test uses.)"""
    import torch
    rng = np.random.default_rng(37)
    n_e, n_r, n_t, b = 3000, 37, 30_000, 32
    s = rng.integers(0, n_e, n_t).astype(np.int32)
    r = rng.integers(0, n_r, n_t).astype(np.int32)
    o = rng.integers(0, n_e, n_t).astype(np.int32)
    gkb = kbf.KB(s, r, o, n_e, n_r)
    X = to_em(rng.standard_normal((b, n_e)).astype(np.float32))
    R = to_em(rng.standard_normal((b, n_r)).astype(np.float32))
    Y = torch.empty_like(X)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        gkb.follow(X, R, out=Y)
    for i in range(3):
        Y.fill_(float("nan"))
        g.replay()
        torch.cuda.synchronize()
        want = gkb.follow(X, R)
        torch.cuda.synchronize()
        assert torch.equal(bits(Y), bits(want)), f"replay {i}"
