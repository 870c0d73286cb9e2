"""The concurrent backward: on large KBs kb_follow_backward runs its dR pass
on a stream the KB owns, forked from the caller's stream and joined back.
Forced on for mid-size KBs here (KBFOLLOW_OVERLAP_BACKWARD=1), it must give
bit for bit the serial results (and the oracle's within tolerance), replay
correctly from a captured graph, and stay correct when two callers on two
streams share the KB (their dR passes then queue on the KB's stream)."""
import numpy as np
import pytest

import kbgen
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


def bits(t):
    import torch
    return t.view(torch.int32)


def workload(tag, batch=32):
    w = kbgen.METAQA.scaled(20_000, 150_000, batch=batch, tag=tag)
    return w, kbgen.make_kb(w)


def make(kbf, w, kb, overlap, monkeypatch):
    monkeypatch.setenv("KBFOLLOW_OVERLAP_BACKWARD", "1" if overlap else "0")
    return kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations)


@pytest.mark.parametrize("gamma", [None, 0.5])
def test_overlap_matches_serial_and_oracle(kbf, gamma, monkeypatch):
    import torch
    w, kb = workload(7)
    X, R, dY = kbgen.make_x(w), kbgen.make_r(w), kbgen.make_dy(w)
    outs = {}
    for overlap in (False, True):
        gkb = make(kbf, w, kb, overlap, monkeypatch)
        dX, dR = gkb.follow_backward(to_em(X), to_em(R), to_em(dY), residual=gamma)
        torch.cuda.synchronize()
        outs[overlap] = (dX, dR)
        gkb.close()
    for a, c in zip(outs[False], outs[True]):
        assert torch.equal(bits(a), bits(c))
    if gamma is None:
        wdX, wdR = oracle.follow_backward(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations,
                                          X, R, dY)
    else:
        wdX, wdR = oracle.follow_backward_residual(kb.subj, kb.rel, kb.obj, w.n_entities,
                                                   w.n_relations, X, R, dY, gamma=gamma)
    assert_close(from_em(outs[True][0]), wdX, "dX")
    assert_close(from_em(outs[True][1]), wdR, "dR")


def test_overlap_graph_replay(kbf, monkeypatch):
    import torch
    w, kb = workload(8)
    gkb = make(kbf, w, kb, True, monkeypatch)
    X, R, dY = to_em(kbgen.make_x(w)), to_em(kbgen.make_r(w)), to_em(kbgen.make_dy(w))
    dX0, dR0 = gkb.follow_backward(X, R, dY)
    torch.cuda.synchronize()
    dX, dR = torch.empty_like(dX0), torch.empty_like(dR0)
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        gkb.follow_backward(X, R, dY, dX=dX, dR=dR)
    torch.cuda.current_stream().wait_stream(side)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        gkb.follow_backward(X, R, dY, dX=dX, dR=dR)
    for i in range(4):
        dX.fill_(float("nan"))
        dR.fill_(float("nan"))
        eX, eR = gkb.follow_backward(X, R, dY)  # eager work between replays
        g.replay()
        torch.cuda.synchronize()
        assert torch.equal(bits(dX), bits(dX0)), f"replay {i}: dX"
        assert torch.equal(bits(dR), bits(dR0)), f"replay {i}: dR"
        assert torch.equal(bits(eR), bits(dR0))


def test_overlap_two_callers_share_the_kb(kbf, monkeypatch):
    import torch
    w, kb = workload(9)
    gkb = make(kbf, w, kb, True, monkeypatch)
    w2 = kbgen.METAQA.scaled(20_000, 150_000, batch=32, tag=10)
    ins = [(to_em(kbgen.make_x(v)), to_em(kbgen.make_r(v)), to_em(kbgen.make_dy(v)))
           for v in (w, w2)]
    alone = [gkb.follow_backward(*i) for i in ins]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    for rep in range(5):
        outs = [None, None]
        for k in (0, 1):
            with torch.cuda.stream(streams[k]):
                outs[k] = gkb.follow_backward(*ins[k])
        torch.cuda.synchronize()
        for k in (0, 1):
            for name, g, e in zip(("dX", "dR"), outs[k], alone[k]):
                assert torch.equal(bits(g), bits(e)), f"rep {rep} caller {k} {name}"


def test_overlap_two_host_threads(kbf, monkeypatch):
    """Two host threads, each with its own stream, call the concurrent
    backward on one KB at the same time: the per-KB lock keeps each call's
    fork / join sequence whole, and every result equals the one computed
    alone."""
    import threading
    import torch
    w, kb = workload(11)
    gkb = make(kbf, w, kb, True, monkeypatch)
    w2 = kbgen.METAQA.scaled(20_000, 150_000, batch=32, tag=12)
    ins = [(to_em(kbgen.make_x(v)), to_em(kbgen.make_r(v)), to_em(kbgen.make_dy(v)))
           for v in (w, w2)]
    alone = [gkb.follow_backward(*i) for i in ins]
    torch.cuda.synchronize()
    results, errors = [[], []], []

    def worker(k):
        try:
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.default_stream())
            with torch.cuda.stream(s):
                for _ in range(20):
                    results[k].append(gkb.follow_backward(*ins[k]))
            s.synchronize()
        except Exception as e:  # reported below, in the main thread
            errors.append(e)

    threads = [threading.Thread(target=worker, args=(k,)) for k in (0, 1)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for k in (0, 1):
        assert len(results[k]) == 20
        for i, (dX, dR) in enumerate(results[k]):
            assert torch.equal(bits(dX), bits(alone[k][0])), f"thread {k} call {i} dX"
            assert torch.equal(bits(dR), bits(alone[k][1])), f"thread {k} call {i} dR"
