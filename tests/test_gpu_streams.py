"""Concurrent calls on different streams.

A KB is immutable after kb_create, so forward and backward passes on two
streams, each with its own workspace (the binding keeps one per stream) and
outputs, may run at the same time.  The passes of two different minibatches
are enqueued interleaved on two streams, several times over, and each result
must equal, bit for bit, the same pass run alone.
"""
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


def test_two_streams(kbf):
    import torch
    w = kbgen.METAQA.scaled(20_000, 150_000, batch=32, tag=5)
    kb = kbgen.make_kb(w)
    gkb = kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations)
    assert gkb.workspace_size(w.batch) > 0  # split rows: the passes use scratch
    w2 = kbgen.METAQA.scaled(20_000, 150_000, batch=32, tag=6)  # other inputs, same shapes
    ins = [(to_em(kbgen.make_x(v)), to_em(kbgen.make_r(v)), to_em(kbgen.make_dy(v)))
           for v in (w, w2)]

    def passes(X, R, dY):
        Y = gkb.follow(X, R)
        dX, dR = gkb.follow_backward(X, R, dY)
        return Y, dX, dR

    alone = [passes(*i) for i in ins]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    for s in streams:
        s.wait_stream(torch.cuda.current_stream())
    bits = lambda t: t.view(torch.int32)
    for rep in range(5):
        outs = [None, None]
        # Enqueue forward of both, then backward of both, alternating streams.
        with torch.cuda.stream(streams[0]):
            y0 = gkb.follow(ins[0][0], ins[0][1])
        with torch.cuda.stream(streams[1]):
            y1 = gkb.follow(ins[1][0], ins[1][1])
        with torch.cuda.stream(streams[0]):
            outs[0] = (y0, *gkb.follow_backward(*ins[0]))
        with torch.cuda.stream(streams[1]):
            outs[1] = (y1, *gkb.follow_backward(*ins[1]))
        torch.cuda.synchronize()
        for k in range(2):
            for name, g, e in zip(("Y", "dX", "dR"), outs[k], alone[k]):
                assert torch.equal(bits(g), bits(e)), f"rep {rep} stream {k}: {name}"
    gkb.close()
