"""Full-size parity on the large (10 M entities / 50 M triples, b = 32) and
training-shaped (2 M entities / 20 M triples, b = 256) workloads, in the
launch configuration bench.py times (default chunk, concurrent dR pass on
the large KB, R staged in LDS in 32-column slices on the training KB).

Every element of Y, dX and dR is compared with the whole oracle (forward and
backward over all b columns; about 3 s for the large KB and 25 s for the
training KB on 16 host threads): bit for bit on integer inputs, within
rtol 1e-5 / atol 1e-7 otherwise.  The largest tolerance ratio
|gpu - oracle| / (atol + rtol |oracle|) of each output is printed.
"""
import numpy as np
import pytest

import kbgen
import oracle
from gpu_util import ATOL, RTOL, assert_bitexact

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


@pytest.fixture(scope="module")
def kbf():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2002_06115_amd as kbf
    return kbf


_KB_CACHE = {}


def to_host_bm(t_em):
    """[N][b] CUDA tensor -> [b][N] numpy (transposed on the GPU)."""
    return t_em.t().contiguous().cpu().numpy()


def compare_all(got, want, integer, what, block=1 << 24):
    """Every element: bit for bit (integer inputs) or within the tolerance;
    returns the largest tolerance ratio.  Blocks of rows keep the float64
    temporaries small."""
    assert got.shape == want.shape, (what, got.shape, want.shape)
    g, w = got.reshape(-1), want.reshape(-1)
    worst = 0.0
    for i in range(0, g.size, block):
        gi, wi = g[i:i + block], w[i:i + block]
        if integer:
            bad = np.nonzero(gi != wi)[0]
            assert bad.size == 0, f"{what}: {bad.size} elements differ in block {i}, " \
                                  f"first at flat index {i + int(bad[0])}"
        assert np.all(np.isfinite(gi)), what
        d = np.abs(gi.astype(np.float64) - wi) / (ATOL + RTOL * np.abs(wi.astype(np.float64)))
        worst = max(worst, float(d.max()) if d.size else 0.0)
    print(f"[fullsize] {what}: {got.size} elements, max tolerance ratio {worst:.3g}", flush=True)
    assert worst <= 1.0, f"{what}: max |gpu-oracle|/(atol+rtol|oracle|) = {worst:.3g}"
    return worst


def run_workload(kbf, w, integer, weighted=False):
    import torch
    print(f"[fullsize] generating {w.label} integer={integer} weighted={weighted}", flush=True)
    if w.name not in _KB_CACHE:
        _KB_CACHE.clear()
        _KB_CACHE[w.name] = kbgen.make_kb(w)
    kb = _KB_CACHE[w.name]
    if integer:
        X, R, dY = kbgen.make_integer_inputs(w)
    else:
        X, R, dY = kbgen.make_x(w), kbgen.make_r(w), kbgen.make_dy(w)
    # Soft-KB weights (App. A): one positive weight per triple.
    wt = (np.random.default_rng(11).uniform(0.1, 2.0, kb.n_triples).astype(np.float32)
          if weighted else None)
    print(f"[fullsize] kb_create {w.label}", flush=True)
    gkb = kbf.KB(kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations, weight=wt)
    em = lambda a: torch.from_numpy(a).cuda().t().contiguous()
    Xe, Re, dYe = em(X), em(R), em(dY)
    Y = gkb.follow(Xe, Re)
    dX, dR = gkb.follow_backward(Xe, Re, dYe)
    # A second call, in the same launch configuration, is bitwise equal.
    Y2 = gkb.follow(Xe, Re)
    dX2, dR2 = gkb.follow_backward(Xe, Re, dYe)
    torch.cuda.synchronize()
    bits = lambda t: t.view(torch.int32)
    for name, t1, t2 in (("Y", Y, Y2), ("dX", dX, dX2), ("dR", dR, dR2)):
        assert torch.equal(bits(t1), bits(t2)), f"{w.name} {name} differs between two calls"
    del Y2, dX2, dR2, Xe, Re, dYe
    got = {"Y": to_host_bm(Y), "dX": to_host_bm(dX), "dR": to_host_bm(dR)}
    del Y, dX, dR
    gkb.close()
    torch.cuda.empty_cache()
    print(f"[fullsize] GPU passes done {w.label}; whole oracle", flush=True)
    args = (kb.subj, kb.rel, kb.obj, w.n_entities, w.n_relations)
    want_y = oracle.follow(*args, X, R, weight=wt)
    compare_all(got["Y"], want_y, integer, f"{w.name} Y")
    del want_y
    want_dx, want_dr = oracle.follow_backward(*args, X, R, dY, weight=wt)
    compare_all(got["dX"], want_dx, integer, f"{w.name} dX")
    compare_all(got["dR"], want_dr, integer, f"{w.name} dR")


@pytest.mark.parametrize("integer", [True, False])
def test_large_fullsize(kbf, integer):
    run_workload(kbf, kbgen.LARGE, integer)


def test_large_fullsize_soft_kb(kbf):
    run_workload(kbf, kbgen.LARGE, False, weighted=True)


@pytest.mark.parametrize("integer", [True, False])
def test_train_fullsize(kbf, integer):
    run_workload(kbf, kbgen.TRAIN, integer)


@pytest.mark.parametrize("layout_sort", ["auto", "counting"])
def test_maximum_entity_ids(kbf, layout_sort, monkeypatch):
    """N_E = 2^30, the largest id space the library takes, at b = 1 (4 GB per
    activation; tables of 4 GB or more take the plain-load path): triples at
    both ends of the id range, integer inputs, every row with a triple and a
    sample of empty rows checked bit for bit against the oracle; layouts built
    by the radix sorts (62-bit keys) and by the counting/comparison sorts."""
    import torch
    if layout_sort == "counting":
        monkeypatch.setenv("KBFOLLOW_LAYOUT_SORT", "counting")
    n_e, n_r, b = 1 << 30, 3, 1
    g = np.random.default_rng(30)
    n_t = 4000
    top = g.integers(n_e - 64, n_e, n_t // 2)
    low = g.integers(0, 64, n_t // 4)
    mid = g.integers(0, n_e, n_t - n_t // 2 - n_t // 4)
    s = np.concatenate([top, low, mid]).astype(np.int32)
    o = np.concatenate([low, mid, top]).astype(np.int32)
    r = g.integers(0, n_r, n_t).astype(np.int32)
    print("[maxsize] kb_create", flush=True)
    gkb = kbf.KB(s, r, o, n_e, n_r)
    gen = torch.Generator(device="cuda")
    gen.manual_seed(30)
    X = torch.randint(0, 4, (n_e, b), device="cuda", generator=gen).float()
    dY = torch.randint(-2, 3, (n_e, b), device="cuda", generator=gen).float()
    R = torch.tensor([[1.0], [2.0], [-1.0]], device="cuda")
    print("[maxsize] GPU passes", flush=True)
    Y = gkb.follow(X, R)
    dX, dR = gkb.follow_backward(X, R, dY)
    torch.cuda.synchronize()
    print("[maxsize] oracle", flush=True)
    Xh, dYh, Rh = (t.t().contiguous().cpu().numpy() for t in (X, dY, R))
    empty = np.setdiff1d(np.array([0, 1, 63, 64, n_e // 2, n_e - 65, n_e - 1], np.int64),
                         np.concatenate([s, o]))
    rand = g.integers(0, n_e, 32)
    objs = np.unique(np.concatenate([o, empty, rand])).astype(np.int32)
    subs = np.unique(np.concatenate([s, empty, rand])).astype(np.int32)
    rels = np.arange(n_r, dtype=np.int32)
    args = (s, r, o, n_e, n_r)
    want_y = oracle.sampled(oracle.SAMPLE_Y, *args, objs, X=Xh, R=Rh)
    want_dx = oracle.sampled(oracle.SAMPLE_DX, *args, subs, R=Rh, dY=dYh)
    want_dr = oracle.sampled(oracle.SAMPLE_DR, *args, rels, X=Xh, dY=dYh)
    idx = lambda t, ids: t[torch.from_numpy(ids.astype(np.int64)).cuda()].t().contiguous().cpu().numpy()
    assert_bitexact(idx(Y, objs), want_y, "max ids Y")
    assert_bitexact(idx(dX, subs), want_dx, "max ids dX")
    assert_bitexact(idx(dR, rels), want_dr, "max ids dR")
    assert gkb.info()["n_empty_rows"][0] == n_e - len(np.unique(o))
    gkb.close()
