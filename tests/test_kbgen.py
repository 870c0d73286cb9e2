"""The seeded workload generators: determinism, shapes and structure."""
import numpy as np

import kbgen


def small(w, n_e, n_t, b=None):
    return w.scaled(n_e, n_t, batch=b)


def test_deterministic_and_distinct():
    for w in (kbgen.TINY, small(kbgen.LARGE, 20_000, 100_000), small(kbgen.TRAIN, 20_000, 100_000)):
        a, c = kbgen.make_kb(w), kbgen.make_kb(w)
        assert a.sha256() == c.sha256()
        assert a.n_triples == w.n_triples
        key = (a.subj.astype(np.int64) * w.n_relations + a.rel) * w.n_entities + a.obj
        assert len(np.unique(key)) == w.n_triples
        for arr, hi in ((a.subj, w.n_entities), (a.obj, w.n_entities), (a.rel, w.n_relations)):
            assert arr.dtype == np.int32 and arr.min() >= 0 and arr.max() < hi


def test_metaqa_shape_has_inverse_pairs():
    w = kbgen.METAQA
    kb = kbgen.make_kb(w)
    assert kb.n_triples == 190_000
    half = w.n_relations // 2
    base = set(zip(kb.subj[kb.rel < half].tolist(), kb.rel[kb.rel < half].tolist(),
                   kb.obj[kb.rel < half].tolist()))
    inv = set(zip(kb.obj[kb.rel >= half].tolist(), (kb.rel[kb.rel >= half] - half).tolist(),
                  kb.subj[kb.rel >= half].tolist()))
    assert base == inv and len(base) == 95_000
    st = kb.stats()
    assert st["max_out_degree"] > 5_000          # Zipf(1.1) head over 43 k entities


def test_zipf_head_and_tail():
    w = small(kbgen.LARGE, 200_000, 1_000_000)
    kb = kbgen.make_kb(w)
    deg = np.sort(np.bincount(kb.subj, minlength=w.n_entities))[::-1]
    # rank-frequency roughly k^-s in the head (distinctness only trims the very top)
    ratio = deg[9] / deg[99]
    assert 5 < ratio < 20
    assert (deg == 0).sum() > w.n_entities // 4


def test_inputs_shapes_and_laws():
    w = small(kbgen.LARGE, 50_000, 200_000)
    X = kbgen.make_x(w)
    assert X.shape == (w.batch, w.n_entities) and X.dtype == np.float32
    assert np.all((X > 0).sum(axis=1) == w.n_entities // 100)
    np.testing.assert_allclose(X.sum(axis=1), 1.0, rtol=1e-5)
    R = kbgen.make_r(w)
    np.testing.assert_allclose(R.sum(axis=1), 1.0, rtol=1e-5)
    assert np.array_equal(X, kbgen.make_x(w))
    Xi, Ri, dYi = kbgen.make_integer_inputs(w)
    assert set(np.unique(Xi).tolist()) <= {0.0, 1.0} and np.all(Ri.sum(axis=1) == 1)


def test_chain_seeds_reach_three_hops():
    w = kbgen.CHAIN3
    kb = kbgen.make_kb(w)
    assert kb.sha256() == kbgen.make_kb(kbgen.TINY).sha256()
    x0, rho, tgt = kbgen.make_chain_inputs(w, kb)
    assert x0.shape == (256, 1000) and np.all(x0.sum(axis=1) == 1)
    assert rho.shape == (3, 256, 10)
    np.testing.assert_allclose(tgt.sum(axis=1), 1.0, rtol=1e-6)


def test_grid_kb_shape():
    s, r, o = kbgen.grid_kb(5)
    assert len(s) == 4 * 5 * 4            # 2 n (n - 1) edges per axis, both directions
    assert set(r.tolist()) == {0, 1, 2, 3}
    for ss, oo in zip(s.tolist(), o.tolist()):
        assert abs(ss // 5 - oo // 5) + abs(ss % 5 - oo % 5) == 1
    s2, r2, o2 = kbgen.grid_kb(5, 50)
    assert np.array_equal(s, s2) and np.array_equal(o, o2) and r2.max() < 50
    x, rr = kbgen.grid_inputs(5, 50, 16)
    assert np.all(x.sum(axis=1) == 1) and np.all((rr >= 1.0) & (rr <= 1.001))
